// Matrix-core GEMMs for gfx950: C[M x N] = A[M x K] * B[N x K]^T, both
// operands K-contiguous, fp32 accumulation, with the epilogues the decoder
// needs fused in (fp32 store, residual add, SwiGLU), and the LM head with a
// full-vocabulary online log-sum-exp epilogue that never writes logits.
//
// Large problems use 256x256 tiles (8 waves, MFMA fragments read one step
// ahead; in the pair mode the hi and lo planes of A share each B tile);
// problems with too few such tiles to fill the 256 CUs use 256x128 tiles
// (8 waves of 64x64, three stages). Both feed
// LDS with direct global->LDS loads, one barrier per K step. Tiles are ordered
// so that each XCD works on a contiguous band (see tile_coords).
#include <algorithm>

#include "gemm_core.h"
#include "kernels.h"

namespace jetk {

template <typename T>
struct GemmArgs {
  const T *A;
  const T *B;
  int64_t lda, ldb;
  int M, N;
  int K, KA, KB;  // K steps over K columns; A column k mod KA, B column k mod KB
  void *out;
  int64_t ldo;
  int pair_out;   // SwiGLU / QKV-RoPE: write (hi, lo) pairs
  float oscale;   // every product is multiplied by oscale before the epilogue
  QkvRope rope;   // EPI_QKV_ROPE only
  // grouped GEMM: row tile t uses B + tile_group[t] * group_stride; tiles
  // with tile_group -1 do nothing (null: one B for all tiles)
  const int *tile_group = nullptr;
  int64_t group_stride = 0;
  // int8 B (LOAD 9 configurations): fp16 scales [K / 32][ceil(N / 128)][32][4]
  const uint16_t *Bs = nullptr;
};

// (hi, lo) split of v stored at p[0] and p[ps] (lo only with pair).
template <typename T>
__device__ __forceinline__ void put_split(T *p, int64_t ps, float v, int pair) {
  const T hi = from_f<T>(v);
  p[0] = hi;
  if (pair) p[ps] = from_f<T>(v - to_f<T>(hi));
}

// Orders a wave's LDS writes before its following LDS reads of other lanes'
// data (a wave's LDS operations complete in order).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// fp32 store, residual add and SwiGLU epilogues through the LDS (free once
// the K loop has ended): each wave writes a slab of its accumulators (16 rows
// of fp32, or 32 rows of T for SwiGLU) into its own LDS region and reads it back as 16-byte
// row chunks, so every global access moves 16 bytes instead of 2 or 4. The
// arithmetic is that of the per-element epilogues in gemm_kernel. Returns
// false (nothing done) for tiles of fewer than 256 rows, where the output rows
// are not 16-byte aligned, or where the LDS is too small.
template <class C, int EPI>
__device__ __forceinline__ bool staged_epilogue(const GemmArgs<typename C::type> &g, int m0, int n0,
                                                f32x16 (&acc)[C::MI][C::NI], uint4 *lds) {
  using T = typename C::type;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  if constexpr (C::BM < 256) {
    // smaller tiles run several workgroups per CU; the staging registers
    // would cost one of them
    return false;
  } else if constexpr (EPI == 0 || EPI == 1) {
    constexpr int SC = C::WN < 64 ? C::WN : 64, LDF = SC + 4;  // slab columns, padded row (floats)
    constexpr int CH = 16 * SC / 4 / 64;                        // float4 chunks per lane per slab
    static_assert(CH >= 1 && (16 * SC / 4) % 64 == 0, "slab of whole chunk rounds");
    if constexpr ((size_t)C::NWAVES * 16 * LDF * 4 > C::LDS_BYTES) {
      return false;
    } else {
      if ((g.ldo & 3) || (g.N & 3)) return false;
      float *wl = reinterpret_cast<float *>(lds) + wave * 16 * LDF;
#pragma unroll
      for (int i = 0; i < C::MI; ++i)
#pragma unroll
        for (int hr = 0; hr < 2; ++hr)  // rows 16 hr .. 16 hr + 15 of the 32-row block
#pragma unroll
          for (int jh = 0; jh < C::WN / SC; ++jh) {
#pragma unroll
            for (int jj = 0; jj < SC / 32; ++jj)
#pragma unroll
              for (int e = 8 * hr; e < 8 * hr + 8; ++e) {
                const int r = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3) - 16 * hr;
                wl[r * LDF + jj * 32 + (lane & 31)] = acc[i][jh * (SC / 32) + jj][e] * g.oscale;
              }
            wave_lds_sync();
#pragma unroll
            for (int t = 0; t < CH; ++t) {
              const int q = t * 64 + lane, r = q / (SC / 4), c4 = q % (SC / 4);
              const int row = m0 + wm * C::WM + i * 32 + 16 * hr + r;
              const int col = n0 + wn * C::WN + jh * SC + 4 * c4;
              if (row < g.M && col < g.N) {
                const float4 v = *reinterpret_cast<const float4 *>(wl + r * LDF + 4 * c4);
                float4 *o = reinterpret_cast<float4 *>((float *)g.out + (int64_t)row * g.ldo + col);
                if constexpr (EPI == 0) {
                  *o = v;
                } else {
                  float4 x = *o;
                  x.x += v.x; x.y += v.y; x.z += v.z; x.w += v.w;
                  *o = x;
                }
              }
            }
            wave_lds_sync();
          }
      return true;
    }
  } else if constexpr (EPI == 2 && sizeof(T) == 2) {
    constexpr int OC = C::WN / 2, LDH = OC + 8;  // output columns of a wave, padded row (elements)
    constexpr int CH = 32 * OC / 8 / 64;         // 16-byte chunks per lane per 32-row slab
    static_assert(CH >= 1 && (32 * OC / 8) % 64 == 0, "slab of whole chunk rounds");
    if constexpr ((size_t)C::NWAVES * 32 * LDH * sizeof(T) > C::LDS_BYTES) {
      return false;
    } else {
      if (g.pair_out || (g.ldo & 7)) return false;
      T *wl = reinterpret_cast<T *>(lds) + wave * 32 * LDH;
      const int f0 = (n0 + wn * C::WN) >> 1;  // first output column of the wave
#pragma unroll
      for (int i = 0; i < C::MI; ++i) {
#pragma unroll
        for (int jp = 0; jp < C::NI / 2; ++jp)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const float gt = acc[i][2 * jp][e] * g.oscale, up = acc[i][2 * jp + 1][e] * g.oscale;
            // silu(g) = g / (1 + e^-g) with the hardware reciprocal (~1 ulp)
            const float v = gt * __builtin_amdgcn_rcpf(1.0f + __expf(-gt)) * up;
            const int r = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            wl[r * LDH + jp * 32 + (lane & 31)] = from_f<T>(v);
          }
        wave_lds_sync();
#pragma unroll
        for (int t = 0; t < CH; ++t) {
          const int q = t * 64 + lane, r = q / (OC / 8), c8 = q % (OC / 8);
          const int row = m0 + wm * C::WM + i * 32 + r;
          const int gcol = n0 + wn * C::WN + 64 * (c8 / 4);  // first gate column of the chunk's block
          if (row < g.M && gcol < g.N)
            *reinterpret_cast<uint4 *>((T *)g.out + (int64_t)row * g.ldo + f0 + 8 * c8) =
                *reinterpret_cast<const uint4 *>(wl + r * LDH + 8 * c8);
        }
        wave_lds_sync();
      }
      return true;
    }
  } else {
    return false;
  }
}

// EPI: 0 = store fp32, 1 = fp32 residual add, 2 = SwiGLU into T (B rows
// interleaved in blocks of 32 gate rows / 32 up rows), 3 = store T, 4 = RoPE
// and scatter of q, K, V (waves of 128 columns = one head).
template <class C, int EPI>
__global__ __launch_bounds__(C::NT) void gemm_kernel(GemmArgs<typename C::type> g) {
  using T = typename C::type;
  extern __shared__ uint4 lds[];
  if (gridDim.y > 1) {
    // split K (plain operands, fp32 store): workgroup row y takes K columns
    // [y Kc, (y + 1) Kc) and writes its partial sums to slice y of out
    const int kc = g.K / (int)gridDim.y;
    g.A += (int64_t)blockIdx.y * kc;
    g.B += (int64_t)blockIdx.y * kc;
    g.K = g.KA = g.KB = kc;
    g.out = (float *)g.out + (int64_t)blockIdx.y * g.M * g.ldo;
  }
  const int nt_m = (g.M + C::BM - 1) / C::BM, nt_n = (g.N + C::BN - 1) / C::BN;
  int tm, tn;
  tile_coords(nt_m, nt_n, &tm, &tn);
  const int m0 = tm * C::BM, n0 = tn * C::BN;
  const T *B = g.B;
  if (g.tile_group) {
    const int grp = g.tile_group[tm];
    if (grp < 0) return;
    B += (int64_t)grp * g.group_stride;
  }
  f32x16 acc[C::MI][C::NI];
  gemm_tile<C>(g.A, g.lda, B, g.ldb, g.M, g.N, g.K, g.KA, g.KB, m0, n0, lds, acc, g.Bs);
  if (staged_epilogue<C, EPI>(g, m0, n0, acc, lds)) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  if constexpr (EPI == 4) {
    static_assert(C::WN == 128 && C::NI == 4, "a wave's columns must be one head of 128");
    const QkvRope &q = g.rope;
    const int head = (n0 + wn * C::WN) >> 7;  // query heads, then key heads, then value heads
    const int64_t ps = head < q.Hq ? q.q_ps : q.kv_ps;
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = m0 + wm * C::WM + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (row >= g.M || head >= q.Hq + 2 * q.Hkv) continue;
        T *dst;
        if (head < q.Hq) dst = (T *)q.q_out + ((int64_t)row * q.Hq + head) * 128;
        else if (head < q.Hq + q.Hkv) dst = (T *)q.k_cache + ((int64_t)(head - q.Hq) * q.S + q.slot0 + row) * 128;
        else dst = (T *)q.v_cache + ((int64_t)(head - q.Hq - q.Hkv) * q.S + q.slot0 + row) * 128;
        if (head < q.Hq + q.Hkv) {
          const int64_t p = q.pos[row];
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int d = j * 32 + (lane & 31);
            const float x1 = acc[i][j][e] * g.oscale, x2 = acc[i][j + 2][e] * g.oscale;
            const float c = q.cos_t[p * 64 + d], s = q.sin_t[p * 64 + d];
            // the same operations as rope_scatter_kernel, so both paths round alike
            put_split<T>(dst + d, ps, fmaf(x1, c, -(x2 * s)), g.pair_out);
            put_split<T>(dst + d + 64, ps, fmaf(x2, c, x1 * s), g.pair_out);
          }
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) put_split<T>(dst + j * 32 + (lane & 31), ps, acc[i][j][e] * g.oscale, g.pair_out);
        }
      }
  } else if constexpr (EPI == 2) {
    T *out = (T *)g.out;
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int jp = 0; jp < C::NI / 2; ++jp) {
        const int gcol = n0 + wn * C::WN + jp * 64;  // first column of the gate block
        const int f = (gcol >> 6) * 32 + (lane & 31);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * C::WM + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          if (row < g.M && gcol < g.N) {
            const float gt = acc[i][2 * jp][e] * g.oscale, up = acc[i][2 * jp + 1][e] * g.oscale;
            // silu(g) = g / (1 + e^-g) with the hardware reciprocal (~1 ulp)
            const float v = gt * __builtin_amdgcn_rcpf(1.0f + __expf(-gt)) * up;
            const T hi = from_f<T>(v);
            out[(int64_t)row * g.ldo + f] = hi;
            if (g.pair_out) out[(int64_t)row * g.ldo + (g.N >> 1) + f] = from_f<T>(v - to_f<T>(hi));
          }
        }
      }
  } else {
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int j = 0; j < C::NI; ++j) {
        const int col = n0 + wn * C::WN + j * 32 + (lane & 31);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * C::WM + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          if (row >= g.M || col >= g.N) continue;
          const int64_t o = (int64_t)row * g.ldo + col;
          const float v = acc[i][j][e] * g.oscale;
          if constexpr (EPI == 0) ((float *)g.out)[o] = v;
          else if constexpr (EPI == 1) ((float *)g.out)[o] += v;
          else ((T *)g.out)[o] = from_f<T>(v);
        }
      }
  }
}

// LM head with online log-sum-exp (Section 3.1 Eq. 2 evaluated over vocabulary
// tiles): logits^T = W[V x K] * F[R x K]^T tile by tile; each lane keeps a
// running (max, sum of exp) in base 2 for its rows of F; one partial per
// (row, vocabulary split) is written. The logits stay in registers.
// F holds R rows of K columns: the final hidden rows, or (hi, lo) pairs of
// them when K = 2 KW (W rows are then read twice).
// With target (one vocabulary index per row of F), the product of a row with
// its target's W row is kept as well, zt[row] (unscaled): the very
// accumulator the log-sum-exp takes in, written by the one lane that holds it.
template <class C>
__global__ __launch_bounds__(C::NT) void lmhead_lse_kernel(const typename C::type *__restrict__ W,
                                                          const typename C::type *__restrict__ F, int V, int R,
                                                          int KW, int K, int tiles_per_split, float zscale,
                                                          float *__restrict__ part_m, float *__restrict__ part_s,
                                                          const int32_t *__restrict__ target,
                                                          float *__restrict__ zt) {
  extern __shared__ uint4 lds[];
  const int n0 = blockIdx.x * C::BN, split = blockIdx.y;
  const int ntiles = (V + C::BM - 1) / C::BM;
  const int vt0 = split * tiles_per_split, vt1 = min(vt0 + tiles_per_split, ntiles);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  float rm[C::NI], rs[C::NI];
  int tj[C::NI];  // this lane's rows' targets (-1: none)
#pragma unroll
  for (int j = 0; j < C::NI; ++j) {
    rm[j] = -INFINITY;
    rs[j] = 0.0f;
    const int row = n0 + wn * C::WN + j * 32 + (lane & 31);
    tj[j] = target && row < R ? target[row] : -1;
  }
  f32x16 acc[C::MI][C::NI];
  for (int vt = vt0; vt < vt1; ++vt) {
    const int m0 = vt * C::BM;
    gemm_tile<C>(W, KW, F, K, V, R, K, KW, K, m0, n0, lds, acc);
    // element e of acc[i][j] is vocabulary index vb + 32 i + 8 (e / 4) + e % 4
    const int vb = m0 + wm * C::WM + 4 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < C::NI; ++j) {
      const int dv = tj[j] - vb;
      if (dv >= 0 && dv < 32 * C::MI && (dv & 4) == 0) {
        const int row = n0 + wn * C::WN + j * 32 + (lane & 31);
        float z = 0.0f;
#pragma unroll
        for (int i = 0; i < C::MI; ++i)
#pragma unroll
          for (int e = 0; e < 16; ++e) z = dv == 32 * i + 8 * (e >> 2) + (e & 3) ? acc[i][j][e] : z;
        zt[row] = z;
      }
    }
#pragma unroll
    for (int j = 0; j < C::NI; ++j) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < C::MI; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int v = m0 + wm * C::WM + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          const float z = v < V ? acc[i][j][e] * zscale : -INFINITY;
          acc[i][j][e] = z;
          mx = fmaxf(mx, z);
        }
      if (mx == -INFINITY) continue;
      const float nm = fmaxf(rm[j], mx);
      float s = rs[j] * exp2f(rm[j] - nm);
#pragma unroll
      for (int i = 0; i < C::MI; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) s += exp2f(acc[i][j][e] - nm);
      rm[j] = nm;
      rs[j] = s;
    }
  }
  // merge the two lane halves that hold the same column, then the waves
  // along the vocabulary dimension through LDS
  float *sm = reinterpret_cast<float *>(lds);  // [WAVES_M][BN] maxima, then sums
#pragma unroll
  for (int j = 0; j < C::NI; ++j) {
    const float om = __shfl_xor(rm[j], 32), os = __shfl_xor(rs[j], 32);
    const float nm = fmaxf(rm[j], om);
    float s = 0.0f;
    if (nm != -INFINITY) s = rs[j] * exp2f(rm[j] - nm) + os * exp2f(om - nm);
    if (lane < 32) {
      const int cl = wn * C::WN + j * 32 + lane;
      sm[wm * C::BN + cl] = nm;
      sm[C::WAVES_M * C::BN + wm * C::BN + cl] = s;
    }
  }
  __syncthreads();
  for (int cl = threadIdx.x; cl < C::BN; cl += C::NT) {
    const int row = n0 + cl;
    if (row >= R) continue;
    float M = -INFINITY;
    for (int w = 0; w < C::WAVES_M; ++w) M = fmaxf(M, sm[w * C::BN + cl]);
    float S = 0.0f;
    if (M != -INFINITY)
      for (int w = 0; w < C::WAVES_M; ++w)
        S += sm[C::WAVES_M * C::BN + w * C::BN + cl] * exp2f(sm[w * C::BN + cl] - M);
    part_m[(int64_t)split * R + row] = M;
    part_s[(int64_t)split * R + row] = S;
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

// Direct-load pipelines with bank-conflict-free swizzles and 128-byte tile
// rows: the 256x256 tiles with fragments read one MFMA step ahead (two stages
// of 64 KB), the 256x128 tiles with three stages.
using BigB = GCfg<bf16, 256, 256, 128, 64, 4, 1, 2, 8>;
// Pair mode: the (hi, lo) planes of A and one B tile per 32-column stage
// (3 x 16 KB, three stages, two tiles in flight, each tile's loads spread
// over the first MFMA step of the step before), waves of 64 x 128 so each B
// fragment serves both planes.
using PairB = GCfg<bf16, 256, 256, 64, 128, 7, 2, 3, 4>;
// ... and for problems with fewer tiles: 128x128 tiles (8 waves of 32x64,
// three 24 KB stages, two workgroups per CU).
using PairS = GCfg<bf16, 128, 128, 32, 64, 7, 2, 3, 4>;
using SmallB = GCfg<bf16, 256, 128, 64, 64, 2, 1, 3, 8>;
using CfgF = GCfg<float, 128, 128, 64, 64, 0, 1>;
using LmB = GCfg<bf16, 256, 256, 128, 64, 4, 1, 2, 8>;
using LmF = GCfg<float, 128, 128, 64, 64, 0, 1>;
// fp16 operands: the LOAD 7 schedule with a single A plane (three 32 KB
// stages of 32-column A and B tiles), 256x256 tiles with waves of 64 x 128,
// or 128x128 tiles for problems with fewer tiles; the LM head on the same
// 256x256 schedule (16% faster than the two-stage 128-byte-row one).
using HalfB = GCfg<f16, 256, 256, 64, 128, 8, 2, 3, 4>;
using HalfS = GCfg<f16, 128, 128, 32, 64, 8, 2, 3, 4>;
// Residual-add GEMMs with a short K loop (the attention output projection):
// 256x128 tiles, two workgroups per CU, so one tile's fp32 read-modify-write
// epilogue overlaps another's K loop (measured 16% faster than 256x256 at
// 134k x 1536 x 1536).
using HalfM = GCfg<f16, 256, 128, 64, 64, 8, 2, 3, 4>;
// (hi, lo) fp16 pair A operands: the bf16 pair schedules with fp16 operands
using HalfPairB = GCfg<f16, 256, 256, 64, 128, 7, 2, 3, 4>;
using HalfPairS = GCfg<f16, 128, 128, 32, 64, 7, 2, 3, 4>;
using LmH = GCfg<f16, 256, 256, 64, 128, 8, 2, 3, 4>;
// int8 B operand (block-quantized weights): the LOAD 8 schedule with int8 B
// tiles and per-block scales (three 24.5 KB stages), 256x256 tiles of 8
// waves, or 128x128 tiles of 4 waves for problems with fewer tiles.
using Q8B = GCfg<f16, 256, 256, 64, 128, 9, 2, 3, 4>;
using Q8S = GCfg<f16, 128, 128, 64, 64, 9, 2, 3, 4>;
// int4 B (packed two per byte), the same schedule
using Q4B = GCfg<f16, 256, 256, 64, 128, 10, 2, 3, 4>;
using Q4S = GCfg<f16, 128, 128, 64, 64, 10, 2, 3, 4>;

// Kernels whose LDS exceeds the default 64 KB limit must opt in once.
template <class C>
static hipError_t allow_lds(const void *fn) {
  if (C::LDS_BYTES <= 65536) return hipSuccess;
  return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS_BYTES);
}

template <class C, int EPI>
static hipError_t run_gemm(const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N, int K, int pair,
                           void *out, int64_t ldo, float oscale, hipStream_t st) {
  using T = typename C::type;
  static const hipError_t once = allow_lds<C>((const void *)gemm_kernel<C, EPI>);
  if (once != hipSuccess) return once;
  GemmArgs<T> g{(const T *)A, (const T *)B, lda, ldb, M, N, pair ? 2 * K : K, pair ? 2 * K : K, K, out, ldo, pair,
                oscale, QkvRope{}};
  const int tiles = ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
  hipLaunchKernelGGL((gemm_kernel<C, EPI>), dim3(tiles), dim3(C::NT), C::LDS_BYTES, st, g);
  return hipGetLastError();
}

template <class C>
static hipError_t run_epi(int epi, const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N, int K,
                          int pair, void *out, int64_t ldo, float oscale, hipStream_t st) {
  switch (epi) {
    case EPI_STORE_F32: return run_gemm<C, 0>(A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st);
    case EPI_RESID_ADD: return run_gemm<C, 1>(A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st);
    case EPI_SWIGLU: return run_gemm<C, 2>(A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st);
    default: return run_gemm<C, 3>(A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st);
  }
}

int gemm_k_step(int dtype) { return dtype == 1 ? CfgF::BK : BigB::BK; }

// Fixed-order sum of the split-K partials: out (+)= sum over s of part[s].
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float *__restrict__ part, int S, int M, int N,
                                                            float *__restrict__ out, int64_t ldo, int add) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)M * N) return;
  const int r = (int)(i / N), c = (int)(i % N);
  float v = 0.0f;
  for (int s = 0; s < S; ++s) v += part[((int64_t)s * M + r) * N + c];
  float *o = out + (int64_t)r * ldo + c;
  *o = add ? *o + v : v;
}

int gemm_splitk_ways(int dtype, int pair, int M, int N, int K) {
  if (dtype != 2 || pair) return 1;
  const int tiles = ((M + HalfS::BM - 1) / HalfS::BM) * ((N + HalfS::BN - 1) / HalfS::BN);
  int s = 1;
  while (s < 16 && tiles * s < 256 && K % (2 * s * HalfS::BK) == 0 && K / (2 * s) >= 512) s *= 2;
  return s;
}

hipError_t launch_gemm_splitk(int epi, const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N, int K,
                              int S, float *part, void *out, int64_t ldo, float oscale, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (S < 2 || K % (S * HalfS::BK) || (epi != EPI_STORE_F32 && epi != EPI_RESID_ADD)) return hipErrorInvalidValue;
  static const hipError_t once = allow_lds<HalfS>((const void *)gemm_kernel<HalfS, 0>);
  if (once != hipSuccess) return once;
  GemmArgs<f16> g{(const f16 *)A, (const f16 *)B, lda, ldb, M, N, K, K, K, part, N, 0, oscale, QkvRope{}};
  const int tiles = ((M + HalfS::BM - 1) / HalfS::BM) * ((N + HalfS::BN - 1) / HalfS::BN);
  hipLaunchKernelGGL((gemm_kernel<HalfS, 0>), dim3(tiles, S), dim3(HalfS::NT), HalfS::LDS_BYTES, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n = (int64_t)M * N;
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, part, S, M, N,
                     (float *)out, ldo, epi == EPI_RESID_ADD ? 1 : 0);
  return hipGetLastError();
}

// Workgroups of gemm_kernel<C, EPI> the device holds at once (0 if unknown).
template <class C, int EPI>
static int resident_groups() {
  static const int n = [] {
    int dev = 0, cus = 0, per_cu = 0;
    if (allow_lds<C>((const void *)gemm_kernel<C, EPI>) != hipSuccess || hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void *)gemm_kernel<C, EPI>, C::NT,
                                                     C::LDS_BYTES) != hipSuccess)
      return 0;
    return cus * per_cu;
  }();
  return n;
}

// fp16 GEMM on the tile configuration C whose last round of tiles would
// leave over half of the device idle: the row tiles holding that round run
// as a second launch of 128x128 tiles (several per CU), which fills the
// device better; every output element is computed alike in both.
template <class C, int EPI>
static hipError_t run_gemm_tail(const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N, int K, void *out,
                                int64_t ldo, float oscale, hipStream_t st) {
  const int nt_m = (M + C::BM - 1) / C::BM, nt_n = (N + C::BN - 1) / C::BN;
  const int64_t tiles = (int64_t)nt_m * nt_n;
  const int slots = resident_groups<C, EPI>();
  const int64_t rem = slots > 0 ? tiles % slots : 0;
  const int tail_mt = rem > 0 ? (int)((rem + nt_n - 1) / nt_n) : 0;
  if (rem == 0 || rem > slots / 2 || tail_mt >= nt_m) return run_gemm<C, EPI>(A, lda, B, ldb, M, N, K, 0, out, ldo, oscale, st);
  const int M1 = (nt_m - tail_mt) * C::BM;
  const size_t osz = EPI == 0 || EPI == 1 ? sizeof(float) : sizeof(f16);
  hipError_t e = run_gemm<C, EPI>(A, lda, B, ldb, M1, N, K, 0, out, ldo, oscale, st);
  if (e != hipSuccess) return e;
  return run_gemm<HalfS, EPI>((const f16 *)A + (int64_t)M1 * lda, lda, B, ldb, M - M1, N, K, 0,
                              (char *)out + (size_t)M1 * (size_t)ldo * osz, ldo, oscale, st);
}

hipError_t launch_gemm(int dtype, int epi, const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N,
                       int K, int pair, void *out, int64_t ldo, float oscale, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  // 256x256 tiles when there are enough of them to fill the chip twice over
  const int64_t big_tiles = (int64_t)((M + 255) / 256) * ((N + 255) / 256);
  if (dtype == 0) {
    if (pair)
      return big_tiles >= 512 ? run_epi<PairB>(epi, A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st)
                              : run_epi<PairS>(epi, A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st);
    if (big_tiles >= 512) return run_epi<BigB>(epi, A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st);
    return run_epi<SmallB>(epi, A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st);
  }
  if (dtype == 2) {
    if (pair)
      return big_tiles >= 512 ? run_epi<HalfPairB>(epi, A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st)
                              : run_epi<HalfPairS>(epi, A, lda, B, ldb, M, N, K, pair, out, ldo, oscale, st);
    if (big_tiles < 512) return run_epi<HalfS>(epi, A, lda, B, ldb, M, N, K, 0, out, ldo, oscale, st);
    if (epi == EPI_RESID_ADD && K <= 2048)
      return run_gemm_tail<HalfM, 1>(A, lda, B, ldb, M, N, K, out, ldo, oscale, st);
    switch (epi) {
      case EPI_STORE_F32: return run_gemm_tail<HalfB, 0>(A, lda, B, ldb, M, N, K, out, ldo, oscale, st);
      case EPI_RESID_ADD: return run_gemm_tail<HalfB, 1>(A, lda, B, ldb, M, N, K, out, ldo, oscale, st);
      case EPI_SWIGLU: return run_gemm_tail<HalfB, 2>(A, lda, B, ldb, M, N, K, out, ldo, oscale, st);
      default: return run_gemm_tail<HalfB, 3>(A, lda, B, ldb, M, N, K, out, ldo, oscale, st);
    }
  }
  return run_epi<CfgF>(epi, A, lda, B, ldb, M, N, K, 0, out, ldo, oscale, st);
}

template <class C, int EPI>
static hipError_t run_gemm_q8(const void *A, int64_t lda, const void *Bq, const uint16_t *Bs, int M, int N, int K,
                              void *out, int64_t ldo, float oscale, hipStream_t st) {
  static const hipError_t once = allow_lds<C>((const void *)gemm_kernel<C, EPI>);
  if (once != hipSuccess) return once;
  GemmArgs<f16> g{(const f16 *)A, (const f16 *)Bq, lda, (int64_t)K * C::QBITS / 8, M, N, K, K, K, out, ldo, 0,
                  oscale, QkvRope{}};
  g.Bs = Bs;
  const int tiles = ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
  hipLaunchKernelGGL((gemm_kernel<C, EPI>), dim3(tiles), dim3(C::NT), C::LDS_BYTES, st, g);
  return hipGetLastError();
}

template <class C>
static hipError_t run_q8_epi(int epi, const void *A, int64_t lda, const void *Bq, const uint16_t *Bs, int M, int N,
                             int K, void *out, int64_t ldo, float oscale, hipStream_t st) {
  switch (epi) {
    case EPI_STORE_F32: return run_gemm_q8<C, 0>(A, lda, Bq, Bs, M, N, K, out, ldo, oscale, st);
    case EPI_RESID_ADD: return run_gemm_q8<C, 1>(A, lda, Bq, Bs, M, N, K, out, ldo, oscale, st);
    case EPI_SWIGLU: return run_gemm_q8<C, 2>(A, lda, Bq, Bs, M, N, K, out, ldo, oscale, st);
    default: return run_gemm_q8<C, 3>(A, lda, Bq, Bs, M, N, K, out, ldo, oscale, st);
  }
}

hipError_t launch_gemm_q8(int epi, const void *A, int64_t lda, const void *Bq, const uint16_t *Bs, int M, int N,
                          int K, void *out, int64_t ldo, float oscale, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K % 32 != 0) return hipErrorInvalidValue;
  const int64_t big_tiles = (int64_t)((M + 255) / 256) * ((N + 255) / 256);
  if (big_tiles >= 512) return run_q8_epi<Q8B>(epi, A, lda, Bq, Bs, M, N, K, out, ldo, oscale, st);
  return run_q8_epi<Q8S>(epi, A, lda, Bq, Bs, M, N, K, out, ldo, oscale, st);
}

hipError_t launch_gemm_q4(int epi, const void *A, int64_t lda, const void *Bq, const uint16_t *Bs, int M, int N,
                          int K, void *out, int64_t ldo, float oscale, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K % 32 != 0) return hipErrorInvalidValue;
  const int64_t big_tiles = (int64_t)((M + 255) / 256) * ((N + 255) / 256);
  if (big_tiles >= 512) return run_q8_epi<Q4B>(epi, A, lda, Bq, Bs, M, N, K, out, ldo, oscale, st);
  return run_q8_epi<Q4S>(epi, A, lda, Bq, Bs, M, N, K, out, ldo, oscale, st);
}

template <class C, int EPI>
static hipError_t run_gemm_grouped(const void *A, int64_t lda, const void *B, int64_t ldb, int64_t group_stride,
                                   const int *tile_group, int M, int N, int K, void *out, int64_t ldo, float oscale,
                                   hipStream_t st) {
  using T = typename C::type;
  static const hipError_t once = allow_lds<C>((const void *)gemm_kernel<C, EPI>);
  if (once != hipSuccess) return once;
  GemmArgs<T> g{(const T *)A, (const T *)B, lda, ldb, M, N, K, K, K, out, ldo, 0, oscale, QkvRope{},
                tile_group, group_stride};
  const int tiles = (M / C::BM) * ((N + C::BN - 1) / C::BN);
  hipLaunchKernelGGL((gemm_kernel<C, EPI>), dim3(tiles), dim3(C::NT), C::LDS_BYTES, st, g);
  return hipGetLastError();
}

template <class C>
static hipError_t run_grouped_epi(int epi, const void *A, int64_t lda, const void *B, int64_t ldb,
                                  int64_t group_stride, const int *tile_group, int M, int N, int K, void *out,
                                  int64_t ldo, float oscale, hipStream_t st) {
  switch (epi) {
    case EPI_STORE_F32:
      return run_gemm_grouped<C, 0>(A, lda, B, ldb, group_stride, tile_group, M, N, K, out, ldo, oscale, st);
    case EPI_RESID_ADD:
      return run_gemm_grouped<C, 1>(A, lda, B, ldb, group_stride, tile_group, M, N, K, out, ldo, oscale, st);
    case EPI_SWIGLU:
      return run_gemm_grouped<C, 2>(A, lda, B, ldb, group_stride, tile_group, M, N, K, out, ldo, oscale, st);
    case EPI_STORE_T:
      return run_gemm_grouped<C, 3>(A, lda, B, ldb, group_stride, tile_group, M, N, K, out, ldo, oscale, st);
    default: return hipErrorInvalidValue;
  }
}

int gemm_group_rows(int dtype, int big) {
  return dtype == 2 ? (big ? HalfB::BM : HalfS::BM) : dtype == 1 ? CfgF::BM : SmallB::BM;
}

hipError_t launch_gemm_grouped(int dtype, int big, int epi, const void *A, int64_t lda, const void *B, int64_t ldb,
                               int64_t group_stride, const int *tile_group, int M, int N, int K, void *out,
                               int64_t ldo, float oscale, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (!tile_group || M % gemm_group_rows(dtype, big)) return hipErrorInvalidValue;
  if (dtype == 2 && big)
    return run_grouped_epi<HalfB>(epi, A, lda, B, ldb, group_stride, tile_group, M, N, K, out, ldo, oscale, st);
  if (dtype == 2)
    return run_grouped_epi<HalfS>(epi, A, lda, B, ldb, group_stride, tile_group, M, N, K, out, ldo, oscale, st);
  if (dtype == 1)
    return run_grouped_epi<CfgF>(epi, A, lda, B, ldb, group_stride, tile_group, M, N, K, out, ldo, oscale, st);
  return run_grouped_epi<SmallB>(epi, A, lda, B, ldb, group_stride, tile_group, M, N, K, out, ldo, oscale, st);
}

template <class C>
static hipError_t run_qkv_rope(const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N, int K,
                               int pair, float oscale, const QkvRope &r, hipStream_t st) {
  using T = typename C::type;
  static const hipError_t once = allow_lds<C>((const void *)gemm_kernel<C, 4>);
  if (once != hipSuccess) return once;
  GemmArgs<T> g{(const T *)A, (const T *)B, lda, ldb, M, N, pair ? 2 * K : K, pair ? 2 * K : K, K, nullptr, 0,
                pair, oscale, r};
  const int tiles = ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
  hipLaunchKernelGGL((gemm_kernel<C, 4>), dim3(tiles), dim3(C::NT), C::LDS_BYTES, st, g);
  return hipGetLastError();
}

bool gemm_qkv_rope_ok(int dtype, int pair, int M, int N, int head_dim) {
  if (head_dim != 128 || N % 128 || M <= 0) return false;
  const int64_t big_tiles = (int64_t)((M + 255) / 256) * ((N + 255) / 256);
  // the 256x256 configurations have waves of 128 columns
  return (dtype == 0 && pair && big_tiles >= 512) || (dtype == 2 && big_tiles >= 512);
}

hipError_t launch_gemm_qkv_rope(int dtype, const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N,
                                int K, int pair, float oscale, const QkvRope &r, hipStream_t st) {
  if (!gemm_qkv_rope_ok(dtype, pair, M, N, 128)) return hipErrorInvalidValue;
  if (dtype == 0) return run_qkv_rope<PairB>(A, lda, B, ldb, M, N, K, pair, oscale, r, st);
  if (pair) return run_qkv_rope<HalfPairB>(A, lda, B, ldb, M, N, K, pair, oscale, r, st);
  return run_qkv_rope<HalfB>(A, lda, B, ldb, M, N, K, 0, oscale, r, st);
}

void lmhead_plan(int dtype, int V, int R, int *tiles_per_split, int *nsplit) {
  (void)R;
  // The split of the vocabulary depends on V only, so that a row's
  // log-sum-exp is merged in the same order whatever batch it is in; about
  // 256 splits keep even a one-row-tile launch spread over the CUs.
  const int bm = dtype == 1 ? LmF::BM : LmB::BM;
  const int vt = (V + bm - 1) / bm;
  const int tps = std::max(1, vt / 256);
  *tiles_per_split = tps;
  *nsplit = (vt + tps - 1) / tps;
}

template <class C>
static hipError_t run_lmhead(const void *W, const void *F, int V, int R, int K, int pair, int tiles_per_split,
                             float wscale, float *part_m, float *part_s, const int32_t *target, float *zt,
                             hipStream_t st) {
  using T = typename C::type;
  static const hipError_t once = allow_lds<C>((const void *)lmhead_lse_kernel<C>);
  if (once != hipSuccess) return once;
  const int nsplit = ((V + C::BM - 1) / C::BM + tiles_per_split - 1) / tiles_per_split;
  dim3 grid((R + C::BN - 1) / C::BN, nsplit);
  hipLaunchKernelGGL((lmhead_lse_kernel<C>), grid, dim3(C::NT), C::LDS_BYTES, st, (const T *)W, (const T *)F, V, R,
                     K, pair ? 2 * K : K, tiles_per_split, wscale * kLog2e, part_m, part_s, target, zt);
  return hipGetLastError();
}

hipError_t launch_lmhead_lse(int dtype, const void *W, const void *F, int V, int R, int K, int pair,
                             int tiles_per_split, float wscale, float *part_m, float *part_s, const int32_t *target,
                             float *zt, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if ((target == nullptr) != (zt == nullptr)) return hipErrorInvalidValue;
  if (dtype == 0)
    return run_lmhead<LmB>(W, F, V, R, K, pair, tiles_per_split, wscale, part_m, part_s, target, zt, st);
  if (dtype == 2) return run_lmhead<LmH>(W, F, V, R, K, 0, tiles_per_split, wscale, part_m, part_s, target, zt, st);
  return run_lmhead<LmF>(W, F, V, R, K, 0, tiles_per_split, wscale, part_m, part_s, target, zt, st);
}

}  // namespace jetk
