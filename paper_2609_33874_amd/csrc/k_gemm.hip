// Matrix-core GEMMs for gfx950: C[M x N] = A[M x K] * B[N x K]^T, both
// operands K-contiguous, fp32 accumulation, with the epilogues the decoder
// needs fused in (fp32 store, residual add, SwiGLU), and the LM head with a
// full-vocabulary online log-sum-exp epilogue that never writes logits.
//
// Tiling: BM x BN output tile per workgroup, K step of 128 bytes per row
// (64 bf16 / 32 fp32), WM x WN per wave built from 32x32 MFMA blocks.
// Global -> registers -> LDS with double buffering (one barrier per K step);
// LDS rows are 8 chunks of 16 B, chunk c of row r stored at c ^ (r & 7) so
// that the MFMA operand reads of 8 consecutive rows hit distinct banks.
#include "device.h"
#include "kernels.h"

namespace jetk {

template <typename T, int BM_, int BN_, int WM_, int WN_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN;
  static constexpr int NT = WAVES_M * WAVES_N * 64;
  static constexpr int MI = WM / 32, NI = WN / 32;
  static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  static constexpr int BK = 8 * EPC;                // elements per K step (128 B)
  static constexpr int A_PT = BM * 8 / NT, B_PT = BN * 8 / NT;
  static constexpr int BUF = (BM + BN) * 8;         // chunks per LDS buffer
  static_assert(BM * 8 % NT == 0 && BN * 8 % NT == 0, "tile/thread mismatch");
};

template <typename T>
__device__ __forceinline__ void lds_frag(Frag<T> &f, const uint4 *row, int c0, int swz);
template <>
__device__ __forceinline__ void lds_frag<bf16>(Frag<bf16> &f, const uint4 *row, int c0, int swz) {
  f.v = __builtin_bit_cast(bf16x8, row[c0 ^ swz]);
}
template <>
__device__ __forceinline__ void lds_frag<float>(Frag<float> &f, const uint4 *row, int c0, int swz) {
  uint4 a = row[c0 ^ swz], b = row[(c0 + 1) ^ swz];
  f.v[0] = __uint_as_float(a.x); f.v[1] = __uint_as_float(a.y);
  f.v[2] = __uint_as_float(a.z); f.v[3] = __uint_as_float(a.w);
  f.v[4] = __uint_as_float(b.x); f.v[5] = __uint_as_float(b.y);
  f.v[6] = __uint_as_float(b.z); f.v[7] = __uint_as_float(b.w);
}

// One output tile: acc = A[m0:m0+BM, :] * B[n0:n0+BN, :]^T. Rows beyond M / N
// read as zero. K must be a multiple of C::BK. Ends with a barrier.
template <typename T, class C>
__device__ __forceinline__ void gemm_tile(const T *__restrict__ A, int64_t lda, const T *__restrict__ B,
                                          int64_t ldb, int M, int N, int K, int m0, int n0, uint4 *lds,
                                          f32x16 (&acc)[C::MI][C::NI]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
#pragma unroll
    for (int j = 0; j < C::NI; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  uint4 ra[C::A_PT], rb[C::B_PT];
  const uint4 zero4 = make_uint4(0, 0, 0, 0);
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::A_PT; ++i) {
      const int ch = tid + i * C::NT, r = ch >> 3, c = ch & 7, gm = m0 + r;
      ra[i] = gm < M ? ld16(A + (int64_t)gm * lda + k0 + c * C::EPC) : zero4;
    }
#pragma unroll
    for (int i = 0; i < C::B_PT; ++i) {
      const int ch = tid + i * C::NT, r = ch >> 3, c = ch & 7, gn = n0 + r;
      rb[i] = gn < N ? ld16(B + (int64_t)gn * ldb + k0 + c * C::EPC) : zero4;
    }
  };
  auto lstore = [&](int buf) {
    uint4 *a = lds + buf * C::BUF, *b = a + C::BM * 8;
#pragma unroll
    for (int i = 0; i < C::A_PT; ++i) {
      const int ch = tid + i * C::NT, r = ch >> 3, c = ch & 7;
      a[r * 8 + (c ^ (r & 7))] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < C::B_PT; ++i) {
      const int ch = tid + i * C::NT, r = ch >> 3, c = ch & 7;
      b[r * 8 + (c ^ (r & 7))] = rb[i];
    }
  };

  const int nk = K / C::BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload((kt + 1) * C::BK);
    const uint4 *a = lds + (kt & 1) * C::BUF, *b = a + C::BM * 8;
#pragma unroll
    for (int kk = 0; kk < C::BK / 16; ++kk) {
      const int c0 = (kk * 16 + (lane >> 5) * 8) / C::EPC;
      Frag<T> fa[C::MI], fb[C::NI];
#pragma unroll
      for (int i = 0; i < C::MI; ++i) {
        const int r = wm * C::WM + i * 32 + (lane & 31);
        lds_frag<T>(fa[i], a + r * 8, c0, r & 7);
      }
#pragma unroll
      for (int j = 0; j < C::NI; ++j) {
        const int r = wn * C::WN + j * 32 + (lane & 31);
        lds_frag<T>(fb[j], b + r * 8, c0, r & 7);
      }
#pragma unroll
      for (int i = 0; i < C::MI; ++i)
#pragma unroll
        for (int j = 0; j < C::NI; ++j) mma32(acc[i][j], fa[i], fb[j]);
    }
    if (kt + 1 < nk) lstore((kt + 1) & 1);
    __syncthreads();
  }
}

template <typename T>
struct GemmArgs {
  const T *A;
  const T *B;
  int64_t lda, ldb;
  int M, N, K;
  void *out;
  int64_t ldo;
};

// EPI: 0 = store fp32, 1 = fp32 residual add, 2 = SwiGLU into T (B rows
// interleaved in blocks of 32 gate rows / 32 up rows), 3 = store T.
template <typename T, class C, int EPI>
__global__ __launch_bounds__(C::NT) void gemm_kernel(GemmArgs<T> g) {
  extern __shared__ uint4 lds[];
  const int n0 = blockIdx.x * C::BN, m0 = blockIdx.y * C::BM;
  f32x16 acc[C::MI][C::NI];
  gemm_tile<T, C>(g.A, g.lda, g.B, g.ldb, g.M, g.N, g.K, m0, n0, lds, acc);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  if constexpr (EPI == 2) {
    T *out = (T *)g.out;
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int jp = 0; jp < C::NI / 2; ++jp) {
        const int gcol = n0 + wn * C::WN + jp * 64;  // first column of the gate block
        if (gcol >= g.N) continue;
        const int f = (gcol >> 6) * 32 + (lane & 31);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * C::WM + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          if (row < g.M) {
            const float gt = acc[i][2 * jp][e], up = acc[i][2 * jp + 1][e];
            out[(int64_t)row * g.ldo + f] = from_f<T>(gt / (1.0f + __expf(-gt)) * up);
          }
        }
      }
  } else {
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int j = 0; j < C::NI; ++j) {
        const int col = n0 + wn * C::WN + j * 32 + (lane & 31);
        if (col >= g.N) continue;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * C::WM + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          if (row >= g.M) continue;
          const int64_t o = (int64_t)row * g.ldo + col;
          if constexpr (EPI == 0) ((float *)g.out)[o] = acc[i][j][e];
          else if constexpr (EPI == 1) ((float *)g.out)[o] += acc[i][j][e];
          else ((T *)g.out)[o] = from_f<T>(acc[i][j][e]);
        }
      }
  }
}

// LM head with online log-sum-exp (Section 3.1 Eq. 2 evaluated over vocabulary
// tiles): logits^T = W[V x K] * F[R x K]^T tile by tile; each lane keeps a
// running (max, sum of exp) in base 2 for its rows of F; one partial per
// (row, vocabulary split) is written. The logits stay in registers.
template <typename T, class C>
__global__ __launch_bounds__(C::NT) void lmhead_lse_kernel(const T *__restrict__ W, const T *__restrict__ F,
                                                          int V, int R, int K, int tiles_per_split,
                                                          float *__restrict__ part_m, float *__restrict__ part_s) {
  extern __shared__ uint4 lds[];
  const int n0 = blockIdx.x * C::BN, split = blockIdx.y;
  const int ntiles = (V + C::BM - 1) / C::BM;
  const int vt0 = split * tiles_per_split, vt1 = min(vt0 + tiles_per_split, ntiles);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  float rm[C::NI], rs[C::NI];
#pragma unroll
  for (int j = 0; j < C::NI; ++j) { rm[j] = -INFINITY; rs[j] = 0.0f; }
  f32x16 acc[C::MI][C::NI];
  for (int vt = vt0; vt < vt1; ++vt) {
    const int m0 = vt * C::BM;
    gemm_tile<T, C>(W, K, F, K, V, R, K, m0, n0, lds, acc);
#pragma unroll
    for (int j = 0; j < C::NI; ++j) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < C::MI; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int v = m0 + wm * C::WM + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          const float z = v < V ? acc[i][j][e] * kLog2e : -INFINITY;
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
  // merge the two lane halves that hold the same column
  float *sm = reinterpret_cast<float *>(lds);  // [WAVES_M][BN] maxima, then sums
#pragma unroll
  for (int j = 0; j < C::NI; ++j) {
    const float om = __shfl_xor(rm[j], 32), os = __shfl_xor(rs[j], 32);
    const float nm = fmaxf(rm[j], om);
    float s = 0.0f;
    if (nm != -INFINITY) s = rs[j] * exp2f(rm[j] - nm) + os * exp2f(om - nm);
    rm[j] = nm;
    rs[j] = s;
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
      for (int w = 0; w < C::WAVES_M; ++w) S += sm[C::WAVES_M * C::BN + w * C::BN + cl] * exp2f(sm[w * C::BN + cl] - M);
    part_m[(int64_t)split * R + row] = M;
    part_s[(int64_t)split * R + row] = S;
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

using CfgB = Cfg<bf16, 128, 128, 64, 64>;
using CfgF = Cfg<float, 128, 128, 64, 64>;

template <typename T, class C, int EPI>
static hipError_t run_gemm(const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N, int K,
                           void *out, int64_t ldo, hipStream_t st) {
  GemmArgs<T> g{(const T *)A, (const T *)B, lda, ldb, M, N, K, out, ldo};
  dim3 grid((N + C::BN - 1) / C::BN, (M + C::BM - 1) / C::BM);
  const size_t lds = sizeof(uint4) * 2 * C::BUF;
  hipLaunchKernelGGL((gemm_kernel<T, C, EPI>), grid, dim3(C::NT), lds, st, g);
  return hipGetLastError();
}

int gemm_k_step(int dtype) { return dtype == 0 ? CfgB::BK : CfgF::BK; }
int gemm_n_step(int) { return 64; }

hipError_t launch_gemm(int dtype, int epi, const void *A, int64_t lda, const void *B, int64_t ldb, int M,
                       int N, int K, void *out, int64_t ldo, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (dtype == 0) {
    switch (epi) {
      case EPI_STORE_F32: return run_gemm<bf16, CfgB, 0>(A, lda, B, ldb, M, N, K, out, ldo, st);
      case EPI_RESID_ADD: return run_gemm<bf16, CfgB, 1>(A, lda, B, ldb, M, N, K, out, ldo, st);
      case EPI_SWIGLU: return run_gemm<bf16, CfgB, 2>(A, lda, B, ldb, M, N, K, out, ldo, st);
      default: return run_gemm<bf16, CfgB, 3>(A, lda, B, ldb, M, N, K, out, ldo, st);
    }
  }
  switch (epi) {
    case EPI_STORE_F32: return run_gemm<float, CfgF, 0>(A, lda, B, ldb, M, N, K, out, ldo, st);
    case EPI_RESID_ADD: return run_gemm<float, CfgF, 1>(A, lda, B, ldb, M, N, K, out, ldo, st);
    case EPI_SWIGLU: return run_gemm<float, CfgF, 2>(A, lda, B, ldb, M, N, K, out, ldo, st);
    default: return run_gemm<float, CfgF, 3>(A, lda, B, ldb, M, N, K, out, ldo, st);
  }
}

int lmhead_tile_rows(int) { return 128; }

int lmhead_num_splits(int V, int tiles_per_split) {
  const int nt = (V + 127) / 128;
  return (nt + tiles_per_split - 1) / tiles_per_split;
}

hipError_t launch_lmhead_lse(int dtype, const void *W, const void *F, int V, int R, int K, int tiles_per_split,
                             float *part_m, float *part_s, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  const int nsplit = lmhead_num_splits(V, tiles_per_split);
  if (dtype == 0) {
    dim3 grid((R + CfgB::BN - 1) / CfgB::BN, nsplit);
    hipLaunchKernelGGL((lmhead_lse_kernel<bf16, CfgB>), grid, dim3(CfgB::NT), sizeof(uint4) * 2 * CfgB::BUF, st,
                       (const bf16 *)W, (const bf16 *)F, V, R, K, tiles_per_split, part_m, part_s);
  } else {
    dim3 grid((R + CfgF::BN - 1) / CfgF::BN, nsplit);
    hipLaunchKernelGGL((lmhead_lse_kernel<float, CfgF>), grid, dim3(CfgF::NT), sizeof(uint4) * 2 * CfgF::BUF, st,
                       (const float *)W, (const float *)F, V, R, K, tiles_per_split, part_m, part_s);
  }
  return hipGetLastError();
}

}  // namespace jetk
