// Grouped-query attention on matrix cores for gfx950.
//
// One workgroup (4 waves) takes up to 64 query slots of one (question, KV
// head): slot s is query head kvh * G + s % G at row s / G, so the G query
// heads that share a KV head share every K/V tile the workgroup stages in
// LDS, a block's rows lie within 64 / G of each other (causal prefix blocks
// stop at nearly the same key), and consecutive lanes read consecutive heads
// of one row of Q and O. Two modes:
//   mode 0, prefix prefill: query i of a question sees prefix keys 0..i.
//   mode 1, candidates: a candidate row sees every key of its question's
//     retained prefix (read-only, staged once per tile for all the slots),
//     then the rows of its own candidate up to itself, and nothing of its
//     siblings, so candidates stay isolated (Section 4.1). The own rows (at
//     most m - 1) are staged as extra tiles aligned to each candidate's first
//     row, so a candidate's score does not depend on where it sits in the
//     batch: candidates with equal text get bitwise-equal scores and the
//     fixed tie order decides between them (Section 3.3).
// Scores are computed transposed, S^T = K Q^T with 16x16x32 MFMAs, so each
// lane owns one query column; the online softmax runs in base 2 and the
// probabilities feed O^T += V^T P^T directly from registers. V is staged
// transposed in LDS (4-key units, XOR-swizzled by d) for that product.
//
// PAIR: q, K, V and the output are (hi, lo) bf16 pairs (value = hi + lo);
// products use hi*hi + lo*hi + hi*lo (the lo*lo term is below fp32 rounding
// of the sum), and the probabilities are split into a pair the same way.
#include "device.h"
#include "kernels.h"

namespace jetk {

template <typename T> __device__ __forceinline__ Frag<T> pack8(const float (&x)[8]) {
  static_assert(sizeof(T) == 2, "16-bit types");
  Frag<T> f;
  const uint4 u = make_uint4(pack2<T>(x[0], x[1]), pack2<T>(x[2], x[3]), pack2<T>(x[4], x[5]), pack2<T>(x[6], x[7]));
  f.v = __builtin_bit_cast(typename Vec8<T>::type, u);
  return f;
}
template <> __device__ __forceinline__ Frag<float> pack8<float>(const float (&x)[8]) {
  Frag<float> f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f.v[j] = x[j];
  return f;
}

template <typename T>
__device__ __forceinline__ void lds_kfrag(Frag<T> &f, const uint4 *row, int c0, int swz) {
  static_assert(sizeof(T) == 2, "16-bit types");
  f.v = __builtin_bit_cast(typename Vec8<T>::type, row[c0 ^ swz]);
}
template <>
__device__ __forceinline__ void lds_kfrag<float>(Frag<float> &f, const uint4 *row, int c0, int swz) {
  const uint4 u0 = row[c0 ^ swz], u1 = row[(c0 + 1) ^ swz];
  f.v[0] = __uint_as_float(u0.x); f.v[1] = __uint_as_float(u0.y);
  f.v[2] = __uint_as_float(u0.z); f.v[3] = __uint_as_float(u0.w);
  f.v[4] = __uint_as_float(u1.x); f.v[5] = __uint_as_float(u1.y);
  f.v[6] = __uint_as_float(u1.z); f.v[7] = __uint_as_float(u1.w);
}

// Transposed V tile: row d holds the KT keys of dim d. Key k = 32 mm + 16 h +
// 4 g + e (mm, h in {0, 1}, g, e in 0..3) sits at position 32 mm + 8 g + 4 h + e,
// so the 8 keys one lane of lane group g needs for the PV product (the keys
// of its probabilities, 32 mm + 4 g + e and 32 mm + 16 + 4 g + e) are one
// contiguous 16-byte (bf16) or 32-byte (fp32) run; 16-byte units are
// XOR-swizzled by d so the 16 lanes of a group (16 consecutive d) hit
// distinct banks.
__device__ __forceinline__ int vt_unit(const bf16 *, int unit, int d) { return unit ^ ((d >> 1) & 7); }
__device__ __forceinline__ int vt_unit(const f16 *, int unit, int d) { return unit ^ ((d >> 1) & 7); }
__device__ __forceinline__ int vt_unit(const float *, int unit, int d) { return unit ^ (d & 15); }

// Writes 4 keys 4u..4u+3 (rows r[0..3], one 16-byte chunk c of dims each).
template <int KT, typename T>
__device__ __forceinline__ void v_put_transposed(T *vt, const uint4 (&r)[4], int u, int c) {
  static_assert(sizeof(T) == 2, "16-bit types");
  const uint32_t *w0 = reinterpret_cast<const uint32_t *>(&r[0]), *w1 = reinterpret_cast<const uint32_t *>(&r[1]);
  const uint32_t *w2 = reinterpret_cast<const uint32_t *>(&r[2]), *w3 = reinterpret_cast<const uint32_t *>(&r[3]);
  const int unit = 4 * (u >> 3) + (u & 3), half = ((u >> 2) & 1) * 4;  // 8-element unit, 4-key half
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int d = c * 8 + j;
    const int sh = (j & 1) * 16;
    const uint32_t e0 = (w0[j >> 1] >> sh) & 0xffffu, e1 = (w1[j >> 1] >> sh) & 0xffffu;
    const uint32_t e2 = (w2[j >> 1] >> sh) & 0xffffu, e3 = (w3[j >> 1] >> sh) & 0xffffu;
    *reinterpret_cast<uint2 *>(vt + d * KT + (vt_unit(vt, unit, d) << 3) + half) =
        make_uint2(e0 | (e1 << 16), e2 | (e3 << 16));
  }
}
template <int KT>
__device__ __forceinline__ void v_put_transposed(float *vt, const uint4 (&r)[4], int u, int c) {
  const int unit = 8 * (u >> 3) + 2 * (u & 3) + ((u >> 2) & 1);  // 4-element unit
  const uint32_t *w0 = reinterpret_cast<const uint32_t *>(&r[0]), *w1 = reinterpret_cast<const uint32_t *>(&r[1]);
  const uint32_t *w2 = reinterpret_cast<const uint32_t *>(&r[2]), *w3 = reinterpret_cast<const uint32_t *>(&r[3]);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int d = c * 4 + j;
    *reinterpret_cast<uint4 *>(vt + d * KT + (vt_unit(vt, unit, d) << 2)) = make_uint4(w0[j], w1[j], w2[j], w3[j]);
  }
}

// PV operand of lane group g for dim d and key half mm (see the layout above).
template <int KT, typename T>
__device__ __forceinline__ void v_frag(Frag<T> &f, const T *vt, int d, int mm, int g) {
  static_assert(sizeof(T) == 2, "16-bit types");
  f.v = __builtin_bit_cast(typename Vec8<T>::type,
                           *reinterpret_cast<const uint4 *>(vt + d * KT + (vt_unit(vt, 4 * mm + g, d) << 3)));
}
template <int KT>
__device__ __forceinline__ void v_frag(Frag<float> &f, const float *vt, int d, int mm, int g) {
  const int unit = 8 * mm + 2 * g;
  const uint4 a = *reinterpret_cast<const uint4 *>(vt + d * KT + (vt_unit(vt, unit, d) << 2));
  const uint4 b = *reinterpret_cast<const uint4 *>(vt + d * KT + (vt_unit(vt, unit + 1, d) << 2));
  f.v[0] = __uint_as_float(a.x); f.v[1] = __uint_as_float(a.y); f.v[2] = __uint_as_float(a.z); f.v[3] = __uint_as_float(a.w);
  f.v[4] = __uint_as_float(b.x); f.v[5] = __uint_as_float(b.y); f.v[6] = __uint_as_float(b.z); f.v[7] = __uint_as_float(b.w);
}

// QB blocks of 16 query slots per wave (64 QB per workgroup): every K and V
// fragment read from LDS feeds QB MFMAs, and every staged tile serves 64 QB
// queries.
template <typename T, int HD, int MODE, bool PAIR, int QB>
__global__ __launch_bounds__(256, 2) void attn_kernel(AttnArgs a) {
  constexpr int KT = 64;                        // keys per tile
  constexpr int EPC = 16 / (int)sizeof(T);      // elements per 16-byte chunk
  constexpr int CPR = HD / EPC;                 // chunks per K row
  constexpr int KSW = CPR < 16 ? CPR : 16;      // XOR range of the K-row swizzle
  constexpr int NP = PAIR ? 2 : 1;              // planes: hi (and lo)
  __shared__ uint4 Ks[NP][KT * CPR];
  __shared__ __align__(16) T Vt[NP][HD * KT];

  const AttnItem it = a.items[blockIdx.x];
  const int G = a.Hq / a.Hkv;
  const int qrow0 = a.qs.qrow0[it.q];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4;
  bool valid[QB];
  int head[QB], qi[QB], row[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int sl = (wave * QB + qb) * 16 + (lane & 15);
    valid[qb] = sl < it.nslots;
    const int slot = it.slot0 + (valid[qb] ? sl : 0);
    head[qb] = it.kvh * G + slot % G;
    qi[qb] = slot / G;
    row[qb] = qrow0 + qi[qb];
  }
  const T *Q = (const T *)a.Q;

  Frag<T> qf[QB][NP][HD / 32];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) {
        if (valid[qb])
          frag_load(qf[qb][p][ks], Q + p * a.q_ps + ((int64_t)row[qb] * a.Hq + head[qb]) * HD + ks * 32 + g * 8);
        else qf[qb][p][ks].zero();
      }
  int my_t[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) my_t[qb] = (MODE == 1 && valid[qb]) ? a.row_t[row[qb]] : 0;

  const float scale2 = a.scale * kLog2e;
  float m_run[QB], l_run[QB];
  f32x4 acc[QB][HD / 16];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = -INFINITY;
    l_run[qb] = 0.0f;
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) acc[qb][d] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  }

  const T *Kp = (const T *)a.Kp, *Vp = (const T *)a.Vp;
  const int64_t pslot = a.qs.pre_slot0[it.q];
  const int npre = MODE == 0 ? it.nkeys_pre : a.qs.pre_len[it.q];
  const int ntile = (npre + KT - 1) / KT;

  // Tiles are software-pipelined: the global loads of tile t + 1 are issued
  // into registers before the MFMAs of tile t and written to LDS after them.
  // Loads always read a valid row (key clamped into the tile); keys beyond
  // the tile are zeroed when the registers are written to LDS, so no load
  // sits in a divergent branch or waits early.
  constexpr int NKC = (KT * CPR + 255) / 256;        // K chunks per thread
  constexpr int NVB = ((KT / 4) * CPR + 255) / 256;  // V 4-key blocks per thread
  constexpr bool KFULL = (KT * CPR) % 256 == 0, VFULL = ((KT / 4) * CPR) % 256 == 0;
  uint4 kreg[NP][NKC], vreg[NP][NVB][4];
  const int64_t ps = a.kp_ps;
  const T *kvbase_k = Kp + ((int64_t)it.kvh * a.s_pre + pslot) * HD;
  const T *kvbase_v = Vp + ((int64_t)it.kvh * a.s_pre + pslot) * HD;
  // loads of rows kb .. kb + nkt - 1 of a [rows][HD] K / V plane pair (plane stride pstride)
  auto issue_tile = [&](const T *kbase_p, const T *vbase_p, int64_t pstride, int kb, int nkt) {
#pragma unroll
    for (int i = 0; i < NKC; ++i) {
      const int ch = tid + i * 256, key = min(ch / CPR, nkt - 1), c = ch % CPR;
#pragma unroll
      for (int p = 0; p < NP; ++p) kreg[p][i] = ld16(kbase_p + p * pstride + (int64_t)(kb + key) * HD + c * EPC);
    }
#pragma unroll
    for (int i = 0; i < NVB; ++i) {
      const int bk = tid + i * 256, u = bk % (KT / 4), c = min(bk / (KT / 4), CPR - 1);
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          vreg[p][i][e] = ld16(vbase_p + p * pstride + (int64_t)(kb + min(4 * u + e, nkt - 1)) * HD + c * EPC);
    }
  };
  // the loaded tile into LDS (keys nk .. KT - 1 zeroed): K as 16-byte
  // chunks, row-swizzled; V transposed: a thread takes 4 keys x one 16-byte
  // chunk of dims and writes each dim's 4 keys as one store; the 16 threads
  // of a group take the 16 key quads of one chunk, so each store of the group
  // fills one 128-byte row of Vt (distinct banks)
  auto store_tile = [&](int nk) {
    const bool tile_full = nk == KT;  // uniform: no key of the tile to zero
#pragma unroll
    for (int i = 0; i < NKC; ++i) {
      const int ch = tid + i * 256, key = ch / CPR, c = ch % CPR;
      if (KFULL || ch < KT * CPR) {
        const bool ok = tile_full || key < nk;
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const uint4 v = kreg[p][i];
          Ks[p][key * CPR + (c ^ (key & (KSW - 1)))] =
              make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < NVB; ++i) {
      const int bk = tid + i * 256, u = bk % (KT / 4), c = bk / (KT / 4);
      if (VFULL || bk < (KT / 4) * CPR) {
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          uint4 r[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool ok = tile_full || 4 * u + e < nk;
            const uint4 v = vreg[p][i][e];
            r[e] = make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
          }
          v_put_transposed<KT>(&Vt[p][0], r, u, c);
        }
      }
    }
  };
  // Scores of the staged tile (keys 0 .. nk - 1), online softmax and the PV
  // product. all_visible(qb): every key of the tile is visible to every
  // query of the wave's block qb (uniform); visible(qb, key): key of the
  // tile is visible to this lane's query of block qb. Groups of 16 keys past
  // nk are skipped: their scores are masked and their products with the
  // zeroed V rows add exact zeros.
  auto tile_compute = [&](int nk, auto all_visible, auto visible) {
    f32x4 s[QB][4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) s[qb][kb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      if (kb * 16 >= nk) continue;
      const int key = kb * 16 + (lane & 15);
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) {
        const int c0 = (ks * 32 + g * 8) / EPC;
        Frag<T> fk;
        lds_kfrag<T>(fk, &Ks[0][key * CPR], c0, key & (KSW - 1));
        Frag<T> fkl;
        if constexpr (PAIR) lds_kfrag<T>(fkl, &Ks[NP - 1][key * CPR], c0, key & (KSW - 1));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          mma16(s[qb][kb], fk, qf[qb][0][ks]);
          if constexpr (PAIR) {
            mma16(s[qb][kb], fkl, qf[qb][0][ks]);
            mma16(s[qb][kb], fk, qf[qb][NP - 1][ks]);
          }
        }
      }
    }
    Frag<T> pf[QB][2], pfl[QB][2];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = -INFINITY;
      if (all_visible(qb)) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            s[qb][kb][e] *= scale2;
            mx = fmaxf(mx, s[qb][kb][e]);
          }
      } else {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float z = visible(qb, kb * 16 + 4 * g + e) ? s[qb][kb][e] * scale2 : -INFINITY;
            s[qb][kb][e] = z;
            mx = fmaxf(mx, z);
          }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      // Every query sees key 0 in the first tile (mode 0) or the whole prefix
      // (mode 1, before any own-key tile), so m_new is finite: exp2 of the
      // (<= 0) differences directly, with exp2(-inf) = 0 for masked keys and
      // for the initial m_run. A tile with no key visible to a query leaves
      // its m_run, l_run and acc bitwise unchanged (alpha = 1, p = 0).
      const float m_new = fmaxf(m_run[qb], mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
      float p[4][4];
      float psum = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          p[kb][e] = __builtin_amdgcn_exp2f(s[qb][kb][e] - m_new);
          psum += p[kb][e];
        }
      l_run[qb] = l_run[qb] * alpha + psum;
      if (__any(alpha != 1.0f)) {
#pragma unroll
        for (int d = 0; d < HD / 16; ++d) acc[qb][d] *= alpha;
      }
      m_run[qb] = m_new;
#pragma unroll
      for (int mm = 0; mm < 2; ++mm) {
        const float x8[8] = {p[2 * mm][0], p[2 * mm][1], p[2 * mm][2], p[2 * mm][3],
                             p[2 * mm + 1][0], p[2 * mm + 1][1], p[2 * mm + 1][2], p[2 * mm + 1][3]};
        pf[qb][mm] = pack8<T>(x8);
        if constexpr (PAIR) {
          float r8[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) r8[j] = x8[j] - (float)pf[qb][mm].v[j];
          pfl[qb][mm] = pack8<T>(r8);
        }
      }
    }
#pragma unroll
    for (int mm = 0; mm < 2; ++mm) {
      if (mm * 32 >= nk) continue;
#pragma unroll
      for (int db = 0; db < HD / 16; ++db) {
        const int d = db * 16 + (lane & 15);
        Frag<T> fv, fvl;
        v_frag<KT>(fv, &Vt[0][0], d, mm, g);
        if constexpr (PAIR) v_frag<KT>(fvl, &Vt[NP - 1][0], d, mm, g);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          mma16(acc[qb][db], fv, pf[qb][mm]);
          if constexpr (PAIR) {
            mma16(acc[qb][db], fvl, pf[qb][mm]);
            mma16(acc[qb][db], fv, pfl[qb][mm]);
          }
        }
      }
    }
  };

  if (ntile > 0) issue_tile(kvbase_k, kvbase_v, ps, 0, min(KT, npre));
  for (int tix = 0; tix < ntile; ++tix) {
    const int kbase = tix * KT;
    const int nk = min(KT, npre - kbase);
    __syncthreads();
    store_tile(nk);
    __syncthreads();
    if (tix + 1 < ntile) issue_tile(kvbase_k, kvbase_v, ps, kbase + KT, min(KT, npre - kbase - KT));
    const bool tile_full = nk == KT;
    // tiles every key of which every query of the wave's block sees skip the mask
    tile_compute(nk, [&](int qb) { return __all(tile_full && (MODE != 0 || kbase + KT - 1 <= qi[qb])); },
                 [&](int qb, int key) { return key < nk && (MODE != 0 || kbase + key <= qi[qb]); });
  }

  if constexpr (MODE == 1) {
    // Own keys of the candidates: the item's rows r_first .. r_last are
    // consecutive body rows of the call, ordered by candidate, then
    // position. Each candidate's keys are staged in tiles that start at its
    // first body row (key j of the tile = its row first + 64 i + j), and a
    // query sees only the tiles of its own candidate (rows up to itself):
    // the tile a query reads and the position of each key in it do not
    // depend on which other candidates share the batch or the item, so a
    // candidate rounds alike alone and among its siblings (Section 3.3: equal
    // text, equal score). Tiles of other candidates leave a query unchanged.
    if (a.s_suf > 0) {
      const int r_first = qrow0 + it.slot0 / G;
      const int r_last = qrow0 + (it.slot0 + it.nslots - 1) / G;
      const T *kown = (const T *)a.Ks + (int64_t)it.kvh * a.s_suf * HD;
      const T *vown = (const T *)a.Vs + (int64_t)it.kvh * a.s_suf * HD;
      int first[QB];  // first body row of this lane's query's candidate
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) first[qb] = valid[qb] ? row[qb] - my_t[qb] + 1 : -1;
      int cs = r_first - a.row_t[r_first] + 1;
      while (cs <= r_last) {
        const int cend = min(cs + a.row_n[cs] - 1, r_last);  // keys after r_last have no query here
        for (int ts = cs; ts <= cend; ts += KT) {
          const int nk = min(KT, cend - ts + 1);
          __syncthreads();
          issue_tile(kown, vown, a.ks_ps, ts, nk);
          store_tile(nk);
          __syncthreads();
          tile_compute(nk, [&](int) { return false; },
                       [&](int qb, int key) { return key < nk && first[qb] == cs && ts + key <= row[qb]; });
        }
        cs += a.row_n[cs];
      }
    }
  }

#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (valid[qb]) {
      const float inv = 1.0f / l_tot;
      T *O = (T *)a.O;
#pragma unroll
      for (int db = 0; db < HD / 16; ++db) {
        // dims 16 db + 4 g .. + 3 of this lane's query, one 8- (bf16) or 16-byte (fp32) store per plane
        float o[4], lo[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = acc[qb][db][e] * inv;
        T *dst = O + (int64_t)row[qb] * a.o_ld + (int64_t)head[qb] * HD + db * 16 + 4 * g;
        if constexpr (sizeof(T) == 2) {
          const uint2 hi = make_uint2(pack2<T>(o[0], o[1]), pack2<T>(o[2], o[3]));
          *reinterpret_cast<uint2 *>(dst) = hi;
          if constexpr (PAIR) {
#pragma unroll
            for (int e = 0; e < 4; ++e) lo[e] = o[e] - to_f<T>(from_f<T>(o[e]));
            *reinterpret_cast<uint2 *>(dst + (int64_t)a.Hq * HD) =
                make_uint2(pack2<T>(lo[0], lo[1]), pack2<T>(lo[2], lo[3]));
          }
        } else {
          *reinterpret_cast<float4 *>(dst) = make_float4(o[0], o[1], o[2], o[3]);
        }
      }
    }
  }
}

// Query blocks per wave: two for single 16-bit planes, one for (hi, lo)
// pairs and fp32 (their fragments take twice the registers).
template <typename T, bool PAIR>
constexpr int attn_qb() {
  return sizeof(T) == 2 && !PAIR ? 2 : 1;
}

int attn_slots_per_item(int dtype, int pair) { return (dtype == 1 || pair) ? 64 : 128; }

template <typename T, int HD, bool PAIR, int QB>
static hipError_t run_attn_qb(const AttnArgs &a, hipStream_t st) {
  if (a.mode == 0) hipLaunchKernelGGL((attn_kernel<T, HD, 0, PAIR, QB>), dim3(a.n_items), dim3(256), 0, st, a);
  else hipLaunchKernelGGL((attn_kernel<T, HD, 1, PAIR, QB>), dim3(a.n_items), dim3(256), 0, st, a);
  return hipGetLastError();
}

template <typename T, int HD, bool PAIR>
static hipError_t run_attn(const AttnArgs &a, hipStream_t st) {
  constexpr int QB = attn_qb<T, PAIR>();
  if (a.n_items <= 0) return hipSuccess;
  if (a.qb < 1 || a.qb > QB) return hipErrorInvalidValue;
  if constexpr (QB == 2) {
    if (a.qb == 2) return run_attn_qb<T, HD, PAIR, 2>(a, st);
  }
  return run_attn_qb<T, HD, PAIR, 1>(a, st);
}

hipError_t launch_attention(int dtype, const AttnArgs &a, hipStream_t st) {
  if (dtype == 0) {
    if (a.pair) {
      if (a.hd == 128) return run_attn<bf16, 128, true>(a, st);
      if (a.hd == 64) return run_attn<bf16, 64, true>(a, st);
      if (a.hd == 32) return run_attn<bf16, 32, true>(a, st);
    } else {
      if (a.hd == 128) return run_attn<bf16, 128, false>(a, st);
      if (a.hd == 64) return run_attn<bf16, 64, false>(a, st);
      if (a.hd == 32) return run_attn<bf16, 32, false>(a, st);
    }
  } else if (dtype == 2) {
    if (a.pair) {
      if (a.hd == 128) return run_attn<f16, 128, true>(a, st);
      if (a.hd == 64) return run_attn<f16, 64, true>(a, st);
      if (a.hd == 32) return run_attn<f16, 32, true>(a, st);
      return hipErrorInvalidValue;
    }
    if (a.hd == 128) return run_attn<f16, 128, false>(a, st);
    if (a.hd == 64) return run_attn<f16, 64, false>(a, st);
    if (a.hd == 32) return run_attn<f16, 32, false>(a, st);
  } else {
    if (a.hd == 128) return run_attn<float, 128, false>(a, st);
    if (a.hd == 64) return run_attn<float, 64, false>(a, st);
    if (a.hd == 32) return run_attn<float, 32, false>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace jetk
