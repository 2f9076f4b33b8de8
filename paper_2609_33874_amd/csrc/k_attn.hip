// Grouped-query attention on matrix cores for gfx950.
//
// One workgroup (4 waves) takes up to 64 query slots of one (question, KV
// head): slot s is query head kvh * G + s / nrows at row s % nrows, so the
// G query heads that share a KV head share every K/V tile the workgroup stages
// in LDS. Two modes:
//   mode 0, prefix prefill: query i of a question sees prefix keys 0..i.
//   mode 1, candidates: a candidate row sees every key of its question's
//     retained prefix (read-only, staged once per tile for all the slots),
//     then the rows of its own candidate up to itself, and nothing of its
//     siblings, so candidates stay isolated (Section 4.1). The own rows (at
//     most m - 1) are walked per query in a fixed order with fp32 FMAs, so a
//     candidate's score does not depend on where it sits in the batch:
//     candidates with equal text get bitwise-equal scores and the fixed
//     tie order decides between them (Section 3.3).
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

template <typename T> __device__ __forceinline__ Frag<T> pack8(const float (&x)[8]);
template <> __device__ __forceinline__ Frag<bf16> pack8<bf16>(const float (&x)[8]) {
  Frag<bf16> f;
  uint4 u;
  u.x = (uint32_t)f2bf(x[0]) | ((uint32_t)f2bf(x[1]) << 16);
  u.y = (uint32_t)f2bf(x[2]) | ((uint32_t)f2bf(x[3]) << 16);
  u.z = (uint32_t)f2bf(x[4]) | ((uint32_t)f2bf(x[5]) << 16);
  u.w = (uint32_t)f2bf(x[6]) | ((uint32_t)f2bf(x[7]) << 16);
  f.v = __builtin_bit_cast(bf16x8, u);
  return f;
}
template <> __device__ __forceinline__ Frag<float> pack8<float>(const float (&x)[8]) {
  Frag<float> f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f.v[j] = x[j];
  return f;
}

// Four consecutive elements from LDS into lanes j0..j0+3 of a fragment.
__device__ __forceinline__ void frag_put4(Frag<bf16> &f, const bf16 *p, int j0) {
  const uint2 u = *reinterpret_cast<const uint2 *>(p);
  bf16x8 v = f.v;
  const __bf16 *h = reinterpret_cast<const __bf16 *>(&u);
  v[j0 + 0] = h[0]; v[j0 + 1] = h[1]; v[j0 + 2] = h[2]; v[j0 + 3] = h[3];
  f.v = v;
}
__device__ __forceinline__ void frag_put4(Frag<float> &f, const float *p, int j0) {
  const uint4 u = *reinterpret_cast<const uint4 *>(p);
  f.v[j0 + 0] = __uint_as_float(u.x); f.v[j0 + 1] = __uint_as_float(u.y);
  f.v[j0 + 2] = __uint_as_float(u.z); f.v[j0 + 3] = __uint_as_float(u.w);
}

template <typename T>
__device__ __forceinline__ void lds_kfrag(Frag<T> &f, const uint4 *row, int c0, int swz);
template <>
__device__ __forceinline__ void lds_kfrag<bf16>(Frag<bf16> &f, const uint4 *row, int c0, int swz) {
  f.v = __builtin_bit_cast(bf16x8, row[c0 ^ swz]);
}
template <>
__device__ __forceinline__ void lds_kfrag<float>(Frag<float> &f, const uint4 *row, int c0, int swz) {
  const uint4 u0 = row[c0 ^ swz], u1 = row[(c0 + 1) ^ swz];
  f.v[0] = __uint_as_float(u0.x); f.v[1] = __uint_as_float(u0.y);
  f.v[2] = __uint_as_float(u0.z); f.v[3] = __uint_as_float(u0.w);
  f.v[4] = __uint_as_float(u1.x); f.v[5] = __uint_as_float(u1.y);
  f.v[6] = __uint_as_float(u1.z); f.v[7] = __uint_as_float(u1.w);
}

template <typename T, int HD, int MODE, bool PAIR>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  constexpr int KT = 64;                        // keys per tile
  constexpr int EPC = 16 / (int)sizeof(T);      // elements per 16-byte chunk
  constexpr int CPR = HD / EPC;                 // chunks per K row
  constexpr int KSW = CPR < 16 ? CPR : 16;      // XOR range of the K-row swizzle
  constexpr int NP = PAIR ? 2 : 1;              // planes: hi (and lo)
  __shared__ uint4 Ks[NP][KT * CPR];
  __shared__ T Vt[NP][HD * KT];

  const AttnItem it = a.items[blockIdx.x];
  const int G = a.Hq / a.Hkv;
  const int nrows = a.qs.nrows[it.q], qrow0 = a.qs.qrow0[it.q];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4;
  const int sl = wave * 16 + (lane & 15);
  const bool valid = sl < it.nslots;
  const int slot = it.slot0 + (valid ? sl : 0);
  const int head = it.kvh * G + slot / nrows;
  const int qi = slot % nrows;
  const int row = qrow0 + qi;
  const T *Q = (const T *)a.Q;

  Frag<T> qf[NP][HD / 32];
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      if (valid) frag_load(qf[p][ks], Q + p * a.q_ps + ((int64_t)row * a.Hq + head) * HD + ks * 32 + g * 8);
      else qf[p][ks].zero();
    }
  int my_t = 0;
  if (MODE == 1 && valid) my_t = a.row_t[row];

  const float scale2 = a.scale * kLog2e;
  float m_run = -INFINITY, l_run = 0.0f;
  f32x4 acc[HD / 16];
#pragma unroll
  for (int d = 0; d < HD / 16; ++d) acc[d] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  const T *Kp = (const T *)a.Kp, *Vp = (const T *)a.Vp;
  const int64_t pslot = a.qs.pre_slot0[it.q];
  const int npre = MODE == 0 ? it.nkeys_pre : a.qs.pre_len[it.q];
  const int ntile = (npre + KT - 1) / KT;

  for (int tix = 0; tix < ntile; ++tix) {
    const int kbase = tix * KT;
    const int nk = min(KT, npre - kbase);
    const int64_t off = ((int64_t)it.kvh * a.s_pre + pslot + kbase) * HD;
    const T *Kb = Kp + off, *Vb = Vp + off;
    const int64_t ps = a.kp_ps;
    __syncthreads();
    for (int ch = tid; ch < KT * CPR; ch += 256) {
      const int key = ch / CPR, c = ch % CPR;
      const int u = key >> 2;
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
        if (key < nk) {
          kv = ld16(Kb + p * ps + (int64_t)key * HD + c * EPC);
          vv = ld16(Vb + p * ps + (int64_t)key * HD + c * EPC);
        }
        Ks[p][key * CPR + (c ^ (key & (KSW - 1)))] = kv;
        const T *ve = reinterpret_cast<const T *>(&vv);
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
          const int d = c * EPC + e;
          Vt[p][d * KT + ((u ^ (d & 15)) << 2) + (key & 3)] = ve[e];
        }
      }
    }
    __syncthreads();

    f32x4 s[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      s[kb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      const int key = kb * 16 + (lane & 15);
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) {
        const int c0 = (ks * 32 + g * 8) / EPC;
        Frag<T> fk;
        lds_kfrag<T>(fk, &Ks[0][key * CPR], c0, key & (KSW - 1));
        mma16(s[kb], fk, qf[0][ks]);
        if constexpr (PAIR) {
          Frag<T> fkl;
          lds_kfrag<T>(fkl, &Ks[NP - 1][key * CPR], c0, key & (KSW - 1));
          mma16(s[kb], fkl, qf[0][ks]);
          mma16(s[kb], fk, qf[NP - 1][ks]);
        }
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = kb * 16 + 4 * g + e;
        bool vis = key < nk;
        if (MODE == 0) vis = vis && (kbase + key <= qi);
        const float z = vis ? s[kb][e] * scale2 : -INFINITY;
        s[kb][e] = z;
        mx = fmaxf(mx, z);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_new == -INFINITY) ? 1.0f : exp2f(m_run - m_new);
    float p[4][4];
    float psum = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float z = s[kb][e];
        p[kb][e] = (z == -INFINITY) ? 0.0f : exp2f(z - m_new);
        psum += p[kb][e];
      }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) acc[d] *= alpha;
    m_run = m_new;
#pragma unroll
    for (int mm = 0; mm < 2; ++mm) {
      const float x8[8] = {p[2 * mm][0], p[2 * mm][1], p[2 * mm][2], p[2 * mm][3],
                           p[2 * mm + 1][0], p[2 * mm + 1][1], p[2 * mm + 1][2], p[2 * mm + 1][3]};
      const Frag<T> pf = pack8<T>(x8);
      Frag<T> pfl;
      if constexpr (PAIR) {
        float r8[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) r8[j] = x8[j] - (float)pf.v[j];
        pfl = pack8<T>(r8);
      }
      const int u1 = 8 * mm + g, u2 = u1 + 4;
#pragma unroll
      for (int db = 0; db < HD / 16; ++db) {
        const int d = db * 16 + (lane & 15);
        Frag<T> fv;
        frag_put4(fv, &Vt[0][d * KT + ((u1 ^ (d & 15)) << 2)], 0);
        frag_put4(fv, &Vt[0][d * KT + ((u2 ^ (d & 15)) << 2)], 4);
        mma16(acc[db], fv, pf);
        if constexpr (PAIR) {
          Frag<T> fvl;
          frag_put4(fvl, &Vt[NP - 1][d * KT + ((u1 ^ (d & 15)) << 2)], 0);
          frag_put4(fvl, &Vt[NP - 1][d * KT + ((u2 ^ (d & 15)) << 2)], 4);
          mma16(acc[db], fvl, pf);
          mma16(acc[db], fv, pfl);
        }
      }
    }
  }

  if constexpr (MODE == 1) {
    // own rows of the candidate: row - my_t + 1 .. row of the call's K / V
    // (rows are ordered by candidate, then position). Lane group g holds the
    // query dims 32 ks + 8 g + j (score) and the output dims 16 db + 4 g + e.
    float qv[HD / 32][8];
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float v = to_f<T>(reinterpret_cast<const T *>(&qf[0][ks].v)[j]);
        if constexpr (PAIR) v += to_f<T>(reinterpret_cast<const T *>(&qf[NP - 1][ks].v)[j]);
        qv[ks][j] = v;
      }
    int tmax = valid ? my_t : 0;
    for (int o = 1; o < 64; o <<= 1) tmax = max(tmax, __shfl_xor(tmax, o));
    const T *Kc = (const T *)a.Ks + (int64_t)it.kvh * a.s_suf * HD;
    const T *Vc = (const T *)a.Vs + (int64_t)it.kvh * a.s_suf * HD;
    for (int i = 0; i < tmax; ++i) {
      const bool act = valid && i < my_t;
      const int64_t krow = (int64_t)row - my_t + 1 + i;
      float part = 0.0f;
      if (act) {
        const T *kr = Kc + krow * HD;
#pragma unroll
        for (int ks = 0; ks < HD / 32; ++ks)
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int d = ks * 32 + g * 8 + j;
            float kv = to_f<T>(kr[d]);
            if constexpr (PAIR) kv += to_f<T>(kr[a.ks_ps + d]);
            part += qv[ks][j] * kv;
          }
      }
      part += __shfl_xor(part, 16);
      part += __shfl_xor(part, 32);
      if (act) {
        const float z = part * scale2;
        const float m_new = fmaxf(m_run, z);
        const float alpha = exp2f(m_run - m_new);
        const float pz = exp2f(z - m_new);
        l_run = l_run * alpha + (g == 0 ? pz : 0.0f);
        const T *vr = Vc + krow * HD;
#pragma unroll
        for (int db = 0; db < HD / 16; ++db)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int d = db * 16 + 4 * g + e;
            float vv = to_f<T>(vr[d]);
            if constexpr (PAIR) vv += to_f<T>(vr[a.ks_ps + d]);
            acc[db][e] = acc[db][e] * alpha + pz * vv;
          }
        m_run = m_new;
      }
    }
  }

  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot += __shfl_xor(l_tot, 32);
  if (!valid) return;
  const float inv = 1.0f / l_tot;
  T *O = (T *)a.O;
#pragma unroll
  for (int db = 0; db < HD / 16; ++db)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int d = db * 16 + 4 * g + e;
      const float o = acc[db][e] * inv;
      const T hi = from_f<T>(o);
      O[(int64_t)row * a.o_ld + (int64_t)head * HD + d] = hi;
      if constexpr (PAIR) O[(int64_t)row * a.o_ld + (int64_t)(a.Hq + head) * HD + d] = from_f<T>(o - to_f<T>(hi));
    }
}

template <typename T, int HD, bool PAIR>
static hipError_t run_attn(const AttnArgs &a, hipStream_t st) {
  if (a.n_items <= 0) return hipSuccess;
  if (a.mode == 0) hipLaunchKernelGGL((attn_kernel<T, HD, 0, PAIR>), dim3(a.n_items), dim3(256), 0, st, a);
  else hipLaunchKernelGGL((attn_kernel<T, HD, 1, PAIR>), dim3(a.n_items), dim3(256), 0, st, a);
  return hipGetLastError();
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
  } else {
    if (a.hd == 128) return run_attn<float, 128, false>(a, st);
    if (a.hd == 64) return run_attn<float, 64, false>(a, st);
    if (a.hd == 32) return run_attn<float, 32, false>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace jetk
