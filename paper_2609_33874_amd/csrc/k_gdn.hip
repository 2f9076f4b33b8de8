// Gated delta-rule (linear attention) layers of the hybrid decoder, gfx950.
//
// Per head (state S of shape [dv][dk], fp32):
//   S <- alpha S;  S <- S + beta (v - S k) k^T;  o = S q
// with q, k l2-normalised (q also scaled by 1/sqrt(dk)) after a causal
// depthwise convolution of width 4 + SiLU, beta = sigmoid(b) and
// alpha = exp(-exp(A_log) softplus(a + dt_bias)); the output is
// RMSNorm(o) * w * silu(z) per head.
//
// The hybrid path keeps the prefix state and the last 3 pre-convolution rows
// of each question (Section 4.1: hybrid models maintain recurrent state that
// must be restored for every candidate). The recurrence kernel starts every
// candidate from a private register copy of its question's state snapshot and
// never writes it back, so candidates cannot see each other (the isolation
// the paper checks in Section 5.6), while all candidates run in one batch.
#include <utility>

#include "device.h"
#include "kernels.h"

namespace jetk {

// Convolution, gates and normalisation of the delta-rule inputs. x:
// projection output [R][ldx] = q~ | k~ | v~ | z | b | a. One half-wave (32
// lanes, 4 channels each) takes one group of 128 channels (one head of q~, k~
// or v~; dk = dv = 128) over a block of GDN_CONV_RB consecutive rows, walked in
// order: the inputs of the previous three rows stay in registers and are
// reused whenever a row's history names the row before it (a row of the same
// sequence), so every input element is read once. The l2 norm of a q / k head
// is a reduction over the 32 lanes of the half-wave.
constexpr int GDN_CONV_RB = 16;

__device__ __forceinline__ float4 ld4f(const float *p, bool aligned) {
  if (aligned) return *reinterpret_cast<const float4 *>(p);
  return make_float4(p[0], p[1], p[2], p[3]);
}

__device__ __forceinline__ float silu_f(float x) { return x / (1.0f + __expf(-x)); }

__global__ __launch_bounds__(256) void gdn_conv_kernel(GdnConvArgs g, int R) {
  const int H = g.H, dk = g.dk, dv = g.dv;
  const int C = 2 * H * dk + H * dv;
  const int ngroups = C / 128;
  const int hw = blockIdx.x * 8 + (threadIdx.x >> 5), lane = threadIdx.x & 31;
  const int nrb = (R + GDN_CONV_RB - 1) / GDN_CONV_RB;
  if (hw >= nrb * ngroups) return;  // no barriers or LDS below
  const int rb = hw / ngroups, cg = hw % ngroups;
  const int c = cg * 128 + lane * 4;
  const bool al = (g.ldx & 3) == 0;
  float4 w[4];  // taps of channels c .. c + 3; tap 3 multiplies the current row
#pragma unroll
  for (int e = 0; e < 4; ++e) w[e] = *reinterpret_cast<const float4 *>(g.conv_w + (int64_t)(c + e) * 4);
  const float qscale = rsqrtf((float)dk);
  const int r0 = rb * GDN_CONV_RB, r1 = min(R, r0 + GDN_CONV_RB);
  float4 win[3] = {};  // inputs of rows r - 1, r - 2, r - 3
  // row r + 1's input and history are fetched while row r is processed
  float4 xn = ld4f(g.x + (int64_t)r0 * g.ldx + c, al);
  int hn[3] = {g.hist[(int64_t)r0 * 3], g.hist[(int64_t)r0 * 3 + 1], g.hist[(int64_t)r0 * 3 + 2]};
  for (int r = r0; r < r1; ++r) {
    const float4 xc = xn;
    const int hc[3] = {hn[0], hn[1], hn[2]};
    if (r + 1 < r1) {
      xn = ld4f(g.x + (int64_t)(r + 1) * g.ldx + c, al);
#pragma unroll
      for (int j = 0; j < 3; ++j) hn[j] = g.hist[(int64_t)(r + 1) * 3 + j];
    }
    float4 src[3];
    bool has[3];
#pragma unroll
    for (int j = 1; j <= 3; ++j) {
      const int h = hc[j - 1];
      has[j - 1] = h != -1;
      if (h == r - j && r - j >= r0) src[j - 1] = win[j - 1];
      else if (h >= 0) src[j - 1] = ld4f(g.x + (int64_t)h * g.ldx + c, al);
      else if (h <= -2) src[j - 1] = *reinterpret_cast<const float4 *>(g.tail + (int64_t)(-2 - h) * C + c);
      else src[j - 1] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
    const float xv[4] = {xc.x, xc.y, xc.z, xc.w};
    float y[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float wt[4] = {w[e].x, w[e].y, w[e].z, w[e].w};
      float acc = wt[3] * xv[e];
#pragma unroll
      for (int j = 1; j <= 3; ++j) {
        const float sv[4] = {src[j - 1].x, src[j - 1].y, src[j - 1].z, src[j - 1].w};
        if (has[j - 1]) acc += wt[3 - j] * sv[e];
      }
      y[e] = silu_f(acc);
    }
    if (g.tail_slot) {
      const int ts = g.tail_slot[r];
      if (ts >= 0) *reinterpret_cast<float4 *>(g.tail + (int64_t)ts * C + c) = xc;
    }
    if (cg < 2 * H) {
      float ss = y[0] * y[0] + y[1] * y[1] + y[2] * y[2] + y[3] * y[3];
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) ss += __shfl_xor(ss, o);
      float inv = rsqrtf(ss + 1e-6f);
      float *out;
      if (cg < H) {
        inv *= qscale;
        out = g.q + ((int64_t)r * H + cg) * dk;
      } else {
        out = g.k + ((int64_t)r * H + cg - H) * dk;
      }
      *reinterpret_cast<float4 *>(out + lane * 4) = make_float4(y[0] * inv, y[1] * inv, y[2] * inv, y[3] * inv);
    } else {
      *reinterpret_cast<float4 *>(g.v + ((int64_t)r * H + cg - 2 * H) * dv + lane * 4) =
          make_float4(y[0], y[1], y[2], y[3]);
    }
    if (cg == 0) {
      const float *xr = g.x + (int64_t)r * g.ldx;
      for (int hh = lane; hh < H; hh += 32) {
        const float b = xr[C + H * dv + hh], a = xr[C + H * dv + H + hh];
        const float xa = a + g.dt_bias[hh];
        const float sp = xa > 20.0f ? xa : log1pf(__expf(xa));
        g.beta[(int64_t)r * H + hh] = 1.0f / (1.0f + __expf(-b));
        g.alpha[(int64_t)r * H + hh] = __expf(-__expf(g.A_log[hh]) * sp);
      }
    }
    win[2] = win[1];
    win[1] = win[0];
    win[0] = xc;
  }
}

// One workgroup of 128 threads per (sequence, head); thread i owns state row
// i (dv = dk = 128 values in registers). Steps are walked in order; k and q of
// 32 steps at a time are staged in LDS. Every product with k or q takes the
// element from a neighbouring lane instead of a private copy: each row of 16
// lanes loads the step's k and q once, lane n holding elements 8n .. 8n + 7,
// and an FMA reads element j from lane j / 8 of its row through the DPP
// row_newbcast operand modifier (16-byte LDS reads per step: 4 instead of 96
// workgroup-wide broadcasts, which bounded the kernel by LDS bandwidth).
//
// The state is held as S = c X with a scalar c (uniform over the workgroup),
// so the decay S <- alpha S costs one multiply of c instead of one per state
// element: with c' = alpha c,
//   S k = c' (X k),  S <- S + delta k^T  is  X <- X + (delta / c') k^T,
//   o = c' (X q).
// X is rescaled into S (c = 1) whenever c' falls below 2^-40, so X stays
// within 2^40 of S, and a vanishing alpha is applied to X directly.
constexpr int GDN_D = 128;
constexpr int GDN_CHUNK = 32;

// acc += (x taken from lane N of this lane's row of 16) * b
template <int N>
__device__ __forceinline__ void fmac_rowbc(float &acc, float x, float b) {
  asm("v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf" : "+v"(acc) : "v"(x), "v"(b), "n"(N));
}

// p[j % 4] += s[j] k[j] (k[j] = kk[j % 8] of lane j / 8)
template <int... J>
__device__ __forceinline__ void gdn_dot(const float (&s)[GDN_D], const float (&kk)[8], float (&p)[4],
                                        std::integer_sequence<int, J...>) {
  (fmac_rowbc<J / 8>(p[J % 4], kk[J % 8], s[J]), ...);
}

// s[j] += e k[j], then p[j % 4] += s[j] q[j] (k[j], q[j] from lane j / 8)
template <int... J>
__device__ __forceinline__ void gdn_update_dot(float (&s)[GDN_D], const float (&kk)[8], const float (&qq)[8], float e,
                                               float (&p)[4], std::integer_sequence<int, J...>) {
  ((fmac_rowbc<J / 8>(s[J], kk[J % 8], e), fmac_rowbc<J / 8>(p[J % 4], qq[J % 8], s[J])), ...);
}

__global__ __launch_bounds__(128) void gdn_recur_kernel(GdnRecurArgs g) {
  __shared__ float4 ks[GDN_CHUNK][GDN_D / 4], qs[GDN_CHUNK][GDN_D / 4];
  __shared__ float al[GDN_CHUNK], be[GDN_CHUNK];
  const int H = g.H;
  const int si = blockIdx.x / H, h = blockIdx.x % H;
  const GdnSeq sq = g.seqs[si];
  const int i = threadIdx.x, ln = i & 15;
  float s[GDN_D];
  if (sq.init >= 0) {
    const float4 *src = reinterpret_cast<const float4 *>(g.S_init + (((int64_t)sq.init * H + h) * GDN_D + i) * GDN_D);
#pragma unroll
    for (int c = 0; c < GDN_D / 4; ++c) {
      const float4 t = src[c];
      s[4 * c] = t.x; s[4 * c + 1] = t.y; s[4 * c + 2] = t.z; s[4 * c + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int c = 0; c < GDN_D; ++c) s[c] = 0.0f;
  }
  float cs = 1.0f;  // the state is cs s
  for (int t0 = 0; t0 < sq.len; t0 += GDN_CHUNK) {
    const int nt = min(GDN_CHUNK, sq.len - t0);
    __syncthreads();
    for (int e = i; e < nt * (GDN_D / 4); e += 128) {
      const int tt = e / (GDN_D / 4), c = e % (GDN_D / 4);
      const int64_t row = sq.row0 + t0 + tt;
      ks[tt][c] = reinterpret_cast<const float4 *>(g.k + (row * H + h) * GDN_D)[c];
      qs[tt][c] = reinterpret_cast<const float4 *>(g.q + (row * H + h) * GDN_D)[c];
    }
    if (i < nt) {
      const int64_t row = sq.row0 + t0 + i;
      al[i] = g.alpha[row * H + h];
      be[i] = g.beta[row * H + h];
    }
    __syncthreads();
    for (int tt = 0; tt < nt; ++tt) {
      const int64_t row = sq.row0 + t0 + tt;
      const float a = al[tt], b = be[tt];
      const float vv = g.v[(row * H + h) * GDN_D + i];
      const float4 k0 = ks[tt][2 * ln], k1 = ks[tt][2 * ln + 1];
      const float4 q0 = qs[tt][2 * ln], q1 = qs[tt][2 * ln + 1];
      const float kk[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
      const float qq[8] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w};
      cs *= a;
      if (cs < 0x1p-40f) {  // uniform: fold c into X
#pragma unroll
        for (int c = 0; c < GDN_D; ++c) s[c] *= cs;
        cs = 1.0f;
      }
      float p[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      gdn_dot(s, kk, p, std::make_integer_sequence<int, GDN_D>{});
      const float pred = cs * ((p[0] + p[1]) + (p[2] + p[3]));
      const float e = b * (vv - pred) / cs;
      float o[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      gdn_update_dot(s, kk, qq, e, o, std::make_integer_sequence<int, GDN_D>{});
      g.o[(row * H + h) * GDN_D + i] = cs * ((o[0] + o[1]) + (o[2] + o[3]));
    }
  }
#pragma unroll
  for (int c = 0; c < GDN_D; ++c) s[c] *= cs;
  if (sq.fin >= 0) {
    float4 *dst = reinterpret_cast<float4 *>(g.S_fin + (((int64_t)sq.fin * H + h) * GDN_D + i) * GDN_D);
#pragma unroll
    for (int c = 0; c < GDN_D / 4; ++c) dst[c] = make_float4(s[4 * c], s[4 * c + 1], s[4 * c + 2], s[4 * c + 3]);
  }
}

// Chunked form of the same recurrence on the matrix cores (the WY / UT
// representation of a product of generalised Householder updates). Within a
// chunk of GC steps t = 0..GC-1 that starts from state S0, with
// g_t = sum_{u <= t} log alpha_u and Gamma[t][s] = exp(g_t - g_s):
//   delta_t = beta_t (v_t - alpha_t S_{t-1} k_t) is the row added at step t,
//   S_t = alpha_t S_{t-1} + delta_t k_t^T, so unrolling the chunk gives
//   (I + A) Delta = diag(beta) (V - diag(e^g) K S0^T),
//     A[t][s] = beta_t Gamma[t][s] (k_t . k_s) for s < t (strictly lower),
//   O = diag(e^g) Q S0^T + (Gamma o Q K^T)_{s <= t} Delta,
//   S_end = e^{g_last} S0 + Delta^T diag(exp(g_last - g)) K.
// The products run as fp16 MFMAs (or, with PAIR, as three bf16 MFMAs over
// (hi, lo) operand pairs) with fp32 accumulation; the triangular solve for
// Delta is a forward substitution in fp32; the state stays in fp32
// accumulators for the whole sequence and is rounded to 16 bits only as an
// operand of the next chunk's products.
//
// One workgroup of 4 waves per (sequence, head); wave w owns columns
// v = 32 w + lane % 32 of the state, of Delta and of the chunk's outputs.
// Everything that is per column stays in that wave's registers:
//   * the state is held transposed, S^T[d][v] in 4 accumulator tiles, and
//     its registers serve directly as the operand of K S0^T and Q S0^T (the
//     accumulator's row order, taken as the contraction order, differs from
//     the operand's by a swap of bits 2 and 3 of d; K and Q are stored in
//     LDS with the same swap);
//   * the right-hand side comes out of K S0^T in the accumulator layout, in
//     which lane half h holds rows t with (t / 4) % 2 = h, and the solve runs
//     on those rows in place;
//   * each row of Delta, once solved, reaches both lane halves of its
//     column, which keep the rows they supply as the operand of the products
//     that follow.
// LDS holds only what is shared across columns: K and Q rows, K~^T, the
// masked Gamma o Q K^T and A. 16-bit rows in LDS are stored in 16-byte chunks
// whose position is XOR-swizzled by the row, so the 32 rows a fragment read
// touches fall in distinct banks.
constexpr int GC = 32;  // chunk length

// element (r, c) of a [*][128] / [*][32] array of 16-bit values
__device__ __forceinline__ int sw128(int r, int c) { return r * 128 + ((((c >> 3) ^ (r & 15)) << 3) | (c & 7)); }
__device__ __forceinline__ int sw32(int r, int c) { return r * 32 + ((((c >> 3) ^ ((r >> 2) & 3)) << 3) | (c & 7)); }
// column d with bits 2 and 3 swapped: within each block of 16, positions
// 0..15 hold d = 0..3, 8..11, 4..7, 12..15
__device__ __forceinline__ int swap23(int d) { return (d & ~12) | ((d & 4) << 1) | ((d & 8) >> 1); }

// Operand storage: single fp16 values, or with PAIR (hi, lo) bf16 pairs whose
// sum carries about 16 significant bits. NP parts of each array are stored
// one after the other.
template <bool PAIR> struct ChunkOp {
  typedef f16 T;
  static constexpr int NP = 1;
};
template <> struct ChunkOp<true> {
  typedef bf16 T;
  static constexpr int NP = 2;
};

// MFMA operand: row r, columns c0 .. c0 + 7 (c0 a multiple of 8)
template <typename T> __device__ __forceinline__ Frag<T> frag128(const T *a, int r, int c0) {
  Frag<T> f;
  f.v = *reinterpret_cast<const typename Vec8<T>::type *>(a + sw128(r, c0));
  return f;
}
template <typename T> __device__ __forceinline__ Frag<T> frag32(const T *a, int r, int c0) {
  Frag<T> f;
  f.v = *reinterpret_cast<const typename Vec8<T>::type *>(a + sw32(r, c0));
  return f;
}
// two values as NP packed words: the rounded values, and with pairs the
// rounded remainders
template <bool PAIR> __device__ __forceinline__ void split2(float a, float b, uint32_t *u) {
  if constexpr (PAIR) {
    const uint32_t hi = f2bf2(a, b);
    u[0] = hi;
    u[1] = f2bf2(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xffff0000u));
  } else {
    u[0] = f2h2(a, b);
  }
}
// MFMA operand (NP parts) from 8 fp32 values
template <bool PAIR> __device__ __forceinline__ void frag_regs(const float *x, Frag<typename ChunkOp<PAIR>::T> *f) {
  typedef typename ChunkOp<PAIR>::T T;
  uint32_t u[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i) split2<PAIR>(x[2 * i], x[2 * i + 1], u[i]);
#pragma unroll
  for (int p = 0; p < ChunkOp<PAIR>::NP; ++p)
    f[p].v = __builtin_bit_cast(typename Vec8<T>::type, make_uint4(u[0][p], u[1][p], u[2][p], u[3][p]));
}
// one value into part 0 at a[i] and, with pairs, its remainder into part 1
// at a[n + i]
template <bool PAIR, typename T> __device__ __forceinline__ void st_parts(T *a, int n, int i, float x) {
  const T hi = from_f<T>(x);
  a[i] = hi;
  if constexpr (PAIR) a[n + i] = from_f<T>(x - to_f<T>(hi));
}
// acc += one 16-wide step of a product; with pairs hi hi + hi lo + lo hi (the
// lo lo term is of the order of the pairs' own rounding)
template <bool PAIR, typename T> __device__ __forceinline__ void mmap(f32x16 &acc, const Frag<T> *a, const Frag<T> *b) {
  mma32(acc, a[0], b[0]);
  if constexpr (PAIR) {
    mma32(acc, a[0], b[1]);
    mma32(acc, a[1], b[0]);
  }
}

// x, as a value the compiler cannot see through: address arithmetic built on
// it is redone in every chunk instead of being held in registers across the
// chunk loop
__device__ __forceinline__ int opaque(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

template <bool PAIR> __global__ __launch_bounds__(256, 2) void gdn_chunk_kernel(GdnRecurArgs g) {
  typedef typename ChunkOp<PAIR>::T T;
  constexpr int NP = ChunkOp<PAIR>::NP;
  constexpr int NKQ = GC * GDN_D, NKT = GDN_D * GC, NPM = GC * GC;  // elements of one part
  __shared__ __align__(16) T kh[NP * NKQ], qh[NP * NKQ];  // K, Q rows [t][swap23(d)]
  __shared__ __align__(16) T kt[NP * NKT];                // K~^T [d][s]
  __shared__ __align__(16) T pm[NP * NPM];                // masked Gamma o Q K^T [t][s]
  // A by columns, each split by lane half: A[t][s] at [s][16 h + e] where
  // lane half h, register e holds row t (t = 8 (e / 4) + 4 h + e % 4)
  __shared__ __align__(16) float al[GC * GC];
  __shared__ float gs[GC], bs[GC];

  const int H = g.H;
  const int si = blockIdx.x / H, h = blockIdx.x % H;
  const GdnSeq sq = g.seqs[si];
  const int tid = threadIdx.x, l = tid & 63, lc = l & 31, lh = l >> 5;
  // the wave index as a scalar: the MFMAs only some waves issue sit behind
  // scalar branches (an MFMA writes its result whatever the execution mask,
  // so masking lanes off would not skip it)
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  // S^T[d][v], v = 32 w + lc, d = 32 j + 8 (e / 4) + 4 lh + e % 4: four
  // consecutive d per quarter of a tile, one 16-byte piece of row v of S
  f32x16 sacc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
      if (sq.init >= 0)
        x = *reinterpret_cast<const float4 *>(g.S_init + (((int64_t)sq.init * H + h) * GDN_D + 32 * w + lc) * GDN_D +
                                              32 * j + 8 * c + 4 * lh);
      sacc[j][4 * c] = x.x;
      sacc[j][4 * c + 1] = x.y;
      sacc[j][4 * c + 2] = x.z;
      sacc[j][4 * c + 3] = x.w;
    }
  // the initial state has arrived before the loop: without this wait the
  // compiler's wait at the top of the loop, made for both ways in, also holds
  // each chunk until the previous chunk's output stores have completed
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)

  for (int c0 = 0; c0 < sq.len; c0 += GC) {
    const int L = min(GC, sq.len - c0);
    const int64_t row0 = sq.row0 + c0;
    const int tid = opaque(threadIdx.x), l = tid & 63, lc = l & 31, lh = l >> 5;
    // every global load of the chunk is issued before the first wait, with no
    // branch between them: rows past L read row L - 1 (in bounds, L >= 1) and
    // are replaced by zeros once they arrive
    float ga, gb;  // gates of step lc (read by every wave, used by wave 0)
    {
      const int64_t r = (row0 + min(lc, L - 1)) * H + h;
      ga = g.alpha[r];
      gb = g.beta[r];
    }
    float4 kr[4], qr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + 256 * i, t = idx >> 5, d = (idx & 31) * 4;
      const int64_t r = ((row0 + min(t, L - 1)) * H + h) * GDN_D + d;
      kr[i] = *reinterpret_cast<const float4 *>(g.k + r);
      qr[i] = *reinterpret_cast<const float4 *>(g.q + r);
    }
    // v for this wave's columns, in the accumulator layout
    float vr[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int t = 8 * (e >> 2) + 4 * lh + (e & 3);
      vr[e] = g.v[((row0 + min(t, L - 1)) * H + h) * GDN_D + 32 * w + lc];
    }
    __syncthreads();  // the previous chunk's readers of every buffer are done
    // ---- stage: K and Q rows, gates; rows past L are zero
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + 256 * i, t = idx >> 5, d = (idx & 31) * 4;
      const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
      if (t >= L) kr[i] = qr[i] = z;
      uint32_t ka[2], kb[2], qa[2], qb[2];
      split2<PAIR>(kr[i].x, kr[i].y, ka);
      split2<PAIR>(kr[i].z, kr[i].w, kb);
      split2<PAIR>(qr[i].x, qr[i].y, qa);
      split2<PAIR>(qr[i].z, qr[i].w, qb);
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        *reinterpret_cast<uint2 *>(kh + p * NKQ + sw128(t, swap23(d))) = make_uint2(ka[p], kb[p]);
        *reinterpret_cast<uint2 *>(qh + p * NKQ + sw128(t, swap23(d))) = make_uint2(qa[p], qb[p]);
      }
    }
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (8 * (e >> 2) + 4 * lh + (e & 3) >= L) vr[e] = 0.0f;
    if (w == 0) {
      // log-decay prefix sums over the chunk (lanes 0..31; the loads were
      // issued first), a vanishing alpha held at e^-80
      float la = lc < L ? fmaxf(__logf(ga), -80.0f) : 0.0f;
#pragma unroll
      for (int off = 1; off < GC; off *= 2) {
        const float y = __shfl_up(la, off, GC);
        if (lc >= off) la += y;
      }
      if (l < GC) {
        gs[l] = la;
        bs[l] = l < L ? gb : 0.0f;
      }
    }
    __syncthreads();
    // K~^T = (K rows scaled by exp(g_last - g_s)) transposed
    const float glast = gs[GC - 1];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + 256 * i, t = idx >> 5, d = (idx & 31) * 4;
      const float f = __expf(glast - gs[t]);
      st_parts<PAIR>(kt, NKT, sw32(d, t), kr[i].x * f);
      st_parts<PAIR>(kt, NKT, sw32(d + 1, t), kr[i].y * f);
      st_parts<PAIR>(kt, NKT, sw32(d + 2, t), kr[i].z * f);
      st_parts<PAIR>(kt, NKT, sw32(d + 3, t), kr[i].w * f);
    }
    // ---- products with S0 (every wave, its 32 state columns from its own
    //      registers) and K K^T (wave 0) / Q K^T (wave 1)
    f32x16 xk, xq, xt;
#pragma unroll
    for (int e = 0; e < 16; ++e) xk[e] = xq[e] = xt[e] = 0.0f;
#pragma unroll
    for (int d0 = 0; d0 < GDN_D; d0 += 16) {
      Frag<T> fk[NP], fq[NP], fs[NP];
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        fk[p] = frag128(kh + p * NKQ, lc, d0 + 8 * lh);
        fq[p] = frag128(qh + p * NKQ, lc, d0 + 8 * lh);
      }
      float sv[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) sv[i] = sacc[d0 >> 5][8 * ((d0 >> 4) & 1) + i];
      frag_regs<PAIR>(sv, fs);
      mmap<PAIR>(xk, fk, fs);
      mmap<PAIR>(xq, fq, fs);
      if (w == 0) mmap<PAIR>(xt, fk, fk);
      if (w == 1) mmap<PAIR>(xt, fq, fk);
    }
    // ---- right-hand side r (in registers), O's first term, A and the masked
    //      Gamma o Q K^T
    float xr[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int t = 8 * (e >> 2) + 4 * lh + (e & 3);
      const float eg = __expf(gs[t]);
      xr[e] = bs[t] * (vr[e] - eg * xk[e]);
      xq[e] *= eg;  // this wave's output tile starts as diag(e^g) Q S0^T
      const int s = lc;
      // K K^T is symmetric: this lane's (t, s) entry also serves as (s, t),
      // so A[s][t] goes to column t of A, 32 lanes to 32 distinct banks
      if (w == 0)
        al[t * GC + 16 * ((s >> 2) & 1) + 4 * (s >> 3) + (s & 3)] =
            t < s ? bs[s] * __expf(gs[s] - gs[t]) * xt[e] : 0.0f;
      if (w == 1) st_parts<PAIR>(pm, NPM, sw32(t, s), s <= t ? __expf(gs[t] - gs[s]) * xt[e] : 0.0f);
    }
    __syncthreads();
    // ---- forward substitution for column v = 32 w + lc of Delta, in the
    //      column-oriented order: once delta_s is final it is taken off every
    //      later row, so the updates of one step are independent of each
    //      other. Each lane half updates the rows it holds; a final delta_s
    //      reaches the other half by a swap of the wave's lane halves. Every
    //      row still takes its terms in the order s = 0, 1, ..., t - 1.
    // Delta[s][v] reaches both lane halves; each keeps the rows it supplies
    // as an MFMA operand, s = 16 c + 8 lh + i in dk[8 c + i]
    float dk[16];
    {
      const float *ap = al + 16 * lh;  // A[t(e)][s] at ap[s * GC + e]
      // column s of A is read one step ahead of its use; register e is
      // updated at step s while its row on the high half, 8 (e / 4) + 4 + e % 4,
      // is above s (a row at or above s on the low half reads A = 0)
      float ac[16], an[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) ac[e] = ap[e];
#pragma unroll
      for (int s = 0; s < GC; ++s) {
        if (s + 1 < GC) {
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (8 * (e >> 2) + 4 + (e & 3) > s + 1) an[e] = ap[(s + 1) * GC + e];
        }
        // row s is final in half (s / 4) % 2, register 4 (s / 8) + s % 4;
        // q[0] holds the low half's value in every lane, q[1] the high half's
        const int es = 4 * (s >> 3) + (s & 3);
        const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(xr[es]), __float_as_uint(xr[es]), false, false);
        const float ds = __uint_as_float(q[(s >> 2) & 1]);
        if (((s >> 3) & 1) == lh) dk[8 * (s >> 4) + (s & 7)] = ds;
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (8 * (e >> 2) + 4 + (e & 3) > s) xr[e] = fmaf(-ac[e], ds, xr[e]);
#pragma unroll
        for (int e = 0; e < 16; ++e) ac[e] = an[e];
      }
    }
    // Delta as an MFMA operand: lane half lh supplies rows 16 c + 8 lh + i
    Frag<T> fd[2][NP];
    frag_regs<PAIR>(dk, fd[0]);
    frag_regs<PAIR>(dk + 8, fd[1]);
    // ---- O += (Gamma o Q K^T) Delta; S^T = e^{g_last} S0^T + K~^T Delta
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      Frag<T> fp[NP];
#pragma unroll
      for (int p = 0; p < NP; ++p) fp[p] = frag32(pm + p * NPM, lc, 16 * c + 8 * lh);
      mmap<PAIR>(xq, fp, fd[c]);
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int t = 8 * (e >> 2) + 4 * lh + (e & 3);
      if (t < L) g.o[((row0 + t) * H + h) * GDN_D + 32 * w + lc] = xq[e];
    }
    const float eg = __expf(glast);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[j][e] *= eg;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        Frag<T> fk[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p) fk[p] = frag32(kt + p * NKT, 32 * j + lc, 16 * c + 8 * lh);
        mmap<PAIR>(sacc[j], fk, fd[c]);
      }
    }
  }
  if (sq.fin >= 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        *reinterpret_cast<float4 *>(g.S_fin + (((int64_t)sq.fin * H + h) * GDN_D + 32 * w + lc) * GDN_D + 32 * j +
                                    8 * c + 4 * lh) =
            make_float4(sacc[j][4 * c], sacc[j][4 * c + 1], sacc[j][4 * c + 2], sacc[j][4 * c + 3]);
  }
}

// y = RMSNorm(o) * w * silu(z) per head, written as the A operand of the
// output projection ([hi | lo] pairs with PAIR).
template <typename T, bool PAIR>
__global__ __launch_bounds__(256) void gdn_out_kernel(const float *__restrict__ o, const float *__restrict__ x,
                                                      int64_t ldx, int zoff, const float *__restrict__ w,
                                                      float eps, int H, int dv, T *__restrict__ y) {
  const int r = blockIdx.x, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float *orow = o + (int64_t)r * H * dv;
  const float *z = x + (int64_t)r * ldx + zoff;
  T *yr = y + (int64_t)r * H * dv * (PAIR ? 2 : 1);
  for (int hh = wave; hh < H; hh += 4) {
    float ss = 0.0f;
    for (int i = lane; i < dv; i += 64) ss += orow[hh * dv + i] * orow[hh * dv + i];
    ss = warp_sum(ss);
    const float inv = rsqrtf(ss / (float)dv + eps);
    for (int i = lane; i < dv; i += 64) {
      const float zz = z[hh * dv + i];
      const float val = orow[hh * dv + i] * inv * w[i] * (zz / (1.0f + __expf(-zz)));
      const T hi = from_f<T>(val);
      yr[hh * dv + i] = hi;
      if constexpr (PAIR) yr[H * dv + hh * dv + i] = from_f<T>(val - to_f<T>(hi));
    }
  }
}

hipError_t launch_gdn_conv(const GdnConvArgs &g, int R, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (g.dk != 128 || g.dv != 128) return hipErrorInvalidValue;
  const int64_t groups = (int64_t)((R + GDN_CONV_RB - 1) / GDN_CONV_RB) * (3 * g.H);
  hipLaunchKernelGGL(gdn_conv_kernel, dim3((unsigned)((groups + 7) / 8)), dim3(256), 0, st, g, R);
  return hipGetLastError();
}

hipError_t launch_gdn_recur(const GdnRecurArgs &g, int nseq, hipStream_t st) {
  if (nseq <= 0) return hipSuccess;
  if (g.dk != GDN_D || g.dv != GDN_D) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gdn_recur_kernel, dim3(nseq * g.H), dim3(128), 0, st, g);
  return hipGetLastError();
}

hipError_t launch_gdn_chunk(const GdnRecurArgs &g, int nseq, int pair, hipStream_t st) {
  if (nseq <= 0) return hipSuccess;
  if (g.dk != GDN_D || g.dv != GDN_D) return hipErrorInvalidValue;
  if (pair)
    hipLaunchKernelGGL(gdn_chunk_kernel<true>, dim3(nseq * g.H), dim3(256), 0, st, g);
  else
    hipLaunchKernelGGL(gdn_chunk_kernel<false>, dim3(nseq * g.H), dim3(256), 0, st, g);
  return hipGetLastError();
}

hipError_t launch_gdn_out(int dtype, int pair, const float *o, const float *x, int64_t ldx, int zoff, const float *w,
                          float eps, int H, int dv, int R, void *y, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (dtype == 0 && pair)
    hipLaunchKernelGGL((gdn_out_kernel<bf16, true>), dim3(R), dim3(256), 0, st, o, x, ldx, zoff, w, eps, H, dv,
                       (bf16 *)y);
  else if (dtype == 0)
    hipLaunchKernelGGL((gdn_out_kernel<bf16, false>), dim3(R), dim3(256), 0, st, o, x, ldx, zoff, w, eps, H, dv,
                       (bf16 *)y);
  else if (dtype == 2)
    hipLaunchKernelGGL((gdn_out_kernel<f16, false>), dim3(R), dim3(256), 0, st, o, x, ldx, zoff, w, eps, H, dv,
                       (f16 *)y);
  else
    hipLaunchKernelGGL((gdn_out_kernel<float, false>), dim3(R), dim3(256), 0, st, o, x, ldx, zoff, w, eps, H, dv,
                       (float *)y);
  return hipGetLastError();
}

}  // namespace jetk
