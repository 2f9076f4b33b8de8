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
