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
#include "device.h"
#include "kernels.h"

namespace jetk {

// One block per row. x: projection output [R][ldx] = q~ | k~ | v~ | z | b | a.
__global__ __launch_bounds__(256) void gdn_conv_kernel(GdnConvArgs g) {
  extern __shared__ float sc[];  // C conv + SiLU outputs of this row
  const int r = blockIdx.x, tid = threadIdx.x;
  const int H = g.H, dk = g.dk, dv = g.dv;
  const int C = 2 * H * dk + H * dv;
  const float *xr = g.x + (int64_t)r * g.ldx;
  const float *src[3];
#pragma unroll
  for (int j = 1; j <= 3; ++j) {
    const int h = g.hist[(int64_t)r * 3 + j - 1];
    src[j - 1] = h >= 0 ? g.x + (int64_t)h * g.ldx : (h == -1 ? nullptr : g.tail + (int64_t)(-2 - h) * C);
  }
  const int ts = g.tail_slot ? g.tail_slot[r] : -1;
  for (int c = tid; c < C; c += 256) {
    float acc = g.conv_w[c * 4 + 3] * xr[c];
#pragma unroll
    for (int j = 1; j <= 3; ++j)
      if (src[j - 1]) acc += g.conv_w[c * 4 + 3 - j] * src[j - 1][c];
    sc[c] = acc / (1.0f + __expf(-acc));
    if (ts >= 0) g.tail[(int64_t)ts * C + c] = xr[c];
  }
  __syncthreads();
  const int wave = tid >> 6, lane = tid & 63;
  const float qscale = rsqrtf((float)dk);
  for (int hh = wave; hh < 2 * H; hh += 4) {
    const int base = hh * dk;
    float ss = 0.0f;
    for (int i = lane; i < dk; i += 64) ss += sc[base + i] * sc[base + i];
    ss = warp_sum(ss);
    float inv = rsqrtf(ss + 1e-6f);
    float *out;
    if (hh < H) {
      inv *= qscale;
      out = g.q + ((int64_t)r * H + hh) * dk;
    } else {
      out = g.k + ((int64_t)r * H + hh - H) * dk;
    }
    for (int i = lane; i < dk; i += 64) out[i] = sc[base + i] * inv;
  }
  for (int i = tid; i < H * dv; i += 256) g.v[(int64_t)r * H * dv + i] = sc[2 * H * dk + i];
  if (tid < H) {
    const float b = xr[C + H * dv + tid], a = xr[C + H * dv + H + tid];
    const float xa = a + g.dt_bias[tid];
    const float sp = xa > 20.0f ? xa : log1pf(__expf(xa));
    g.beta[(int64_t)r * H + tid] = 1.0f / (1.0f + __expf(-b));
    g.alpha[(int64_t)r * H + tid] = __expf(-__expf(g.A_log[tid]) * sp);
  }
}

// One workgroup of 128 threads per (sequence, head); thread i owns state row
// i (dv = dk = 128 values in registers). Steps are walked in order; k and q of
// 32 steps at a time are staged in LDS and read by all threads.
constexpr int GDN_D = 128;
constexpr int GDN_CHUNK = 32;

__global__ __launch_bounds__(128) void gdn_recur_kernel(GdnRecurArgs g) {
  __shared__ float4 ks[GDN_CHUNK][GDN_D / 4], qs[GDN_CHUNK][GDN_D / 4];
  __shared__ float al[GDN_CHUNK], be[GDN_CHUNK];
  const int H = g.H;
  const int si = blockIdx.x / H, h = blockIdx.x % H;
  const GdnSeq sq = g.seqs[si];
  const int i = threadIdx.x;
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
      float pred = 0.0f;
#pragma unroll
      for (int c = 0; c < GDN_D / 4; ++c) {
        const float4 kk = ks[tt][c];
        s[4 * c] *= a; s[4 * c + 1] *= a; s[4 * c + 2] *= a; s[4 * c + 3] *= a;
        pred += s[4 * c] * kk.x + s[4 * c + 1] * kk.y + s[4 * c + 2] * kk.z + s[4 * c + 3] * kk.w;
      }
      const float delta = b * (vv - pred);
      float out = 0.0f;
#pragma unroll
      for (int c = 0; c < GDN_D / 4; ++c) {
        const float4 kk = ks[tt][c], qq = qs[tt][c];
        s[4 * c] += delta * kk.x; s[4 * c + 1] += delta * kk.y;
        s[4 * c + 2] += delta * kk.z; s[4 * c + 3] += delta * kk.w;
        out += s[4 * c] * qq.x + s[4 * c + 1] * qq.y + s[4 * c + 2] * qq.z + s[4 * c + 3] * qq.w;
      }
      g.o[(row * H + h) * GDN_D + i] = out;
    }
  }
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
  const size_t lds = sizeof(float) * (size_t)(2 * g.H * g.dk + g.H * g.dv);
  if (lds > 65536) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gdn_conv_kernel, dim3(R), dim3(256), lds, st, g);
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
