// Row-wise and gather kernels of the scoring path: embedding gather, RMSNorm,
// RoPE + KV-cache scatter, log-sum-exp merge, target log-probability gather
// (Section 3.1 Eq. 2), per-candidate sums (Section 3.2 Eq. 3), id checks.
// All are memory-bound; each reads its rows once with 16-byte accesses where
// the layout allows.
#include "device.h"
#include "kernels.h"

namespace jetk {

template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(const T *__restrict__ E, const int32_t *__restrict__ ids,
                                                     const int32_t *__restrict__ idx, int d,
                                                     float *__restrict__ resid) {
  const int r = blockIdx.x;
  const int64_t tok = ids[idx ? idx[r] : r];
  const T *src = E + tok * d;
  float *dst = resid + (int64_t)r * d;
  for (int i = threadIdx.x; i < d; i += 256) dst[i] = to_f<T>(src[i]);
}

template <typename T, bool PAIR>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float *__restrict__ x, const int32_t *__restrict__ map,
                                                       const float *__restrict__ g, int d, float eps,
                                                       T *__restrict__ out) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const int64_t src = map ? map[r] : r;
  const float *xr = x + src * d;
  float ss = 0.0f;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float v = xr[i];
    ss += v * v;
  }
  ss = warp_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = rsqrtf(tot / (float)d + eps);
  T *o = out + (int64_t)r * d * (PAIR ? 2 : 1);
  for (int i = threadIdx.x; i < d; i += 256) {
    const float v = xr[i] * inv * g[i];
    const T hi = from_f<T>(v);
    o[i] = hi;
    if constexpr (PAIR) o[d + i] = from_f<T>(v - to_f<T>(hi));
  }
}

// One wave per row, 4 rows per block: the row is read once with 16-byte loads
// into registers (NV float4 per lane, d <= 256 NV, d a multiple of 4), then
// normalised and written with 8-byte (16-bit T) or 16-byte (fp32) stores.
template <typename T, bool PAIR, int NV>
__global__ __launch_bounds__(256) void rmsnorm_rows_kernel(const float *__restrict__ x,
                                                            const int32_t *__restrict__ map,
                                                            const float *__restrict__ g, int R, int d, float eps,
                                                            T *__restrict__ out) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= R) return;
  const int64_t src = map ? map[r] : r;
  const float4 *xr = reinterpret_cast<const float4 *>(x + src * d);
  const float4 *g4 = reinterpret_cast<const float4 *>(g);
  const int n4 = d >> 2;
  float4 v[NV];
  float ss = 0.0f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = j * 64 + lane;
    v[j] = i < n4 ? xr[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
  }
  ss = warp_sum(ss);
  const float inv = rsqrtf(ss / (float)d + eps);
  T *o = out + (int64_t)r * d * (PAIR ? 2 : 1);
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = j * 64 + lane;
    if (i >= n4) break;
    const float4 gg = g4[i];
    const float y[4] = {v[j].x * inv * gg.x, v[j].y * inv * gg.y, v[j].z * inv * gg.z, v[j].w * inv * gg.w};
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<float4 *>(o + 4 * i) = make_float4(y[0], y[1], y[2], y[3]);
    } else {
      T hi[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) hi[e] = from_f<T>(y[e]);
      *reinterpret_cast<uint2 *>(o + 4 * i) =
          make_uint2(pack2<T>(to_f<T>(hi[0]), to_f<T>(hi[1])), pack2<T>(to_f<T>(hi[2]), to_f<T>(hi[3])));
      if constexpr (PAIR)
        *reinterpret_cast<uint2 *>(o + d + 4 * i) =
            make_uint2(pack2<T>(y[0] - to_f<T>(hi[0]), y[1] - to_f<T>(hi[1])),
                       pack2<T>(y[2] - to_f<T>(hi[2]), y[3] - to_f<T>(hi[3])));
    }
  }
}

// One block per row; thread t handles rotation pairs (i, i + hd/2).
template <typename T, bool PAIR>
__device__ __forceinline__ void put_val(T *p, int64_t ps, float v) {
  const T hi = from_f<T>(v);
  p[0] = hi;
  if constexpr (PAIR) p[ps] = from_f<T>(v - to_f<T>(hi));
}

template <typename T, bool PAIR>
__global__ __launch_bounds__(256) void rope_scatter_kernel(const float *__restrict__ qkv, const int32_t *__restrict__ pos,
                                                            const float *__restrict__ cos_t,
                                                            const float *__restrict__ sin_t, int Hq, int Hkv,
                                                            int hd, T *__restrict__ q_out, int64_t q_ps,
                                                            T *__restrict__ kc, T *__restrict__ vc, int64_t kv_ps,
                                                            int64_t S, int64_t slot0) {
  const int r = blockIdx.x;
  const int half = hd / 2;
  const int W = (Hq + 2 * Hkv) * hd;
  const float *src = qkv + (int64_t)r * W;
  const int64_t p = pos[r];
  const float *cs = cos_t + p * half, *sn = sin_t + p * half;
  const int64_t slot = slot0 + r;
  for (int t = threadIdx.x; t < (Hq + Hkv) * half; t += 256) {
    const int h = t / half, i = t % half;
    const float x1 = src[h * hd + i], x2 = src[h * hd + i + half];
    const float c = cs[i], s = sn[i];
    // the same operations as the QKV GEMM's RoPE epilogue, so both paths round alike
    const float y1 = fmaf(x1, c, -(x2 * s)), y2 = fmaf(x2, c, x1 * s);
    if (h < Hq) {
      T *o = q_out + ((int64_t)r * Hq + h) * hd;
      put_val<T, PAIR>(o + i, q_ps, y1);
      put_val<T, PAIR>(o + i + half, q_ps, y2);
    } else {
      T *o = kc + ((int64_t)(h - Hq) * S + slot) * hd;
      put_val<T, PAIR>(o + i, kv_ps, y1);
      put_val<T, PAIR>(o + i + half, kv_ps, y2);
    }
  }
  for (int t = threadIdx.x; t < Hkv * hd; t += 256) {
    const int h = t / hd, i = t % hd;
    put_val<T, PAIR>(vc + ((int64_t)h * S + slot) * hd + i, kv_ps, src[(Hq + Hkv) * hd + t]);
  }
}

__global__ __launch_bounds__(256) void lse_merge_kernel(const float *__restrict__ pm, const float *__restrict__ ps,
                                                         int nsplit, int R, float *__restrict__ lse,
                                                         const float *__restrict__ zt, float wscale,
                                                         float *__restrict__ ell) {
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= R) return;
  float M = -INFINITY;
  for (int s = 0; s < nsplit; ++s) M = fmaxf(M, pm[(int64_t)s * R + r]);
  float S = 0.0f;
  for (int s = 0; s < nsplit; ++s) S += ps[(int64_t)s * R + r] * exp2f(pm[(int64_t)s * R + r] - M);
  const float l = (M + log2f(S)) * kLn2;
  lse[r] = l;
  if (zt) ell[r] = zt[r] * wscale - l;
}

// Rows of the final hidden states in scored-token order: a candidate body
// row, or the question's last prefix row for a candidate's first token.
__global__ __launch_bounds__(256) void token_rows_kernel(const int32_t *__restrict__ lm_row, int row_base,
                                                          const uint4 *__restrict__ f_body,
                                                          const uint4 *__restrict__ f_last, int64_t row_chunks,
                                                          uint4 *__restrict__ dst) {
  const int i = blockIdx.x, r = lm_row[i];
  const uint4 *s = r < 0 ? f_last + (int64_t)(-r - 1) * row_chunks : f_body + (int64_t)(r - row_base) * row_chunks;
  uint4 *d = dst + (int64_t)i * row_chunks;
  for (int64_t c = threadIdx.x; c < row_chunks; c += 256) d[c] = s[c];
}

__global__ __launch_bounds__(256) void segment_sum_kernel(const float *__restrict__ ell, const int64_t *__restrict__ off,
                                                           int n, float *__restrict__ s) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= n) return;
  const int64_t b = off[0];
  float acc = 0.0f;
  for (int64_t i = off[c]; i < off[c + 1]; ++i) acc += ell[i - b];
  s[c] = acc;
}

__global__ __launch_bounds__(256) void count_bad_ids_kernel(const int32_t *__restrict__ ids, int64_t n, int V,
                                                             int *__restrict__ bad) {
  int cnt = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    cnt += (ids[i] < 0 || ids[i] >= V) ? 1 : 0;
  cnt = (int)warp_sum((float)cnt);
  if ((threadIdx.x & 63) == 0 && cnt) atomicAdd(bad, cnt);
}

template <typename T>
__global__ __launch_bounds__(256) void convert_f32_kernel(const float *__restrict__ src, int64_t n, T *__restrict__ dst) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = from_f<T>(src[i]);
}

// bf16 * scale (a power of two: exact in fp32) rounded to fp16; values the
// rounding changed are counted into *inexact.
__global__ __launch_bounds__(256) void bf16_to_f16_kernel(const uint16_t *__restrict__ src, int64_t n, float scale,
                                                           f16 *__restrict__ dst, unsigned long long *inexact) {
  unsigned long long cnt = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const float v = bf2f(src[i]) * scale;
    const f16 h = (f16)v;
    cnt += ((float)h != v);
    dst[i] = h;
  }
  if (cnt) atomicAdd(inexact, cnt);
}

__global__ __launch_bounds__(256) void bf16_to_f32_kernel(const uint16_t *__restrict__ src, int64_t n,
                                                           float *__restrict__ dst) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = bf2f(src[i]);
}

// ---------------------------------------------------------------------------

hipError_t launch_embed(int dtype, const void *E, const int32_t *ids, const int32_t *idx, int R, int d,
                        float *resid, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (dtype == 0) hipLaunchKernelGGL(embed_kernel<bf16>, dim3(R), dim3(256), 0, st, (const bf16 *)E, ids, idx, d, resid);
  else hipLaunchKernelGGL(embed_kernel<float>, dim3(R), dim3(256), 0, st, (const float *)E, ids, idx, d, resid);
  return hipGetLastError();
}

template <typename T, bool PAIR>
static bool rmsnorm_rows(const float *x, const int32_t *map, const float *g, int R, int d, float eps, T *out,
                         hipStream_t st) {
  if (d % 4) return false;
  const dim3 grid((R + 3) / 4), block(256);
  const int nv = (d + 255) / 256;
  if (nv <= 2) hipLaunchKernelGGL((rmsnorm_rows_kernel<T, PAIR, 2>), grid, block, 0, st, x, map, g, R, d, eps, out);
  else if (nv <= 4) hipLaunchKernelGGL((rmsnorm_rows_kernel<T, PAIR, 4>), grid, block, 0, st, x, map, g, R, d, eps, out);
  else if (nv <= 8) hipLaunchKernelGGL((rmsnorm_rows_kernel<T, PAIR, 8>), grid, block, 0, st, x, map, g, R, d, eps, out);
  else if (nv <= 12) hipLaunchKernelGGL((rmsnorm_rows_kernel<T, PAIR, 12>), grid, block, 0, st, x, map, g, R, d, eps, out);
  else if (nv <= 20) hipLaunchKernelGGL((rmsnorm_rows_kernel<T, PAIR, 20>), grid, block, 0, st, x, map, g, R, d, eps, out);
  else if (nv <= 32) hipLaunchKernelGGL((rmsnorm_rows_kernel<T, PAIR, 32>), grid, block, 0, st, x, map, g, R, d, eps, out);
  else return false;
  return true;
}

hipError_t launch_rmsnorm(int dtype, int pair, const float *x, const int32_t *map, const float *g, int R, int d,
                          float eps, void *out, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  // one wave per row with the row in registers (d <= 8192, d % 4 == 0)
  bool done = false;
  if (dtype == 0 && pair) done = rmsnorm_rows<bf16, true>(x, map, g, R, d, eps, (bf16 *)out, st);
  else if (dtype == 0) done = rmsnorm_rows<bf16, false>(x, map, g, R, d, eps, (bf16 *)out, st);
  else if (dtype == 2 && pair) done = rmsnorm_rows<f16, true>(x, map, g, R, d, eps, (f16 *)out, st);
  else if (dtype == 2) done = rmsnorm_rows<f16, false>(x, map, g, R, d, eps, (f16 *)out, st);
  else done = rmsnorm_rows<float, false>(x, map, g, R, d, eps, (float *)out, st);
  if (done) return hipGetLastError();
  if (dtype == 0 && pair)
    hipLaunchKernelGGL((rmsnorm_kernel<bf16, true>), dim3(R), dim3(256), 0, st, x, map, g, d, eps, (bf16 *)out);
  else if (dtype == 0)
    hipLaunchKernelGGL((rmsnorm_kernel<bf16, false>), dim3(R), dim3(256), 0, st, x, map, g, d, eps, (bf16 *)out);
  else if (dtype == 2 && pair)
    hipLaunchKernelGGL((rmsnorm_kernel<f16, true>), dim3(R), dim3(256), 0, st, x, map, g, d, eps, (f16 *)out);
  else if (dtype == 2)
    hipLaunchKernelGGL((rmsnorm_kernel<f16, false>), dim3(R), dim3(256), 0, st, x, map, g, d, eps, (f16 *)out);
  else
    hipLaunchKernelGGL((rmsnorm_kernel<float, false>), dim3(R), dim3(256), 0, st, x, map, g, d, eps, (float *)out);
  return hipGetLastError();
}

hipError_t launch_rope_scatter(int dtype, int pair, const float *qkv, const int32_t *pos, const float *cos_t,
                               const float *sin_t, int R, int Hq, int Hkv, int hd, void *q_out, int64_t q_ps,
                               void *k_cache, void *v_cache, int64_t kv_ps, int64_t S, int64_t slot0,
                               hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (dtype == 0 && pair)
    hipLaunchKernelGGL((rope_scatter_kernel<bf16, true>), dim3(R), dim3(256), 0, st, qkv, pos, cos_t, sin_t, Hq,
                       Hkv, hd, (bf16 *)q_out, q_ps, (bf16 *)k_cache, (bf16 *)v_cache, kv_ps, S, slot0);
  else if (dtype == 0)
    hipLaunchKernelGGL((rope_scatter_kernel<bf16, false>), dim3(R), dim3(256), 0, st, qkv, pos, cos_t, sin_t, Hq,
                       Hkv, hd, (bf16 *)q_out, q_ps, (bf16 *)k_cache, (bf16 *)v_cache, kv_ps, S, slot0);
  else if (dtype == 2 && pair)
    hipLaunchKernelGGL((rope_scatter_kernel<f16, true>), dim3(R), dim3(256), 0, st, qkv, pos, cos_t, sin_t, Hq,
                       Hkv, hd, (f16 *)q_out, q_ps, (f16 *)k_cache, (f16 *)v_cache, kv_ps, S, slot0);
  else if (dtype == 2)
    hipLaunchKernelGGL((rope_scatter_kernel<f16, false>), dim3(R), dim3(256), 0, st, qkv, pos, cos_t, sin_t, Hq,
                       Hkv, hd, (f16 *)q_out, q_ps, (f16 *)k_cache, (f16 *)v_cache, kv_ps, S, slot0);
  else
    hipLaunchKernelGGL((rope_scatter_kernel<float, false>), dim3(R), dim3(256), 0, st, qkv, pos, cos_t, sin_t, Hq,
                       Hkv, hd, (float *)q_out, q_ps, (float *)k_cache, (float *)v_cache, kv_ps, S, slot0);
  return hipGetLastError();
}

hipError_t launch_lse_merge(const float *pm, const float *ps, int nsplit, int R, float *lse, const float *zt,
                            float wscale, float *ell, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (zt && !ell) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lse_merge_kernel, dim3((R + 255) / 256), dim3(256), 0, st, pm, ps, nsplit, R, lse, zt, wscale,
                     ell);
  return hipGetLastError();
}

hipError_t launch_token_rows(const int32_t *lm_row, int n, int row_base, const void *f_body, const void *f_last,
                             int64_t row_bytes, void *dst, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  if (row_bytes % 16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(token_rows_kernel, dim3(n), dim3(256), 0, st, lm_row, row_base, (const uint4 *)f_body,
                     (const uint4 *)f_last, row_bytes / 16, (uint4 *)dst);
  return hipGetLastError();
}

// dst row i = src row idx[i] (rows of row_bytes bytes, a multiple of 16).
__global__ __launch_bounds__(256) void gather_rows_kernel(const uint4 *__restrict__ src, int64_t row_chunks,
                                                          const int32_t *__restrict__ idx, uint4 *__restrict__ dst) {
  const int i = blockIdx.x;
  const uint4 *s = src + (int64_t)idx[i] * row_chunks;
  uint4 *d = dst + (int64_t)i * row_chunks;
  for (int64_t c = threadIdx.x; c < row_chunks; c += 256) d[c] = s[c];
}

hipError_t launch_gather_rows(const void *src, int64_t row_bytes, const int32_t *idx, int n, void *dst,
                              hipStream_t st) {
  if (n <= 0) return hipSuccess;
  if (row_bytes % 16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(n), dim3(256), 0, st, (const uint4 *)src, row_bytes / 16, idx,
                     (uint4 *)dst);
  return hipGetLastError();
}

hipError_t launch_segment_sum(const float *ell, const int64_t *off, int n, float *s, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(segment_sum_kernel, dim3((n + 255) / 256), dim3(256), 0, st, ell, off, n, s);
  return hipGetLastError();
}

hipError_t launch_count_bad_ids(const int32_t *ids, int64_t n, int V, int *bad, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 1024);
  hipLaunchKernelGGL(count_bad_ids_kernel, dim3(blocks), dim3(256), 0, st, ids, n, V, bad);
  return hipGetLastError();
}

hipError_t launch_convert_f32(int dtype, const float *src, int64_t n, void *dst, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 8192);
  if (dtype == 0) hipLaunchKernelGGL(convert_f32_kernel<bf16>, dim3(blocks), dim3(256), 0, st, src, n, (bf16 *)dst);
  else hipLaunchKernelGGL(convert_f32_kernel<float>, dim3(blocks), dim3(256), 0, st, src, n, (float *)dst);
  return hipGetLastError();
}

hipError_t launch_convert_bf16_to_f16(const uint16_t *src, int64_t n, float scale, void *dst,
                                      unsigned long long *inexact, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 8192);
  hipLaunchKernelGGL(bf16_to_f16_kernel, dim3(blocks), dim3(256), 0, st, src, n, scale, (f16 *)dst, inexact);
  return hipGetLastError();
}

hipError_t launch_convert_bf16_to_f32(const uint16_t *src, int64_t n, float *dst, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 8192);
  hipLaunchKernelGGL(bf16_to_f32_kernel, dim3(blocks), dim3(256), 0, st, src, n, dst);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// reasoning trace: cache layout, K/V append, sampling
// ---------------------------------------------------------------------------

// Question q's rows [offs[q], offs[q+1]) of every block of an [nblk][S_old]
// row cache go to rows offs[q] + q extra + i of the [nblk][S_new] cache.
__global__ __launch_bounds__(256) void kv_relayout_kernel(const uint4 *__restrict__ src, uint4 *__restrict__ dst,
                                                          const int64_t *__restrict__ offs, int64_t S_old,
                                                          int64_t S_new, int64_t row_chunks, int extra) {
  const int q = blockIdx.x, blk = blockIdx.y;
  const int64_t r0 = offs[q], n = (offs[q + 1] - r0) * row_chunks;
  const uint4 *s = src + ((int64_t)blk * S_old + r0) * row_chunks;
  uint4 *d = dst + ((int64_t)blk * S_new + r0 + (int64_t)q * extra) * row_chunks;
  for (int64_t c = threadIdx.x; c < n; c += 256) d[c] = s[c];
}

hipError_t launch_kv_relayout(const void *src, void *dst, const int64_t *offs, int n_q, int nblk, int64_t S_old,
                              int64_t S_new, int64_t row_bytes, int extra, hipStream_t st) {
  if (n_q <= 0 || nblk <= 0) return hipSuccess;
  if (row_bytes % 16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(kv_relayout_kernel, dim3(n_q, nblk), dim3(256), 0, st, (const uint4 *)src, (uint4 *)dst, offs,
                     S_old, S_new, row_bytes / 16, extra);
  return hipGetLastError();
}

// Row r of every block of tmp [nblk][R] goes to row slot[r] of the same block
// of cache [nblk][S].
__global__ __launch_bounds__(64) void kv_append_kernel(const uint4 *__restrict__ tmp, uint4 *__restrict__ cache,
                                                       const int32_t *__restrict__ slot, int R, int64_t S,
                                                       int64_t row_chunks) {
  const int r = blockIdx.x, blk = blockIdx.y;
  const uint4 *s = tmp + ((int64_t)blk * R + r) * row_chunks;
  uint4 *d = cache + ((int64_t)blk * S + slot[r]) * row_chunks;
  for (int64_t c = threadIdx.x; c < row_chunks; c += 64) d[c] = s[c];
}

hipError_t launch_kv_append(const void *tmp, void *cache, const int32_t *slot, int R, int nblk, int64_t S,
                            int64_t row_bytes, hipStream_t st) {
  if (R <= 0 || nblk <= 0) return hipSuccess;
  if (row_bytes % 16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(kv_append_kernel, dim3(R, nblk), dim3(64), 0, st, (const uint4 *)tmp, (uint4 *)cache, slot, R,
                     S, row_bytes / 16);
  return hipGetLastError();
}

// SplitMix64 (Steele, Lea and Flood, 2014): output i + 1 of the generator
// seeded with `seed`, i.e. the mix of seed + (i + 1) * golden gamma.
__device__ __forceinline__ uint64_t splitmix64_at(uint64_t seed, uint64_t i) {
  uint64_t z = seed + (i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Gumbel noise of (question q, step t, token v): -log(-log U), U the top 53
// bits of the counter's output mapped to the open interval (0, 1).
__device__ __forceinline__ double gumbel_at(uint64_t seed, int q, int t, int v) {
  const uint64_t i = ((uint64_t)q << 38) | ((uint64_t)t << 18) | (uint64_t)v;
  const double u = ((double)(splitmix64_at(seed, i) >> 11) + 0.5) * 0x1p-53;
  return -log(-log(u));
}

// Row r, slice y of the vocabulary (gridDim.y slices): the slice's largest
// key_v = z_v / tau + G_v (tau > 0) or z_v (tau = 0) and its token, the
// lowest v among equal keys, v = -1 if no key is a number.
constexpr int kSampleSplit = 32;

__global__ __launch_bounds__(256) void sample_part_kernel(const float *__restrict__ logits, int64_t ldl, int V,
                                                          double tau, uint64_t seed, int q0, int t,
                                                          double *__restrict__ pk, int *__restrict__ pv) {
  __shared__ double bk[256];
  __shared__ int bv[256];
  const int r = blockIdx.x, y = blockIdx.y, tid = threadIdx.x;
  const int per = (V + kSampleSplit - 1) / kSampleSplit, v0 = y * per, v1 = min(V, v0 + per);
  const float *z = logits + (int64_t)r * ldl;
  double best = 0.0;
  int arg = -1;
  for (int v = v0 + tid; v < v1; v += 256) {
    const double key = tau > 0.0 ? (double)z[v] / tau + gumbel_at(seed, q0 + r, t, v) : (double)z[v];
    if (key == key && (arg < 0 || key > best)) {  // v ascends: equal keys keep the lower v
      best = key;
      arg = v;
    }
  }
  bk[tid] = best;
  bv[tid] = arg;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (tid < o) {
      const int va = bv[tid], vb = bv[tid + o];
      const double ka = bk[tid], kb = bk[tid + o];
      if (vb >= 0 && (va < 0 || kb > ka || (kb == ka && vb < va))) {
        bk[tid] = kb;
        bv[tid] = vb;
      }
    }
    __syncthreads();
  }
  if (tid == 0) {
    pk[(int64_t)r * kSampleSplit + y] = bk[0];
    pv[(int64_t)r * kSampleSplit + y] = bv[0];
  }
}

// The row's token: the best of its slices (slices in vocabulary order, so
// the first of equal keys has the lowest v).
__global__ __launch_bounds__(64) void sample_pick_kernel(const double *__restrict__ pk, const int *__restrict__ pv,
                                                         int R, int32_t *__restrict__ tokens, int64_t ld_tok) {
  const int r = blockIdx.x * 64 + threadIdx.x;
  if (r >= R) return;
  double best = 0.0;
  int arg = -1;
  for (int y = 0; y < kSampleSplit; ++y) {
    const int v = pv[(int64_t)r * kSampleSplit + y];
    const double k = pk[(int64_t)r * kSampleSplit + y];
    if (v >= 0 && (arg < 0 || k > best)) {
      best = k;
      arg = v;
    }
  }
  tokens[(int64_t)r * ld_tok] = arg;
}

int sample_scratch_bytes(int R) { return R * kSampleSplit * (int)(sizeof(double) + sizeof(int)); }

hipError_t launch_sample(const float *logits, int64_t ldl, int R, int V, double tau, uint64_t seed, int q0, int t,
                         void *scratch, int32_t *tokens, int64_t ld_tok, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  double *pk = (double *)scratch;
  int *pv = (int *)(pk + (int64_t)R * kSampleSplit);
  hipLaunchKernelGGL(sample_part_kernel, dim3(R, kSampleSplit), dim3(256), 0, st, logits, ldl, V, tau, seed, q0, t,
                     pk, pv);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_pick_kernel, dim3((R + 63) / 64), dim3(64), 0, st, pk, pv, R, tokens, ld_tok);
  return hipGetLastError();
}

}  // namespace jetk
