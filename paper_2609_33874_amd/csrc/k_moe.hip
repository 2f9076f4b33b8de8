// Mixture-of-experts FFN pieces around the grouped expert GEMMs: top-k
// routing, placement of each (row, choice) in its expert's segment, the row
// scatter into that segment, and the weighted combine back into the residual.
//
// Layout: every expert owns a segment of the permuted row buffer that starts
// at a multiple of the grouped GEMM's tile rows (bm), so each row tile of the
// grouped GEMM belongs to one expert (tile_group[tile] = expert, -1 past the
// last segment). Places are given in (row, choice) order within each
// expert's segment (a counting sort over chunks of the choice list), so the
// permuted layout, and with it every result, is the same on every run; the
// combine adds a row's choices in the order of its top-k list.
#include "device.h"
#include "kernels.h"

namespace jetk {

// One wave per row: top_k experts by router logit (lowest index first among
// equal logits), their weights softmax over the kept logits, and the shared
// expert's gate sigmoid(logit[E]) when present.
__global__ __launch_bounds__(256) void moe_route_kernel(MoeRouteArgs a) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= a.R) return;
  const float *z = a.logits + (int64_t)r * a.ldl;
  constexpr int PER = kMoeMaxExperts / 64;
  float v[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = i * 64 + lane;
    v[i] = e < a.E ? z[e] : -INFINITY;
  }
  float zsel[kMoeMaxTopK];
  int esel[kMoeMaxTopK];
  for (int j = 0; j < a.top_k; ++j) {
    // lane-local best, ties to the lower index (indices grow with i)
    float bv = -INFINITY;
    int be = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = i * 64 + lane;
      if (e < a.E && (v[i] > bv || (v[i] == bv && e < be))) {
        bv = v[i];
        be = e;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o);
      const int oe = __shfl_xor(be, o);
      if (ov > bv || (ov == bv && oe < be)) {
        bv = ov;
        be = oe;
      }
    }
    if (be < 0 || be >= a.E) be = 0;  // only when no finite logit is left (NaN input)
    zsel[j] = bv;
    esel[j] = be;
#pragma unroll
    for (int i = 0; i < PER; ++i)
      if (i * 64 + lane == be) v[i] = -INFINITY;
  }
  if (lane != 0) return;
  // zsel[0] is the largest kept logit
  float s = 0.0f;
  for (int j = 0; j < a.top_k; ++j) s += __expf(zsel[j] - zsel[0]);
  const float inv = 1.0f / s;
  for (int j = 0; j < a.top_k; ++j) {
    a.sel[(int64_t)r * a.top_k + j] = esel[j];
    a.wts[(int64_t)r * a.top_k + j] = __expf(zsel[j] - zsel[0]) * inv;
  }
  if (a.shared_gate) a.shared_gate[r] = 1.0f / (1.0f + __expf(-z[a.E]));
}

// One workgroup: per-expert totals from the chunk counts, segment starts
// (totals rounded up to bm), the first place of each expert's entries in each
// chunk, and the expert of every row tile.
__global__ __launch_bounds__(256) void moe_plan_kernel(int E, int bm, int max_tiles, int *__restrict__ tile_group,
                                                       const int *__restrict__ chunk_hist, int nchunks,
                                                       int *__restrict__ chunk_base) {
  __shared__ int off[kMoeMaxExperts + 1];
  for (int e = threadIdx.x; e < E; e += 256) {
    int t = 0;
    for (int c = 0; c < nchunks; ++c) t += chunk_hist[(int64_t)c * E + e];
    off[e] = t;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int e = 0; e < E; ++e) {
      const int t = off[e];
      off[e] = acc;
      acc += (t + bm - 1) / bm * bm;
    }
    off[E] = acc;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += 256) {
    int acc = off[e];
    for (int c = 0; c < nchunks; ++c) {
      chunk_base[(int64_t)c * E + e] = acc;
      acc += chunk_hist[(int64_t)c * E + e];
    }
  }
  for (int t = threadIdx.x; t < max_tiles; t += 256) {
    const int row = t * bm;
    int g = -1;
    if (row < off[E]) {
      int lo = 0, hi = E - 1;  // last e with off[e] <= row
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (off[mid] <= row) lo = mid;
        else hi = mid - 1;
      }
      g = lo;
    }
    tile_group[t] = g;
  }
}

// Entries of the choice list (i = row * top_k + j) per expert in each chunk of
// kMoeChunk entries (one wave per chunk).
__global__ __launch_bounds__(64) void moe_count_kernel(const int *__restrict__ sel, int n, int E,
                                                       int *__restrict__ chunk_hist) {
  __shared__ int h[kMoeMaxExperts];
  const int lane = threadIdx.x, c = blockIdx.x;
  for (int e = lane; e < E; e += 64) h[e] = 0;
  __syncthreads();
  const int i0 = c * kMoeChunk, i1 = min(n, i0 + kMoeChunk);
  for (int i = i0 + lane; i < i1; i += 64) atomicAdd(&h[sel[i]], 1);
  __syncthreads();
  for (int e = lane; e < E; e += 64) chunk_hist[(int64_t)c * E + e] = h[e];
}

// Places in list order (one wave per chunk): entry i of expert e gets
// chunk_base[chunk][e] + (entries of e before i in the chunk).
__global__ __launch_bounds__(64) void moe_assign_kernel(const int *__restrict__ sel, int n, int E,
                                                        const int *__restrict__ chunk_base,
                                                        int *__restrict__ slot_of) {
  __shared__ int cnt[kMoeMaxExperts];
  __shared__ int eb[64];
  const int lane = threadIdx.x, c = blockIdx.x;
  for (int e = lane; e < E; e += 64) cnt[e] = chunk_base[(int64_t)c * E + e];
  __syncthreads();
  const int i0 = c * kMoeChunk, i1 = min(n, i0 + kMoeChunk);
  for (int b = i0; b < i1; b += 64) {
    const int i = b + lane;
    const int e = i < i1 ? sel[i] : -1;
    eb[lane] = e;
    __syncthreads();
    int before = 0, after = 0;
    for (int j = 0; j < 64; ++j) {
      const int ej = eb[j];
      before += (j < lane && ej == e);
      after += (j > lane && ej == e);
    }
    if (e >= 0) slot_of[i] = cnt[e] + before;
    __syncthreads();
    if (e >= 0 && after == 0) cnt[e] += before + 1;  // the last entry of e in this step
    __syncthreads();
  }
}

// One wave per entry: row i / top_k of x copied to row slot_of[i] of xp
// (row_chunks 16-byte chunks per row).
__global__ __launch_bounds__(256) void moe_scatter_kernel(const uint4 *__restrict__ x, int64_t row_chunks, int n,
                                                          int top_k, const int *__restrict__ slot_of,
                                                          uint4 *__restrict__ xp) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= n) return;
  const uint4 *src = x + (int64_t)(i / top_k) * row_chunks;
  uint4 *dst = xp + (int64_t)slot_of[i] * row_chunks;
  for (int64_t c = lane; c < row_chunks; c += 64) dst[c] = src[c];
}

// One workgroup per row: resid += sum_j w_j y[slot_j] (j in top-k order)
// + g * y_shared, the mixture summed first, in fp32 (expert outputs y are
// stored in the compute type).
template <typename T>
__global__ __launch_bounds__(256) void moe_combine_kernel(const T *__restrict__ y, const int *__restrict__ slot_of,
                                                          const float *__restrict__ wts, int top_k,
                                                          const float *__restrict__ ys,
                                                          const float *__restrict__ gate, int d,
                                                          float *__restrict__ resid) {
  const int r = blockIdx.x;
  const int *sl = slot_of + (int64_t)r * top_k;
  const float *w = wts + (int64_t)r * top_k;
  for (int c = threadIdx.x * 4; c < d; c += 1024) {
    float o[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int j = 0; j < top_k; ++j) {
      const T *v = y + (int64_t)sl[j] * d + c;
      const float wj = w[j];
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] += wj * to_f<T>(v[q]);
    }
    if (ys) {
      const float g = gate[r];
      const float4 v = *(const float4 *)(ys + (int64_t)r * d + c);
      o[0] += g * v.x;
      o[1] += g * v.y;
      o[2] += g * v.z;
      o[3] += g * v.w;
    }
    float4 *dst = (float4 *)(resid + (int64_t)r * d + c);
    float4 x = *dst;
    x.x += o[0];
    x.y += o[1];
    x.z += o[2];
    x.w += o[3];
    *dst = x;
  }
}

hipError_t launch_moe_route(const MoeRouteArgs &a, hipStream_t st) {
  if (a.R <= 0) return hipSuccess;
  if (a.E < 1 || a.E > kMoeMaxExperts || a.top_k < 1 || a.top_k > kMoeMaxTopK || a.top_k > a.E)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(moe_route_kernel, dim3((a.R + 3) / 4), dim3(256), 0, st, a);
  return hipGetLastError();
}

int moe_chunks(int R, int top_k) { return (R * top_k + kMoeChunk - 1) / kMoeChunk; }

hipError_t launch_moe_plan(const int *sel, int R, int top_k, int E, int bm, int max_tiles, int *tile_group,
                           int *chunk_hist, int *chunk_base, int *slot_of, hipStream_t st) {
  if (E < 1 || E > kMoeMaxExperts || bm < 1 || max_tiles < 0 || R < 0 || top_k < 1) return hipErrorInvalidValue;
  const int n = R * top_k, nchunks = moe_chunks(R, top_k);
  if (nchunks > 0) hipLaunchKernelGGL(moe_count_kernel, dim3(nchunks), dim3(64), 0, st, sel, n, E, chunk_hist);
  hipLaunchKernelGGL(moe_plan_kernel, dim3(1), dim3(256), 0, st, E, bm, max_tiles, tile_group, chunk_hist, nchunks,
                     chunk_base);
  if (nchunks > 0) hipLaunchKernelGGL(moe_assign_kernel, dim3(nchunks), dim3(64), 0, st, sel, n, E, chunk_base, slot_of);
  return hipGetLastError();
}

hipError_t launch_moe_scatter(const void *x, int64_t row_bytes, int R, int top_k, const int *slot_of, void *xp,
                              hipStream_t st) {
  const int n = R * top_k;
  if (n <= 0) return hipSuccess;
  if (row_bytes % 16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(moe_scatter_kernel, dim3((n + 3) / 4), dim3(256), 0, st, (const uint4 *)x, row_bytes / 16, n,
                     top_k, slot_of, (uint4 *)xp);
  return hipGetLastError();
}

hipError_t launch_moe_combine(int dtype, const void *y, const int *slot_of, const float *wts, int top_k,
                              const float *ys, const float *gate, int R, int d, float *resid, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (d % 4) return hipErrorInvalidValue;
  if (dtype == 2)
    hipLaunchKernelGGL(moe_combine_kernel<f16>, dim3(R), dim3(256), 0, st, (const f16 *)y, slot_of, wts, top_k, ys,
                       gate, d, resid);
  else if (dtype == 0)
    hipLaunchKernelGGL(moe_combine_kernel<bf16>, dim3(R), dim3(256), 0, st, (const bf16 *)y, slot_of, wts, top_k, ys,
                       gate, d, resid);
  else
    hipLaunchKernelGGL(moe_combine_kernel<float>, dim3(R), dim3(256), 0, st, (const float *)y, slot_of, wts, top_k,
                       ys, gate, d, resid);
  return hipGetLastError();
}

}  // namespace jetk
