// Matrix-core GEMM core for gfx950: acc = A[m0:m0+BM, :] * B[n0:n0+BN, :]^T
// with A [M][K] and B [N][K] both K-contiguous, fp32 accumulation in 32x32
// MFMA blocks.
//
// Per K step every row of the A and B tiles contributes 128 bytes (64 bf16 /
// 32 fp32) = 8 chunks of 16 B. In LDS, chunk c of tile row r is stored at
// position c ^ swz(r) of that row, so the MFMA operand reads (one row per
// lane, same logical chunk) spread over all banks. Two LDS buffers alternate.
// Tiles reach LDS either through registers (global load, then ds_write) or
// directly (global_load_lds_dwordx4: each wave instruction fills 1 KB = 8
// tile rows, lane L filling physical chunk L % 8 of row L / 8, so it fetches
// the logical chunk (L % 8) ^ swz(row)).
#pragma once

#include "device.h"

namespace jetk {

template <typename T, int BM_, int BN_, int WM_, int WN_, int LOAD_ = 0, int SWZ_ = 0>
struct GCfg {
  using type = T;
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, LOAD = LOAD_, SWZ = SWZ_;
  static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN, NWAVES = WAVES_M * WAVES_N;
  static constexpr int NT = NWAVES * 64;
  static constexpr int MI = WM / 32, NI = WN / 32;
  static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  static constexpr int BK = 8 * EPC;                // elements per K step (128 B per row)
  static constexpr int A_PT = BM * 8 / NT, B_PT = BN * 8 / NT;  // chunks per thread per K step
  static constexpr int BUF = (BM + BN) * 8;                      // chunks per LDS buffer
  static constexpr size_t LDS_BYTES = sizeof(uint4) * 2 * BUF;
  static_assert(BM * 8 % NT == 0 && BN * 8 % NT == 0, "tile/thread mismatch");
  static_assert(BM % (8 * NWAVES) == 0 && BN % (8 * NWAVES) == 0, "direct loads fill 8 rows per wave");
};

template <int SWZ>
__device__ __forceinline__ int lds_swz(int r) {
  if constexpr (SWZ == 0) return r & 7;
  else return (r >> 1) & 7;
}

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

typedef __attribute__((address_space(3))) void lds_void;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Tile order: blockIdx.x enumerates tiles; workgroups are dealt round-robin to
// the 8 XCDs, so tile ids are remapped to give each XCD a contiguous band of
// tiles (which share A rows in its L2), and inside the band tiles run in
// groups of GM row-tiles so consecutive tiles also share B columns.
template <int GM>
__device__ __forceinline__ void tile_coords(int nt_m, int nt_n, int *tm, int *tn) {
  const int ntiles = nt_m * nt_n;
  int id = blockIdx.x;
  const int per = ntiles / 8;  // tiles per XCD (the remainder keeps its id)
  if (id < per * 8) id = (id & 7) * per + (id >> 3);
  const int group = GM * nt_n;
  const int g = id / group, first_m = g * GM;
  const int gm = min(nt_m - first_m, GM);
  const int in = id % group;
  *tm = first_m + in % gm;
  *tn = in / gm;
}

template <class C>
__device__ __forceinline__ void zero_acc(f32x16 (&acc)[C::MI][C::NI]) {
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
#pragma unroll
    for (int j = 0; j < C::NI; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;
}

// One K step of MFMAs from LDS buffer `buf`.
template <class C>
__device__ __forceinline__ void tile_compute(const uint4 *__restrict__ lds, int buf, int lane, int wm, int wn,
                                             f32x16 (&acc)[C::MI][C::NI]) {
  using T = typename C::type;
  const uint4 *a = lds + buf * C::BUF, *b = a + C::BM * 8;
#pragma unroll
  for (int kk = 0; kk < C::BK / 16; ++kk) {
    const int c0 = (kk * 16 + (lane >> 5) * 8) / C::EPC;
    Frag<T> fa[C::MI], fb[C::NI];
#pragma unroll
    for (int i = 0; i < C::MI; ++i) {
      const int r = wm * C::WM + i * 32 + (lane & 31);
      lds_frag<T>(fa[i], a + r * 8, c0, lds_swz<C::SWZ>(r));
    }
#pragma unroll
    for (int j = 0; j < C::NI; ++j) {
      const int r = wn * C::WN + j * 32 + (lane & 31);
      lds_frag<T>(fb[j], b + r * 8, c0, lds_swz<C::SWZ>(r));
    }
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int j = 0; j < C::NI; ++j) mma32(acc[i][j], fa[i], fb[j]);
  }
}

// Register path: global -> registers.
template <class C>
__device__ __forceinline__ void tile_gload(const typename C::type *__restrict__ A, int64_t lda,
                                           const typename C::type *__restrict__ B, int64_t ldb, int M, int N,
                                           int m0, int n0, int ka, int kb, int tid, uint4 (&ra)[C::A_PT],
                                           uint4 (&rb)[C::B_PT]) {
  const uint4 zero4 = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int i = 0; i < C::A_PT; ++i) {
    const int ch = tid + i * C::NT, r = ch >> 3, c = ch & 7, gm = m0 + r;
    ra[i] = gm < M ? ld16(A + (int64_t)gm * lda + ka + c * C::EPC) : zero4;
  }
#pragma unroll
  for (int i = 0; i < C::B_PT; ++i) {
    const int ch = tid + i * C::NT, r = ch >> 3, c = ch & 7, gn = n0 + r;
    rb[i] = gn < N ? ld16(B + (int64_t)gn * ldb + kb + c * C::EPC) : zero4;
  }
}

// Register path: registers -> LDS buffer `buf` (swizzled).
template <class C>
__device__ __forceinline__ void tile_lstore(uint4 *__restrict__ lds, int buf, int tid, const uint4 (&ra)[C::A_PT],
                                            const uint4 (&rb)[C::B_PT]) {
  uint4 *a = lds + buf * C::BUF, *b = a + C::BM * 8;
#pragma unroll
  for (int i = 0; i < C::A_PT; ++i) {
    const int ch = tid + i * C::NT, r = ch >> 3, c = ch & 7;
    a[r * 8 + (c ^ lds_swz<C::SWZ>(r))] = ra[i];
  }
#pragma unroll
  for (int i = 0; i < C::B_PT; ++i) {
    const int ch = tid + i * C::NT, r = ch >> 3, c = ch & 7;
    b[r * 8 + (c ^ lds_swz<C::SWZ>(r))] = rb[i];
  }
}

// Direct path: global -> LDS buffer `buf`; rows beyond M / N are clamped to
// the last valid row (their outputs are discarded by the caller).
template <class C>
__device__ __forceinline__ void tile_issue_direct(const typename C::type *__restrict__ A, int64_t lda,
                                                  const typename C::type *__restrict__ B, int64_t ldb, int M,
                                                  int N, int m0, int n0, int ka, int kb, uint4 *lds, int buf,
                                                  int wave, int lane) {
  uint4 *a = lds + buf * C::BUF, *b = a + C::BM * 8;
  const int sub_r = lane >> 3;
#pragma unroll
  for (int i = 0; i < C::A_PT; ++i) {
    const int blk = i * C::NWAVES + wave;
    const int r = blk * 8 + sub_r;
    const int c = (lane & 7) ^ lds_swz<C::SWZ>(r);
    const int gm = min(m0 + r, M - 1);
    __builtin_amdgcn_global_load_lds((const void *)(A + (int64_t)gm * lda + ka + c * C::EPC),
                                     (lds_void *)(a + blk * 64), 16, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < C::B_PT; ++i) {
    const int blk = i * C::NWAVES + wave;
    const int r = blk * 8 + sub_r;
    const int c = (lane & 7) ^ lds_swz<C::SWZ>(r);
    const int gn = min(n0 + r, N - 1);
    __builtin_amdgcn_global_load_lds((const void *)(B + (int64_t)gn * ldb + kb + c * C::EPC),
                                     (lds_void *)(b + blk * 64), 16, 0, 0);
  }
}

// acc = sum over k < K of A[m0 + r][k mod KA] * B[n0 + c][k mod KB]: a plain
// GEMM when K = KA = KB; with K = 2 KB and KA = K the A rows hold a (hi, lo)
// bf16 pair of each activation, [a_hi | a_lo], and B is read twice, so the
// product is B (a_hi + a_lo) (and symmetrically with A read twice). K, KA and
// KB must be multiples of C::BK. Ends with a barrier, so the caller may reuse
// the LDS right after.
template <class C>
__device__ __forceinline__ void gemm_tile(const typename C::type *__restrict__ A, int64_t lda,
                                          const typename C::type *__restrict__ B, int64_t ldb, int M, int N,
                                          int K, int KA, int KB, int m0, int n0, uint4 *lds,
                                          f32x16 (&acc)[C::MI][C::NI]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  zero_acc<C>(acc);
  const int nk = K / C::BK;
  auto kmod = [](int k, int kk) { return k >= kk ? k - kk : k; };
  if constexpr (C::LOAD == 0) {
    uint4 ra[C::A_PT], rb[C::B_PT];
    tile_gload<C>(A, lda, B, ldb, M, N, m0, n0, 0, 0, tid, ra, rb);
    tile_lstore<C>(lds, 0, tid, ra, rb);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const bool more = kt + 1 < nk;
      const int k1 = (kt + 1) * C::BK;
      if (more) tile_gload<C>(A, lda, B, ldb, M, N, m0, n0, kmod(k1, KA), kmod(k1, KB), tid, ra, rb);
      tile_compute<C>(lds, kt & 1, lane, wm, wn, acc);
      if (more) tile_lstore<C>(lds, (kt + 1) & 1, tid, ra, rb);
      __syncthreads();
    }
  } else {
    tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, 0, 0, lds, 0, wave, lane);
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) {
        const int k1 = (kt + 1) * C::BK;
        tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, kmod(k1, KA), kmod(k1, KB), lds, (kt + 1) & 1, wave,
                             lane);
        wait_vmcnt<C::A_PT + C::B_PT>();
      } else {
        wait_vmcnt<0>();
      }
      __syncthreads();
      tile_compute<C>(lds, kt & 1, lane, wm, wn, acc);
      __syncthreads();
    }
  }
}

}  // namespace jetk
