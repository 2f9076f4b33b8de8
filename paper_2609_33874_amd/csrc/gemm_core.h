// Matrix-core GEMM core for gfx950: acc = A[m0:m0+BM, :] * B[n0:n0+BN, :]^T
// with A [M][K] and B [N][K] both K-contiguous, fp32 accumulation in 32x32
// MFMA blocks.
//
// Per K step every row of the A and B tiles contributes CPR chunks of 16 B
// (CPR = 8: 64 bf16 / 32 fp32; CPR = 4: half of that). In LDS, chunk c of tile
// row r is stored at position c ^ swz(r) of that row, so that the 16 lanes
// the LDS serves per clock (one row each, same logical chunk) hit distinct
// banks. Tiles reach LDS either through registers (global load, then
// ds_write; LOAD 0, two stages) or directly (global_load_lds_dwordx4: each
// wave instruction fills 1 KB = 64 / CPR tile rows, lane L filling physical
// chunk L % CPR, so it fetches logical chunk (L % CPR) ^ swz(row); LOAD 1 with
// two stages, LOAD 2 with NSTAGE stages and one barrier per K step).
// Rows beyond M / N load a clamped valid row; their outputs are discarded.
#pragma once

#include "device.h"

namespace jetk {

template <typename T, int BM_, int BN_, int WM_, int WN_, int LOAD_ = 0, int SWZ_ = 0, int NSTAGE_ = 2,
          int CPR_ = 8>
struct GCfg {
  using type = T;
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, LOAD = LOAD_, SWZ = SWZ_;
  static constexpr int NSTAGE = NSTAGE_, CPR = CPR_;
  static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN, NWAVES = WAVES_M * WAVES_N;
  static constexpr int NT = NWAVES * 64;
  static constexpr int MI = WM / 32, NI = WN / 32;
  static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  static constexpr int BK = CPR * EPC;              // elements per K step
  static constexpr int A_PT = BM * CPR / NT, B_PT = BN * CPR / NT;  // chunks per thread per K step
  static constexpr int BUF = (BM + BN) * CPR;                        // chunks per LDS stage
  static constexpr size_t LDS_BYTES = sizeof(uint4) * NSTAGE * BUF;
  static constexpr int RPI = 64 / CPR;  // tile rows per direct-load wave instruction
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile/thread mismatch");
  static_assert(BM % (RPI * NWAVES) == 0 && BN % (RPI * NWAVES) == 0, "direct loads fill whole row groups");
  static_assert(BK % 16 == 0, "K step must hold whole MFMA steps");
  static_assert(LOAD >= 2 ? NSTAGE >= 3 : NSTAGE == 2, "pipeline depth");
  static_assert(LOAD != 3 || NWAVES == 8, "ping-pong needs two groups of four waves");
};

// SWZ 0: c ^ (r mod CPR). SWZ 1 (CPR 8): c ^ ((r >> 1) & 7). SWZ 2 (CPR 4):
// c ^ ((r >> 2) & 3). With 256-byte LDS lines, 1 and 2 give 16 consecutive
// rows distinct banks for one logical chunk.
template <class C>
__device__ __forceinline__ int lds_swz(int r) {
  if constexpr (C::SWZ == 0) return r & (C::CPR - 1);
  else if constexpr (C::SWZ == 1) return (r >> 1) & 7;
  else return (r >> 2) & 3;
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

__device__ __forceinline__ void wait_lgkmcnt0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Waits until at most `tiles` K steps of direct loads (PT each) are in flight.
template <int PT, int MAXT>
__device__ __forceinline__ void wait_tiles(int tiles) {
  if constexpr (MAXT >= 3) {
    if (tiles >= 3) { wait_vmcnt<3 * PT>(); return; }
  }
  if constexpr (MAXT >= 2) {
    if (tiles == 2) { wait_vmcnt<2 * PT>(); return; }
  }
  if constexpr (MAXT >= 1) {
    if (tiles == 1) { wait_vmcnt<PT>(); return; }
  }
  wait_vmcnt<0>();
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
  const uint4 *a = lds + buf * C::BUF, *b = a + C::BM * C::CPR;
#pragma unroll
  for (int kk = 0; kk < C::BK / 16; ++kk) {
    const int c0 = (kk * 16 + (lane >> 5) * 8) / C::EPC;
    Frag<T> fa[C::MI], fb[C::NI];
#pragma unroll
    for (int i = 0; i < C::MI; ++i) {
      const int r = wm * C::WM + i * 32 + (lane & 31);
      lds_frag<T>(fa[i], a + r * C::CPR, c0, lds_swz<C>(r));
    }
#pragma unroll
    for (int j = 0; j < C::NI; ++j) {
      const int r = wn * C::WN + j * 32 + (lane & 31);
      lds_frag<T>(fb[j], b + r * C::CPR, c0, lds_swz<C>(r));
    }
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int j = 0; j < C::NI; ++j) mma32(acc[i][j], fa[i], fb[j]);
  }
}

// Fragments of one K step from LDS stage `buf` into registers.
template <class C>
__device__ __forceinline__ void tile_frags(const uint4 *__restrict__ lds, int buf, int lane, int wm, int wn,
                                           Frag<typename C::type> (&fa)[C::BK / 16][C::MI],
                                           Frag<typename C::type> (&fb)[C::BK / 16][C::NI]) {
  using T = typename C::type;
  const uint4 *a = lds + buf * C::BUF, *b = a + C::BM * C::CPR;
#pragma unroll
  for (int kk = 0; kk < C::BK / 16; ++kk) {
    const int c0 = (kk * 16 + (lane >> 5) * 8) / C::EPC;
#pragma unroll
    for (int i = 0; i < C::MI; ++i) {
      const int r = wm * C::WM + i * 32 + (lane & 31);
      lds_frag<T>(fa[kk][i], a + r * C::CPR, c0, lds_swz<C>(r));
    }
#pragma unroll
    for (int j = 0; j < C::NI; ++j) {
      const int r = wn * C::WN + j * 32 + (lane & 31);
      lds_frag<T>(fb[kk][j], b + r * C::CPR, c0, lds_swz<C>(r));
    }
  }
}

template <class C>
__device__ __forceinline__ void tile_mma(const Frag<typename C::type> (&fa)[C::BK / 16][C::MI],
                                         const Frag<typename C::type> (&fb)[C::BK / 16][C::NI],
                                         f32x16 (&acc)[C::MI][C::NI]) {
#pragma unroll
  for (int kk = 0; kk < C::BK / 16; ++kk)
#pragma unroll
    for (int i = 0; i < C::MI; ++i)
#pragma unroll
      for (int j = 0; j < C::NI; ++j) mma32(acc[i][j], fa[kk][i], fb[kk][j]);
}

// Register path: global -> registers.
template <class C>
__device__ __forceinline__ void tile_gload(const typename C::type *__restrict__ A, int64_t lda,
                                           const typename C::type *__restrict__ B, int64_t ldb, int M, int N,
                                           int m0, int n0, int ka, int kb, int tid, uint4 (&ra)[C::A_PT],
                                           uint4 (&rb)[C::B_PT]) {
#pragma unroll
  for (int i = 0; i < C::A_PT; ++i) {
    const int ch = tid + i * C::NT, r = ch / C::CPR, c = ch % C::CPR, gm = min(m0 + r, M - 1);
    ra[i] = ld16(A + (int64_t)gm * lda + ka + c * C::EPC);
  }
#pragma unroll
  for (int i = 0; i < C::B_PT; ++i) {
    const int ch = tid + i * C::NT, r = ch / C::CPR, c = ch % C::CPR, gn = min(n0 + r, N - 1);
    rb[i] = ld16(B + (int64_t)gn * ldb + kb + c * C::EPC);
  }
}

// Register path: registers -> LDS buffer `buf` (swizzled).
template <class C>
__device__ __forceinline__ void tile_lstore(uint4 *__restrict__ lds, int buf, int tid, const uint4 (&ra)[C::A_PT],
                                            const uint4 (&rb)[C::B_PT]) {
  uint4 *a = lds + buf * C::BUF, *b = a + C::BM * C::CPR;
#pragma unroll
  for (int i = 0; i < C::A_PT; ++i) {
    const int ch = tid + i * C::NT, r = ch / C::CPR, c = ch % C::CPR;
    a[r * C::CPR + (c ^ lds_swz<C>(r))] = ra[i];
  }
#pragma unroll
  for (int i = 0; i < C::B_PT; ++i) {
    const int ch = tid + i * C::NT, r = ch / C::CPR, c = ch % C::CPR;
    b[r * C::CPR + (c ^ lds_swz<C>(r))] = rb[i];
  }
}

// Direct path: global -> LDS buffer `buf`; rows beyond M / N are clamped to
// the last valid row (their outputs are discarded by the caller).
template <class C>
__device__ __forceinline__ void tile_issue_direct(const typename C::type *__restrict__ A, int64_t lda,
                                                  const typename C::type *__restrict__ B, int64_t ldb, int M,
                                                  int N, int m0, int n0, int ka, int kb, uint4 *lds, int buf,
                                                  int wave, int lane) {
  uint4 *a = lds + buf * C::BUF, *b = a + C::BM * C::CPR;
  const int sub_r = lane / C::CPR, pc = lane % C::CPR;
#pragma unroll
  for (int i = 0; i < C::A_PT; ++i) {
    const int blk = i * C::NWAVES + wave;
    const int r = blk * C::RPI + sub_r;
    const int c = pc ^ lds_swz<C>(r);
    const int gm = min(m0 + r, M - 1);
    __builtin_amdgcn_global_load_lds((const void *)(A + (int64_t)gm * lda + ka + c * C::EPC),
                                     (lds_void *)(a + blk * 64), 16, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < C::B_PT; ++i) {
    const int blk = i * C::NWAVES + wave;
    const int r = blk * C::RPI + sub_r;
    const int c = pc ^ lds_swz<C>(r);
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
  } else if constexpr (C::LOAD == 2) {
    // NSTAGE-deep pipeline, one barrier per K step: the barrier of step kt
    // certifies that every wave's loads of tile kt have landed and that every
    // wave is done reading the stage that tile kt + NSTAGE - 1 overwrites.
    constexpr int PT = C::A_PT + C::B_PT, AHEAD = C::NSTAGE - 1;
#pragma unroll
    for (int s = 0; s < AHEAD; ++s)
      if (s < nk)
        tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, kmod(s * C::BK, KA), kmod(s * C::BK, KB), lds, s, wave,
                             lane);
    for (int kt = 0; kt < nk; ++kt) {
      wait_tiles<PT, AHEAD - 1>(min(AHEAD - 1, nk - 1 - kt));
      wait_lgkmcnt0();
      __builtin_amdgcn_s_barrier();
      const int kn = kt + AHEAD;
      if (kn < nk)
        tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, kmod(kn * C::BK, KA), kmod(kn * C::BK, KB), lds,
                             kn % C::NSTAGE, wave, lane);
      tile_compute<C>(lds, kt % C::NSTAGE, lane, wm, wn, acc);
    }
    wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
  } else if constexpr (C::LOAD == 3) {
    // Ping-pong: waves 0-3 and 4-7 (one per SIMD in each group) alternate
    // between a load phase (direct loads of a later tile, LDS -> registers for
    // this tile) and an MFMA phase, one phase apart, with one barrier per
    // phase; so on every SIMD one wave feeds the matrix core while the other
    // loads. Hazards: a wave issues the loads of tile kt + NSTAGE - 1 into the
    // stage of tile kt - 1 during its load phase of tile kt, after both groups
    // finished reading tile kt - 1 (each waited for its LDS reads before the
    // barrier that ended its load phase of kt - 1); every wave waits for its
    // own loads of tile kt + 1 before its load phase of kt ends, and the
    // barrier after that phase precedes any read of tile kt + 1.
    constexpr int PT = C::A_PT + C::B_PT, AHEAD = C::NSTAGE - 1;
    const int grp = wave >> 2;
#pragma unroll
    for (int s = 0; s < AHEAD; ++s)
      if (s < nk)
        tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, kmod(s * C::BK, KA), kmod(s * C::BK, KB), lds, s, wave,
                             lane);
    wait_tiles<PT, AHEAD - 1>(min(AHEAD - 1, nk - 1));
    __builtin_amdgcn_s_barrier();
    if (grp == 1) __builtin_amdgcn_s_barrier();
    Frag<typename C::type> fa[C::BK / 16][C::MI], fb[C::BK / 16][C::NI];
    for (int kt = 0; kt < nk; ++kt) {
      tile_frags<C>(lds, kt % C::NSTAGE, lane, wm, wn, fa, fb);
      const int kn = kt + AHEAD;
      if (kn < nk)
        tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, kmod(kn * C::BK, KA), kmod(kn * C::BK, KB), lds,
                             kn % C::NSTAGE, wave, lane);
      wait_tiles<PT, AHEAD - 1>(max(0, min(AHEAD - 1, nk - 2 - kt)));
      wait_lgkmcnt0();
      __builtin_amdgcn_s_barrier();
      tile_mma<C>(fa, fb, acc);
      __builtin_amdgcn_s_barrier();
    }
    if (grp == 0) __builtin_amdgcn_s_barrier();
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
