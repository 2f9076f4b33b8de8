// Matrix-core GEMM core for gfx950: acc = A[m0:m0+BM, :] * B[n0:n0+BN, :]^T
// with A [M][K] and B [N][K] both K-contiguous, fp32 accumulation in 32x32
// MFMA blocks.
//
// Per K step every row of the A and B tiles contributes CPR chunks of 16 B
// (CPR = 8: 64 bf16 / 32 fp32; CPR = 4: half of that). In LDS, chunk c of tile
// row r is stored at position c ^ swz(r) of that row, so that the 16 lanes
// the LDS serves per clock (one row each, same logical chunk) hit distinct
// banks. Tile schedules:
//   LOAD 0  global -> registers -> ds_write, two stages (any element type);
//   LOAD 2  global_load_lds_dwordx4 straight into LDS (each wave instruction
//           fills 1 KB = 64 / CPR tile rows, lane L filling physical chunk
//           L % CPR, so it fetches logical chunk (L % CPR) ^ swz(row)),
//           NSTAGE stages, NSTAGE - 1 K steps in flight, one barrier per step;
//   LOAD 4  as LOAD 2 with the MFMA fragments read one MFMA step ahead into
//           registers (bf16), all NSTAGE stages in flight;
//   LOAD 7  for a (hi, lo) pair A operand: a stage holds the hi and lo tiles
//           of A and one B tile, so every B fragment feeds both products;
//           NSTAGE - 1 K steps in flight, each step's loads interleaved with
//           the MFMAs of the step before it (fixed by scheduling groups);
//   LOAD 8  the LOAD 7 schedule for a plain (single-plane) A operand.
//   LOAD 9  the LOAD 8 schedule with an int8 B operand: the stored values q
//           of a block-quantized weight matrix (blocks of 32 along K) and one
//           fp16 scale per (row, block), a power of two; a stage holds the A
//           tile, the B tile as [K chunk][row] 16-byte units and the tile's
//           scales, and each B fragment is turned into fp16 q * scale in
//           registers (exact) before its MFMAs.
// Rows beyond M / N load a clamped valid row; their outputs are discarded.
#pragma once

#include <utility>

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
  // LOAD 7 (pair-aware): A holds (hi, lo) planes and both are staged, B once
  static constexpr bool PAIRA = LOAD == 7;
  static constexpr bool INTERLEAVED = LOAD == 7 || LOAD == 8;  // the LOAD 7 / 8 schedule
  // block-quantized B with per-block scales: int8 (LOAD 9) or int4 (LOAD 10)
  static constexpr int QBITS = LOAD == 9 ? 8 : LOAD == 10 ? 4 : 0;
  static constexpr bool Q8B = QBITS > 0;
  static constexpr int BROW0 = PAIRA ? 2 * BM : BM;                  // first B row of a stage
  static constexpr int B_CH = Q8B ? BK * QBITS / 128 : BK / 16;     // quantized B: 16-byte chunks per row per K step
  static constexpr int A_PT = BM * CPR / NT;                         // chunks per thread per K step (per plane)
  // quantized B: B_CH * BN chunks per K step, 64 per wave (one direct load
  // each) or, for int4 tiles of 32 per wave, one load with half the lanes
  static constexpr int B_PT = Q8B ? (B_CH * BN >= NT ? B_CH * BN / NT : 1) : BN * CPR / NT;
  static constexpr int BUF = Q8B ? BM * CPR + B_CH * BN + BN / 8 : (BROW0 + BN) * CPR;  // chunks per LDS stage
  static constexpr size_t LDS_BYTES = sizeof(uint4) * NSTAGE * BUF;
  static constexpr int RPI = 64 / CPR;  // tile rows per direct-load wave instruction
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile/thread mismatch");
  static_assert(BM % (RPI * NWAVES) == 0 && BN % (RPI * NWAVES) == 0, "direct loads fill whole row groups");
  static_assert(BK % 16 == 0, "K step must hold whole MFMA steps");
  static_assert(LOAD == 0 || LOAD == 2 || LOAD == 4 || LOAD == 7 || LOAD == 8 || LOAD == 9 || LOAD == 10,
                "tile load schedule");
  static_assert(!Q8B || (BK == 32 && (B_CH * BN % (64 * NWAVES) == 0 || B_CH * BN == 32 * NWAVES) &&
                         BN / 8 == 4 * NWAVES && WN <= 128 && 128 % WN == 0),
                "quantized B: one quantization block per K step, whole direct-load rounds, 4 scale chunks per wave");
  static_assert(INTERLEAVED || Q8B ? NSTAGE >= 2 : LOAD >= 4 ? NSTAGE >= 2 : LOAD == 2 ? NSTAGE >= 3 : NSTAGE == 2,
                "pipeline depth");
  static_assert(LOAD < 4 || (BK / 16) % 2 == 0, "fragment pipelining alternates two register sets");
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
__device__ __forceinline__ void lds_frag<f16>(Frag<f16> &f, const uint4 *row, int c0, int swz) {
  f.v = __builtin_bit_cast(f16x8, row[c0 ^ swz]);
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

// LDS reads issued as inline asm, so that their completion is waited for
// explicitly (wait_frags) instead of by the compiler's conservative
// lgkmcnt(0) in front of the first use. The offset is an immediate.
template <int OFF, typename V>
__device__ __forceinline__ void ds_read16(V &v, uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF) : "memory");
}

template <int STRIDE, typename T, int N, int... I>
__device__ __forceinline__ void ds_read_rows(Frag<T> (&f)[N], uint32_t addr, std::integer_sequence<int, I...>) {
  (ds_read16<I * STRIDE>(f[I].v, addr), ...);
}

// Waits until at most N LDS reads are in flight, then ties the fragments to
// that wait so that no use of them is scheduled above it.
template <int N, typename T, int MI, int NI>
__device__ __forceinline__ void wait_frags(Frag<T> (&fa)[MI], Frag<T> (&fb)[NI]) {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
#pragma unroll
  for (int i = 0; i < MI; ++i) asm volatile("" : "+v"(fa[i].v));
#pragma unroll
  for (int j = 0; j < NI; ++j) asm volatile("" : "+v"(fb[j].v));
}

template <int N, typename T, int MI, int NI>
__device__ __forceinline__ void wait_frags(Frag<T> (&fa)[MI], Frag<T> (&fl)[MI], Frag<T> (&fb)[NI]) {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
#pragma unroll
  for (int i = 0; i < MI; ++i) asm volatile("" : "+v"(fa[i].v), "+v"(fl[i].v));
#pragma unroll
  for (int j = 0; j < NI; ++j) asm volatile("" : "+v"(fb[j].v));
}

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
// tiles, and inside the band tiles run in groups of 4 row-tiles (row-tile
// fastest): the 32 tiles an XCD runs at once then share 4 A row panels and
// 8 B column panels in its L2 (measured best against groups of 1, 2, 5, 8
// and of all columns, on every decoder GEMM shape).
__host__ __device__ __forceinline__ int tile_group_rows(int) { return 4; }

__device__ __forceinline__ void tile_coords(int nt_m, int nt_n, int *tm, int *tn) {
  const int ntiles = nt_m * nt_n;
  int id = blockIdx.x;
  const int per = ntiles / 8;  // tiles per XCD (the remainder keeps its id)
  if (id < per * 8) id = (id & 7) * per + (id >> 3);
  const int GM = tile_group_rows(nt_n);
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

// Fragments of MFMA step kk of stage `buf`, read as inline asm (16-bit types):
// one base address per operand, the 32-row blocks at immediate offsets (the
// swizzle depends on the row modulo 32 only).
template <class C>
__device__ __forceinline__ void kk_frags_asm(uint32_t lds_addr, int buf, int kk, int lane, int wm, int wn,
                                             Frag<typename C::type> (&fa)[C::MI],
                                             Frag<typename C::type> (&fb)[C::NI]) {
  static_assert(sizeof(typename C::type) == 2, "asm fragment reads are 16-bit only");
  const int c0 = (kk * 16 + (lane >> 5) * 8) / C::EPC;
  const int ra = wm * C::WM + (lane & 31), rb = C::BROW0 + wn * C::WN + (lane & 31);
  const uint32_t stage = lds_addr + (uint32_t)(buf * C::BUF) * 16u;
  const uint32_t a = stage + (uint32_t)(ra * C::CPR + (c0 ^ lds_swz<C>(ra))) * 16u;
  const uint32_t b = stage + (uint32_t)(rb * C::CPR + (c0 ^ lds_swz<C>(rb - C::BROW0))) * 16u;
  ds_read_rows<32 * C::CPR * 16>(fa, a, std::make_integer_sequence<int, C::MI>{});
  ds_read_rows<32 * C::CPR * 16>(fb, b, std::make_integer_sequence<int, C::NI>{});
}

// Pair mode: the lo-plane fragments of A (the tile BM rows after the hi tile).
template <class C>
__device__ __forceinline__ void kk_frags_lo_asm(uint32_t lds_addr, int buf, int kk, int lane, int wm,
                                                Frag<typename C::type> (&fl)[C::MI]) {
  const int c0 = (kk * 16 + (lane >> 5) * 8) / C::EPC;
  const int ra = wm * C::WM + (lane & 31);
  const uint32_t a = lds_addr + (uint32_t)(buf * C::BUF + (C::BM + ra) * C::CPR + (c0 ^ lds_swz<C>(ra))) * 16u;
  ds_read_rows<32 * C::CPR * 16>(fl, a, std::make_integer_sequence<int, C::MI>{});
}

template <class C>
__device__ __forceinline__ void kk_mma(const Frag<typename C::type> (&fa)[C::MI],
                                       const Frag<typename C::type> (&fb)[C::NI], f32x16 (&acc)[C::MI][C::NI]) {
#pragma unroll
  for (int i = 0; i < C::MI; ++i)
#pragma unroll
    for (int j = 0; j < C::NI; ++j) mma32(acc[i][j], fa[i], fb[j]);
}

// ---------------------------------------------------------------------------
// int8 B operand (LOAD 9)
// ---------------------------------------------------------------------------

typedef _Float16 h2v __attribute__((ext_vector_type(2)));

template <int OFF>
__device__ __forceinline__ void ds_read8(uint2 &v, uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  asm volatile("ds_read_b64 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF) : "memory");
}
template <int OFF>
__device__ __forceinline__ void ds_read4(uint32_t &v, uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF) : "memory");
}
template <int STRIDE, int N, int... I>
__device__ __forceinline__ void ds_read8_rows(uint2 (&r)[N], uint32_t addr, std::integer_sequence<int, I...>) {
  (ds_read8<I * STRIDE>(r[I], addr), ...);
}
template <int STRIDE, int N, int... I>
__device__ __forceinline__ void ds_read4_rows(uint2 (&r)[N], uint32_t addr, std::integer_sequence<int, I...>) {
  (ds_read4<I * STRIDE>(r[I].x, addr), ...);
}

// fp16 fragment of 8 int8 values q (K order) times the power-of-two scale s:
// (0x6400 | (q + 128)) is the fp16 number 1024 + q + 128, so subtracting
// 1152 gives q exactly, and q * s is exact for every scale the loader stores.
__device__ __forceinline__ Frag<f16> q8_frag(uint2 raw, uint32_t sbits) {
  const uint32_t x0 = raw.x ^ 0x80808080u, x1 = raw.y ^ 0x80808080u;
  const _Float16 s = __builtin_bit_cast(_Float16, (uint16_t)sbits);
  const h2v bias = {(_Float16)1152.0f, (_Float16)1152.0f}, sc = {s, s};
  const uint32_t p[4] = {__builtin_amdgcn_perm(0x64646464u, x0, 0x04010400u),
                         __builtin_amdgcn_perm(0x64646464u, x0, 0x04030402u),
                         __builtin_amdgcn_perm(0x64646464u, x1, 0x04010400u),
                         __builtin_amdgcn_perm(0x64646464u, x1, 0x04030402u)};
  Frag<f16> f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const h2v v = (__builtin_bit_cast(h2v, p[i]) - bias) * sc;
    f.v[2 * i] = v.x;
    f.v[2 * i + 1] = v.y;
  }
  return f;
}

// fp16 fragment of 8 int4 values q (K order, two per byte, low nibble first)
// times the power-of-two scale s: flipping each nibble's sign bit gives
// u = q + 8 in 0..15, (0x6400 | u) is the fp16 number 1024 + u, so
// subtracting 1032 gives q exactly, and q * s is exact.
__device__ __forceinline__ Frag<f16> q4_frag(uint32_t raw, uint32_t sbits) {
  const uint32_t x = raw ^ 0x88888888u;
  const uint32_t lo = x & 0x0F0F0F0Fu, hi = (x >> 4) & 0x0F0F0F0Fu;  // values 0, 2, 4, 6 / 1, 3, 5, 7
  const _Float16 s = __builtin_bit_cast(_Float16, (uint16_t)sbits);
  const h2v bias = {(_Float16)1032.0f, (_Float16)1032.0f}, sc = {s, s};
  // pair i = (value 2i, value 2i + 1) = (byte i of lo, byte i of hi); selector 0x0c gives a zero byte
  const uint32_t p[4] = {__builtin_amdgcn_perm(hi, lo, 0x0c040c00u) | 0x64006400u,
                         __builtin_amdgcn_perm(hi, lo, 0x0c050c01u) | 0x64006400u,
                         __builtin_amdgcn_perm(hi, lo, 0x0c060c02u) | 0x64006400u,
                         __builtin_amdgcn_perm(hi, lo, 0x0c070c03u) | 0x64006400u};
  Frag<f16> f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const h2v v = (__builtin_bit_cast(h2v, p[i]) - bias) * sc;
    f.v[2 * i] = v.x;
    f.v[2 * i + 1] = v.y;
  }
  return f;
}

// Fragment reads of MFMA step kk of stage `buf`: the A rows (fp16) and the
// wave's NI raw int8 B fragments (8 bytes each).
template <class C>
__device__ __forceinline__ void kk_frags_q8(uint32_t lds_addr, int buf, int kk, int lane, int wm, int wn,
                                           Frag<f16> (&fa)[C::MI], uint2 (&rb)[C::NI]) {
  const int c0 = (kk * 16 + (lane >> 5) * 8) / C::EPC;
  const int ra = wm * C::WM + (lane & 31), rbw = wn * C::WN + (lane & 31);
  const uint32_t stage = lds_addr + (uint32_t)(buf * C::BUF) * 16u;
  const uint32_t a = stage + (uint32_t)(ra * C::CPR + (c0 ^ lds_swz<C>(ra))) * 16u;
  ds_read_rows<32 * C::CPR * 16>(fa, a, std::make_integer_sequence<int, C::MI>{});
  if constexpr (C::QBITS == 8) {
    // chunk kk of the row holds the step's 16 values; 8 bytes per lane half
    const uint32_t b = stage + (uint32_t)(C::BM * C::CPR + kk * C::BN + rbw) * 16u + (uint32_t)((lane >> 5) * 8);
    ds_read8_rows<32 * 16>(rb, b, std::make_integer_sequence<int, C::NI>{});
  } else {
    // one chunk holds the K step's 32 values (low nibble first); 4 bytes per lane half
    const uint32_t b = stage + (uint32_t)(C::BM * C::CPR + rbw) * 16u + (uint32_t)(kk * 8 + (lane >> 5) * 4);
    ds_read4_rows<32 * 16>(rb, b, std::make_integer_sequence<int, C::NI>{});
  }
}

// The scales of the wave's NI fragment rows for stage `buf` (NI consecutive
// fp16 values: the stage holds [row group of 128][row % 32][(row / 32) % 4]).
// The read and its wait are one statement: a result register of an
// asynchronous read must not be live across compiler-scheduled code (the
// compiler may copy it before the data has arrived).
template <class C>
__device__ __forceinline__ void scale_read_q8(uint32_t lds_addr, int buf, int lane, int wn, uint2 &sc) {
  const int n = wn * C::WN + (lane & 31);
  const int off = (n >> 7) * 128 + (n & 31) * 4 + ((wn * C::WN) >> 5) % 4;
  const uint32_t a = lds_addr + (uint32_t)(buf * C::BUF + C::BM * C::CPR + C::B_CH * C::BN) * 16u + (uint32_t)off * 2u;
  if constexpr (C::NI == 4) {
    asm volatile("ds_read_b64 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(sc) : "v"(a) : "memory");
  } else {
    static_assert(C::NI == 2, "2 or 4 fragments per wave row block");
    asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(sc.x) : "v"(a) : "memory");
    sc.y = 0u;
  }
}

template <int N, int MI, int NI>
__device__ __forceinline__ void wait_frags_q8(Frag<f16> (&fa)[MI], uint2 (&rb)[NI]) {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
#pragma unroll
  for (int i = 0; i < MI; ++i) asm volatile("" : "+v"(fa[i].v));
#pragma unroll
  for (int j = 0; j < NI; ++j) asm volatile("" : "+v"(rb[j]));
}

// Direct loads of one K step (k: first K column) of the int8 B operand:
// A as tile_issue_direct; B rows as [chunk][row] 16-byte units; the tile's
// scales from Bs [K / 32][NG][32][4] (fp16 bits; NG = row groups of 128),
// four 16-byte units per wave.
template <class C>
__device__ __forceinline__ void tile_issue_direct_q8(const f16 *__restrict__ A, int64_t lda,
                                                     const int8_t *__restrict__ B, int64_t ldb,
                                                     const uint16_t *__restrict__ Bs, int NG, int M, int N, int m0,
                                                     int n0, int k, uint4 *lds, int buf, int wave, int lane) {
  uint4 *a = lds + buf * C::BUF, *b = a + C::BM * C::CPR, *s = b + C::B_CH * C::BN;
  const int sub_r = lane / C::CPR, pc = lane % C::CPR;
#pragma unroll
  for (int i = 0; i < C::A_PT; ++i) {
    const int blk = i * C::NWAVES + wave;
    const int r = blk * C::RPI + sub_r;
    const int c = pc ^ lds_swz<C>(r);
    const int gm = min(m0 + r, M - 1);
    __builtin_amdgcn_global_load_lds((const void *)(A + (int64_t)gm * lda + k + c * C::EPC),
                                     (lds_void *)(a + blk * 64), 16, 0, 0);
  }
  if constexpr (C::B_CH * C::BN >= 64 * C::NWAVES) {
#pragma unroll
    for (int i = 0; i < C::B_PT; ++i) {
      const int blk = i * C::NWAVES + wave;
      const int u = blk * 64 + lane, c = u / C::BN, r = u % C::BN;
      const int gn = min(n0 + r, N - 1);
      __builtin_amdgcn_global_load_lds((const void *)(B + (int64_t)gn * ldb + k * C::QBITS / 8 + c * 16),
                                       (lds_void *)(b + blk * 64), 16, 0, 0);
    }
  } else {
    // 32 chunks per wave: one load, lanes 0..31 (every wave issues it, so
    // each wave's count of loads in flight stays B_PT per K step)
    constexpr int BPW = C::B_CH * C::BN / C::NWAVES;
    if (lane < BPW) {
      const int u = wave * BPW + lane, c = u / C::BN, r = u % C::BN;
      const int gn = min(n0 + r, N - 1);
      __builtin_amdgcn_global_load_lds((const void *)(B + (int64_t)gn * ldb + k * C::QBITS / 8 + c * 16),
                                       (lds_void *)(b + wave * BPW), 16, 0, 0);
    }
  }
  if (lane < 4) {
    const int u = wave * 4 + lane, gg = min((n0 >> 7) + (u >> 4), NG - 1);
    const char *src = (const char *)Bs + ((int64_t)(k >> 5) * NG + gg) * 256 + (u & 15) * 16;
    __builtin_amdgcn_global_load_lds((const void *)src, (lds_void *)(s + wave * 4), 16, 0, 0);
  }
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
                                                  int wave, int lane, int klo = 0) {
  uint4 *a = lds + buf * C::BUF, *b = a + C::BROW0 * C::CPR;
  const int sub_r = lane / C::CPR, pc = lane % C::CPR;
#pragma unroll
  for (int pl = 0; pl < (C::PAIRA ? 2 : 1); ++pl) {
    // plane pl of A: columns ka (hi) or klo + ka (lo), LDS block pl
#pragma unroll
    for (int i = 0; i < C::A_PT; ++i) {
      const int blk = i * C::NWAVES + wave;
      const int r = blk * C::RPI + sub_r;
      const int c = pc ^ lds_swz<C>(r);
      const int gm = min(m0 + r, M - 1);
      __builtin_amdgcn_global_load_lds((const void *)(A + (int64_t)gm * lda + pl * klo + ka + c * C::EPC),
                                       (lds_void *)(a + pl * C::BM * C::CPR + blk * 64), 16, 0, 0);
    }
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
                                          f32x16 (&acc)[C::MI][C::NI], const uint16_t *__restrict__ Bs = nullptr) {
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
  } else if constexpr (C::LOAD == 4) {
    // As LOAD 2, with the fragments of every MFMA step read into registers
    // one step ahead: the reads for step kk + 1 (for the last step: the first
    // step of the next tile, after the barrier) are issued before the MFMAs of
    // step kk, which wait only for the older reads. When the barrier of tile
    // kt is passed every wave has its last fragments of tile kt in registers,
    // so tile kt + NSTAGE is loaded straight into kt's stage: all NSTAGE
    // stages hold tiles in flight.
    constexpr int PT = C::A_PT + C::B_PT, NS = C::NSTAGE, KK = C::BK / 16, NR = C::MI + C::NI;
    const uint32_t lds_addr = (uint32_t)(uintptr_t)(lds_void *)lds;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      if (s < nk)
        tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, kmod(s * C::BK, KA), kmod(s * C::BK, KB), lds, s, wave,
                             lane);
    wait_tiles<PT, NS - 1>(min(NS - 1, nk - 1));
    __builtin_amdgcn_s_barrier();
    Frag<typename C::type> fa[2][C::MI], fb[2][C::NI];
    kk_frags_asm<C>(lds_addr, 0, 0, lane, wm, wn, fa[0], fb[0]);
    for (int kt = 0; kt < nk; ++kt) {
      const int st = kt % NS;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const int cur = kk & 1, nx = cur ^ 1;
        if (kk + 1 < KK) {
          kk_frags_asm<C>(lds_addr, st, kk + 1, lane, wm, wn, fa[nx], fb[nx]);
          wait_frags<NR>(fa[cur], fb[cur]);
        } else if (kt + 1 < nk) {
          // tiles kt + 2 .. min(kt + NS - 1, nk - 1) may still be in flight
          wait_tiles<PT, NS - 2>(min(NS - 2, nk - 2 - kt));
          wait_frags<0>(fa[cur], fb[cur]);
          __builtin_amdgcn_s_barrier();
          const int kn = kt + NS;
          if (kn < nk)
            tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, kmod(kn * C::BK, KA), kmod(kn * C::BK, KB), lds, st,
                                 wave, lane);
          kk_frags_asm<C>(lds_addr, (kt + 1) % NS, 0, lane, wm, wn, fa[nx], fb[nx]);
        } else {
          wait_frags<0>(fa[cur], fb[cur]);
        }
        kk_mma<C>(fa[cur], fb[cur], acc);
      }
    }
    __builtin_amdgcn_s_barrier();
  } else if constexpr (C::INTERLEAVED) {
    // Pair-aware: K steps over the KB columns of B; A rows hold [hi | lo]
    // with the lo plane KB columns after the hi plane, and each stage holds
    // A_hi, A_lo and B, so every B fragment feeds acc += A_hi B + A_lo B.
    // (LOAD 8: A is a single plane, the lo parts drop out.)
    // NSTAGE - 1 tiles are in flight: the stage of tile kt - 1 is free once
    // the barrier inside step kt - 1 has passed, and tile kt + NSTAGE - 1 is
    // loaded into it during the first MFMA step of tile kt, its loads
    // interleaved with the MFMAs (a share of the step's MFMAs before each
    // load) rather than issued by all waves in one burst. Each K step is one
    // basic block: past the last tile the loads fetch the last tile again
    // into the free stage (which no MFMA reads any more) and the first
    // fragments of the next tile are read anyway (and not used), so the
    // vmcnt wait is a constant and no register copies join two paths.
    constexpr int NPL = C::PAIRA ? 2 : 1;  // planes of A
    constexpr int PT = NPL * C::A_PT + C::B_PT, NS = C::NSTAGE, KK = C::BK / 16, NR = NPL * C::MI + C::NI;
    // MFMAs of one step, and how many go before each load
    constexpr int NMMA = NPL * C::MI * C::NI, R = NMMA >= PT ? NMMA / PT : 1, NG = NMMA >= PT ? PT : NMMA;
    constexpr int PRE = NS - 1;  // tiles loaded before the loop
    const int nk5 = KB / C::BK;
    const uint32_t lds_addr = (uint32_t)(uintptr_t)(lds_void *)lds;
#pragma unroll
    for (int s = 0; s < PRE; ++s) {
      const int ks = min(s, nk5 - 1) * C::BK;
      tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, ks, ks, lds, s, wave, lane, KB);
    }
    wait_vmcnt<(PRE - 1) * PT>();
    __builtin_amdgcn_s_barrier();
    Frag<typename C::type> fa[2][C::MI], fl[2][C::MI], fb[2][C::NI];
    kk_frags_asm<C>(lds_addr, 0, 0, lane, wm, wn, fa[0], fb[0]);
    if constexpr (C::PAIRA) kk_frags_lo_asm<C>(lds_addr, 0, 0, lane, wm, fl[0]);
    int st = 0, sl = NS - 1;  // stage of tile kt; stage of tile kt + NS - 1
    for (int kt = 0; kt < nk5; ++kt) {
      const int kn = min(kt + PRE, nk5 - 1) * C::BK;
      const int snext = st + 1 == NS ? 0 : st + 1;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const int cur = kk & 1, nx = cur ^ 1;
        if (kk + 1 < KK) {
          kk_frags_asm<C>(lds_addr, st, kk + 1, lane, wm, wn, fa[nx], fb[nx]);
          if constexpr (C::PAIRA) {
            kk_frags_lo_asm<C>(lds_addr, st, kk + 1, lane, wm, fl[nx]);
            wait_frags<NR>(fa[cur], fl[cur], fb[cur]);
          } else {
            wait_frags<NR>(fa[cur], fb[cur]);
          }
        } else {
          // own loads of tile kt + 1 have landed; after the barrier every
          // wave's have, and no wave reads stage kt any more
          wait_vmcnt<(NS - 2) * PT>();
          if constexpr (C::PAIRA) wait_frags<0>(fa[cur], fl[cur], fb[cur]);
          else wait_frags<0>(fa[cur], fb[cur]);
          __builtin_amdgcn_s_barrier();
          kk_frags_asm<C>(lds_addr, snext, 0, lane, wm, wn, fa[nx], fb[nx]);
          if constexpr (C::PAIRA) kk_frags_lo_asm<C>(lds_addr, snext, 0, lane, wm, fl[nx]);
        }
        if (kk == 0) {
          __builtin_amdgcn_sched_barrier(0);
          kk_mma<C>(fa[cur], fb[cur], acc);
          if constexpr (C::PAIRA) kk_mma<C>(fl[cur], fb[cur], acc);
          tile_issue_direct<C>(A, lda, B, ldb, M, N, m0, n0, kn, kn, lds, sl, wave, lane, KB);
#pragma unroll
          for (int i = 0; i < PT; ++i) {
            if (i < NG) __builtin_amdgcn_sched_group_barrier(0x008, R, 0);  // MFMA
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);              // VMEM read
          }
          if constexpr (NMMA > R * NG) __builtin_amdgcn_sched_group_barrier(0x008, NMMA - R * NG, 0);
          __builtin_amdgcn_sched_barrier(0);
        } else {
          kk_mma<C>(fa[cur], fb[cur], acc);
          if constexpr (C::PAIRA) kk_mma<C>(fl[cur], fb[cur], acc);
          __builtin_amdgcn_sched_barrier(0);  // the step's MFMAs stay on their side of the barrier
        }
      }
      st = snext;
      sl = sl + 1 == NS ? 0 : sl + 1;
    }
    wait_vmcnt<0>();
    // The last step also read fragments past the last tile (unused). Wait for
    // those reads with both fragment buffers held live: otherwise the
    // compiler may give their registers to the caller's epilogue while the
    // reads are still in flight, and a late read overwrites its values.
    if constexpr (C::PAIRA) {
      wait_frags<0>(fa[0], fl[0], fb[0]);
      wait_frags<0>(fa[1], fl[1], fb[1]);
    } else {
      wait_frags<0>(fa[0], fb[0]);
      wait_frags<0>(fa[1], fb[1]);
    }
    __builtin_amdgcn_s_barrier();
  } else if constexpr (C::Q8B) {
    // The LOAD 8 schedule (see above) with an int8 B operand: B is int8
    // [N][KB] (ldb bytes per row) with fp16 scales Bs; a stage's scales are
    // read with the first fragments of the stage and serve both MFMA steps
    // of its K step (one quantization block).
    static_assert(sizeof(typename C::type) == 2, "fp16 A with int8 B");
    constexpr int PT = C::A_PT + C::B_PT + 1, NS = C::NSTAGE, KK = C::BK / 16, NR = C::MI + C::NI;
    constexpr int NMMA = C::MI * C::NI, R = NMMA >= PT ? NMMA / PT : 1, NG = NMMA >= PT ? PT : NMMA;
    constexpr int PRE = NS - 1;
    const int nk5 = KB / C::BK, ngroups = (N + 127) / 128;
    const int8_t *Bq = reinterpret_cast<const int8_t *>(B);
    const uint32_t lds_addr = (uint32_t)(uintptr_t)(lds_void *)lds;
#pragma unroll
    for (int s = 0; s < PRE; ++s)
      tile_issue_direct_q8<C>(A, lda, Bq, ldb, Bs, ngroups, M, N, m0, n0, min(s, nk5 - 1) * C::BK, lds, s, wave,
                              lane);
    wait_vmcnt<(PRE - 1) * PT>();
    __builtin_amdgcn_s_barrier();
    static_assert(KK == 2, "two MFMA steps per K step");
    Frag<f16> fa[2][C::MI];
    uint2 rb[2][C::NI], sc;
    kk_frags_q8<C>(lds_addr, 0, 0, lane, wm, wn, fa[0], rb[0]);
    int st = 0, sl = NS - 1;  // stage of tile kt; stage of tile kt + NS - 1
    for (int kt = 0; kt < nk5; ++kt) {
      const int kn = min(kt + PRE, nk5 - 1) * C::BK;
      const int snext = st + 1 == NS ? 0 : st + 1;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const int cur = kk & 1, nx = cur ^ 1;
        if (kk == 0) {
          // this step's fragments (read at the stage boundary), then the
          // stage's scales, read and waited for at once
          wait_frags_q8<0>(fa[cur], rb[cur]);
          scale_read_q8<C>(lds_addr, st, lane, wn, sc);
        } else {
          // own loads of tile kt + 1 have landed; after the barrier every
          // wave's have, and no wave reads stage kt any more
          wait_vmcnt<(NS - 2) * PT>();
          wait_frags_q8<0>(fa[cur], rb[cur]);
          __builtin_amdgcn_s_barrier();
          kk_frags_q8<C>(lds_addr, snext, 0, lane, wm, wn, fa[nx], rb[nx]);
        }
        Frag<f16> fb[C::NI];
#pragma unroll
        for (int j = 0; j < C::NI; ++j) {
          const uint32_t w = (j >> 1) ? sc.y : sc.x;
          const uint32_t sb = (j & 1) ? w >> 16 : w & 0xffffu;
          if constexpr (C::QBITS == 8) fb[j] = q8_frag(rb[cur][j], sb);
          else fb[j] = q4_frag(rb[cur][j].x, sb);
        }
        if (kk == 0) kk_frags_q8<C>(lds_addr, st, 1, lane, wm, wn, fa[nx], rb[nx]);
        if (kk == 0) {
          __builtin_amdgcn_sched_barrier(0);
          kk_mma<C>(fa[cur], fb, acc);
          tile_issue_direct_q8<C>(A, lda, Bq, ldb, Bs, ngroups, M, N, m0, n0, kn, lds, sl, wave, lane);
#pragma unroll
          for (int i = 0; i < PT; ++i) {
            if (i < NG) __builtin_amdgcn_sched_group_barrier(0x008, R, 0);  // MFMA
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);              // VMEM read
          }
          if constexpr (NMMA > R * NG) __builtin_amdgcn_sched_group_barrier(0x008, NMMA - R * NG, 0);
          __builtin_amdgcn_sched_barrier(0);
        } else {
          kk_mma<C>(fa[cur], fb, acc);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      st = snext;
      sl = sl + 1 == NS ? 0 : sl + 1;
    }
    wait_vmcnt<0>();
    wait_frags_q8<0>(fa[0], rb[0]);
    wait_frags_q8<0>(fa[1], rb[1]);
    __builtin_amdgcn_s_barrier();
  }
}

}  // namespace jetk
