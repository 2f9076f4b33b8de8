// Device-side building blocks for gfx950 (CDNA4): storage types, bf16
// rounding, and matrix-core (MFMA) wrappers.
//
// Every MFMA wrapper takes operands in one per-lane layout, "8 consecutive K
// elements per lane": for a 32x32 product lane l holds
//   A[row = l % 32][k0 + 8 * (l / 32) + j],  B[col = l % 32][k0 + 8 * (l / 32) + j]
// for j = 0..7 (16 K elements per call), and for a 16x16 product
//   A[row = l % 16][k0 + 8 * (l / 16) + j],  B[col = l % 16][k0 + 8 * (l / 16) + j]
// (32 K elements per call). In bf16 (fp16) this is exactly one
// v_mfma_f32_32x32x16_bf16 (_f16) / v_mfma_f32_16x16x32_bf16 (_f16). In fp32 the same
// registers feed eight v_mfma_f32_32x32x2f32 / v_mfma_f32_16x16x4f32, call j
// taking element j of every lane, so both dtypes share all indexing code.
// Accumulator layouts: 32x32: acc[e] = C[8*(e/4) + 4*(l/32) + e%4][l % 32];
// 16x16: acc[e] = C[4*(l/16) + e][l % 16].
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jetk {

typedef uint16_t bf16;  // bfloat16 bits in memory
typedef _Float16 f16;   // IEEE binary16
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf2f(bf16 h) { return __uint_as_float(((uint32_t)h) << 16); }

// float -> bfloat16, round to nearest even (NaN stays NaN): the gfx950
// conversion instruction (v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16 f2bf(float f) { return __builtin_bit_cast(bf16, (__bf16)f); }

// Two floats -> two bfloat16 in one 32-bit word (a in the low half).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f2bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// Two floats -> two binary16 values in one 32-bit word (a in the low half),
// round to nearest even.
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f2h2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, f16x2_t));
}

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16>(bf16 v) { return bf2f(v); }
template <> __device__ __forceinline__ float to_f<f16>(f16 v) { return (float)v; }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return f2bf(v); }
template <> __device__ __forceinline__ f16 from_f<f16>(float v) { return (f16)v; }

// Two floats -> two 16-bit values of type T in one 32-bit word.
template <typename T> __device__ __forceinline__ uint32_t pack2(float a, float b);
template <> __device__ __forceinline__ uint32_t pack2<bf16>(float a, float b) { return f2bf2(a, b); }
template <> __device__ __forceinline__ uint32_t pack2<f16>(float a, float b) { return f2h2(a, b); }

// The 8-element vector type of a 16-bit storage type (MFMA operands).
template <typename T> struct Vec8;
template <> struct Vec8<bf16> { typedef bf16x8 type; };
template <> struct Vec8<f16> { typedef f16x8 type; };

// Eight consecutive K elements of one lane.
template <typename T> struct Frag;
template <> struct Frag<bf16> {
  bf16x8 v;
  __device__ __forceinline__ void zero() {
    for (int j = 0; j < 8; ++j) v[j] = (__bf16)0.0f;
  }
};
template <> struct Frag<f16> {
  f16x8 v;
  __device__ __forceinline__ void zero() {
    for (int j = 0; j < 8; ++j) v[j] = (_Float16)0.0f;
  }
};
template <> struct Frag<float> {
  f32x8 v;
  __device__ __forceinline__ void zero() {
    for (int j = 0; j < 8; ++j) v[j] = 0.0f;
  }
};

__device__ __forceinline__ void mma32(f32x16 &acc, const Frag<bf16> &a, const Frag<bf16> &b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma32(f32x16 &acc, const Frag<f16> &a, const Frag<f16> &b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma32(f32x16 &acc, const Frag<float> &a, const Frag<float> &b) {
#pragma unroll
  for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v[j], b.v[j], acc, 0, 0, 0);
}
__device__ __forceinline__ void mma16(f32x4 &acc, const Frag<bf16> &a, const Frag<bf16> &b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma16(f32x4 &acc, const Frag<f16> &a, const Frag<f16> &b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma16(f32x4 &acc, const Frag<float> &a, const Frag<float> &b) {
#pragma unroll
  for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], acc, 0, 0, 0);
}

// 16-byte vector load/store helpers.
__device__ __forceinline__ uint4 ld16(const void *p) { return *reinterpret_cast<const uint4 *>(p); }
__device__ __forceinline__ void st16(void *p, uint4 v) { *reinterpret_cast<uint4 *>(p) = v; }

// Frag from memory holding 8 consecutive elements (16 B bf16 / 32 B fp32).
__device__ __forceinline__ void frag_load(Frag<bf16> &f, const bf16 *p) {
  uint4 u = ld16(p);
  f.v = __builtin_bit_cast(bf16x8, u);
}
__device__ __forceinline__ void frag_load(Frag<f16> &f, const f16 *p) {
  uint4 u = ld16(p);
  f.v = __builtin_bit_cast(f16x8, u);
}
__device__ __forceinline__ void frag_load(Frag<float> &f, const float *p) {
  uint4 a = ld16(p), b = ld16(p + 4);
  f.v[0] = __uint_as_float(a.x); f.v[1] = __uint_as_float(a.y);
  f.v[2] = __uint_as_float(a.z); f.v[3] = __uint_as_float(a.w);
  f.v[4] = __uint_as_float(b.x); f.v[5] = __uint_as_float(b.y);
  f.v[6] = __uint_as_float(b.z); f.v[7] = __uint_as_float(b.w);
}

__device__ __forceinline__ float warp_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float warp_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

}  // namespace jetk
