// Device-side building blocks for the gfx950 kernels: MFMA atoms, type
// conversions, the E4M3 encoder and GELU.  Everything here is __device__
// inline; nothing allocates.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cf_internal.h"

namespace cf {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2_t;

typedef uint16_t bf16_t;  // storage type of bfloat16 values

// ---------------------------------------------------------------------------
// Conversions
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint32_t h) {
  return __uint_as_float(h << 16);
}

// fp32 -> bf16, round to nearest even (finite inputs; NaN stays NaN because
// the quiet bit survives the rounding add for every NaN payload we produce).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// Two fp32 -> packed bf16 pair (lo in bits 0..15), round to nearest even:
// one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef float f32x2_v __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
  const f32x2_v v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_v));
}

// z / s rounded to nearest fp32, from r = 1 / s rounded to nearest (one IEEE
// division per row): the product z r is corrected by one fused step on its
// exact remainder z - q s (Markstein's division theorem: with r within half
// an ulp of 1/s and q within one ulp of z/s, q + (z - q s) r rounds to the
// correctly rounded quotient).  For s > 0 and quotients in the normal range.
// The sign is copied from z: for z = -0 the correction would add opposite
// zeros and return +0.
__device__ __forceinline__ float div_rn(float z, float s, float r) {
  const float q = z * r;
  return copysignf(fmaf(fmaf(-q, s, z), r, q), z);
}

// Four fp32 values -> four OCP E4M3FN codes (byte q from the q-th value) by
// gfx950's packed conversion: round to nearest, ties to even mantissa,
// subnormals m * 2^-9.  Callers pass quotients x / s with s = amax / 448 of
// the values' own row, so |x / s| stays below 464 and the conversion never
// reaches its overflow range (448 is the largest finite code).  Over every
// fp32 pattern in [-448, 448] it gives the same code as an integer encoder
// written from the OCP FP8 specification.
__device__ __forceinline__ uint32_t e4m3x4(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);   // bytes 0, 1
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);          // bytes 2, 3
  return (uint32_t)w;
}

// erf by Abramowitz and Stegun, Handbook of Mathematical Functions, 7.1.26:
// erf(x) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-x^2) with
// t = 1 / (1 + p x) for x >= 0, |error| <= 1.5e-7; odd extension.  Branch-free
// (one reciprocal, one exp), so a wave never runs two code paths.
__device__ __forceinline__ float erf_as(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
  float y = fmaf(1.061405429f, t, -1.453152027f);
  y = fmaf(y, t, 1.421413741f);
  y = fmaf(y, t, -0.284496736f);
  y = fmaf(y, t, 0.254829592f);
  const float e = __builtin_amdgcn_exp2f(-(ax * ax) * 1.4426950408889634f);   // exp(-x^2)
  return copysignf(fmaf(-(y * t), e, 1.0f), x);
}

// GELU, erf form: x * Phi(x) = x/2 (1 + erf(x / sqrt 2)).
__device__ __forceinline__ float gelu_erf(float x) {
  return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f));
}
// GELU, tanh approximation.
__device__ __forceinline__ float gelu_tanh(float x) {
  const float c = 0.79788456080286536f;  // sqrt(2/pi)
  return 0.5f * x * (1.0f + tanhf(c * (x + 0.044715f * x * x * x)));
}

// ---------------------------------------------------------------------------
// MFMA atoms.  Both operate on 16-byte operand chunks read from LDS rows that
// are contiguous along k; lane group g = lane/32 holds the g-th chunk of a
// 2-chunk k step.  Because the instruction pairs A and B k-indices the same
// way, any fixed k assignment inside a step gives the right dot product.
//
// Accumulator layout of a 32x32 block (D = A.B, A 32 x k, B k x 32):
//   lane l holds column (l % 32) and rows 8*(i/4) + 4*(l/32) + (i%4),
//   i = 0..15.
// ---------------------------------------------------------------------------
template <typename T> struct Mma;

template <> struct Mma<bf16_t> {
  static constexpr int kPerChunk = 8;   // bf16 values per 16-byte chunk
  static constexpr int kInstrs = 1;     // MFMA instructions per run()
  __device__ __forceinline__ static void run(f32x16_t& acc, u32x4_t a, u32x4_t b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
};

template <> struct Mma<float> {
  static constexpr int kPerChunk = 4;   // fp32 values per 16-byte chunk
  static constexpr int kInstrs = 4;     // MFMA instructions per run()
  // Four k=2 MFMAs: step j pairs element j of lane group 0 with element j of
  // lane group 1, so the four together cover the 8 k values of the chunk pair.
  __device__ __forceinline__ static void run(f32x16_t& acc, u32x4_t a, u32x4_t b) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[j]), __uint_as_float(b[j]),
                                                 acc, 0, 0, 0);
  }
};

// Row index (inside a 32x32 block) held by accumulator element i of lane l.
__device__ __forceinline__ int acc_row(int i, int lane) {
  return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
}

// ---------------------------------------------------------------------------
// LDS / global helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ u32x4_t lds_read16(const char* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}
__device__ __forceinline__ void lds_write16(char* p, u32x4_t v) {
  *reinterpret_cast<u32x4_t*>(p) = v;
}
__device__ __forceinline__ u32x4_t gload16(const void* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

// ---------------------------------------------------------------------------
// Four consecutive row elements: load (bf16 or fp32), activation, store.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void load4(const T* p, float (&v)[4]);
template <>
__device__ __forceinline__ void load4<bf16_t>(const bf16_t* p, float (&v)[4]) {
  const u32x2_t u = *reinterpret_cast<const u32x2_t*>(p);
  v[0] = bf16_to_f32(u[0] & 0xFFFFu);
  v[1] = bf16_to_f32(u[0] >> 16);
  v[2] = bf16_to_f32(u[1] & 0xFFFFu);
  v[3] = bf16_to_f32(u[1] >> 16);
}
template <>
__device__ __forceinline__ void load4<float>(const float* p, float (&v)[4]) {
  const f32x4_t u = *reinterpret_cast<const f32x4_t*>(p);
  v[0] = u[0]; v[1] = u[1]; v[2] = u[2]; v[3] = u[3];
}
// The same for data read once (row-pass inputs, residuals): non-temporal
// loads, so the lines do not displace reused operands in the caches.
template <typename T>
__device__ __forceinline__ void load4_once(const T* p, float (&v)[4]);
template <>
__device__ __forceinline__ void load4_once<bf16_t>(const bf16_t* p, float (&v)[4]) {
  const u32x2_t u = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
  v[0] = bf16_to_f32(u[0] & 0xFFFFu);
  v[1] = bf16_to_f32(u[0] >> 16);
  v[2] = bf16_to_f32(u[1] & 0xFFFFu);
  v[3] = bf16_to_f32(u[1] >> 16);
}
template <>
__device__ __forceinline__ void load4_once<float>(const float* p, float (&v)[4]) {
  const f32x4_t u = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p));
  v[0] = u[0]; v[1] = u[1]; v[2] = u[2]; v[3] = u[3];
}

// tanh(z) = sign(z) (1 - t) / (1 + t), t = exp(-2 |z|): no overflow for any z;
// near 0 the absolute error stays at the fp32 rounding of 1 - t (~6e-8).
__device__ __forceinline__ float tanh_exp(float z) {
  const float t = __builtin_amdgcn_exp2f(-2.8853900817779268f * fabsf(z));   // 2 log2(e)
  return copysignf((1.0f - t) * __builtin_amdgcn_rcpf(1.0f + t), z);
}

__device__ __forceinline__ void store4(void* base, int64_t off, int f32, const float (&v)[4]) {
  if (f32) {
    f32x4_t o = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(o, reinterpret_cast<f32x4_t*>(reinterpret_cast<float*>(base) + off));
  } else {
    u32x2_t o = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
    __builtin_nontemporal_store(o, reinterpret_cast<u32x2_t*>(reinterpret_cast<bf16_t*>(base) + off));
  }
}

}  // namespace cf
