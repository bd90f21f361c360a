// Device-side helpers shared by the gfx950 kernels: element types, 16-byte
// vector access, bf16 conversion and wavefront reductions.
#pragma once

#include <hip/hip_runtime.h>

#include "gelu_poly.h"
#include <stdint.h>

namespace dsf {

constexpr int kWave = 64;  // CDNA wavefront width

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// bf16 is carried as raw uint16_t bits in memory.
__device__ __forceinline__ float bf2f(uint16_t u) { return __uint_as_float(uint32_t(u) << 16); }

// fp32 -> bf16, round to nearest even (gfx950 converts in hardware).
__device__ __forceinline__ uint16_t f2bf(float f) {
  __bf16 b = (__bf16)f;
  return __builtin_bit_cast(uint16_t, b);
}

// Element traits: how many elements form one 16-byte vector and how to widen.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int kVec = 4;
  __device__ static __forceinline__ float to_f(float v) { return v; }
  __device__ static __forceinline__ float from_f(float v) { return v; }
};
template <> struct Elem<uint16_t> {
  static constexpr int kVec = 8;
  __device__ static __forceinline__ float to_f(uint16_t v) { return bf2f(v); }
  __device__ static __forceinline__ uint16_t from_f(float v) { return f2bf(v); }
};

// Load one 16-byte vector and widen it to fp32 (kVec values).
template <typename T>
__device__ __forceinline__ void load_vec(const T* p, float* out) {
  u32x4 raw = *reinterpret_cast<const u32x4*>(p);
  if constexpr (sizeof(T) == 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = __uint_as_float(raw[i]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out[2 * i] = __uint_as_float(raw[i] << 16);
      out[2 * i + 1] = __uint_as_float(raw[i] & 0xffff0000u);
    }
  }
}

// Round kVec fp32 values to T and store them as one 16-byte vector.
template <typename T>
__device__ __forceinline__ void store_vec(T* p, const float* v) {
  u32x4 raw;
  if constexpr (sizeof(T) == 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) raw[i] = __float_as_uint(v[i]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) raw[i] = uint32_t(f2bf(v[2 * i])) | (uint32_t(f2bf(v[2 * i + 1])) << 16);
  }
  *reinterpret_cast<u32x4*>(p) = raw;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Reductions over the four 16-lane rows of a wavefront (lanes l, l^16, l^32,
// l^48) with gfx950's row-swap permutes: VALU only, no LDS round trip. After
// the 32-swap each lane holds its own value and that of lane l^32 (in either
// order), after the 16-swap those of lane l^16; max and + are symmetric.
__device__ __forceinline__ float rows4_max(float v) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows4_sum(float v) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// MI355X dispatches consecutive workgroup ids round-robin over its 8 XCDs,
// each with its own L2. xcd_remap turns launch index L (of W) into a work
// index so that every XCD receives one contiguous range of work items (a
// bijection on [0, W)): neighbouring items, which share operands, then share
// an L2.
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_remap(int L, int W) {
  const int q = W / kXcds, r = W % kXcds, x = L % kXcds;
  return x * q + (x < r ? x : r) + L / kXcds;
}

// Sum over the 16 lanes of each row with DPP lane moves (VALU only):
// xor 1 and xor 2 via quad permutes, then the half-row mirror pairs the two
// quads of each 8 lanes and the row mirror the two halves of the row. Every
// lane of the row ends with the same value (+ is commutative).
#define DSF_DPP(v, ctrl) __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), (ctrl), 0xF, 0xF, false))
__device__ __forceinline__ float row16_sum(float v) {
  v += DSF_DPP(v, 0xB1);   // quad_perm [1,0,3,2]: lane ^ 1
  v += DSF_DPP(v, 0x4E);   // quad_perm [2,3,0,1]: lane ^ 2
  v += DSF_DPP(v, 0x141);  // row_half_mirror
  v += DSF_DPP(v, 0x140);  // row_mirror
  return v;
}
__device__ __forceinline__ float wave_sum_fast(float v) { return rows4_sum(row16_sum(v)); }

// Positions supplied by a caller are clamped into [0, T) so that a bad index
// cannot address memory outside the hidden-state rows.
__device__ __forceinline__ int clamp_pos(int p, int T) { return p < 0 ? 0 : (p >= T ? T - 1 : p); }

// erf by Abramowitz & Stegun, Handbook of Mathematical Functions, formula
// 7.1.26: erf(z) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-z^2),
// t = 1 / (1 + p z), for z >= 0 (odd extension below), |error| <= 1.5e-7.
__device__ __forceinline__ float erf_as7126(float x) {
  const float z = fabsf(x);
  const float t = 1.0f / fmaf(0.3275911f, z, 1.0f);
  float poly = fmaf(1.061405429f, t, -1.453152027f);
  poly = fmaf(poly, t, 1.421413741f);
  poly = fmaf(poly, t, -0.284496736f);
  poly = fmaf(poly, t, 0.254829592f);
  const float y = 1.0f - poly * t * __expf(-z * z);
  return copysignf(y, x);
}
// GELU(x) = x Phi(x) = x (1 + erf(x / sqrt 2)) / 2
__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erf_as7126(x * 0.70710678118654752f)); }
__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

// d/dx GELU(x) = Phi(x) + x phi(x) for gradients stored as bf16: Phi from the
// same fitted polynomial as gelu_bf16, phi from the hardware exp2.
__device__ __forceinline__ float gelu_grad_bf16(float x) {
  const float xc = __builtin_amdgcn_fmed3f(x, -kGeluPolyXmax, kGeluPolyXmax);
  const float u = xc * xc;
  float q = kGeluPolyQ[0];
#pragma unroll
  for (int i = 1; i < int(sizeof(kGeluPolyQ) / sizeof(float)); ++i) q = fmaf(q, u, kGeluPolyQ[i]);
  const float cdf = fmaf(0.5f, xc * q, 0.5f);
  const float pdf = 0.3989422804014327f * __builtin_amdgcn_exp2f(-0.5f * 1.4426950408889634f * x * x);
  return fmaf(x, pdf, cdf);
}

// SiLU for outputs stored as bf16: x * 1 / (1 + 2^(-x log2 e)) with the
// hardware exp2 and reciprocal (each within about 1 ulp of fp32), a relative
// error near 1e-6, far below a bf16 ulp of the result; three transcendental-
// unit operations instead of expf's range reduction and an IEEE division.
// Large negative x gives 2^(+big) = inf, a zero reciprocal and -0 (SiLU
// tends to 0 from below); NaN propagates.
__device__ __forceinline__ float silu_bf16(float x) {
  const float e = __builtin_amdgcn_exp2f(-x * 1.4426950408889634f);
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}
// sigmoid(x) and d/dx SiLU(x) = s (1 + x (1 - s)) with the same primitives
__device__ __forceinline__ float sigmoid_bf16(float x) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-x * 1.4426950408889634f));
}
__device__ __forceinline__ float silu_grad_bf16(float x) {
  const float s = sigmoid_bf16(x);
  return s * fmaf(x, 1.0f - s, 1.0f);
}

// GELU for outputs stored as bf16: erf(x / sqrt 2) = x Q(x^2) on the clamped
// argument (a degree-8 polynomial, gelu_poly.h), within 2e-5 in fp32, so
// Phi(x) is within 1e-5, far below a bf16 ulp of the result. 13 VALU
// operations against the reciprocal and exponential of gelu_erf.
__device__ __forceinline__ float gelu_bf16(float x) {
  const float xc = __builtin_amdgcn_fmed3f(x, -kGeluPolyXmax, kGeluPolyXmax);
  const float u = xc * xc;
  float q = kGeluPolyQ[0];
#pragma unroll
  for (int i = 1; i < int(sizeof(kGeluPolyQ) / sizeof(float)); ++i) q = fmaf(q, u, kGeluPolyQ[i]);
  const float h = 0.5f * x;
  return fmaf(h, xc * q, h);
}

}  // namespace dsf
