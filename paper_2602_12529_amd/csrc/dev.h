// Device-side helpers shared by the kernels: bf16 conversion, vector loads, reductions.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace ff {

typedef uint16_t bf16_t;   // bfloat16 storage word

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// Round to nearest, ties to even; NaN stays NaN.
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return bf16_t((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return bf16_t(u >> 16);
}

// Scalar load/store of a dtype element as float.
template <bool BF16>
__device__ __forceinline__ float ld1(const void* p, int64_t i) {
  if constexpr (BF16) return bf2f(static_cast<const bf16_t*>(p)[i]);
  else return static_cast<const float*>(p)[i];
}
template <bool BF16>
__device__ __forceinline__ void st1(void* p, int64_t i, float v) {
  if constexpr (BF16) static_cast<bf16_t*>(p)[i] = f2bf(v);
  else static_cast<float*>(p)[i] = v;
}
// Value after rounding to the storage dtype.
template <bool BF16>
__device__ __forceinline__ float round_dt(float v) {
  if constexpr (BF16) return bf2f(f2bf(v));
  else return v;
}

// 8 consecutive elements (16 bytes of bf16 or 32 bytes of f32) as floats.
template <bool BF16>
__device__ __forceinline__ void ld8(const void* p, int64_t i, float (&o)[8]) {
  if constexpr (BF16) {
    uint4 u = *reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(p) + i);
    uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      o[2 * j] = __uint_as_float(w[j] << 16);
      o[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
    }
  } else {
    const float4* q = reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
    float4 a = q[0], b = q[1];
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  }
}
// ld8 / st8 with non-temporal accesses: for streams touched exactly once (the SDE step's x, v,
// eps and x'), so they bypass the caches' retention instead of displacing other data.
typedef unsigned int nt_u32x4 __attribute__((ext_vector_type(4)));
typedef float nt_f32x4 __attribute__((ext_vector_type(4)));
template <bool BF16>
__device__ __forceinline__ void ld8_nt(const void* p, int64_t i, float (&o)[8]) {
  if constexpr (BF16) {
    const nt_u32x4 u = __builtin_nontemporal_load(reinterpret_cast<const nt_u32x4*>(static_cast<const bf16_t*>(p) + i));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      o[2 * j] = __uint_as_float(u[j] << 16);
      o[2 * j + 1] = __uint_as_float(u[j] & 0xffff0000u);
    }
  } else {
    const nt_f32x4* q = reinterpret_cast<const nt_f32x4*>(static_cast<const float*>(p) + i);
    const nt_f32x4 a = __builtin_nontemporal_load(q), b = __builtin_nontemporal_load(q + 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) { o[j] = a[j]; o[4 + j] = b[j]; }
  }
}
template <bool BF16>
__device__ __forceinline__ void st8_nt(void* p, int64_t i, const float (&v)[8]);
// Eight values stored as bf16 with one non-temporal 16-byte store: for outputs written once and
// read by a later kernel, so they stream out without displacing cached inputs.
__device__ __forceinline__ void st8_bf16_nt(void* p, int64_t i, const float (&v)[8]) {
  typedef uint32_t u32x4_nt __attribute__((ext_vector_type(4)));
  u32x4_nt u;
  u.x = uint32_t(f2bf(v[0])) | (uint32_t(f2bf(v[1])) << 16);
  u.y = uint32_t(f2bf(v[2])) | (uint32_t(f2bf(v[3])) << 16);
  u.z = uint32_t(f2bf(v[4])) | (uint32_t(f2bf(v[5])) << 16);
  u.w = uint32_t(f2bf(v[6])) | (uint32_t(f2bf(v[7])) << 16);
  __builtin_nontemporal_store(u, reinterpret_cast<u32x4_nt*>(static_cast<bf16_t*>(p) + i));
}
template <bool BF16>
__device__ __forceinline__ void st8_nt(void* p, int64_t i, const float (&v)[8]) {
  if constexpr (BF16) {
    st8_bf16_nt(p, i, v);
  } else {
    nt_f32x4* q = reinterpret_cast<nt_f32x4*>(static_cast<float*>(p) + i);
    const nt_f32x4 a = {v[0], v[1], v[2], v[3]}, b = {v[4], v[5], v[6], v[7]};
    __builtin_nontemporal_store(a, q);
    __builtin_nontemporal_store(b, q + 1);
  }
}
template <bool BF16>
__device__ __forceinline__ void st8(void* p, int64_t i, const float (&v)[8]) {
  if constexpr (BF16) {
    uint4 u;
    u.x = uint32_t(f2bf(v[0])) | (uint32_t(f2bf(v[1])) << 16);
    u.y = uint32_t(f2bf(v[2])) | (uint32_t(f2bf(v[3])) << 16);
    u.z = uint32_t(f2bf(v[4])) | (uint32_t(f2bf(v[5])) << 16);
    u.w = uint32_t(f2bf(v[6])) | (uint32_t(f2bf(v[7])) << 16);
    *reinterpret_cast<uint4*>(static_cast<bf16_t*>(p) + i) = u;
  } else {
    float4* q = reinterpret_cast<float4*>(static_cast<float*>(p) + i);
    q[0] = make_float4(v[0], v[1], v[2], v[3]);
    q[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// x * sigmoid(x), with the sigmoid from the hardware exp2 and reciprocal (about 1 ulp each;
// an IEEE divide is a ten-instruction sequence).
__device__ __forceinline__ float silu_f(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * x));
}

// GELU, tanh approximation: 0.5 x (1 + tanh(u)) with u = sqrt(2/pi) (x + 0.044715 x^3), written
// as x * sigmoid(2u) and evaluated like silu_f.
__device__ __forceinline__ float gelu_tanh_f(float x) {
  const float k = -2.0f * 0.7978845608028654f * 1.4426950408889634f;   // -2 sqrt(2/pi) log2(e)
  const float e = __builtin_amdgcn_exp2f(k * fmaf(0.044715f * x, x * x, x));
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

}  // namespace ff
