// Internal helpers shared by the library's HIP sources (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "moe.h"

namespace moe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two fp32 -> packed bf16x2, round-to-nearest-even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

// A 16-byte load of data read once and not again soon (a routed row on its way through a copy or
// a combine, a weight on its way to its codes): non-temporal, i.e. streamed past the caches
// instead of displacing what they hold.  Measured on the layer's copies and combines: 5-17%
// shorter than plain loads.  Stores stay plain (non-temporal stores measured slower).
__device__ __forceinline__ u32x4 ld_stream(const u32x4* p) { return __builtin_nontemporal_load(p); }
template <bool NT> __device__ __forceinline__ u32x4 ld_maybe_stream(const u32x4* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

// 8 bf16 in a 16-byte vector <-> 8 floats.
__device__ __forceinline__ void unpack8(const u32x4& v, float* f) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = bf16_lo(v[i]);
    f[2 * i + 1] = bf16_hi(v[i]);
  }
}
__device__ __forceinline__ u32x4 pack8(const float* f) {
  u32x4 v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = pack_bf16(f[2 * i], f[2 * i + 1]);
  return v;
}

// sigmoid(g) = 1 / (1 + exp(-g)) and silu(g) = g * sigmoid(g) in fp32, from the hardware base-2
// exponential and reciprocal (each within 1 ulp): exp(-g) = 2^(-g * log2(e)).  The results are
// stored as bf16, whose rounding step is 2^16 times coarser than these errors.  Limits: g -> -inf
// gives exp -> inf, sigmoid -> 0, silu -> -0; g -> +inf gives sigmoid -> 1, silu -> g.
__device__ __forceinline__ float sigmoid_f32(float g) {
  constexpr float LOG2E = 1.4426950408889634f;
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-g * LOG2E));
}
__device__ __forceinline__ float silu_f32(float g) { return g * sigmoid_f32(g); }

// SwiGLU backward for one element (the same arithmetic everywhere it is computed):
// dh_up = d * g * s, dh_gate = d * u * s * (1 + g * (1 - s)), s = sigmoid(g).
__device__ __forceinline__ void swiglu_bwd1(float g, float u, float d, float& dh_gate, float& dh_up) {
  const float s = sigmoid_f32(g);
  dh_up = d * g * s;
  dh_gate = d * u * s * (1.0f + g * (1.0f - s));
}

}  // namespace moe

// ---- host-side status plumbing (defined in status.hip) ----
namespace moe {
moe_status fail(moe_status s, const char* fmt, ...);
moe_status check_launch(const char* what);
int device_cu_count();
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
}  // namespace moe
