// Per-row quantization of bf16 rows to OCP E4M3 with an fp32 scale per row (the operand format of
// the FP8 grouped product): amax = max |x[r, :]|, scale[r] = amax / 448, and each element becomes
// the E4M3 code nearest to x * (448 / amax), ties to the even mantissa, magnitudes beyond 448
// saturating; an all-zero row gets scale 1 and zero codes.  The quotients and the product are
// single fp32 operations (IEEE round to nearest), so the codes are a function of the inputs alone.
#include "common.h"

namespace moe {
namespace {

// E4M3 code of an fp32 value: sign from the input, magnitude clamped to 448, then rounded to 3
// mantissa bits (normal range, 2^-6 and up) or to a multiple of 2^-9 (subnormals).
__device__ __forceinline__ uint32_t e4m3_code(float y) {
  const uint32_t sign = (__float_as_uint(y) >> 24) & 0x80u;
  if (y != y) return 0x7Fu;
  const float a = fminf(fabsf(y), 448.0f);
  if (a < 0.015625f) {                                   // below 2^-6: multiples of 2^-9, 0 .. 8
    return sign | (uint32_t)__builtin_rintf(a * 512.0f); // 8 is the code of 2^-6 itself
  }
  const uint32_t b = __float_as_uint(a);
  const uint32_t r = (b + 0x7FFFFu + ((b >> 20) & 1u)) & ~0xFFFFFu;   // ties to even at bit 20
  const uint32_t e = (r >> 23) - 127u + 7u;             // biased E4M3 exponent, 1 .. 15
  return sign | (e << 3) | ((r >> 20) & 7u);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// One workgroup (256 threads) per row; each thread handles 8 elements (16 bytes) at a time.
__global__ __launch_bounds__(256) void quantize_fp8_rows_kernel(const u32x4* __restrict__ x, int64_t K8,
                                                                uint2* __restrict__ q, float* __restrict__ scale) {
  __shared__ float s_max[4];
  const int64_t r = blockIdx.x;
  const u32x4* row = x + r * K8;
  float m = 0.0f;
  for (int64_t c = threadIdx.x; c < K8; c += 256) {
    const u32x4 v = row[c];
#pragma unroll
    for (int e = 0; e < 4; ++e) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[e])), fabsf(bf16_hi(v[e]))));
  }
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) s_max[threadIdx.x >> 6] = m;
  __syncthreads();
  const float amax = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
  const bool nz = amax > 0.0f;
  const float inv = nz ? __fdiv_rn(448.0f, amax) : 1.0f;
  if (threadIdx.x == 0) scale[r] = nz ? __fdiv_rn(amax, 448.0f) : 1.0f;
  uint2* qrow = q + r * K8;
  for (int64_t c = threadIdx.x; c < K8; c += 256) {
    const u32x4 v = row[c];
    uint32_t w[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      w[h] = e4m3_code(__fmul_rn(bf16_lo(v[2 * h]), inv)) | (e4m3_code(__fmul_rn(bf16_hi(v[2 * h]), inv)) << 8) |
             (e4m3_code(__fmul_rn(bf16_lo(v[2 * h + 1]), inv)) << 16) |
             (e4m3_code(__fmul_rn(bf16_hi(v[2 * h + 1]), inv)) << 24);
    }
    qrow[c] = make_uint2(w[0], w[1]);
  }
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status moe_quantize_fp8_rows(const moe_bf16* x, int64_t M, int64_t K, uint8_t* q, float* scale,
                                            hipStream_t stream) {
  const char* fn = "moe_quantize_fp8_rows";
  if (M < 0 || K <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (K % 16) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K must be a multiple of 16", fn);
  if (M >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: M >= 2^31", fn);
  if (M == 0) return MOE_SUCCESS;
  if (!x || !q || !scale) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (!aligned16(x) || (reinterpret_cast<uintptr_t>(q) & 7) || (reinterpret_cast<uintptr_t>(scale) & 3))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: x must be 16-byte, q 8-byte, scale 4-byte aligned", fn);
  quantize_fp8_rows_kernel<<<(unsigned)M, 256, 0, stream>>>(reinterpret_cast<const u32x4*>(x), K / 8,
                                                             reinterpret_cast<uint2*>(q), scale);
  return check_launch("quantize_fp8_rows_kernel");
}
