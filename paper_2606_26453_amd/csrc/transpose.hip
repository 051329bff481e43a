// Grouped transpose into the contraction-major layout of the weight-gradient products:
// dst[c][p] = src[row(p)][c], where the rows of each group g (offsets[g] .. offsets[g+1]) land at
// columns pstart[g] .. pstart[g] + rows_g of dst and the group's segment is zero-padded to a
// multiple of 32 columns (pstart = exclusive prefix of the padded group sizes).  With both dW
// operands in this layout, the contraction of each group is contiguous in memory and the dW GEMM
// reads its tiles with plain 16-byte LDS reads instead of transposing ones.
#include "common.h"

namespace moe {
namespace {

constexpr int TP = 64;       // tile: 64 padded rows x 64 columns through LDS

// Padded group starts over <= 256 groups, computed by every workgroup (256 threads) into LDS:
// s_p[g] = sum_{h<g} ceil32(rows_h), s_p[G] = padded total (inclusive scan of the padded sizes,
// shifted by one).
__device__ __forceinline__ void padded_prefix(const int32_t* __restrict__ offsets, int G, int* s_p,
                                              int* s_off) {
  const int tid = threadIdx.x;
  for (int i = tid; i <= G; i += blockDim.x) s_off[i] = offsets[i];
  __syncthreads();
  int v = tid < G ? ((s_off[tid + 1] - s_off[tid] + 31) & ~31) : 0;
  s_p[tid + 1] = v;
  if (tid == 0) s_p[0] = 0;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {
    const int add = tid >= o ? s_p[tid + 1 - o] : 0;
    __syncthreads();
    s_p[tid + 1] += add;
    __syncthreads();
  }
}

// Workgroup: 256 threads, one 64 x 64 tile of dst (64 padded positions p x 64 columns c).
__global__ __launch_bounds__(256) void transpose_grouped_kernel(const uint16_t* __restrict__ src,
                                                                const int32_t* __restrict__ offsets, int G,
                                                                int64_t C, int64_t ld_dst,
                                                                uint16_t* __restrict__ dst) {
  __shared__ int s_p[257], s_off[257];
  __shared__ uint16_t tile[TP][TP + 2];
  padded_prefix(offsets, G, s_p, s_off);
  const int64_t p0 = (int64_t)blockIdx.x * TP;
  const int64_t c0 = (int64_t)blockIdx.y * TP;
  if (p0 >= s_p[G]) return;                      // uniform: past the padded total
  const int tid = threadIdx.x;
  // load: thread -> (row p = p0 + tid/4, 16 columns (tid%4)*16 ..); rows past their group's real
  // rows (padding) read as zeros
  {
    const int pl = tid >> 2, cq = (tid & 3) * 16;
    const int64_t p = p0 + pl;
    int64_t r = -1;
    if (p < s_p[G]) {
      int lo = 0, hi = G;                        // group g with s_p[g] <= p < s_p[g+1]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_p[mid] <= p) lo = mid; else hi = mid;
      }
      const int64_t within = p - s_p[lo];
      if (within < s_off[lo + 1] - s_off[lo]) r = s_off[lo] + within;
    }
    u32x4 v0 = {0, 0, 0, 0}, v1 = {0, 0, 0, 0};
    if (r >= 0 && c0 + cq < C) {
      const u32x4* s = reinterpret_cast<const u32x4*>(src + r * C + c0 + cq);
      v0 = s[0];
      v1 = s[1];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      tile[pl][cq + 2 * q] = (uint16_t)(v0[q] & 0xffff);
      tile[pl][cq + 2 * q + 1] = (uint16_t)(v0[q] >> 16);
      tile[pl][cq + 8 + 2 * q] = (uint16_t)(v1[q] & 0xffff);
      tile[pl][cq + 8 + 2 * q + 1] = (uint16_t)(v1[q] >> 16);
    }
  }
  __syncthreads();
  // store: thread -> (column c = c0 + tid/4, 16 positions (tid%4)*16 ..): 32 contiguous bytes
  {
    const int cl = tid >> 2, pq = (tid & 3) * 16;
    if (c0 + cl < C) {
      u32x4 w0, w1;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        w0[q] = (uint32_t)tile[pq + 2 * q][cl] | ((uint32_t)tile[pq + 2 * q + 1][cl] << 16);
        w1[q] = (uint32_t)tile[pq + 8 + 2 * q][cl] | ((uint32_t)tile[pq + 8 + 2 * q + 1][cl] << 16);
      }
      u32x4* d = reinterpret_cast<u32x4*>(dst + (c0 + cl) * ld_dst + p0 + pq);
      d[0] = w0;
      d[1] = w1;
    }
  }
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" int64_t moe_transposed_cols_bound(int64_t R, int32_t G) {
  if (R < 0 || G < 1) return 0;
  return ((R + 31) & ~(int64_t)31) + 32 * (int64_t)G;
}

extern "C" moe_status moe_transpose_grouped(const moe_bf16* src, const int32_t* offsets, int32_t G, int64_t R,
                                            int64_t C, moe_bf16* dst, int64_t ld_dst, hipStream_t stream) {
  const char* fn = "moe_transpose_grouped";
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: need 1 <= G <= 256", fn);
  if (R < 0 || C <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (C % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: C must be a multiple of 64", fn);
  const int64_t bound = moe_transposed_cols_bound(R, G);
  if (ld_dst < bound || ld_dst % 64)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: ld_dst must be a multiple of 64 and >= %lld", fn, (long long)bound);
  if (!offsets || !dst || (R > 0 && !src)) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if ((src && !aligned16(src)) || !aligned16(dst))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: pointers must be 16-byte aligned", fn);
  if (bound / TP >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: too large", fn);
  dim3 grid((unsigned)((bound + TP - 1) / TP), (unsigned)(C / TP));
  transpose_grouped_kernel<<<grid, 256, 0, stream>>>(src, offsets, G, C, ld_dst, dst);
  return check_launch("transpose_grouped");
}
