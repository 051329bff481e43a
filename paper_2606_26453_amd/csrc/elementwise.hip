// HBM-bound kernels of the layer: SwiGLU forward/backward (elementwise over [rows, f]) and the
// weighted unpermute-combine with its backward (one wavefront per token; each token's rows of
// the permuted buffer are whole 16-byte-vector rows, so every access is a coalesced row copy).
#include "common.h"

namespace moe {
namespace {

__global__ __launch_bounds__(256) void swiglu_kernel(const u32x4* __restrict__ hg,
                                                     const u32x4* __restrict__ hu,
                                                     u32x4* __restrict__ act, int64_t n8) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n8; i += (int64_t)gridDim.x * 256) {
    float g[8], u[8], a[8];
    unpack8(hg[i], g);
    unpack8(hu[i], u);
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = silu_f32(g[j]) * u[j];
    act[i] = pack8(a);
  }
}

__device__ __forceinline__ void swiglu_bwd8(const u32x4& hg, const u32x4& hu, const u32x4& da,
                                            u32x4& dhg, u32x4& dhu) {
  float g[8], u[8], d[8], og[8], ou[8];
  unpack8(hg, g);
  unpack8(hu, u);
  unpack8(da, d);
#pragma unroll
  for (int j = 0; j < 8; ++j) swiglu_bwd1(g[j], u[j], d[j], og[j], ou[j]);
  dhg = pack8(og);
  dhu = pack8(ou);
}

// one 16-byte vector (8 elements) per thread, no grid-stride loop
__global__ __launch_bounds__(256) void swiglu_bwd_kernel(const u32x4* __restrict__ hg,
                                                         const u32x4* __restrict__ hu,
                                                         const u32x4* __restrict__ da,
                                                         u32x4* __restrict__ dhg,
                                                         u32x4* __restrict__ dhu, int64_t n8) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  u32x4 a, b;
  swiglu_bwd8(hg[i], hu[i], da[i], a, b);
  dhg[i] = a;
  dhu[i] = b;
}

// y[t] = bf16(sum_j w[t,j] * y_perm[row_of_slot[t*k+j]] + add[t]).  KK > 0: k == KK.  NT: the
// permuted rows (and add) are read with streaming loads.
template <int U, int KK, bool NT>
__global__ __launch_bounds__(256) void combine_kernel(const u32x4* __restrict__ y_perm,
                                                      const float* __restrict__ w,
                                                      const int32_t* __restrict__ row_of_slot,
                                                      const u32x4* __restrict__ add, int64_t T,
                                                      int64_t chunks, int k,
                                                      u32x4* __restrict__ y) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  if constexpr (KK > 0) {
    // k known at compile time: the chunks of all k source rows are loaded before any is summed
    // (KK*U loads in flight per lane instead of U), summed in the same order as below
    const u32x4* src[KK];
    float wj[KK];
#pragma unroll
    for (int j = 0; j < KK; ++j) {
      src[j] = y_perm + (int64_t)row_of_slot[t * KK + j] * chunks;
      wj[j] = w ? w[t * KK + j] : 1.0f;
    }
    for (int64_t c0 = 0; c0 < chunks; c0 += 64 * U) {
      u32x4 v[KK][U];
#pragma unroll
      for (int j = 0; j < KK; ++j)
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int64_t c = c0 + u * 64 + lane;
          v[j][u] = c < chunks ? ld_maybe_stream<NT>(src[j] + c) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 64 + lane;
        float acc[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = 0.f;
#pragma unroll
        for (int j = 0; j < KK; ++j) {
          float f[8];
          unpack8(v[j][u], f);
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[i] += wj[j] * f[i];
        }
        if (c < chunks) {
          if (add) {
            float f[8];
            unpack8(ld_maybe_stream<NT>(add + t * chunks + c), f);
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] += f[i];
          }
          y[t * chunks + c] = pack8(acc);
        }
      }
    }
    return;
  }
  for (int64_t c0 = 0; c0 < chunks; c0 += 64 * U) {
    float acc[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[u][i] = 0.f;
    for (int j = 0; j < k; ++j) {
      const int64_t r = row_of_slot[t * k + j];
      const float wj = w ? w[t * k + j] : 1.0f;
      const u32x4* src = y_perm + r * chunks;
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 64 + lane;
        if (c < chunks) v[u] = ld_maybe_stream<NT>(src + c);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float f[8];
        unpack8(v[u], f);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[u][i] += wj * f[i];
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t c = c0 + u * 64 + lane;
      if (c < chunks) {
        if (add) {
          float f[8];
          unpack8(ld_maybe_stream<NT>(add + t * chunks + c), f);
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[u][i] += f[i];
        }
        y[t * chunks + c] = pack8(acc[u]);
      }
    }
  }
}

// dy_perm[row] = bf16(w * dy[t]); d_w[t,j] = <dy[t], y_perm[row]>.  The token's choices are taken
// eight at a time; for each group the dY row is read once per chunk and the partial dot products
// stay in registers until one wavefront reduction per choice at the end.  KK > 0: k == KK, and U
// chunks of dY and of every Y_perm row are loaded per lane before any is used (the same sums).
template <int U, int KK>
__global__ __launch_bounds__(256) void combine_bwd_kernel(const u32x4* __restrict__ dy,
                                                          const float* __restrict__ w,
                                                          const int32_t* __restrict__ row_of_slot,
                                                          const u32x4* __restrict__ y_perm,
                                                          int64_t T, int64_t chunks, int k,
                                                          u32x4* __restrict__ dy_perm,
                                                          float* __restrict__ d_w) {
  constexpr int J = 8;
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const u32x4* src = dy + t * chunks;
  if constexpr (KK > 0) {
    static_assert(KK <= J, "one group of choices");
    int64_t row[KK];
    float wj[KK], dot[KK];
#pragma unroll
    for (int j = 0; j < KK; ++j) {
      row[j] = row_of_slot[t * KK + j];
      wj[j] = w[t * KK + j];
      dot[j] = 0.f;
    }
    for (int64_t c0 = lane; c0 < chunks; c0 += 64 * U) {
      u32x4 dv[U], yv[KK][U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + 64 * u;
        dv[u] = c < chunks ? ld_stream(src + c) : u32x4{0u, 0u, 0u, 0u};
        if (y_perm) {
#pragma unroll
          for (int j = 0; j < KK; ++j) yv[j][u] = c < chunks ? ld_stream(y_perm + row[j] * chunks + c) : u32x4{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + 64 * u;
        if (c < chunks) {
          float f[8];
          unpack8(dv[u], f);
#pragma unroll
          for (int j = 0; j < KK; ++j) {
            float o[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) o[i] = wj[j] * f[i];
            dy_perm[row[j] * chunks + c] = pack8(o);
            if (y_perm) {
              float yf[8];
              unpack8(yv[j][u], yf);
#pragma unroll
              for (int i = 0; i < 8; ++i) dot[j] += f[i] * yf[i];
            }
          }
        }
      }
    }
    if (y_perm && d_w) {
#pragma unroll
      for (int j = 0; j < KK; ++j) {
        float v = dot[j];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
        if (lane == 0) d_w[t * KK + j] = v;
      }
    }
    return;
  }
  for (int j0 = 0; j0 < k; j0 += J) {
    const int nj = k - j0 < J ? k - j0 : J;
    int64_t row[J];
    float wj[J], dot[J];
#pragma unroll
    for (int j = 0; j < J; ++j) {
      row[j] = j < nj ? row_of_slot[t * k + j0 + j] : 0;
      wj[j] = j < nj ? w[t * k + j0 + j] : 0.f;
      dot[j] = 0.f;
    }
    for (int64_t c = lane; c < chunks; c += 64) {
      float f[8];
      unpack8(ld_stream(src + c), f);
#pragma unroll
      for (int j = 0; j < J; ++j) {
        if (j < nj) {
          float o[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) o[i] = wj[j] * f[i];
          dy_perm[row[j] * chunks + c] = pack8(o);
          if (y_perm) {
            float yf[8];
            unpack8(ld_stream(y_perm + row[j] * chunks + c), yf);
#pragma unroll
            for (int i = 0; i < 8; ++i) dot[j] += f[i] * yf[i];
          }
        }
      }
    }
    if (y_perm && d_w) {
#pragma unroll
      for (int j = 0; j < J; ++j) {
        if (j < nj) {
          float v = dot[j];
#pragma unroll
          for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
          if (lane == 0) d_w[t * k + j0 + j] = v;
        }
      }
    }
  }
}

unsigned elementwise_grid(int64_t n8) {
  const int64_t want = (n8 + 255) / 256;
  const int64_t cap = (int64_t)device_cu_count() * 16;
  return (unsigned)(want < cap ? (want > 0 ? want : 1) : cap);
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status moe_swiglu(const moe_bf16* h_gate, const moe_bf16* h_up, moe_bf16* act,
                                 int64_t rows, int64_t f, hipStream_t stream) {
  if (rows < 0 || f < 0) return fail(MOE_ERROR_INVALID_VALUE, "moe_swiglu: negative size");
  if (f % 64 != 0) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_swiglu: f must be a multiple of 64");
  if (rows == 0 || f == 0) return MOE_SUCCESS;
  if (!h_gate || !h_up || !act) return fail(MOE_ERROR_INVALID_VALUE, "moe_swiglu: NULL pointer");
  if (!aligned16(h_gate) || !aligned16(h_up) || !aligned16(act))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_swiglu: pointers must be 16-byte aligned");
  const int64_t n8 = rows * f / 8;
  swiglu_kernel<<<elementwise_grid(n8), 256, 0, stream>>>(
      reinterpret_cast<const u32x4*>(h_gate), reinterpret_cast<const u32x4*>(h_up),
      reinterpret_cast<u32x4*>(act), n8);
  return check_launch("swiglu_kernel");
}

extern "C" moe_status moe_swiglu_bwd(const moe_bf16* h_gate, const moe_bf16* h_up,
                                     const moe_bf16* d_act, moe_bf16* dh_gate, moe_bf16* dh_up,
                                     int64_t rows, int64_t f, hipStream_t stream) {
  if (rows < 0 || f < 0) return fail(MOE_ERROR_INVALID_VALUE, "moe_swiglu_bwd: negative size");
  if (f % 64 != 0) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_swiglu_bwd: f must be a multiple of 64");
  if (rows == 0 || f == 0) return MOE_SUCCESS;
  if (!h_gate || !h_up || !d_act || !dh_gate || !dh_up)
    return fail(MOE_ERROR_INVALID_VALUE, "moe_swiglu_bwd: NULL pointer");
  if (!aligned16(h_gate) || !aligned16(h_up) || !aligned16(d_act) || !aligned16(dh_gate) ||
      !aligned16(dh_up))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_swiglu_bwd: pointers must be 16-byte aligned");
  const int64_t n8 = rows * f / 8;
  if ((n8 + 255) / 256 > 0x7fffffff)
    return fail(MOE_ERROR_NOT_SUPPORTED, "moe_swiglu_bwd: rows*f too large");
  swiglu_bwd_kernel<<<(unsigned)((n8 + 255) / 256), 256, 0, stream>>>(
      reinterpret_cast<const u32x4*>(h_gate), reinterpret_cast<const u32x4*>(h_up),
      reinterpret_cast<const u32x4*>(d_act), reinterpret_cast<u32x4*>(dh_gate),
      reinterpret_cast<u32x4*>(dh_up), n8);
  return check_launch("swiglu_bwd_kernel");
}

// about eight 16-byte loads in flight per lane for the common k
template <bool NT>
static void launch_combine(unsigned grid, hipStream_t stream, const u32x4* yp, const float* w, const int32_t* rows,
                    const u32x4* ad, int64_t T, int64_t chunks, int k, u32x4* yo) {
  switch (k) {
    case 1: combine_kernel<8, 1, NT><<<grid, 256, 0, stream>>>(yp, w, rows, ad, T, chunks, k, yo); break;
    case 2: combine_kernel<4, 2, NT><<<grid, 256, 0, stream>>>(yp, w, rows, ad, T, chunks, k, yo); break;
    case 4: combine_kernel<2, 4, NT><<<grid, 256, 0, stream>>>(yp, w, rows, ad, T, chunks, k, yo); break;
    case 6: combine_kernel<1, 6, NT><<<grid, 256, 0, stream>>>(yp, w, rows, ad, T, chunks, k, yo); break;
    case 8: combine_kernel<1, 8, NT><<<grid, 256, 0, stream>>>(yp, w, rows, ad, T, chunks, k, yo); break;
    default: combine_kernel<4, 0, NT><<<grid, 256, 0, stream>>>(yp, w, rows, ad, T, chunks, k, yo); break;
  }
}

extern "C" moe_status moe_unpermute_combine(const moe_bf16* y_perm, const float* topk_w,
                                            const int32_t* row_of_slot, const moe_bf16* add,
                                            int64_t T, int64_t d, int32_t k, moe_bf16* y,
                                            hipStream_t stream) {
  if (T < 0 || d < 0) return fail(MOE_ERROR_INVALID_VALUE, "moe_unpermute_combine: negative size");
  if (k < 1 || k > 256) return fail(MOE_ERROR_INVALID_VALUE, "moe_unpermute_combine: need 1 <= k <= 256");
  if (d % 64 != 0) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_unpermute_combine: d must be a multiple of 64");
  if (T == 0 || d == 0) return MOE_SUCCESS;
  if (!y_perm || !row_of_slot || !y)
    return fail(MOE_ERROR_INVALID_VALUE, "moe_unpermute_combine: NULL pointer");
  if (!aligned16(y_perm) || !aligned16(y) || (add && !aligned16(add)))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_unpermute_combine: pointers must be 16-byte aligned");
  const int64_t chunks = d / 8;
  const unsigned grid = (unsigned)((T + 3) / 4);
  const u32x4* yp = reinterpret_cast<const u32x4*>(y_perm);
  const u32x4* ad = reinterpret_cast<const u32x4*>(add);
  u32x4* yo = reinterpret_cast<u32x4*>(y);
  // Without weights this is the unpermute-sum of dX: its input was just written and is read once,
  // so it streams.  The weighted forward combine streams Y_perm only when Y_perm is too large to
  // stay in the 256 MiB Infinity Cache until the backward reads it again (taken as over half of
  // it); a smaller one is read with plain loads, which leave it there (measured on the
  // Mixtral-shaped layer, Y_perm 128 MiB: streaming made the combine 2 us shorter and its
  // backward 8 us longer; on the fine-grained layer, Y_perm 384 MiB, the combine 111 -> 94 us).
  constexpr int64_t kCacheHalf = (int64_t)128 << 20;
  if (topk_w && T * k * d * 2 <= kCacheHalf)
    launch_combine<false>(grid, stream, yp, topk_w, row_of_slot, ad, T, chunks, k, yo);
  else
    launch_combine<true>(grid, stream, yp, topk_w, row_of_slot, ad, T, chunks, k, yo);
  return check_launch("combine_kernel");
}

extern "C" moe_status moe_unpermute_combine_bwd(const moe_bf16* dy, const float* topk_w,
                                                const int32_t* row_of_slot, const moe_bf16* y_perm,
                                                int64_t T, int64_t d, int32_t k, moe_bf16* dy_perm,
                                                float* d_topk_w, hipStream_t stream) {
  if (T < 0 || d < 0) return fail(MOE_ERROR_INVALID_VALUE, "moe_unpermute_combine_bwd: negative size");
  if (k < 1 || k > 256) return fail(MOE_ERROR_INVALID_VALUE, "moe_unpermute_combine_bwd: need 1 <= k <= 256");
  if (d % 64 != 0) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_unpermute_combine_bwd: d must be a multiple of 64");
  if (T == 0 || d == 0) return MOE_SUCCESS;
  if (!dy || !topk_w || !row_of_slot || !dy_perm)
    return fail(MOE_ERROR_INVALID_VALUE, "moe_unpermute_combine_bwd: NULL pointer");
  if (!aligned16(dy) || !aligned16(dy_perm) || (y_perm && !aligned16(y_perm)))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_unpermute_combine_bwd: pointers must be 16-byte aligned");
  const int64_t chunks = d / 8;
  const unsigned grid = (unsigned)((T + 3) / 4);
  const u32x4* dyp = reinterpret_cast<const u32x4*>(dy);
  const u32x4* yp = reinterpret_cast<const u32x4*>(y_perm);
  u32x4* dpo = reinterpret_cast<u32x4*>(dy_perm);
  switch (k) {
    case 1: combine_bwd_kernel<4, 1><<<grid, 256, 0, stream>>>(dyp, topk_w, row_of_slot, yp, T, chunks, k, dpo, d_topk_w); break;
    case 2: combine_bwd_kernel<4, 2><<<grid, 256, 0, stream>>>(dyp, topk_w, row_of_slot, yp, T, chunks, k, dpo, d_topk_w); break;
    case 4: combine_bwd_kernel<2, 4><<<grid, 256, 0, stream>>>(dyp, topk_w, row_of_slot, yp, T, chunks, k, dpo, d_topk_w); break;
    case 6: combine_bwd_kernel<1, 6><<<grid, 256, 0, stream>>>(dyp, topk_w, row_of_slot, yp, T, chunks, k, dpo, d_topk_w); break;
    case 8: combine_bwd_kernel<1, 8><<<grid, 256, 0, stream>>>(dyp, topk_w, row_of_slot, yp, T, chunks, k, dpo, d_topk_w); break;
    default: combine_bwd_kernel<1, 0><<<grid, 256, 0, stream>>>(dyp, topk_w, row_of_slot, yp, T, chunks, k, dpo, d_topk_w); break;
  }
  return check_launch("combine_bwd_kernel");
}
