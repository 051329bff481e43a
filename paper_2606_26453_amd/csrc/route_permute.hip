// Routing (top-k + softmax), expert grouping (histogram + scan), stable permutation and gather.
//
// Section 5.4 names top-k routing; Appendix H packs the routed rows into one buffer ordered by
// expert with the per-expert row counts given as a cumulative sum.  Every result here is integer
// or a bit copy except topk_w, and all of it is deterministic: counts use integer LDS atomics
// (order-free), ranks come from wave ballots over slots taken in slot order.
#include "common.h"

namespace moe {
namespace {

constexpr int kMaxE = 256;

__device__ __forceinline__ bool better(float v1, int i1, float v2, int i2) {
  return v1 > v2 || (v1 == v2 && i1 < i2);
}

// L lanes cooperate on one token; lane i of the group holds experts i, i+L, i+2L, i+3L.
template <int L>
__global__ __launch_bounds__(256) void route_topk_kernel(const float* __restrict__ logits,
                                                         int64_t T, int E, int k, int normalize,
                                                         int32_t* __restrict__ topk_idx,
                                                         float* __restrict__ topk_w) {
  constexpr int P = (L == 64) ? kMaxE / 64 : 1;  // L < 64 only when E <= L
  const int gl = threadIdx.x % L;
  const int64_t t = (int64_t)blockIdx.x * (256 / L) + threadIdx.x / L;
  const bool live = t < T;
  float v[P];
  int rank[P];
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const int e = gl + L * p;
    v[p] = (live && e < E) ? logits[t * E + e] : -INFINITY;
    if (v[p] != v[p]) v[p] = -INFINITY;  // NaN is not supported; keep every selection valid
    rank[p] = (e < E) ? -1 : -2;  // -1 available, -2 no such expert, >= 0 selected at that rank
  }
  float m = 0.f;
  for (int j = 0; j < k; ++j) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int p = 0; p < P; ++p)
      if (rank[p] == -1 && better(v[p], gl + L * p, bv, bi)) { bv = v[p]; bi = gl + L * p; }
#pragma unroll
    for (int off = L / 2; off > 0; off >>= 1) {
      const float ov = __shfl_xor(bv, off);
      const int oi = __shfl_xor(bi, off);
      if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    if (j == 0) m = bv;
#pragma unroll
    for (int p = 0; p < P; ++p)
      if (gl + L * p == bi) rank[p] = j;
  }
  float s = 0.f;
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (rank[p] >= 0 || (!normalize && rank[p] == -1)) s += expf(v[p] - m);
#pragma unroll
  for (int off = L / 2; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (!live) return;
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (rank[p] >= 0) {
      topk_idx[t * k + rank[p]] = gl + L * p;
      topk_w[t * k + rank[p]] = expf(v[p] - m) / s;
    }
}

// Per-range expert histogram: hist[e * nranges + range].
__global__ __launch_bounds__(256) void hist_kernel(const int32_t* __restrict__ topk_idx, int64_t R,
                                                   int E, int64_t S, int nranges,
                                                   int32_t* __restrict__ hist) {
  __shared__ int cnt[kMaxE];
  for (int e = threadIdx.x; e < E; e += 256) cnt[e] = 0;
  __syncthreads();
  const int64_t lo = (int64_t)blockIdx.x * S;
  const int64_t hi = lo + S < R ? lo + S : R;
  for (int64_t s = lo + threadIdx.x; s < hi; s += 256) atomicAdd(&cnt[topk_idx[s]], 1);
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += 256) hist[(int64_t)e * nranges + blockIdx.x] = cnt[e];
}

// Exclusive scan of hist (e-major) in place -> base[e][range]; offsets[e] = base[e][0].
__global__ __launch_bounds__(1024) void scan_kernel(int32_t* __restrict__ hist, int64_t n,
                                                    int nranges, int E, int64_t R,
                                                    int32_t* __restrict__ offsets) {
  __shared__ int part[1024];
  const int tid = threadIdx.x;
  const int64_t per = (n + 1023) / 1024;
  const int64_t lo = tid * per;
  const int64_t hi = lo + per < n ? lo + per : n;
  int sum = 0;
  for (int64_t i = lo; i < hi; ++i) sum += hist[i];
  part[tid] = sum;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int add = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += add;
    __syncthreads();
  }
  int run = part[tid] - sum;  // exclusive prefix of this thread's segment
  for (int64_t i = lo; i < hi; ++i) {
    const int c = hist[i];
    hist[i] = run;
    run += c;
  }
  __syncthreads();
  for (int e = tid; e < E; e += 1024) offsets[e] = hist[(int64_t)e * nranges];
  if (tid == 0) offsets[E] = (int32_t)R;
}

// One wave per range of S slots, walked in slot order 64 at a time: the rank of a slot among
// the earlier slots of the same expert comes from a ballot match on the expert id bits.
__global__ __launch_bounds__(64) void scatter_kernel(const int32_t* __restrict__ topk_idx, int64_t R,
                                                     int k, int E, int nbits, int64_t S,
                                                     int nranges,
                                                     const int32_t* __restrict__ base,
                                                     int32_t* __restrict__ row_of_slot,
                                                     int32_t* __restrict__ token_of_row) {
  __shared__ int running[kMaxE];
  const int lane = threadIdx.x;
  for (int e = lane; e < E; e += 64) running[e] = 0;
  __syncthreads();
  const int64_t lo = (int64_t)blockIdx.x * S;
  const int64_t hi = lo + S < R ? lo + S : R;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int64_t c0 = lo; c0 < hi; c0 += 64) {
    const int64_t s = c0 + lane;
    const bool act = s < hi;
    const int e = act ? topk_idx[s] : 0;
    uint64_t peers = __ballot(act);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t bal = __ballot(act && bit);
      peers &= bit ? bal : ~bal;
    }
    const int rank = __popcll(peers & below);
    const int cnt = __popcll(peers);
    int row = 0;
    if (act) {
      row = base[(int64_t)e * nranges + blockIdx.x] + running[e] + rank;
      row_of_slot[s] = row;
      token_of_row[row] = (int32_t)(s / k);
    }
    __syncthreads();
    if (act && rank == cnt - 1) running[e] += cnt;
    __syncthreads();
  }
}

// One wave per token: read x[t] once, write it to the token's k rows of x_perm.
template <int U>
__global__ __launch_bounds__(256) void gather_kernel(const u32x4* __restrict__ x, int64_t T,
                                                     int64_t chunks, int k,
                                                     const int32_t* __restrict__ row_of_slot,
                                                     u32x4* __restrict__ x_perm) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const u32x4* src = x + t * chunks;
  for (int64_t c0 = 0; c0 < chunks; c0 += 64 * U) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t c = c0 + u * 64 + lane;
      if (c < chunks) v[u] = src[c];
    }
    for (int j = 0; j < k; ++j) {
      u32x4* dst = x_perm + (int64_t)row_of_slot[t * k + j] * chunks;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 64 + lane;
        if (c < chunks) dst[c] = v[u];
      }
    }
  }
}

__global__ void fill_i32_kernel(int32_t* p, int n, int32_t v) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = v;
}

struct RangePlan {
  int64_t S;
  int nranges;
};

RangePlan plan_ranges(int64_t R) {
  // ranges of S slots (a multiple of 256), at most 4096 of them: short ranges keep the
  // sequential part of the ballot ranking short and give the scatter many wavefronts
  int64_t S = 256 * ((R + 256 * 4096 - 1) / (256 * 4096));
  if (S < 256) S = 256;
  return {S, (int)((R + S - 1) / S)};
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" size_t moe_route_permute_workspace_bytes(int64_t T, int32_t E, int32_t k) {
  if (T <= 0 || E <= 0 || k <= 0) return 0;
  const RangePlan p = plan_ranges(T * (int64_t)k);
  return (size_t)E * p.nranges * sizeof(int32_t);
}

extern "C" moe_status moe_route_permute(const float* logits, const moe_bf16* x, int64_t T,
                                        int64_t d, int32_t E, int32_t k, int32_t normalize_topk,
                                        int32_t* topk_idx, float* topk_w, int32_t* offsets,
                                        int32_t* row_of_slot, int32_t* token_of_row,
                                        moe_bf16* x_perm, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  if (T < 0) return fail(MOE_ERROR_INVALID_VALUE, "moe_route_permute: T < 0");
  if (E < 1 || k < 1 || k > E) return fail(MOE_ERROR_INVALID_VALUE, "moe_route_permute: need 1 <= k <= E");
  if (E > kMaxE) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_route_permute: E > 256");
  if (normalize_topk != 0 && normalize_topk != 1)
    return fail(MOE_ERROR_INVALID_VALUE, "moe_route_permute: normalize_topk must be 0 or 1");
  if ((x == nullptr) != (x_perm == nullptr))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_route_permute: x and x_perm must both be set or both NULL");
  if (x && (d <= 0 || d % 64 != 0))
    return fail(MOE_ERROR_NOT_SUPPORTED, "moe_route_permute: d must be a positive multiple of 64");
  const int64_t R = T * (int64_t)k;
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_route_permute: T*k >= 2^31");
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "moe_route_permute: offsets is NULL");
  if (T == 0) {
    // every group is empty: offsets = 0 (a fill kernel, no memset node)
    fill_i32_kernel<<<1, 256, 0, stream>>>(offsets, E + 1, 0);
    return check_launch("moe_route_permute(T=0)");
  }
  if (!logits || !topk_idx || !topk_w || !row_of_slot || !token_of_row)
    return fail(MOE_ERROR_INVALID_VALUE, "moe_route_permute: NULL pointer");
  if (x && (!aligned16(x) || !aligned16(x_perm)))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_route_permute: x/x_perm not 16-byte aligned");
  const size_t need = moe_route_permute_workspace_bytes(T, E, k);
  if (!workspace || workspace_bytes < need)
    return fail(MOE_ERROR_WORKSPACE, "moe_route_permute: workspace needs %zu bytes", need);

  // A1: top-k + softmax
  int L = 1;
  while (L < E && L < 64) L <<= 1;
  const int tpb = 256 / L;
  const unsigned gr = (unsigned)((T + tpb - 1) / tpb);
  switch (L) {
    case 1: route_topk_kernel<1><<<gr, 256, 0, stream>>>(logits, T, E, k, normalize_topk, topk_idx, topk_w); break;
    case 2: route_topk_kernel<2><<<gr, 256, 0, stream>>>(logits, T, E, k, normalize_topk, topk_idx, topk_w); break;
    case 4: route_topk_kernel<4><<<gr, 256, 0, stream>>>(logits, T, E, k, normalize_topk, topk_idx, topk_w); break;
    case 8: route_topk_kernel<8><<<gr, 256, 0, stream>>>(logits, T, E, k, normalize_topk, topk_idx, topk_w); break;
    case 16: route_topk_kernel<16><<<gr, 256, 0, stream>>>(logits, T, E, k, normalize_topk, topk_idx, topk_w); break;
    case 32: route_topk_kernel<32><<<gr, 256, 0, stream>>>(logits, T, E, k, normalize_topk, topk_idx, topk_w); break;
    default: route_topk_kernel<64><<<gr, 256, 0, stream>>>(logits, T, E, k, normalize_topk, topk_idx, topk_w); break;
  }
  moe_status st = check_launch("route_topk_kernel");
  if (st != MOE_SUCCESS) return st;

  // A2: histogram + scan -> offsets and per-range bases
  const RangePlan p = plan_ranges(R);
  int32_t* hist = static_cast<int32_t*>(workspace);
  hist_kernel<<<p.nranges, 256, 0, stream>>>(topk_idx, R, E, p.S, p.nranges, hist);
  if ((st = check_launch("hist_kernel")) != MOE_SUCCESS) return st;
  scan_kernel<<<1, 1024, 0, stream>>>(hist, (int64_t)E * p.nranges, p.nranges, E, R, offsets);
  if ((st = check_launch("scan_kernel")) != MOE_SUCCESS) return st;

  // A3: stable scatter
  int nbits = 0;
  while ((1 << nbits) < E) ++nbits;
  scatter_kernel<<<p.nranges, 64, 0, stream>>>(topk_idx, R, k, E, nbits, p.S, p.nranges, hist,
                                               row_of_slot, token_of_row);
  if ((st = check_launch("scatter_kernel")) != MOE_SUCCESS) return st;

  // A4: gather
  if (x) {
    const int64_t chunks = d / 8;
    gather_kernel<4><<<(unsigned)((T + 3) / 4), 256, 0, stream>>>(
        reinterpret_cast<const u32x4*>(x), T, chunks, k, row_of_slot, reinterpret_cast<u32x4*>(x_perm));
    if ((st = check_launch("gather_kernel")) != MOE_SUCCESS) return st;
  }
  return MOE_SUCCESS;
}

extern "C" moe_status moe_gather_rows(const moe_bf16* x, int64_t T, int64_t d, int32_t k,
                                      const int32_t* row_of_slot, moe_bf16* x_perm, hipStream_t stream) {
  const char* fn = "moe_gather_rows";
  if (T < 0 || k < 1) return fail(MOE_ERROR_INVALID_VALUE, "%s: need T >= 0 and k >= 1", fn);
  if (d <= 0 || d % 64 != 0) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: d must be a positive multiple of 64", fn);
  if (T * (int64_t)k >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: T*k >= 2^31", fn);
  if (T == 0) return MOE_SUCCESS;
  if (!x || !row_of_slot || !x_perm) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (!aligned16(x) || !aligned16(x_perm)) return fail(MOE_ERROR_INVALID_VALUE, "%s: x/x_perm not 16-byte aligned", fn);
  gather_kernel<4><<<(unsigned)((T + 3) / 4), 256, 0, stream>>>(
      reinterpret_cast<const u32x4*>(x), T, d / 8, k, row_of_slot, reinterpret_cast<u32x4*>(x_perm));
  return check_launch("gather_kernel");
}
