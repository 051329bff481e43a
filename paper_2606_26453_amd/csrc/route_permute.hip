// Routing (top-k + softmax), expert grouping (histogram + scan), stable permutation and gather.
//
// Section 5.4 names top-k routing; Appendix H packs the routed rows into one buffer ordered by
// expert with the per-expert row counts given as a cumulative sum.  Every result here is integer
// or a bit copy except topk_w, and all of it is deterministic: ranks come from wave ballots over
// slots taken in slot order, counts and offsets from integer sums in a fixed order.
#include "common.h"

#include <mutex>

namespace moe {
namespace {

constexpr int kMaxE = 256;
typedef int i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bool better(float v1, int i1, float v2, int i2) {
  return v1 > v2 || (v1 == v2 && i1 < i2);
}

// ---- routing in two launches -------------------------------------------------------------------
// The tokens are split into ranges of TR consecutive tokens (slots t*k + j of those tokens).
//
// Launch 1 (route_rank_kernel, one workgroup per range): top-k and softmax of the range's tokens
// (topk_one), then each slot's rank among the range's earlier slots of the same expert
// (stored in row_of_slot for launch 2) and the range's per-expert count hist[range * E + e].
// The range's slots are split into four contiguous quarters, one per wavefront: a wave ranks its
// quarter with ballots (64 slots at a time, in slot order), the counts of the earlier quarters are
// added after one barrier, so the rank is the slot's position in slot order (stable).
//
// Launch 2 (route_rows_kernel, one workgroup per range): every workgroup reduces the histogram
// (expert-major, nranges x E integers) to the per-expert totals -- an exclusive scan of which gives
// offsets -- and to the counts of the ranges before its own; a slot's row is then
// offsets[e] + (slots of e in earlier ranges) + (its rank inside the range).  The workgroup then
// copies its tokens' rows of x to x_perm (one wavefront per token, x read once per token).  Integer
// sums only: no atomics, nothing depends on the order in which workgroups run.
constexpr int kRankWaves = 4;
constexpr int kMaxRangeSlots = 4096;

// Top-k of one token by L cooperating lanes (gl = lane within the group); lane i of the group holds
// experts i, i+L, ..., i+(P-1)L (L*P >= E): k rounds of a local then butterfly arg-max with an index
// tie-break, then the softmax over the selected logits (or over all E with normalize = 0).
template <int L, int P>
__device__ __forceinline__ void topk_one(const float* __restrict__ logits, int64_t t, bool live, int E, int k,
                                         int normalize, int gl, int32_t* __restrict__ topk_idx,
                                         float* __restrict__ topk_w, int32_t* sel /* LDS, k entries or NULL */) {
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
      if (sel) sel[rank[p]] = gl + L * p;
    }
}

template <int L, int P>
__global__ __launch_bounds__(256) void route_rank_kernel(const float* __restrict__ logits, int64_t T, int E, int k,
                                                         int normalize, int TR, int nranges, int nbits,
                                                         int32_t* __restrict__ topk_idx, float* __restrict__ topk_w,
                                                         int32_t* __restrict__ rank_of_slot,
                                                         int32_t* __restrict__ hist) {
  __shared__ int sel[kMaxRangeSlots];             // expert of each slot of the range
  __shared__ int rk[kMaxRangeSlots];              // rank of the slot inside its wave's quarter
  __shared__ int cnt[kRankWaves][kMaxE];          // per-quarter expert counts
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * TR;
  const int ntok = (int)(T - t0 < TR ? T - t0 : TR);
  for (int i = tid; i < kRankWaves * kMaxE; i += 256) (&cnt[0][0])[i] = 0;
  // top-k: L lanes per token, 256 / L tokens per pass
  for (int i0 = 0; i0 < ntok; i0 += 256 / L) {
    const int i = i0 + tid / L;
    const bool live = i < ntok;
    topk_one<L, P>(logits, t0 + (live ? i : 0), live, E, k, normalize, tid % L, topk_idx, topk_w,
                live ? sel + i * k : nullptr);
  }
  __syncthreads();
  // rank inside each wave's quarter (slot order), counting the quarter's slots per expert
  const int n = ntok * k;
  const int q0 = (int)((int64_t)n * wave / kRankWaves), q1 = (int)((int64_t)n * (wave + 1) / kRankWaves);
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int c0 = q0; c0 < q1; c0 += 64) {
    const int s = c0 + lane;
    const bool act = s < q1;
    const int e = act ? sel[s] : 0;
    uint64_t peers = __ballot(act);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t bal = __ballot(act && bit);
      peers &= bit ? bal : ~bal;
    }
    const int r = __popcll(peers & below);
    const int c = __popcll(peers);
    if (act) rk[s] = cnt[wave][e] + r;
    __builtin_amdgcn_wave_barrier();
    if (act && r == c - 1) cnt[wave][e] += c;   // one lane per expert present
    __builtin_amdgcn_wave_barrier();
  }
  __syncthreads();
  // the range's counts, and each slot's rank among the range's slots of its expert
  for (int e = tid; e < E; e += 256) {
    int tot = 0;
#pragma unroll
    for (int w = 0; w < kRankWaves; ++w) tot += cnt[w][e];
    hist[(int64_t)blockIdx.x * E + e] = tot;
  }
  for (int s = tid; s < n; s += 256) {
    int w = 0;   // quarter holding s
    while (w < kRankWaves - 1 && (int)((int64_t)n * (w + 1) / kRankWaves) <= s) ++w;
    int add = 0;
    const int e = sel[s];
    for (int w2 = 0; w2 < w; ++w2) add += cnt[w2][e];
    rank_of_slot[t0 * k + s] = add + rk[s];
  }
}

// Launch 2 (512 threads).  The histogram is reduced to per-expert totals (all ranges) and counts of
// the ranges before this workgroup's.  When E divides 2048 and is a multiple of 4, thread t reads the
// 16-byte chunks t, t + 512, ... of hist (all of them holding experts (4t) mod E .. +3), lanes of a
// wave holding the same experts are summed by shuffles and the eight waves through LDS; otherwise
// S = 512 / E threads per expert each sum a segment of the expert's column.
constexpr int kRowsThreads = 512;

template <int U>
__global__ __launch_bounds__(kRowsThreads) void route_rows_kernel(const int32_t* __restrict__ hist, int nranges,
                                                                  int E, int64_t T, int k, int TR,
                                                                  const int32_t* __restrict__ topk_idx,
                                                                  int32_t* __restrict__ offsets,
                                                                  int32_t* __restrict__ row_of_slot,
                                                                  int32_t* __restrict__ token_of_row,
                                                                  const u32x4* __restrict__ x, int64_t chunks,
                                                                  u32x4* __restrict__ x_perm) {
  constexpr int NT = kRowsThreads, NW = NT / 64;
  __shared__ int red_all[NW][kMaxE], red_pre[NW][kMaxE];
  __shared__ int off_e[kMaxE + 1], base_e[kMaxE];
  __shared__ int rows[kMaxRangeSlots];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = blockIdx.x;
  if ((E & 3) == 0 && (2048 % E) == 0) {
    const int nvec = nranges * (E >> 2);
    const i32x4* hv = reinterpret_cast<const i32x4*>(hist);
    int a0 = 0, a1 = 0, a2 = 0, a3 = 0, b0 = 0, b1 = 0, b2 = 0, b3 = 0;
#pragma unroll 8
    for (int c = tid; c < nvec; c += NT) {
      const i32x4 v = hv[c];
      const bool before = (4 * c) / E < r;
      a0 += v[0]; a1 += v[1]; a2 += v[2]; a3 += v[3];
      if (before) { b0 += v[0]; b1 += v[1]; b2 += v[2]; b3 += v[3]; }
    }
    // lanes l and l + E/4 (mod 64) hold the same experts
    for (int off = E >> 2; off < 64; off <<= 1) {
      a0 += __shfl_xor(a0, off); a1 += __shfl_xor(a1, off); a2 += __shfl_xor(a2, off); a3 += __shfl_xor(a3, off);
      b0 += __shfl_xor(b0, off); b1 += __shfl_xor(b1, off); b2 += __shfl_xor(b2, off); b3 += __shfl_xor(b3, off);
    }
    if (lane < (E >> 2) || (E >> 2) >= 64) {
      const int e0 = (4 * tid) % E;
      red_all[wave][e0] = a0; red_all[wave][e0 + 1] = a1; red_all[wave][e0 + 2] = a2; red_all[wave][e0 + 3] = a3;
      red_pre[wave][e0] = b0; red_pre[wave][e0 + 1] = b1; red_pre[wave][e0 + 2] = b2; red_pre[wave][e0 + 3] = b3;
    }
    __syncthreads();
    if (tid < E) {
      int all = 0, pre = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) { all += red_all[w][tid]; pre += red_pre[w][tid]; }
      off_e[tid + 1] = all;   // the inclusive scan below turns these into offsets[tid + 1]
      base_e[tid] = pre;
    }
  } else {
    const int S = NT / E;
    const int e = tid / S, seg = tid - e * S;
    int all = 0, pre = 0;
    if (e < E) {
      const int lo = (int)((int64_t)nranges * seg / S), hi = (int)((int64_t)nranges * (seg + 1) / S);
      for (int i = lo; i < hi; ++i) {
        const int v = hist[(int64_t)i * E + e];
        all += v;
        pre += i < r ? v : 0;
      }
    }
    int* ra = &red_all[0][0];
    int* rp = &red_pre[0][0];
    ra[tid] = all;
    rp[tid] = pre;
    __syncthreads();
    if (tid < E) {
      int sa = 0, sp = 0;
      for (int j = 0; j < S; ++j) { sa += ra[tid * S + j]; sp += rp[tid * S + j]; }
      off_e[tid + 1] = sa;
      base_e[tid] = sp;
    }
  }
  if (tid == 0) off_e[0] = 0;
  __syncthreads();
  for (int d = 1; d < E; d <<= 1) {   // inclusive scan of off_e[1..E]
    const int v = (tid < E && tid >= d) ? off_e[tid + 1 - d] : 0;
    __syncthreads();
    if (tid < E) off_e[tid + 1] += v;
    __syncthreads();
  }
  if (r == 0)
    for (int e = tid; e <= E; e += NT) offsets[e] = off_e[e];
  // rows of the range's slots
  const int64_t t0 = (int64_t)r * TR;
  const int ntok = (int)(T - t0 < TR ? T - t0 : TR);
  const int n = ntok * k;
  for (int s = tid; s < n; s += NT) {
    const int64_t slot = t0 * k + s;
    const int e = topk_idx[slot];
    const int row = off_e[e] + base_e[e] + row_of_slot[slot];
    row_of_slot[slot] = row;
    token_of_row[row] = (int32_t)(slot / k);
    rows[s] = row;
  }
  if (x == nullptr) return;
  __syncthreads();
  // gather: one wavefront per token, U chunks per lane in flight, each x row read once
  for (int i = wave; i < ntok; i += NW) {
    const u32x4* src = x + (t0 + i) * chunks;
    for (int64_t c0 = 0; c0 < chunks; c0 += 64 * U) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 64 + lane;
        if (c < chunks) v[u] = ld_stream(src + c);
      }
      for (int j = 0; j < k; ++j) {
        u32x4* dst = x_perm + (int64_t)rows[i * k + j] * chunks;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int64_t c = c0 + u * 64 + lane;
          if (c < chunks) dst[c] = v[u];
        }
      }
    }
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
      if (c < chunks) v[u] = ld_stream(src + c);
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
  int TR;        // tokens per range
  int nranges;
};

// Ranges of TR tokens: a multiple of 16, sized so that the histogram (nranges x E integers, which
// every workgroup of launch 2 reads) stays near 64 KiB, and at most kMaxRangeSlots slots.
RangePlan plan_ranges(int64_t T, int E, int k) {
  int64_t tr = (T * E + 16383) / 16384;
  tr = (tr + 15) / 16 * 16;
  if (tr < 16) tr = 16;
  int64_t cap = kMaxRangeSlots / k / 16 * 16;   // k <= 256 keeps this >= 16
  if (cap > 1024) cap = 1024;
  if (tr > cap) tr = cap;
  return {(int)tr, (int)((T + tr - 1) / tr)};
}

size_t route_workspace_bytes(int64_t T, int E, int k) {
  if (T <= 0 || E <= 0 || k <= 0 || k > kMaxE) return 0;
  const RangePlan p = plan_ranges(T, E, k);
  return (size_t)E * p.nranges * sizeof(int32_t);
}

// Shared body of moe_route_permute and its allocation-free variant; hist is the caller's scratch
// of at least route_workspace_bytes(T, E, k) bytes (contents on entry ignored).
moe_status route_permute_impl(const char* fn, const float* logits, const moe_bf16* x, int64_t T, int64_t d,
                              int32_t E, int32_t k, int32_t normalize_topk, int32_t* topk_idx, float* topk_w,
                              int32_t* offsets, int32_t* row_of_slot, int32_t* token_of_row, moe_bf16* x_perm,
                              int32_t* hist, hipStream_t stream) {
  const RangePlan p = plan_ranges(T, E, k);
  // lanes per token: the next power of two >= E up to 16, then P = E / 16 (rounded up to a power of
  // two) experts per lane
  int L = 1;
  while (L < E && L < 16) L <<= 1;
  int P = 1;
  while (L * P < E) P <<= 1;
  int nbits = 0;
  while ((1 << nbits) < E) ++nbits;
  // launch 1: top-k, softmax, ranks inside each range, per-range counts
#define MOE_RANK(LL, PP)                                                                                        \
  route_rank_kernel<LL, PP><<<p.nranges, 256, 0, stream>>>(logits, T, E, k, normalize_topk, p.TR, p.nranges, \
                                                           nbits, topk_idx, topk_w, row_of_slot, hist)
  switch (L * 100 + P) {
    case 101: MOE_RANK(1, 1); break;
    case 201: MOE_RANK(2, 1); break;
    case 401: MOE_RANK(4, 1); break;
    case 801: MOE_RANK(8, 1); break;
    case 1601: MOE_RANK(16, 1); break;
    case 1602: MOE_RANK(16, 2); break;
    case 1604: MOE_RANK(16, 4); break;
    case 1608: MOE_RANK(16, 8); break;
    default: MOE_RANK(16, 16); break;
  }
#undef MOE_RANK
  moe_status st = check_launch("route_rank_kernel");
  if (st != MOE_SUCCESS) return st;
  // launch 2: offsets, rows, and the gather (U 16-byte chunks per lane and token in flight)
  const int64_t chunks = x ? d / 8 : 0;
  const u32x4* xs = reinterpret_cast<const u32x4*>(x);
  u32x4* xp = reinterpret_cast<u32x4*>(x_perm);
#define MOE_ROWS(UU) \
  route_rows_kernel<UU><<<p.nranges, kRowsThreads, 0, stream>>>(hist, p.nranges, E, T, k, p.TR, topk_idx, offsets, \
                                                               row_of_slot, token_of_row, xs, chunks, xp)
  if (chunks >= 512) MOE_ROWS(8);
  else if (chunks >= 256) MOE_ROWS(4);
  else if (chunks >= 128) MOE_ROWS(2);
  else MOE_ROWS(1);
#undef MOE_ROWS
  (void)fn;
  return check_launch("route_rows_kernel");
}

moe_status route_check(const char* fn, const float* logits, const moe_bf16* x, int64_t T, int64_t d, int32_t E,
                       int32_t k, int32_t normalize_topk, int32_t* topk_idx, float* topk_w, int32_t* offsets,
                       int32_t* row_of_slot, int32_t* token_of_row, moe_bf16* x_perm) {
  if (T < 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: T < 0", fn);
  if (E < 1 || k < 1 || k > E) return fail(MOE_ERROR_INVALID_VALUE, "%s: need 1 <= k <= E", fn);
  if (E > kMaxE) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: E > 256", fn);
  if (normalize_topk != 0 && normalize_topk != 1)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: normalize_topk must be 0 or 1", fn);
  if ((x == nullptr) != (x_perm == nullptr))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: x and x_perm must both be set or both NULL", fn);
  if (x && (d <= 0 || d % 64 != 0))
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: d must be a positive multiple of 64", fn);
  if (T * (int64_t)k >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: T*k >= 2^31", fn);
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "%s: offsets is NULL", fn);
  if (T == 0) return MOE_SUCCESS;
  if (!logits || !topk_idx || !topk_w || !row_of_slot || !token_of_row)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (x && (!aligned16(x) || !aligned16(x_perm)))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: x/x_perm not 16-byte aligned", fn);
  return MOE_SUCCESS;
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" size_t moe_route_permute_workspace_bytes(int64_t T, int32_t E, int32_t k) {
  return route_workspace_bytes(T, E, k);
}

extern "C" moe_status moe_route_permute(const float* logits, const moe_bf16* x, int64_t T,
                                        int64_t d, int32_t E, int32_t k, int32_t normalize_topk,
                                        int32_t* topk_idx, float* topk_w, int32_t* offsets,
                                        int32_t* row_of_slot, int32_t* token_of_row,
                                        moe_bf16* x_perm, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  const char* fn = "moe_route_permute";
  moe_status st = route_check(fn, logits, x, T, d, E, k, normalize_topk, topk_idx, topk_w, offsets, row_of_slot,
                              token_of_row, x_perm);
  if (st != MOE_SUCCESS) return st;
  if (T == 0) {
    // every group is empty: offsets = 0 (a fill kernel, no memset node)
    fill_i32_kernel<<<1, 256, 0, stream>>>(offsets, E + 1, 0);
    return check_launch("moe_route_permute(T=0)");
  }
  const size_t need = route_workspace_bytes(T, E, k);
  if (!workspace || workspace_bytes < need || !aligned16(workspace))
    return fail(MOE_ERROR_WORKSPACE, "%s: a 16-byte aligned workspace of %zu bytes is needed", fn, need);
  return route_permute_impl(fn, logits, x, T, d, E, k, normalize_topk, topk_idx, topk_w, offsets, row_of_slot,
                            token_of_row, x_perm, static_cast<int32_t*>(workspace), stream);
}

// ---- allocation-free variant -----------------------------------------------------------------
// Scratch for moe_route_permute_noalloc: the per-range histogram lives in this file-scope device
// array instead of a caller workspace.  In host code `route_scratch` names a host-side stand-in,
// not device memory: its device address is looked up once per device (hipGetSymbolAddress, with
// that device current) and only that address is passed to kernels.  Every device holds its own
// copy until the process ends; calls on one device share it (overlapping calls race).
constexpr size_t kNoAllocScratchBytes = 256 * 1024;
static __device__ __align__(256) int32_t route_scratch[kNoAllocScratchBytes / sizeof(int32_t)];

namespace moe {
namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of route_scratch, looked up on the first call on that device.
moe_status route_scratch_ptr(const char* fn, int32_t** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(MOE_ERROR_HIP, "%s: no current device (or device index >= %d)", fn, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(route_scratch));
    if (e != hipSuccess || ptr == nullptr)
      return fail(MOE_ERROR_HIP, "%s: hipGetSymbolAddress(route_scratch) failed: %s", fn, hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = static_cast<int32_t*>(g_scratch_ptr[dev]);
  return MOE_SUCCESS;
}
}  // namespace
}  // namespace moe

extern "C" size_t moe_route_permute_noalloc_max_scratch_bytes(void) { return kNoAllocScratchBytes; }

extern "C" moe_status moe_route_permute_noalloc(const float* logits, const moe_bf16* x, int64_t T, int64_t d,
                                                int32_t E, int32_t k, int32_t normalize_topk, int32_t* topk_idx,
                                                float* topk_w, int32_t* offsets, int32_t* row_of_slot,
                                                int32_t* token_of_row, moe_bf16* x_perm, hipStream_t stream) {
  const char* fn = "moe_route_permute_noalloc";
  moe_status st = route_check(fn, logits, x, T, d, E, k, normalize_topk, topk_idx, topk_w, offsets, row_of_slot,
                              token_of_row, x_perm);
  if (st != MOE_SUCCESS) return st;
  if (T == 0) {
    fill_i32_kernel<<<1, 256, 0, stream>>>(offsets, E + 1, 0);
    return check_launch("moe_route_permute_noalloc(T=0)");
  }
  const size_t need = route_workspace_bytes(T, E, k);
  if (need > kNoAllocScratchBytes)
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: these sizes need %zu bytes of scratch, more than the %zu it holds "
                "(use moe_route_permute with a workspace)", fn, need, kNoAllocScratchBytes);
  int32_t* hist = nullptr;
  if ((st = route_scratch_ptr(fn, &hist)) != MOE_SUCCESS) return st;
  return route_permute_impl(fn, logits, x, T, d, E, k, normalize_topk, topk_idx, topk_w, offsets, row_of_slot,
                            token_of_row, x_perm, hist, stream);
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
