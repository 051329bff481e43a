// Router of the MoE layer on the GPU: logits = x . Wr (+ bias), the backward through the routing
// weights (d_topk_w -> dlogits, plus an optional Switch-style load-balancing loss), and the
// router map's backward (dWr = x^T . dlogits, dX += dlogits . Wr^T).
//
// The contractions are tiny (E <= 256 experts) and their fp32 operands must stay fp32, so these
// are vector-ALU kernels, not MFMA.  At the usual sizes (E <= 16, d <= 4096) a lane owns 8
// consecutive hidden columns and streams x or dX rows in 1 KiB wavefront accesses (the
// column-parallel kernels below); per-token work over the experts (softmax, dlogits) takes one
// lane per token.  Other sizes use the general kernels: one lane per token (logits) or per pair of
// hidden columns (dX, dWr), with the operand that is the same for the whole wavefront (rows of
// Wr, a block of tokens' dlogits) staged in LDS and read as broadcasts.
#include "common.h"

namespace moe {
namespace {

constexpr int RL_WAVES = 8;     // logits: wavefronts per workgroup, each a slice of the hidden dim
constexpr int RL_ROWS = 32;     // logits: rows of Wr staged per wavefront at a time
constexpr int RB_EC = 32;       // backward: experts per register chunk
constexpr int RB_TOK = 64;      // dX / dWr: tokens per workgroup block
constexpr int RB_SUB = 16;      // tokens per LDS-staged block of dlogits

// logits[t, e] = sum_i x[t, i] * wr[i, e] (+ bias[e]), fp32.  Workgroup: 128 tokens (lane =
// tokens t and t + 64) x RL_WAVES slices of the hidden dimension; each wavefront stages RL_ROWS
// rows of its slice of Wr (EG experts) in LDS, loading the next rows into registers while it
// works on the current ones, and reads them as broadcasts; the slices' partial sums are added in
// slice order through LDS, so the result does not depend on the launch.  EG experts per pass (8,
// 16 or 32, the smallest that covers E up to 32; grid.y covers the rest).
template <int EG>
__global__ __launch_bounds__(64 * RL_WAVES) void router_logits_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ wr, const float* __restrict__ bias,
    int64_t T, int64_t d, int E, float* __restrict__ logits) {
  constexpr int PER = RL_ROWS * EG / 64;        // staged values per lane
  __shared__ __attribute__((aligned(16))) float s_w[RL_WAVES][RL_ROWS][EG];
  __shared__ float part[EG][128];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int e0 = blockIdx.y * EG;
  const int64_t ta = (int64_t)blockIdx.x * 128 + lane, tb = ta + 64;
  const int64_t tca = ta < T ? ta : T - 1, tcb = tb < T ? tb : T - 1;
  const int64_t slice = d / RL_WAVES;           // a multiple of 8 (d is a multiple of 64)
  const int64_t i_begin = w * slice, i_end = i_begin + slice;
  float acc[2][EG];
#pragma unroll
  for (int e = 0; e < EG; ++e) acc[0][e] = acc[1][e] = 0.0f;
  const u32x4* xa = reinterpret_cast<const u32x4*>(x + tca * d);
  const u32x4* xb = reinterpret_cast<const u32x4*>(x + tcb * d);
  float nxt[PER];
  auto fetch = [&](int64_t r0) {                // rows r0 .. of the slice (0 past its end or E)
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int o = lane + 64 * q, rr = o / EG, e = o - rr * EG;
      nxt[q] = (r0 + rr < i_end && e0 + e < E) ? wr[(r0 + rr) * E + e0 + e] : 0.0f;
    }
  };
  fetch(i_begin);
  for (int64_t r0 = i_begin; r0 < i_end; r0 += RL_ROWS) {
    const int rows = (int)((i_end - r0) < RL_ROWS ? (i_end - r0) : RL_ROWS);   // a multiple of 8
#pragma unroll
    for (int q = 0; q < PER; ++q) (&s_w[w][0][0])[lane + 64 * q] = nxt[q];
    __builtin_amdgcn_s_waitcnt(0xc07f);          // lgkmcnt(0): this wave's LDS writes landed
    __builtin_amdgcn_wave_barrier();
    if (r0 + RL_ROWS < i_end) fetch(r0 + RL_ROWS);
    for (int rb = 0; rb < rows; rb += 8) {
      float xv[2][8];
      unpack8(xa[(r0 + rb) >> 3], xv[0]);
      unpack8(xb[(r0 + rb) >> 3], xv[1]);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const f32x4* wrow = reinterpret_cast<const f32x4*>(&s_w[w][rb + u][0]);
#pragma unroll
        for (int q = 0; q < EG / 4; ++q) {
          const f32x4 wv = wrow[q];
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[h][4 * q + c] = __builtin_fmaf(xv[h][u], wv[c], acc[h][4 * q + c]);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();             // every lane is done with the staged rows
  }
  // slices added in slice order: wavefront 0 stores its sums, then 1 .. RL_WAVES-1 add theirs
  for (int ww = 0; ww < RL_WAVES; ++ww) {
    if (w == ww) {
#pragma unroll
      for (int e = 0; e < EG; ++e) {
        part[e][lane] = ww ? part[e][lane] + acc[0][e] : acc[0][e];
        part[e][lane + 64] = ww ? part[e][lane + 64] + acc[1][e] : acc[1][e];
      }
    }
    __syncthreads();
  }
  for (int o = threadIdx.x; o < EG * 128; o += 64 * RL_WAVES) {
    const int e = o >> 7, tl = o & 127;
    const int64_t tt = (int64_t)blockIdx.x * 128 + tl;
    if (tt >= T || e0 + e >= E) continue;
    float s = part[e][tl];
    if (bias) s += bias[e0 + e];
    logits[tt * E + e0 + e] = s;
  }
}

constexpr int RD_TPW = 4;       // dlogits: tokens per wavefront
constexpr int RA_TPW = 16;      // load-balancing loss: tokens per wavefront
constexpr int RD_EPL = 4;       // experts per lane (E <= 64 * RD_EPL = 256)

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Full softmax of one token's logits across the wavefront: lane l holds experts l, l+64, ...
// (q = 0 past E).
__device__ __forceinline__ void wave_softmax(const float* __restrict__ L, int E, int lane, float* q) {
  float v[RD_EPL];
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < RD_EPL; ++j) {
    const int e = lane + 64 * j;
    v[j] = e < E ? L[e] : -INFINITY;
    m = fmaxf(m, v[j]);
  }
  m = wave_max(m);
  float z = 0.0f;
#pragma unroll
  for (int j = 0; j < RD_EPL; ++j) {
    q[j] = lane + 64 * j < E ? expf(v[j] - m) : 0.0f;
    z += q[j];
  }
  z = wave_sum(z);
#pragma unroll
  for (int j = 0; j < RD_EPL; ++j) q[j] = q[j] / z;
}

// dlogits of a token: the routing weights' backward (with p the probabilities the weights were
// read from: the k weights themselves when normalized, the full softmax otherwise), plus the
// load-balancing loss's gradient when alpha != 0:
//   dl[e] = p[e] * (G[e] - sum_j g_j w_j)  +  alpha*E/T * q[e] * (f[e] - sum_e' f[e'] q[e'])
// with G[e] = g_j if e = topk_idx[j] (else 0), q the full softmax, f[e] = counts[e] / (T*k).
// One wavefront per RD_TPW tokens, lane l owning experts l, l+64, ... (coalesced rows; the
// softmax reductions are wavefront reductions).
__global__ __launch_bounds__(256) void router_dlogits_kernel(
    const float* __restrict__ logits, const int32_t* __restrict__ topk_idx,
    const float* __restrict__ topk_w, const float* __restrict__ d_topk_w,
    const int32_t* __restrict__ offsets, int64_t T, int E, int k, int normalize, float alpha,
    float* __restrict__ dlogits) {
  const int lane = threadIdx.x & 63;
  const int64_t wv = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const bool full = !normalize || alpha != 0.0f;
  const float inv_slots = 1.0f / (float)(T * k);
  const float aux = alpha * (float)E / (float)T;
  float f[RD_EPL];
#pragma unroll
  for (int j = 0; j < RD_EPL; ++j) {
    const int e = lane + 64 * j;
    f[j] = (alpha != 0.0f && e < E) ? (float)(offsets[e + 1] - offsets[e]) * inv_slots : 0.0f;
  }
  for (int64_t t = wv * RD_TPW; t < (wv + 1) * RD_TPW && t < T; ++t) {
    const float* L = logits + t * E;
    float q[RD_EPL] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (full) wave_softmax(L, E, lane, q);
    float gw = 0.0f;                       // sum_j g_j w_j (the same in every lane)
    for (int j = 0; j < k; ++j) gw += d_topk_w[t * k + j] * topk_w[t * k + j];
    float fq = 0.0f;
    if (alpha != 0.0f) {
#pragma unroll
      for (int j = 0; j < RD_EPL; ++j) fq += f[j] * q[j];
      fq = wave_sum(fq);
    }
    float out[RD_EPL];
#pragma unroll
    for (int j = 0; j < RD_EPL; ++j) {
      out[j] = normalize ? 0.0f : -q[j] * gw;          // the G = 0 part of p * (G - gw)
      if (alpha != 0.0f) out[j] += aux * q[j] * (f[j] - fq);
    }
    // selected experts: + p_e * G_e (normalized: p_e = w_j, and the -p_e * gw term lives there)
    for (int j = 0; j < k; ++j) {
      const int e = topk_idx[t * k + j];
      const float g = d_topk_w[t * k + j];
#pragma unroll
      for (int jj = 0; jj < RD_EPL; ++jj)
        if (e == lane + 64 * jj) out[jj] += normalize ? topk_w[t * k + j] * (g - gw) : q[jj] * g;
    }
#pragma unroll
    for (int j = 0; j < RD_EPL; ++j)
      if (lane + 64 * j < E) dlogits[t * E + lane + 64 * j] = out[j];
  }
}

// A block of dlogits, dl[t0 .. t0+RB_SUB-1][ec .. ec+EC-1] (0 past T or E), fetched into
// registers by one wavefront (PER values per lane) and later stored to LDS for broadcast reads.
template <int EC>
struct DlBlock {
  static constexpr int PER = RB_SUB * EC / 64;
  float v[PER];
  __device__ __forceinline__ void fetch(const float* __restrict__ dl, int64_t t0, int64_t T, int ec, int E,
                                        int lane) {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int o = lane + 64 * q, t = o / EC, e = o - t * EC;
      v[q] = (t0 + t < T && ec + e < E) ? dl[(t0 + t) * E + ec + e] : 0.0f;
    }
  }
  __device__ __forceinline__ void store(float* s, int lane) const {
#pragma unroll
    for (int q = 0; q < PER; ++q) s[lane + 64 * q] = v[q];
    __builtin_amdgcn_s_waitcnt(0xc07f);          // lgkmcnt(0): the writes landed
    __builtin_amdgcn_wave_barrier();
  }
};

// Wr^T [E, d] from Wr [d, E] (so that a wavefront reads a row of experts' weights for 128
// consecutive hidden columns in one access).
__global__ __launch_bounds__(256) void router_transpose_kernel(const float* __restrict__ wr, int64_t d, int E,
                                                             float* __restrict__ wrt) {
  const int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (o >= d * E) return;
  const int64_t e = o / d, i = o - e * d;
  wrt[o] = wr[i * E + e];
}

// dX[t, i] = bf16(dX[t, i] + sum_e dl[t, e] * wr[i, e]) for the 2 hidden columns i, i+1 of each
// lane (a one-wavefront workgroup covers 128 columns) and RB_TOK tokens, in blocks of RB_SUB
// tokens whose sums stay in registers; Wr's columns stay in registers for RB_DXE experts at
// a time, and each block's dlogits are read from LDS as broadcasts while the next block is being
// fetched.
constexpr int RB_DXE = 32;
__global__ __launch_bounds__(64) void router_dx_kernel(
    const float* __restrict__ dl, const float* __restrict__ wrt, int64_t T, int64_t d, int E,
    uint16_t* __restrict__ dx) {
  __shared__ __attribute__((aligned(16))) float s_dl[RB_SUB][RB_DXE];
  const int lane = threadIdx.x;
  const int64_t i = (int64_t)blockIdx.x * 128 + 2 * lane;      // d is a multiple of 64: i+1 < d or
  const bool col_ok = i < d;                                   // both columns are out of range
  const int64_t ic = col_ok ? i : 0;
  const int64_t t_beg = (int64_t)blockIdx.y * RB_TOK;
  const int64_t t_end = t_beg + RB_TOK < T ? t_beg + RB_TOK : T;
  const int nch = (E + RB_DXE - 1) / RB_DXE;
  float w0[RB_DXE], w1[RB_DXE];
  auto load_w = [&](int ec) {                    // Wr^T rows: 64 lanes read 512 contiguous bytes
#pragma unroll
    for (int e = 0; e < RB_DXE; ++e) {
      const bool ok = ec + e < E;
      const f32x2 v = ok ? *reinterpret_cast<const f32x2*>(wrt + (int64_t)(ec + e) * d + ic) : f32x2{0.0f, 0.0f};
      w0[e] = v[0];
      w1[e] = v[1];
    }
  };
  load_w(0);
  DlBlock<RB_DXE> blk;
  blk.fetch(dl, t_beg, t_end, 0, E, lane);
  for (int64_t tb = t_beg; tb < t_end; tb += RB_SUB) {
    float acc0[RB_SUB], acc1[RB_SUB];
#pragma unroll
    for (int t = 0; t < RB_SUB; ++t) acc0[t] = acc1[t] = 0.0f;
    for (int ci = 0; ci < nch; ++ci) {
      if (nch > 1 && (ci > 0 || tb > t_beg)) load_w(ci * RB_DXE);
      blk.store(&s_dl[0][0], lane);
      // fetch the next block: the next expert chunk of these tokens, or the next tokens
      if (ci + 1 < nch) blk.fetch(dl, tb, t_end, (ci + 1) * RB_DXE, E, lane);
      else if (tb + RB_SUB < t_end) blk.fetch(dl, tb + RB_SUB, t_end, 0, E, lane);
#pragma unroll
      for (int t = 0; t < RB_SUB; ++t) {
        const f32x4* g = reinterpret_cast<const f32x4*>(&s_dl[t][0]);
#pragma unroll
        for (int q = 0; q < RB_DXE / 4; ++q) {
          const f32x4 gv = g[q];
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            acc0[t] = __builtin_fmaf(gv[c], w0[4 * q + c], acc0[t]);
            acc1[t] = __builtin_fmaf(gv[c], w1[4 * q + c], acc1[t]);
          }
        }
      }
      __builtin_amdgcn_wave_barrier();           // every lane is done with this block of s_dl
    }
    if (col_ok) {
#pragma unroll
      for (int t = 0; t < RB_SUB; ++t) {
        if (tb + t < t_end) {
          uint32_t* p = reinterpret_cast<uint32_t*>(dx + (tb + t) * d + i);
          const uint32_t v = *p;
          *p = pack_bf16(bf16_lo(v) + acc0[t], bf16_hi(v) + acc1[t]);
        }
      }
    }
  }
}

// Partial dWr over token chunk c: part[c][i][e] = sum_{t in chunk c} x[t, i] * dl[t, e]; lane = 2
// hidden columns, RB_EC experts per pass (grid.z); the chunk's dlogits are read from LDS as
// broadcasts in blocks of RB_SUB tokens while the next block (and its x values) is fetched.
__global__ __launch_bounds__(64) void router_dwr_partial_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ dl, int64_t T, int64_t d, int E,
    int64_t chunk, float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) float s_dl[RB_SUB][RB_EC];
  const int lane = threadIdx.x;
  const int64_t i = (int64_t)blockIdx.x * 128 + 2 * lane;
  const bool col_ok = i < d;
  const int64_t ic = col_ok ? i : 0;
  const int c = blockIdx.y;
  const int ec = blockIdx.z * RB_EC;
  const int64_t tb0 = (int64_t)c * chunk;
  const int64_t te = (tb0 + chunk) < T ? (tb0 + chunk) : T;
  float a0[RB_EC], a1[RB_EC];
#pragma unroll
  for (int e = 0; e < RB_EC; ++e) a0[e] = a1[e] = 0.0f;
  uint32_t xn[RB_SUB];
  auto fetch_x = [&](int64_t tb) {
#pragma unroll
    for (int t = 0; t < RB_SUB; ++t)
      xn[t] = (tb + t < te) ? *reinterpret_cast<const uint32_t*>(x + (tb + t) * d + ic) : 0u;
  };
  DlBlock<RB_EC> blk;
  if (tb0 < te) {
    fetch_x(tb0);
    blk.fetch(dl, tb0, te, ec, E, lane);
  }
  for (int64_t tb = tb0; tb < te; tb += RB_SUB) {
    uint32_t xv[RB_SUB];
#pragma unroll
    for (int t = 0; t < RB_SUB; ++t) xv[t] = xn[t];
    blk.store(&s_dl[0][0], lane);
    if (tb + RB_SUB < te) {
      fetch_x(tb + RB_SUB);
      blk.fetch(dl, tb + RB_SUB, te, ec, E, lane);
    }
#pragma unroll
    for (int t = 0; t < RB_SUB; ++t) {
      const float x0 = bf16_lo(xv[t]), x1 = bf16_hi(xv[t]);
      const f32x4* g = reinterpret_cast<const f32x4*>(&s_dl[t][0]);
#pragma unroll
      for (int q = 0; q < RB_EC / 4; ++q) {
        const f32x4 gv = g[q];
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
          a0[4 * q + cc] = __builtin_fmaf(x0, gv[cc], a0[4 * q + cc]);
          a1[4 * q + cc] = __builtin_fmaf(x1, gv[cc], a1[4 * q + cc]);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  if (!col_ok) return;
  float* o0 = part + ((int64_t)c * d + i) * E;
#pragma unroll
  for (int e = 0; e < RB_EC; ++e) {
    if (ec + e < E) {
      o0[ec + e] = a0[e];
      o0[E + ec + e] = a1[e];
    }
  }
}

// dWr[i, e] = sum_c part[c][i][e], chunks added in order.
__global__ __launch_bounds__(256) void router_dwr_reduce_kernel(const float* __restrict__ part, int nchunk,
                                                              int64_t n, float* __restrict__ dwr) {
  const int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (o >= n) return;
  float s = part[o];
  int c = 1;
  for (; c + 8 <= nchunk; c += 8) {       // eight loads in flight, then added in chunk order
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = part[(int64_t)(c + u) * n + o];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  for (; c < nchunk; ++c) s += part[(int64_t)c * n + o];
  dwr[o] = s;
}

// Load-balancing loss, first stage: each wavefront sums the full softmax of its RA_TPW tokens per
// expert (lane l owning experts l, l+64, ...) in token order; the workgroup's four sums are added
// in wavefront order and stored as one row of partials.
__global__ __launch_bounds__(256) void router_aux_partial_kernel(const float* __restrict__ logits, int64_t T,
                                                                 int E, float* __restrict__ part) {
  __shared__ float s_acc[4][64 * RD_EPL];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t wv = (int64_t)blockIdx.x * 4 + w;
  float acc[RD_EPL] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t t = wv * RA_TPW; t < (wv + 1) * RA_TPW && t < T; ++t) {
    float q[RD_EPL];
    wave_softmax(logits + t * E, E, lane, q);
#pragma unroll
    for (int j = 0; j < RD_EPL; ++j) acc[j] += q[j];
  }
#pragma unroll
  for (int j = 0; j < RD_EPL; ++j) s_acc[w][lane + 64 * j] = acc[j];
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += 256)
    part[(int64_t)blockIdx.x * E + e] = ((s_acc[0][e] + s_acc[1][e]) + s_acc[2][e]) + s_acc[3][e];
}

// Second stage: loss = alpha * E * sum_e f_e * P_e, P_e = (sum of the partial rows) / T.  Thread
// (e, h) of 4 per expert sums rows h, h+4, ... (eight independent running sums, added in a fixed
// order), then the four are added in order.
__global__ __launch_bounds__(256) void router_aux_final_kernel(const float* __restrict__ part, int nrow,
                                                               const int32_t* __restrict__ offsets,
                                                               int64_t T, int E, int k, float alpha,
                                                               float* __restrict__ loss) {
  __shared__ float s_p[4][64];
  __shared__ float s_v[64];
  float total = 0.0f;
  for (int eb = 0; eb < E; eb += 64) {
    const int e = eb + (threadIdx.x & 63), h = threadIdx.x >> 6;
    float r[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (e < E)
      for (int b = h; b < nrow; b += 32) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (b + 4 * u < nrow) r[u] += part[(int64_t)(b + 4 * u) * E + e];
      }
    s_p[h][threadIdx.x & 63] = ((r[0] + r[1]) + (r[2] + r[3])) + ((r[4] + r[5]) + (r[6] + r[7]));
    __syncthreads();
    if (threadIdx.x < 64) {
      const float P = (((s_p[0][threadIdx.x] + s_p[1][threadIdx.x]) + s_p[2][threadIdx.x]) + s_p[3][threadIdx.x]) / (float)T;
      s_v[threadIdx.x] = e < E ? (float)(offsets[e + 1] - offsets[e]) / (float)(T * k) * P : 0.0f;
    }
    __syncthreads();
    if (threadIdx.x == 0)
      for (int j = 0; j < 64; ++j) total += s_v[j];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = alpha * (float)E * total;
}

// ---------------------------------------------------------------------------------------------
// Column-parallel forms for the router's usual sizes (E <= 16 experts, d <= 4096): a lane owns 8
// consecutive hidden columns, so every wavefront access to x or dX is 1 KiB of one row, and the
// lane keeps its columns' rows of Wr (8 x EG fp32) in registers.  At E = 8 the contractions do
// about 8 flops per byte of x, under the fp32 vector-ALU / HBM ridge: these kernels are meant to
// stream x (or dX) at HBM speed.
// ---------------------------------------------------------------------------------------------
template <int N>
struct Log2 { static constexpr int v = 1 + Log2<N / 2>::v; };
template <>
struct Log2<1> { static constexpr int v = 0; };

// a + b across lane halves (v_permlane32_swap): lanes 0-31 get a[l] + a[l + 32], lanes 32-63 get
// b[l - 32] + b[l]; the same across the 16-lane rows of each half (v_permlane16_swap).
__device__ __forceinline__ float pair_sum32(float a, float b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair_sum16(float a, float b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sum of N (4 <= N <= 64, a power of 2) per-lane values over the 64 lanes of a wavefront,
// scattered: afterwards v[0] of lane l holds the wavefront's total of value l >> (6 - log2 N) (the
// 64/N lanes of a group hold the same total).  log2 N halving steps (lane offsets 32, 16, ...: the
// lanes with the offset bit set keep the upper half of the values), the first two by lane-swap
// instructions, the rest by two shuffles and a choice between the two sums; then full sums over the
// remaining offsets.  A fixed pattern of adds.
template <int N>
__device__ __forceinline__ float wave_reduce_scatter(float (&v)[N], int lane) {
  static_assert(N >= 4 && N <= 64 && (N & (N - 1)) == 0, "4..64 values, a power of 2");
  constexpr int LOG = Log2<N>::v;
#pragma unroll
  for (int i = 0; i < N / 2; ++i) v[i] = pair_sum32(v[i], v[i + N / 2]);
#pragma unroll
  for (int i = 0; i < N / 4; ++i) v[i] = pair_sum16(v[i], v[i + N / 4]);
#pragma unroll
  for (int s = 2; s < 6; ++s) {
    const int o = 32 >> s;
    if (s < LOG) {
      const int half = N >> (s + 1);
      const bool up = (lane & o) != 0;
#pragma unroll
      for (int i = 0; i < N / 8; ++i) {
        if (i < half) {
          const float a = v[i], b = v[i + half];
          const float sa = a + __shfl_xor(a, o, 64), sb = b + __shfl_xor(b, o, 64);
          v[i] = up ? sb : sa;
        }
      }
    } else {
      v[0] += __shfl_xor(v[0], o, 64);
    }
  }
  return v[0];
}

// Rows col .. col+7 of wr [d, E], experts e0 .. e0+EG-1 (0 past E or for an idle lane); 16-byte
// loads when the whole group is in range and aligned.
template <int EG>
__device__ __forceinline__ void load_wr_rows(const float* __restrict__ wr, int64_t col, bool ok, int E, int e0,
                                             float (&wv)[8][EG]) {
  const bool vec = e0 + EG <= E && (E & 3) == 0 && (reinterpret_cast<uintptr_t>(wr) & 15) == 0;
  if (vec) {
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
      for (int q = 0; q < EG / 4; ++q) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(wr + (col + c) * E + e0 + 4 * q);
#pragma unroll
        for (int i = 0; i < 4; ++i) wv[c][4 * q + i] = ok ? v[i] : 0.0f;
      }
  } else {
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
      for (int e = 0; e < EG; ++e) wv[c][e] = (ok && e0 + e < E) ? wr[(col + c) * E + e0 + e] : 0.0f;
  }
}

// DPP-moved copy of v: lane l gets v of lane l ^ 8 (row_ror:8 within rows of 16), of lane
// (l & ~7) | (7 - (l & 7)) (row_half_mirror), of l ^ 2 or of l ^ 1 (quad_perm).
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, true));
}
constexpr int DPP_ROR8 = 0x128, DPP_HALF_MIRROR = 0x141, DPP_XOR2 = 0x4e, DPP_XOR1 = 0xb1;

// One halving step inside a row of 16 lanes: pairs (v[i], v[i + H]) for i < H; the lane whose
// bit (up) is set keeps the upper value plus its partner's upper value, the other the lower pair.
template <int H, int CTRL>
__device__ __forceinline__ void dpp_halve(float* v, bool up) {
#pragma unroll
  for (int i = 0; i < H; ++i) {
    const float a = v[i], b = v[i + H];
    const float send = up ? a : b, keep = up ? b : a;
    v[i] = keep + dpp_mov<CTRL>(send);
  }
}

// Transposing sum over the wavefront: 64 values per lane in, lane l out with the wavefront's
// total of value l.  Six halving steps (lane offsets 32 and 16 by lane swaps; 8 by a rotation of
// each 16-lane row; then the mirror of each half-row and the quad swaps, each of which pairs every
// lane with one across the step's bit), all on the vector ALU with no LDS round trip, and the 64
// totals come out spread one per lane.  A fixed pattern of adds.
__device__ __forceinline__ float wave_transpose_sum64(float (&v)[64], int lane) {
#pragma unroll
  for (int i = 0; i < 32; ++i) v[i] = pair_sum32(v[i], v[i + 32]);
#pragma unroll
  for (int i = 0; i < 16; ++i) v[i] = pair_sum16(v[i], v[i + 16]);
  dpp_halve<8, DPP_ROR8>(v, (lane & 8) != 0);
  dpp_halve<4, DPP_HALF_MIRROR>(v, (lane & 4) != 0);
  dpp_halve<2, DPP_XOR2>(v, (lane & 2) != 0);
  dpp_halve<1, DPP_XOR1>(v, (lane & 1) != 0);
  return v[0];
}

constexpr int RC_ROUND = 8;     // logits: tokens per round (one LDS exchange per round)

// logits[t, e0 + e] for EG experts e0 = blockIdx.y * EG and the tpb tokens of block blockIdx.x.
// The NW wavefronts of a workgroup cover d = 512 * NW columns (lanes past d/8 hold zeros); per
// round of RC_ROUND tokens each lane sums its 8 columns' products (column order) for every
// (token, expert), the wavefront adds them across its lanes with wave_transpose_sum64, and the NW
// wavefront totals are added in wavefront order through LDS.  The next round's x values are loaded
// while the current round is summed.
template <int EG, int NW>
__global__ __launch_bounds__(64 * NW) void router_logits_cols_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ wr, const float* __restrict__ bias,
    int64_t T, int64_t d, int E, int64_t tpb, float* __restrict__ logits) {
  static_assert(RC_ROUND * EG == 64, "a round's token x expert sums fill one value per lane");
  __shared__ float part[2][RC_ROUND][NW][EG];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int e0 = blockIdx.y * EG;
  const bool cok = tid < d / 8;
  const int64_t col = cok ? 8 * (int64_t)tid : 0;
  float wv[8][EG];
  load_wr_rows<EG>(wr, col, cok, E, e0, wv);
  // the finishing thread of (token u, expert e) of a round: its bias, loaded before the loop
  const int fe = tid - (tid / EG) * EG;
  const float fb = (bias && tid < RC_ROUND * EG && e0 + fe < E) ? bias[e0 + fe] : 0.0f;
  const int64_t t0 = (int64_t)blockIdx.x * tpb;
  const int64_t t1 = t0 + tpb < T ? t0 + tpb : T;
  // Loads without branches or uses right behind them (token index clamped into range; an idle
  // lane's values are zeroed where they are used, a clamped token's results are never stored),
  // into two register buffers used in turn, so the next round's rows are in flight while a round
  // is summed and nothing waits for them before they are used.
  auto fetch = [&](u32x4 (&xb)[RC_ROUND], int64_t tb) {
#pragma unroll
    for (int u = 0; u < RC_ROUND; ++u) {
      const int64_t tt = tb + u < t1 ? tb + u : T - 1;
      xb[u] = *reinterpret_cast<const u32x4*>(x + tt * d + col);
    }
  };
  auto round = [&](const u32x4 (&xc)[RC_ROUND], u32x4 (&xnext)[RC_ROUND], int64_t tb, int buf) {
    fetch(xnext, tb + RC_ROUND);      // the next round (past the end: clamped, unused)
    __builtin_amdgcn_sched_barrier(0);  // issue those loads before this round's sums
    float v[RC_ROUND * EG];           // [token u][expert e]: this lane's 8 columns
#pragma unroll
    for (int u = 0; u < RC_ROUND; ++u) {
      float xf[8];
      unpack8(cok ? xc[u] : u32x4{0u, 0u, 0u, 0u}, xf);
#pragma unroll
      for (int e = 0; e < EG; ++e) v[u * EG + e] = 0.0f;
#pragma unroll
      for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int e = 0; e < EG; ++e) v[u * EG + e] = __builtin_fmaf(xf[c], wv[c][e], v[u * EG + e]);
    }
    // lane l: the wavefront's total for token l / EG, expert l % EG
    (&part[buf][0][0][0])[((lane / EG) * NW + w) * EG + lane % EG] = wave_transpose_sum64(v, lane);
    __syncthreads();
    if (tid < RC_ROUND * EG) {
      const int u = tid / EG;
      const int64_t t = tb + u;
      if (t < t1 && e0 + fe < E) {
        float s = part[buf][u][0][fe];
#pragma unroll
        for (int ww = 1; ww < NW; ++ww) s += part[buf][u][ww][fe];
        if (bias) s += fb;
        logits[t * E + e0 + fe] = s;
      }
    }
  };
  u32x4 xa[RC_ROUND], xb[RC_ROUND];
  fetch(xa, t0);
  // rounds in pairs, both always run (a round past the end stores nothing), so no branch sits
  // between a round's loads and the round that uses them
  for (int64_t tb = t0; tb < t1; tb += 2 * RC_ROUND) {
    round(xa, xb, tb, 0);
    round(xb, xa, tb + RC_ROUND, 1);
  }
}

constexpr int RW_WAVES = 8;     // dWr: wavefronts per workgroup, splitting the tokens
constexpr int RW_ROUND = 8;     // dWr: tokens per wavefront and round

// Partial dWr over token chunk blockIdx.y: part[c][i][e0 + e] = sum_{t in chunk c} x[t, i] *
// dl[t, e0 + e] for the 512 columns i of block blockIdx.x (8 per lane) and EG experts e0 =
// blockIdx.z * EG.  The RW_WAVES wavefronts take turns over the chunk's tokens (round r: wavefront
// w the RW_ROUND tokens from (r * RW_WAVES + w) * RW_ROUND), each token's dlogits read from LDS as
// broadcasts (staged one round ahead); then the wavefronts' sums are added pairwise through LDS
// in a fixed tree (w + 4 into w, w + 2 into w, 1 into 0) and wavefront 0 stores the partial row.
template <int EG>
__global__ __launch_bounds__(64 * RW_WAVES) void router_dwr_cols_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ dl, int64_t T, int64_t d, int E,
    int64_t chunk, float* __restrict__ part) {
  constexpr int RT = RW_WAVES * RW_ROUND;                 // tokens per round
  constexpr int DPT = RT * EG / (64 * RW_WAVES);          // staged dlogits per thread (1 or 2)
  __shared__ __attribute__((aligned(16))) float pool[4 * 16 * 64 * 4];   // 64 KiB
  float (*s_dl)[RT][EG] = reinterpret_cast<float (*)[RT][EG]>(pool);  // [2][RT][EG] while summing
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t col = (int64_t)blockIdx.x * 512 + 8 * lane;
  const bool cok = col < d;
  const int e0 = blockIdx.z * EG;
  const int64_t t0 = (int64_t)blockIdx.y * chunk;
  const int64_t t1 = t0 + chunk < T ? t0 + chunk : T;
  float acc[8][EG];
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int e = 0; e < EG; ++e) acc[c][e] = 0.0f;
  float dn[DPT];
  // Loads without branches or uses right behind them (indices clamped into range, values past
  // the end zeroed where they are used), into two register buffers used in turn: the next
  // round's dlogits and x are in flight while a round is summed, and storing the dlogits to LDS
  // at the end of the round waits for them only (they are issued first).
  const int64_t xcol = cok ? col : 0;
  auto fetch = [&](u32x4 (&xb)[RW_ROUND], int64_t tb) {   // this wavefront's tokens of a round
    const int64_t tw = tb + (int64_t)w * RW_ROUND;
#pragma unroll
    for (int u = 0; u < RW_ROUND; ++u) {
      const int64_t tt = tw + u < t1 ? tw + u : T - 1;
      xb[u] = *reinterpret_cast<const u32x4*>(x + tt * d + xcol);
    }
  };
  auto dl_ok = [&](int64_t tb, int q) {
    const int o = tid + 64 * RW_WAVES * q, u = o / EG, e = o - (o / EG) * EG;
    return tb + u < t1 && e0 + e < E;
  };
  auto fetch_dl = [&](int64_t tb) {   // the whole round's dlogits, one or two values per thread
#pragma unroll
    for (int q = 0; q < DPT; ++q) {
      const int o = tid + 64 * RW_WAVES * q, u = o / EG, e = o - (o / EG) * EG;
      const bool ok = dl_ok(tb, q);
      dn[q] = dl[(ok ? tb + u : T - 1) * E + (ok ? e0 + e : E - 1)];
    }
  };
  auto store_dl = [&](int64_t tb, int b) {
#pragma unroll
    for (int q = 0; q < DPT; ++q) (&s_dl[b][0][0])[tid + 64 * RW_WAVES * q] = dl_ok(tb, q) ? dn[q] : 0.0f;
  };
  auto round = [&](const u32x4 (&xc)[RW_ROUND], u32x4 (&xnext)[RW_ROUND], int64_t tb, int buf) {
    __syncthreads();                  // s_dl[buf] is complete; s_dl[buf ^ 1] is no longer read
    fetch_dl(tb + RT);                // the next round (past the end: clamped, stored as zeros)
    fetch(xnext, tb + RT);
    __builtin_amdgcn_sched_barrier(0);  // issue those loads before this round's sums
    const int64_t tw = tb + (int64_t)w * RW_ROUND;
#pragma unroll
    for (int u = 0; u < RW_ROUND; ++u) {
      float xf[8];
      unpack8((cok && tw + u < t1) ? xc[u] : u32x4{0u, 0u, 0u, 0u}, xf);
      const f32x4* g = reinterpret_cast<const f32x4*>(&s_dl[buf][w * RW_ROUND + u][0]);
#pragma unroll
      for (int q = 0; q < EG / 4; ++q) {
        const f32x4 gv = g[q];
#pragma unroll
        for (int c = 0; c < 8; ++c)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[c][4 * q + i] = __builtin_fmaf(xf[c], gv[i], acc[c][4 * q + i]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // the sums first, then wait for the staged dlogits
    store_dl(tb + RT, buf ^ 1);
  };
  u32x4 xa[RW_ROUND], xb[RW_ROUND];
  fetch_dl(t0);
  store_dl(t0, 0);
  fetch(xa, t0);
  // rounds in pairs, both always run (a round past the end adds zeros), so no branch sits
  // between a round's loads and the round that uses them
  for (int64_t tb = t0; tb < t1; tb += 2 * RT) {
    round(xa, xb, tb, 0);
    round(xb, xa, tb + RT, 1);
  }
  // wavefront sums added pairwise through LDS, 8 experts (64 values per lane) at a time
  f32x4* red = reinterpret_cast<f32x4*>(pool);        // [slot 0..3][16][64 lanes]
#pragma unroll
  for (int h = 0; h < EG / 8; ++h) {
#pragma unroll
    for (int step = RW_WAVES / 2; step >= 1; step >>= 1) {
      __syncthreads();
      if (w >= step && w < 2 * step) {
        f32x4* dst = red + (w - step) * 16 * 64 + lane;
#pragma unroll
        for (int c = 0; c < 8; ++c)
#pragma unroll
          for (int q = 0; q < 2; ++q)
            dst[(2 * c + q) * 64] = f32x4{acc[c][8 * h + 4 * q], acc[c][8 * h + 4 * q + 1], acc[c][8 * h + 4 * q + 2],
                                          acc[c][8 * h + 4 * q + 3]};
      }
      __syncthreads();
      if (w < step) {
        const f32x4* src = red + w * 16 * 64 + lane;
#pragma unroll
        for (int c = 0; c < 8; ++c)
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const f32x4 v = src[(2 * c + q) * 64];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[c][8 * h + 4 * q + i] += v[i];
          }
      }
    }
  }
  if (w == 0 && cok) {
    float* o = part + ((int64_t)blockIdx.y * d + col) * E + e0;
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
      for (int e = 0; e < EG; ++e)
        if (e0 + e < E) o[(int64_t)c * E + e] = acc[c][e];
  }
}

// dlogits with one lane per token (E <= EP): the same formula as router_dlogits_kernel, the
// softmax and the sums over experts taken in expert order inside the lane.
template <int EP>
__global__ __launch_bounds__(256) void router_dlogits_lanes_kernel(
    const float* __restrict__ logits, const int32_t* __restrict__ topk_idx,
    const float* __restrict__ topk_w, const float* __restrict__ d_topk_w,
    const int32_t* __restrict__ offsets, int64_t T, int E, int k, int normalize, float alpha,
    float* __restrict__ dlogits) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  const bool full = !normalize || alpha != 0.0f;
  float l[EP], q[EP], out[EP];
#pragma unroll
  for (int e = 0; e < EP; ++e) {
    l[e] = e < E ? logits[t * E + e] : -INFINITY;
    q[e] = 0.0f;
  }
  if (full) {
    float m = l[0];
#pragma unroll
    for (int e = 1; e < EP; ++e) m = fmaxf(m, l[e]);
    float z = 0.0f;
#pragma unroll
    for (int e = 0; e < EP; ++e) {
      q[e] = e < E ? expf(l[e] - m) : 0.0f;
      z += q[e];
    }
#pragma unroll
    for (int e = 0; e < EP; ++e) q[e] = q[e] / z;
  }
  float gw = 0.0f;
  for (int j = 0; j < k; ++j) gw += d_topk_w[t * k + j] * topk_w[t * k + j];
  const float aux = alpha * (float)E / (float)T;
  float f[EP];
  float fq = 0.0f;
#pragma unroll
  for (int e = 0; e < EP; ++e) {
    f[e] = (alpha != 0.0f && e < E) ? (float)(offsets[e + 1] - offsets[e]) / (float)(T * k) : 0.0f;
    fq += f[e] * q[e];
  }
#pragma unroll
  for (int e = 0; e < EP; ++e) {
    out[e] = normalize ? 0.0f : -q[e] * gw;
    if (alpha != 0.0f) out[e] += aux * q[e] * (f[e] - fq);
  }
  for (int j = 0; j < k; ++j) {
    const int s = topk_idx[t * k + j];
    const float g = d_topk_w[t * k + j], wj = topk_w[t * k + j];
#pragma unroll
    for (int e = 0; e < EP; ++e)
      if (e == s) out[e] += normalize ? wj * (g - gw) : q[e] * g;
  }
#pragma unroll
  for (int e = 0; e < EP; ++e)
    if (e < E) dlogits[t * E + e] = out[e];
}

// Load-balancing loss, first stage with one lane per token (E <= EP): the workgroup's 256 full
// softmax rows summed per expert (wave_reduce_scatter, then the four wavefronts in order) into
// one row of partials.
template <int EP>
__global__ __launch_bounds__(256) void router_aux_lanes_kernel(const float* __restrict__ logits, int64_t T,
                                                               int E, float* __restrict__ part) {
  constexpr int G = 64 / EP;
  __shared__ float s_acc[4][EP];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  float q[EP];
#pragma unroll
  for (int e = 0; e < EP; ++e) q[e] = 0.0f;
  if (t < T) {
    float l[EP];
#pragma unroll
    for (int e = 0; e < EP; ++e) l[e] = e < E ? logits[t * E + e] : -INFINITY;
    float m = l[0];
#pragma unroll
    for (int e = 1; e < EP; ++e) m = fmaxf(m, l[e]);
    float z = 0.0f;
#pragma unroll
    for (int e = 0; e < EP; ++e) {
      q[e] = e < E ? expf(l[e] - m) : 0.0f;
      z += q[e];
    }
#pragma unroll
    for (int e = 0; e < EP; ++e) q[e] = q[e] / z;
  }
  const float s = wave_reduce_scatter<EP>(q, lane);
  if ((lane & (G - 1)) == 0) s_acc[w][lane / G] = s;
  __syncthreads();
  if (threadIdx.x < E)
    part[(int64_t)blockIdx.x * E + threadIdx.x] =
        ((s_acc[0][threadIdx.x] + s_acc[1][threadIdx.x]) + s_acc[2][threadIdx.x]) + s_acc[3][threadIdx.x];
}

// dX[t] = bf16(bf16(sum_j src[row_of_slot[t*k + j]] + add[t]) + sum_e dl[t, e] * wr[:, e]): the
// experts' unpermute-sum rounded to bf16 exactly as combine_kernel stores it (w = 1, the rows in
// slot order, then add), then the router's share (a fused multiply-add chain over e in expert
// order from 0) added and rounded again, which is what router_dx_kernel does to a stored dX.  K =
// k at compile time, K < 0 for any k at run time, K = 0 for no source rows (then add is the stored
// dX and may alias out).  One lane per 8 columns (the NW wavefronts cover 512 * NW columns), the
// lane's rows of Wr in registers; tokens in rounds (DxRound) whose dlogits are staged in LDS and
// whose rows are loaded one round ahead.
// Tokens per round: about 8 (EG = 8) or 4 (EG = 16) rows of 16 bytes in flight per lane.
template <int EG, int K>
struct DxRound {
  static constexpr int rows = K > 0 ? K : 2;
  static constexpr int v = (EG == 8 ? 8 : 4) / rows > 0 ? (EG == 8 ? 8 : 4) / rows : 1;
};
template <int EG, int K, bool A, int NW>
__global__ __launch_bounds__(64 * NW) void router_dx_rows_kernel(
    const uint16_t* __restrict__ src, const int32_t* __restrict__ row_of_slot, const uint16_t* add,
    const float* __restrict__ dl, const float* __restrict__ wr, int64_t T, int64_t d, int k, int E,
    int64_t tpb, uint16_t* out) {
  static_assert(K != 0 || A, "without source rows the stored dX comes in as add");
  constexpr int RX_ROUND = DxRound<EG, K>::v;
  constexpr int KR = K > 0 ? K : 1;     // rows loaded ahead per token (run-time k: the first)
  __shared__ __attribute__((aligned(16))) float s_dl[2][RX_ROUND][EG];
  const int tid = threadIdx.x;
  const bool cok = tid < d / 8;
  const int64_t col = cok ? 8 * (int64_t)tid : 0;
  float wv[8][EG];
  load_wr_rows<EG>(wr, col, cok, E, 0, wv);
  const int64_t t0 = (int64_t)blockIdx.x * tpb;
  const int64_t t1 = t0 + tpb < T ? t0 + tpb : T;
  float dn = 0.0f;
  // Loads without branches or uses right behind them (token index clamped into range: a clamped
  // token's results are never stored; an idle lane stores nothing), into two register buffers
  // used in turn, so the next round's rows are in flight while a round is summed.
  struct Rows {
    u32x4 r[RX_ROUND][KR];
    u32x4 a[RX_ROUND];
  };
  auto fetch = [&](Rows& b, int64_t tb) {   // the round's rows (and added rows) for this lane's columns
#pragma unroll
    for (int u = 0; u < RX_ROUND; ++u) {
      const int64_t tt = tb + u < t1 ? tb + u : T - 1;
      if constexpr (K != 0) {
#pragma unroll
        for (int j = 0; j < KR; ++j) {   // the slot index is the same in every lane: a scalar load
          const int64_t r = row_of_slot[__builtin_amdgcn_readfirstlane((int)(tt * k + j))];
          b.r[u][j] = ld_stream(reinterpret_cast<const u32x4*>(src + r * d + col));
        }
      }
      if constexpr (A) b.a[u] = ld_stream(reinterpret_cast<const u32x4*>(add + tt * d + col));
    }
  };
  auto dl_ok = [&](int64_t tb) {
    const int u = tid / EG, e = tid - (tid / EG) * EG;
    return tid < RX_ROUND * EG && tb + u < t1 && e < E;
  };
  auto fetch_dl = [&](int64_t tb) {     // one value of the round's dlogits per staging thread
    const int u = tid / EG, e = tid - (tid / EG) * EG;
    const bool ok = dl_ok(tb);
    dn = dl[(ok ? tb + u : T - 1) * E + (ok ? e : E - 1)];
  };
  auto store_dl = [&](int64_t tb, int b) {
    if (tid < RX_ROUND * EG) (&s_dl[b][0][0])[tid] = dl_ok(tb) ? dn : 0.0f;
  };
  auto round = [&](const Rows& cur, Rows& nxt, int64_t tb, int buf) {
    __syncthreads();                  // s_dl[buf] is complete; s_dl[buf ^ 1] is no longer read
    fetch_dl(tb + RX_ROUND);          // the next round (past the end: clamped, staged as zeros)
    fetch(nxt, tb + RX_ROUND);
    __builtin_amdgcn_sched_barrier(0);  // issue those loads before this round's sums
#pragma unroll
    for (int u = 0; u < RX_ROUND; ++u) {
      const int64_t t = tb + u;
      if (t >= t1) break;
      float base[8];
      if constexpr (K == 0) {
        unpack8(cur.a[u], base);        // the stored dX itself
      } else {
        float acc[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
#pragma unroll
        for (int j = 0; j < KR; ++j) {
          float f[8];
          unpack8(cur.r[u][j], f);
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[i] += f[i];
        }
        if constexpr (K < 0) {
          for (int j = 1; j < k; ++j) {
            const int64_t r = row_of_slot[t * k + j];
            float f[8];
            unpack8(ld_stream(reinterpret_cast<const u32x4*>(src + r * d + col)), f);
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] += f[i];
          }
        }
        if constexpr (A) {
          float f[8];
          unpack8(cur.a[u], f);
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[i] += f[i];
        }
        unpack8(pack8(acc), base);      // the experts' dX as stored in bf16
      }
      float sh[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) sh[i] = 0.0f;
      const f32x4* g = reinterpret_cast<const f32x4*>(&s_dl[buf][u][0]);
#pragma unroll
      for (int q = 0; q < EG / 4; ++q) {
        const f32x4 gv = g[q];
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          if (4 * q + c4 < E) {
#pragma unroll
            for (int i = 0; i < 8; ++i) sh[i] = __builtin_fmaf(gv[c4], wv[i][4 * q + c4], sh[i]);
          }
        }
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) base[i] += sh[i];
      if (cok) *reinterpret_cast<u32x4*>(out + t * d + col) = pack8(base);
    }
    __builtin_amdgcn_sched_barrier(0);  // the sums first, then wait for the staged dlogits
    store_dl(tb + RX_ROUND, buf ^ 1);
  };
  Rows ra, rb;
  fetch_dl(t0);
  store_dl(t0, 0);
  fetch(ra, t0);
  // rounds in pairs, both always run (a round past the end stores nothing), so no branch sits
  // between a round's loads and the round that uses them
  for (int64_t tb = t0; tb < t1; tb += 2 * RX_ROUND) {
    round(ra, rb, tb, 0);
    round(rb, ra, tb + RX_ROUND, 1);
  }
}

int64_t dwr_chunks(int64_t T) {
  int64_t c = (T + 255) / 256;
  return c < 1 ? 1 : (c > 64 ? 64 : c);
}

// Tokens per workgroup of the column-parallel kernels: about T/256 (one workgroup per compute
// unit), a multiple of the round size.
int64_t cols_tokens_per_block(int64_t T, int round) {
  const int64_t t = (T + 255) / 256;
  return (t + round - 1) / round * round;
}

// The column-parallel forms serve d <= 4096: with any E for logits and dWr (8 experts per pass),
// with E <= 16 for dX (all experts' rows of Wr in registers); the lane-per-token forms E <= 16.
bool cols_ok(int64_t d) { return d <= 4096; }

template <int EG, bool A>
void launch_dx_rows_a(int K, const uint16_t* src, const int32_t* ros, const uint16_t* add, const float* dl,
                      const float* wr, int64_t T, int64_t d, int k, int E, uint16_t* out, hipStream_t stream) {
  const int64_t tpb = cols_tokens_per_block(T, 8);   // a multiple of every round size
  const unsigned grid = (unsigned)((T + tpb - 1) / tpb);
  switch (K) {
    case 1: router_dx_rows_kernel<EG, 1, A, 8><<<grid, 512, 0, stream>>>(src, ros, add, dl, wr, T, d, k, E, tpb, out); break;
    case 2: router_dx_rows_kernel<EG, 2, A, 8><<<grid, 512, 0, stream>>>(src, ros, add, dl, wr, T, d, k, E, tpb, out); break;
    case 4: router_dx_rows_kernel<EG, 4, A, 8><<<grid, 512, 0, stream>>>(src, ros, add, dl, wr, T, d, k, E, tpb, out); break;
    case 8: router_dx_rows_kernel<EG, 8, A, 8><<<grid, 512, 0, stream>>>(src, ros, add, dl, wr, T, d, k, E, tpb, out); break;
    default: router_dx_rows_kernel<EG, -1, A, 8><<<grid, 512, 0, stream>>>(src, ros, add, dl, wr, T, d, k, E, tpb, out); break;
  }
}

// K = 0: dx (given as add, also the output) += the router's share; otherwise the fused unpermute.
template <int EG>
void launch_dx_rows(int K, const uint16_t* src, const int32_t* ros, const uint16_t* add, const float* dl,
                    const float* wr, int64_t T, int64_t d, int k, int E, uint16_t* out, hipStream_t stream) {
  if (K == 0) {
    const int64_t tpb = cols_tokens_per_block(T, 8);
    router_dx_rows_kernel<EG, 0, true, 8><<<(unsigned)((T + tpb - 1) / tpb), 512, 0, stream>>>(
        src, ros, add, dl, wr, T, d, k, E, tpb, out);
  } else if (add) {
    launch_dx_rows_a<EG, true>(K, src, ros, add, dl, wr, T, d, k, E, out, stream);
  } else {
    launch_dx_rows_a<EG, false>(K, src, ros, add, dl, wr, T, d, k, E, out, stream);
  }
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status moe_router_logits(const moe_bf16* x, const float* wr, const float* bias, int64_t T,
                                        int64_t d, int32_t E, float* logits, hipStream_t stream) {
  if (T < 0 || d <= 0 || E < 1 || E > 256) return fail(MOE_ERROR_INVALID_VALUE, "moe_router_logits: bad size");
  if (d % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_router_logits: d must be a multiple of 64");
  if (T == 0) return MOE_SUCCESS;
  if (!x || !wr || !logits) return fail(MOE_ERROR_INVALID_VALUE, "moe_router_logits: NULL pointer");
  if (!aligned16(x)) return fail(MOE_ERROR_INVALID_VALUE, "moe_router_logits: x must be 16-byte aligned");
  if (T > ((int64_t)1 << 31) / 64) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_router_logits: T too large");
  if (cols_ok(d)) {
    // 8 experts per pass (grid.y passes over x for larger E)
    const int64_t tpb = cols_tokens_per_block(T, RC_ROUND);
    const dim3 grid((unsigned)((T + tpb - 1) / tpb), (unsigned)((E + 7) / 8));
    if (d <= 2048) router_logits_cols_kernel<8, 4><<<grid, 256, 0, stream>>>(x, wr, bias, T, d, E, tpb, logits);
    else router_logits_cols_kernel<8, 8><<<grid, 512, 0, stream>>>(x, wr, bias, T, d, E, tpb, logits);
    return check_launch("router_logits_cols");
  }
  const unsigned gx = (unsigned)((T + 127) / 128);
  if (E <= 8) router_logits_kernel<8><<<dim3(gx, 1), 64 * RL_WAVES, 0, stream>>>(x, wr, bias, T, d, E, logits);
  else if (E <= 16) router_logits_kernel<16><<<dim3(gx, 1), 64 * RL_WAVES, 0, stream>>>(x, wr, bias, T, d, E, logits);
  else router_logits_kernel<32><<<dim3(gx, (unsigned)((E + 31) / 32)), 64 * RL_WAVES, 0, stream>>>(x, wr, bias, T, d, E, logits);
  return check_launch("router_logits");
}

extern "C" size_t moe_router_bwd_workspace_bytes(int64_t T, int64_t d, int32_t E) {
  if (T <= 0 || d <= 0 || E <= 0) return 0;
  return (size_t)((dwr_chunks(T) + 1) * d * E * (int64_t)sizeof(float));   // dWr partials, then Wr^T
}

extern "C" moe_status moe_router_bwd(const moe_bf16* x, const float* wr, const float* logits,
                                     const int32_t* topk_idx, const float* topk_w, const float* d_topk_w,
                                     const int32_t* offsets, int64_t T, int64_t d, int32_t E, int32_t k,
                                     int32_t normalize_topk, float aux_alpha, void* workspace,
                                     size_t workspace_bytes, float* dlogits, float* dwr, moe_bf16* dx,
                                     hipStream_t stream) {
  const char* fn = "moe_router_bwd";
  if (T < 0 || d <= 0 || E < 1 || E > 256 || k < 1 || k > E) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (d % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: d must be a multiple of 64", fn);
  if (T == 0) return MOE_SUCCESS;
  if (!x || !wr || !logits || !topk_idx || !topk_w || !d_topk_w || !dlogits || !dwr)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (aux_alpha != 0.0f && !offsets) return fail(MOE_ERROR_INVALID_VALUE, "%s: the auxiliary loss needs offsets", fn);
  if (!aligned16(x) || (dx && !aligned16(dx))) return fail(MOE_ERROR_INVALID_VALUE, "%s: x and dx must be 16-byte aligned", fn);
  if (T > ((int64_t)1 << 31) / 64) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: T too large", fn);
  const size_t need = moe_router_bwd_workspace_bytes(T, d, E);
  if (!workspace || workspace_bytes < need)
    return fail(MOE_ERROR_WORKSPACE, "%s: workspace of %zu bytes needed", fn, need);
  moe_status st;
  if (E <= 16) {
    const unsigned g = (unsigned)((T + 255) / 256);
    if (E <= 8)
      router_dlogits_lanes_kernel<8><<<g, 256, 0, stream>>>(logits, topk_idx, topk_w, d_topk_w, offsets, T, E, k,
                                                           normalize_topk, aux_alpha, dlogits);
    else
      router_dlogits_lanes_kernel<16><<<g, 256, 0, stream>>>(logits, topk_idx, topk_w, d_topk_w, offsets, T, E, k,
                                                            normalize_topk, aux_alpha, dlogits);
    if ((st = check_launch("router_dlogits_lanes")) != MOE_SUCCESS) return st;
  } else {
    const int64_t waves = (T + RD_TPW - 1) / RD_TPW;
    router_dlogits_kernel<<<(unsigned)((waves + 3) / 4), 256, 0, stream>>>(
        logits, topk_idx, topk_w, d_topk_w, offsets, T, E, k, normalize_topk, aux_alpha, dlogits);
    if ((st = check_launch("router_dlogits")) != MOE_SUCCESS) return st;
  }
  const int64_t chunks = dwr_chunks(T);
  const int64_t chunk = (T + chunks - 1) / chunks;
  float* part = static_cast<float*>(workspace);
  if (cols_ok(d)) {
    const dim3 grid((unsigned)((d + 511) / 512), (unsigned)chunks, (unsigned)((E + 7) / 8));   // 8 experts per pass
    router_dwr_cols_kernel<8><<<grid, 64 * RW_WAVES, 0, stream>>>(x, dlogits, T, d, E, chunk, part);
    if ((st = check_launch("router_dwr_cols")) != MOE_SUCCESS) return st;
  } else {
    router_dwr_partial_kernel<<<dim3((unsigned)((d + 127) / 128), (unsigned)chunks, (unsigned)((E + RB_EC - 1) / RB_EC)),
                                64, 0, stream>>>(x, dlogits, T, d, E, chunk, part);
    if ((st = check_launch("router_dwr_partial")) != MOE_SUCCESS) return st;
  }
  const int64_t n = d * E;
  router_dwr_reduce_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(part, (int)chunks, n, dwr);
  if ((st = check_launch("router_dwr_reduce")) != MOE_SUCCESS) return st;
  if (dx) {
    if (E <= 16 && cols_ok(d)) {
      // in place: each lane reads its 8 columns of a token's stored dX, then overwrites them
      if (E <= 8) launch_dx_rows<8>(0, nullptr, nullptr, dx, dlogits, wr, T, d, 0, E, dx, stream);
      else launch_dx_rows<16>(0, nullptr, nullptr, dx, dlogits, wr, T, d, 0, E, dx, stream);
      return check_launch("router_dx_rows");
    }
    float* wrt = part + chunks * n;
    router_transpose_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(wr, d, E, wrt);
    if ((st = check_launch("router_transpose")) != MOE_SUCCESS) return st;
    router_dx_kernel<<<dim3((unsigned)((d + 127) / 128), (unsigned)((T + RB_TOK - 1) / RB_TOK)), 64, 0, stream>>>(
        dlogits, wrt, T, d, E, dx);
    if ((st = check_launch("router_dx")) != MOE_SUCCESS) return st;
  }
  return MOE_SUCCESS;
}

extern "C" moe_status moe_unpermute_router_dx(const moe_bf16* dx_perm, const int32_t* row_of_slot,
                                              const moe_bf16* add, const float* dlogits, const float* wr,
                                              int64_t T, int64_t d, int32_t k, int32_t E, moe_bf16* dx,
                                              hipStream_t stream) {
  const char* fn = "moe_unpermute_router_dx";
  if (T < 0 || d < 0 || k < 1 || k > 256 || E < 1) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (d % 64 != 0) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: d must be a multiple of 64", fn);
  if (E > 16 || !cols_ok(d)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: needs E <= 16 and d <= 4096", fn);
  if (T * (int64_t)k >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: T*k must fit in int32", fn);
  if (T == 0 || d == 0) return MOE_SUCCESS;
  if (!dx_perm || !row_of_slot || !dlogits || !wr || !dx) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (!aligned16(dx_perm) || !aligned16(dx) || (add && !aligned16(add)))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: dx_perm, add and dx must be 16-byte aligned", fn);
  const int K = (k == 1 || k == 2 || k == 4 || k == 8) ? k : -1;
  if (E <= 8) launch_dx_rows<8>(K, dx_perm, row_of_slot, add, dlogits, wr, T, d, k, E, dx, stream);
  else launch_dx_rows<16>(K, dx_perm, row_of_slot, add, dlogits, wr, T, d, k, E, dx, stream);
  return check_launch("router_dx_rows");
}

extern "C" size_t moe_router_aux_loss_workspace_bytes(int64_t T, int32_t E) {
  if (T <= 0 || E <= 0) return 0;
  const int64_t waves = (T + RA_TPW - 1) / RA_TPW;
  return (size_t)((waves + 3) / 4) * (size_t)E * sizeof(float);
}

extern "C" moe_status moe_router_aux_loss(const float* logits, const int32_t* offsets, int64_t T, int32_t E,
                                          int32_t k, float alpha, void* workspace, size_t workspace_bytes,
                                          float* loss, hipStream_t stream) {
  const char* fn = "moe_router_aux_loss";
  if (T <= 0 || E < 1 || E > 256 || k < 1 || k > E) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (!logits || !offsets || !loss) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  const size_t need = moe_router_aux_loss_workspace_bytes(T, E);
  if (!workspace || workspace_bytes < need)
    return fail(MOE_ERROR_WORKSPACE, "%s: workspace of %zu bytes needed", fn, need);
  float* part = static_cast<float*>(workspace);
  int64_t nblk;
  moe_status st;
  if (E <= 16) {                      // one lane per token: 256 tokens per partial row
    nblk = (T + 255) / 256;
    if (nblk > ((int64_t)1 << 30)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: T too large", fn);
    if (E <= 8) router_aux_lanes_kernel<8><<<(unsigned)nblk, 256, 0, stream>>>(logits, T, E, part);
    else router_aux_lanes_kernel<16><<<(unsigned)nblk, 256, 0, stream>>>(logits, T, E, part);
    if ((st = check_launch("router_aux_lanes")) != MOE_SUCCESS) return st;
  } else {
    const int64_t waves = (T + RA_TPW - 1) / RA_TPW;
    nblk = (waves + 3) / 4;
    if (nblk > ((int64_t)1 << 30)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: T too large", fn);
    router_aux_partial_kernel<<<(unsigned)nblk, 256, 0, stream>>>(logits, T, E, part);
    if ((st = check_launch("router_aux_partial")) != MOE_SUCCESS) return st;
  }
  router_aux_final_kernel<<<1, 256, 0, stream>>>(part, (int)nblk, offsets, T, E, k, alpha, loss);
  return check_launch("router_aux_final");
}
