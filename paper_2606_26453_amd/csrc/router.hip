// Router of the MoE layer on the GPU: logits = x . Wr (+ bias), the backward through the routing
// weights (d_topk_w -> dlogits, plus an optional Switch-style load-balancing loss), and the
// router map's backward (dWr = x^T . dlogits, dX += dlogits . Wr^T).
//
// The contractions are tiny (E <= 256 experts) and their fp32 operands must stay fp32, so these
// are vector-ALU kernels, not MFMA: one lane per token (logits) or per pair of hidden columns
// (dX, dWr).  The operand that is the same for the whole wavefront (rows of Wr, a block of
// tokens' dlogits) is staged in LDS and read as broadcasts (every lane the same address, 16
// bytes per read for 8 fused multiply-adds per lane).
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
  for (int c = 1; c < nchunk; ++c) s += part[(int64_t)c * n + o];
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

int64_t dwr_chunks(int64_t T) {
  int64_t c = (T + 255) / 256;
  return c < 1 ? 1 : (c > 64 ? 64 : c);
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
  const int64_t waves = (T + RD_TPW - 1) / RD_TPW;
  router_dlogits_kernel<<<(unsigned)((waves + 3) / 4), 256, 0, stream>>>(
      logits, topk_idx, topk_w, d_topk_w, offsets, T, E, k, normalize_topk, aux_alpha, dlogits);
  moe_status st = check_launch("router_dlogits");
  if (st != MOE_SUCCESS) return st;
  const int64_t chunks = dwr_chunks(T);
  const int64_t chunk = (T + chunks - 1) / chunks;
  float* part = static_cast<float*>(workspace);
  router_dwr_partial_kernel<<<dim3((unsigned)((d + 127) / 128), (unsigned)chunks, (unsigned)((E + RB_EC - 1) / RB_EC)),
                              64, 0, stream>>>(x, dlogits, T, d, E, chunk, part);
  if ((st = check_launch("router_dwr_partial")) != MOE_SUCCESS) return st;
  const int64_t n = d * E;
  router_dwr_reduce_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(part, (int)chunks, n, dwr);
  if ((st = check_launch("router_dwr_reduce")) != MOE_SUCCESS) return st;
  if (dx) {
    float* wrt = part + chunks * n;
    router_transpose_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(wr, d, E, wrt);
    if ((st = check_launch("router_transpose")) != MOE_SUCCESS) return st;
    router_dx_kernel<<<dim3((unsigned)((d + 127) / 128), (unsigned)((T + RB_TOK - 1) / RB_TOK)), 64, 0, stream>>>(
        dlogits, wrt, T, d, E, dx);
    if ((st = check_launch("router_dx")) != MOE_SUCCESS) return st;
  }
  return MOE_SUCCESS;
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
  const int64_t waves = (T + RA_TPW - 1) / RA_TPW;
  const int64_t nblk = (waves + 3) / 4;
  if (nblk > ((int64_t)1 << 30)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: T too large", fn);
  float* part = static_cast<float*>(workspace);
  router_aux_partial_kernel<<<(unsigned)nblk, 256, 0, stream>>>(logits, T, E, part);
  moe_status st = check_launch("router_aux_partial");
  if (st != MOE_SUCCESS) return st;
  router_aux_final_kernel<<<1, 256, 0, stream>>>(part, (int)nblk, offsets, T, E, k, alpha, loss);
  return check_launch("router_aux_final");
}
