// Grouped GEMMs over ragged expert row groups on gfx950 bf16 MFMA (fp32 accumulation).
//
// One kernel template serves the three products of the layer:
//   FWD  C[r, n]      = sum_c A[r, c]  * B[g][c, n]      rows r of group g (ragged), c < K
//   DX   dA[r, kk]    = sum_c dC[r, c] * B[g][kk, c]     rows r of group g (ragged), c < N (or 2N)
//   DW   dB[g][m, n]  = sum_r A[r, m]  * dC[r, n]        r over group g (ragged contraction)
// DW is the paper's dW1_e = X_e^T G_e (section 5.4, Appendix H).
//
// Work decomposition.  A 256-thread workgroup (4 wavefronts in a 2x2 grid) owns a BM x BN output
// tile and walks the contraction in steps of BK = 64.  Both operand tiles are staged in LDS in
// one layout, [row][64 contraction elements] with the contraction contiguous, which is what a
// lane of v_mfma_f32_32x32x16_bf16 consumes (8 consecutive contraction elements of one row, one
// ds_read_b128).  An operand whose contraction index is its memory row (B in FWD, both operands
// in DW) is loaded as 8x8 bf16 blocks (eight 16-byte row segments per thread, coalesced along
// the memory row) and transposed in registers before the LDS store; the other operands are
// copied 16 bytes per thread.  16-byte LDS chunks are XOR-swizzled by row so that both the
// MFMA reads (8 consecutive rows, same chunk) and the transposed stores (rows 8 apart, same
// chunk) hit distinct banks.  LDS is double buffered: global loads for step s+1 are in flight
// while step s runs on the matrix cores, with one barrier per step.
//
// MFMA operand roles: the N-side operand is the MFMA "A" (32 MFMA rows = 32 output columns) and
// the M-side operand the MFMA "B", so each lane's accumulator holds one output row and runs of
// 4 consecutive output columns, stored as 8-byte (bf16) or 16-byte (fp32) vectors.
//
// Dual mode (FWD gate/up, DW gate/up): the N side of a tile is split into two halves fed from two
// sources at the same output columns; each wave's 128 N-columns are 64 from each source, so the
// accumulators for the same (row, column) of both products sit in the same lane, which is what
// the fused SwiGLU epilogue needs.  DX dual mode appends the second pair to the contraction.
#include "common.h"

namespace moe {
namespace {

constexpr int NT = 256;
constexpr int BK = 64;

enum { KIND_FWD = 0, KIND_DX = 1, KIND_DW = 2 };

struct GemmParams {
  const uint16_t* a;   // M side: FWD A [R,K]; DX dC [R,N]; DW A [R,K]
  const uint16_t* a2;  // DX: dC2
  const uint16_t* b;   // N side: FWD B [G,K,N]; DX B [G,K,N]; DW dC [R,N]
  const uint16_t* b2;  // FWD B2; DX B2; DW dC2
  const int32_t* offsets;
  void* out;           // FWD C; DX dA; DW dB
  void* out2;          // FWD C2; DW dB2
  uint16_t* act;       // FWD SwiGLU output
  int G;
  int64_t R, K, N;
  int mt_bound;        // FWD/DX: upper bound on the number of row tiles (grid extent)
  int m_tiles;         // DW: tiles over K
  int n_tiles;         // tiles over the output columns
};

// LDS element offset of (row, 16-byte chunk) in a [rows][64] bf16 tile.
__device__ __forceinline__ int lds_off(int row, int ch) {
  return row * BK + ((ch ^ (row & 7) ^ ((row >> 3) & 7)) << 3);
}

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// 8x8 bf16 transpose: in[i] holds 8 elements of row i; out[j] gets element j of rows 0..7.
__device__ __forceinline__ void transpose8x8(const u32x4* in, u32x4* out) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t x = in[2 * p][j >> 1];
      const uint32_t y = in[2 * p + 1][j >> 1];
      out[j][p] = (j & 1) ? ((x >> 16) | (y & 0xffff0000u)) : ((x & 0xffffu) | (y << 16));
    }
  }
}

template <int KIND, int BM, int BN, bool DUAL, bool ACT>
__global__ __launch_bounds__(NT, 1) void grouped_gemm_kernel(GemmParams p) {
  constexpr int WM = BM / 2, WN = BN / 2;     // per-wave tile
  constexpr int MB = WM / 32, NB = WN / 32;   // 32x32 MFMA blocks per wave
  constexpr bool M_T = (KIND == KIND_DW);     // M-side operand stored contraction-major
  constexpr bool N_T = (KIND != KIND_DX);     // N-side operand stored contraction-major
  static_assert(BM % 64 == 0 && BN % 64 == 0 && BM <= 256 && BN <= 256, "tile");

  __shared__ __attribute__((aligned(16))) uint16_t lds[2][(BM + BN) * BK];
  __shared__ int s_scan[256];
  __shared__ int s_tile[2];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // ---------------- tile -> (group, row range, column range, contraction range) ------------
  int g, mt, nt;
  int64_t row_lo = 0, row_hi = 0;    // FWD/DX: output rows; DW: contraction rows
  if constexpr (KIND == KIND_DW) {
    const int per_g = p.m_tiles * p.n_tiles;
    g = blockIdx.x / per_g;
    const int rem = blockIdx.x - g * per_g;
    mt = rem % p.m_tiles;
    nt = rem / p.m_tiles;
    row_lo = p.offsets[g];
    row_hi = p.offsets[g + 1];
  } else {
    const int mt_glob = blockIdx.x % p.mt_bound;
    nt = blockIdx.x / p.mt_bound;
    // inclusive scan of per-group row-tile counts (G <= 256)
    int cnt = 0;
    if (tid < p.G) {
      const int lo = p.offsets[tid], hi = p.offsets[tid + 1];
      cnt = (hi - lo + BM - 1) / BM;
    }
    s_scan[tid] = cnt;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
      const int add = tid >= off ? s_scan[tid - off] : 0;
      __syncthreads();
      s_scan[tid] += add;
      __syncthreads();
    }
    const int total = s_scan[255];
    if (mt_glob >= total) return;  // uniform over the workgroup
    const int ng = __syncthreads_count(tid < p.G && s_scan[tid] <= mt_glob);
    g = ng;
    mt = mt_glob - (g > 0 ? s_scan[g - 1] : 0);
    row_lo = (int64_t)p.offsets[g] + (int64_t)mt * BM;
    row_hi = p.offsets[g + 1];
  }

  // ---------------- per-thread load descriptors ----------------------------------------------
  // M side
  constexpr int M_DIRECT_LOADS = BM / 32;     // direct: 16-byte chunks per thread
  int64_t m_off[M_T ? 1 : M_DIRECT_LOADS];    // element offset of each loaded row
  const uint16_t* mt_ptr = nullptr;           // transposed: column base
  bool mt_live = false;
  int m_kb = 0, m_mb = 0;
  if constexpr (!M_T) {
    const int64_t ld = (KIND == KIND_FWD) ? p.K : p.N;
#pragma unroll
    for (int i = 0; i < M_DIRECT_LOADS; ++i) {
      int64_t r = row_lo + tid / 8 + 32 * i;
      if (r > row_hi - 1) r = row_hi - 1;
      m_off[i] = r * ld + 8 * (tid & 7);
    }
  } else {
    // DW: A[r, m], columns m in [mt*BM, mt*BM+BM)
    mt_live = tid < BM;
    m_mb = tid % (BM / 8);
    m_kb = tid / (BM / 8);
    int64_t col = (int64_t)mt * BM + 8 * m_mb;
    if (col > p.K - 8) col = p.K - 8;
    mt_ptr = p.a + col;
  }
  // N side
  constexpr int N_DIRECT_LOADS = BN / 32;
  int64_t n_off[N_T ? 1 : N_DIRECT_LOADS];
  const uint16_t* nt_ptr = nullptr;
  bool nt_live = false;
  int n_kb = 0, n_mb = 0;
  if constexpr (!N_T) {
    // DX: B[g][kk, c], kk = output column
#pragma unroll
    for (int i = 0; i < N_DIRECT_LOADS; ++i) {
      int64_t kk = (int64_t)nt * BN + tid / 8 + 32 * i;
      if (kk > p.K - 1) kk = p.K - 1;
      n_off[i] = (int64_t)g * p.K * p.N + kk * p.N + 8 * (tid & 7);
    }
  } else {
    nt_live = tid < BN;
    n_mb = tid % (BN / 8);
    n_kb = tid / (BN / 8);
    const int v0 = 8 * n_mb;  // virtual column of this thread's block
    const int64_t ncols = (KIND == KIND_FWD) ? p.N : p.N;
    int64_t col;
    const uint16_t* src = p.b;
    if constexpr (DUAL) {
      const int w = v0 / WN, u = v0 % WN;
      col = (int64_t)nt * (BN / 2) + w * (WN / 2) + (u % (WN / 2));
      if (u >= WN / 2) src = p.b2;
    } else {
      col = (int64_t)nt * BN + v0;
    }
    if (col > ncols - 8) col = ncols - 8;
    nt_ptr = src + col + ((KIND == KIND_FWD) ? (int64_t)g * p.K * p.N : 0);
  }

  // contraction extent
  int64_t c_len;
  if constexpr (KIND == KIND_FWD) c_len = p.K;
  else if constexpr (KIND == KIND_DX) c_len = DUAL ? 2 * p.N : p.N;
  else c_len = row_hi - row_lo;
  const int nsteps = (int)((c_len + BK - 1) / BK);

  // ---------------- global -> register loads for one k-step ----------------------------------
  u32x4 mreg[M_T ? 8 : M_DIRECT_LOADS];
  u32x4 nreg[N_T ? 8 : N_DIRECT_LOADS];

  auto load_step = [&](int s) {
    const int64_t c0 = (int64_t)s * BK;
    if constexpr (!M_T) {
      const uint16_t* base = p.a;
      int64_t cc = c0;
      if constexpr (KIND == KIND_DX && DUAL) {
        if (c0 >= p.N) { base = p.a2; cc = c0 - p.N; }
      }
#pragma unroll
      for (int i = 0; i < M_DIRECT_LOADS; ++i) mreg[i] = ld16(base + m_off[i] + cc);
    } else {
      if (mt_live) {
        const int64_t r0 = row_lo + c0 + 8 * m_kb;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int64_t r = r0 + i;
          mreg[i] = (r < row_hi) ? ld16(mt_ptr + r * p.K) : u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
    if constexpr (!N_T) {
      const uint16_t* base = p.b;
      int64_t cc = c0;
      if constexpr (DUAL) {
        if (c0 >= p.N) { base = p.b2; cc = c0 - p.N; }
      }
#pragma unroll
      for (int i = 0; i < N_DIRECT_LOADS; ++i) nreg[i] = ld16(base + n_off[i] + cc);
    } else {
      if (nt_live) {
        if constexpr (KIND == KIND_FWD) {
          const int64_t r0 = c0 + 8 * n_kb;
#pragma unroll
          for (int i = 0; i < 8; ++i) nreg[i] = ld16(nt_ptr + (r0 + i) * p.N);
        } else {
          const int64_t r0 = row_lo + c0 + 8 * n_kb;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int64_t r = r0 + i;
            nreg[i] = (r < row_hi) ? ld16(nt_ptr + r * p.N) : u32x4{0u, 0u, 0u, 0u};
          }
        }
      }
    }
  };

  auto store_step = [&](int buf) {
    uint16_t* ms = &lds[buf][0];
    uint16_t* ns = &lds[buf][BM * BK];
    if constexpr (!M_T) {
#pragma unroll
      for (int i = 0; i < M_DIRECT_LOADS; ++i)
        *reinterpret_cast<u32x4*>(ms + lds_off(tid / 8 + 32 * i, tid & 7)) = mreg[i];
    } else {
      if (mt_live) {
        u32x4 t[8];
        transpose8x8(mreg, t);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          *reinterpret_cast<u32x4*>(ms + lds_off(8 * m_mb + j, m_kb)) = t[j];
      }
    }
    if constexpr (!N_T) {
#pragma unroll
      for (int i = 0; i < N_DIRECT_LOADS; ++i)
        *reinterpret_cast<u32x4*>(ns + lds_off(tid / 8 + 32 * i, tid & 7)) = nreg[i];
    } else {
      if (nt_live) {
        u32x4 t[8];
        transpose8x8(nreg, t);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          *reinterpret_cast<u32x4*>(ns + lds_off(8 * n_mb + j, n_kb)) = t[j];
      }
    }
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x16{};

  const int frag_row = lane & 31;
  const int frag_ch = lane >> 5;

  if (nsteps > 0) {
    load_step(0);
    store_step(0);
    __syncthreads();
  }
  for (int s = 0; s < nsteps; ++s) {
    const int buf = s & 1;
    if (s + 1 < nsteps) load_step(s + 1);
    const uint16_t* ms = &lds[buf][0];
    const uint16_t* ns = &lds[buf][BM * BK];
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = 2 * ks + frag_ch;
      bf16x8 af[NB], bfr[MB];
#pragma unroll
      for (int j = 0; j < NB; ++j)
        af[j] = *reinterpret_cast<const bf16x8*>(ns + lds_off(wn * WN + 32 * j + frag_row, ch));
#pragma unroll
      for (int i = 0; i < MB; ++i)
        bfr[i] = *reinterpret_cast<const bf16x8*>(ms + lds_off(wm * WM + 32 * i + frag_row, ch));
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[j], bfr[i], acc[i][j], 0, 0, 0);
    }
    if (s + 1 < nsteps) store_step(buf ^ 1);
    __syncthreads();
  }

  // ---------------- epilogue ------------------------------------------------------------------
  // lane holds output row (wm*WM + 32*i + lane%32) and columns wn*WN + 32*j + 8*q + 4*(lane/32) + 0..3
  const int col_in = 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < MB; ++i) {
    const int mrow = wm * WM + 32 * i + frag_row;
    if constexpr (KIND == KIND_DW) {
      const int64_t m = (int64_t)mt * BM + mrow;
      if (m >= p.K) continue;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        float* dst;
        int64_t col;
        if constexpr (DUAL) {
          const int half = (j >= NB / 2);
          col = (int64_t)nt * (BN / 2) + wn * (WN / 2) + 32 * (j % (NB / 2));
          dst = static_cast<float*>(half ? p.out2 : p.out);
        } else {
          col = (int64_t)nt * BN + wn * WN + 32 * j;
          dst = static_cast<float*>(p.out);
        }
        dst += (int64_t)g * p.K * p.N + m * p.N;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int64_t n = col + 8 * q + col_in;
          if (n < p.N) {
            f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            *reinterpret_cast<f32x4*>(dst + n) = v;
          }
        }
      }
    } else {
      const int64_t r = row_lo + mrow;
      if (r >= row_hi) continue;
      if constexpr (KIND == KIND_DX) {
        uint16_t* dst = static_cast<uint16_t*>(p.out) + r * p.K;
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int64_t n = (int64_t)nt * BN + wn * WN + 32 * j + 8 * q + col_in;
            if (n < p.K) {
              uint2 v;
              v.x = pack_bf16(acc[i][j][4 * q], acc[i][j][4 * q + 1]);
              v.y = pack_bf16(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
              *reinterpret_cast<uint2*>(dst + n) = v;
            }
          }
      } else if constexpr (DUAL) {
        uint16_t* c1 = static_cast<uint16_t*>(p.out) + r * p.N;
        uint16_t* c2 = static_cast<uint16_t*>(p.out2) + r * p.N;
        uint16_t* ca = p.act + r * p.N;
#pragma unroll
        for (int j = 0; j < NB / 2; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int64_t n = (int64_t)nt * (BN / 2) + wn * (WN / 2) + 32 * j + 8 * q + col_in;
            if (n < p.N) {
              uint2 vg, vu;
              vg.x = pack_bf16(acc[i][j][4 * q], acc[i][j][4 * q + 1]);
              vg.y = pack_bf16(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
              vu.x = pack_bf16(acc[i][j + NB / 2][4 * q], acc[i][j + NB / 2][4 * q + 1]);
              vu.y = pack_bf16(acc[i][j + NB / 2][4 * q + 2], acc[i][j + NB / 2][4 * q + 3]);
              *reinterpret_cast<uint2*>(c1 + n) = vg;
              *reinterpret_cast<uint2*>(c2 + n) = vu;
              if constexpr (ACT) {
                uint2 va;
                va.x = pack_bf16(silu_f32(bf16_lo(vg.x)) * bf16_lo(vu.x),
                                 silu_f32(bf16_hi(vg.x)) * bf16_hi(vu.x));
                va.y = pack_bf16(silu_f32(bf16_lo(vg.y)) * bf16_lo(vu.y),
                                 silu_f32(bf16_hi(vg.y)) * bf16_hi(vu.y));
                *reinterpret_cast<uint2*>(ca + n) = va;
              }
            }
          }
      } else {
        uint16_t* dst = static_cast<uint16_t*>(p.out) + r * p.N;
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int64_t n = (int64_t)nt * BN + wn * WN + 32 * j + 8 * q + col_in;
            if (n < p.N) {
              uint2 v;
              v.x = pack_bf16(acc[i][j][4 * q], acc[i][j][4 * q + 1]);
              v.y = pack_bf16(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
              *reinterpret_cast<uint2*>(dst + n) = v;
            }
          }
      }
    }
  }
}

constexpr int kBM = 256;
constexpr int kBN = 256;

template <int KIND, bool DUAL, bool ACT>
moe_status launch(const GemmParams& p, unsigned grid, hipStream_t stream, const char* name) {
  if (grid == 0) return MOE_SUCCESS;
  grouped_gemm_kernel<KIND, kBM, kBN, DUAL, ACT><<<grid, NT, 0, stream>>>(p);
  return check_launch(name);
}

bool bad_ptr(const void* q) { return q != nullptr && !aligned16(q); }

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status moe_grouped_gemm_fwd(const moe_bf16* A, const moe_bf16* B, const moe_bf16* B2,
                                           const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                           int64_t N, moe_bf16* C, moe_bf16* C2, moe_bf16* act,
                                           hipStream_t stream) {
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_fwd: need 1 <= G <= 256");
  if (R < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_fwd: bad size");
  if (K % 64 || N % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_fwd: K and N must be multiples of 64");
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_fwd: R >= 2^31");
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_fwd: offsets is NULL");
  if ((B2 == nullptr) != (C2 == nullptr))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_fwd: B2 and C2 must both be set or both NULL");
  if (act && !B2) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_fwd: act needs B2");
  if (R == 0) return MOE_SUCCESS;
  if (!A || !B || !C) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_fwd: NULL pointer");
  if (bad_ptr(A) || bad_ptr(B) || bad_ptr(B2) || bad_ptr(C) || bad_ptr(C2) || bad_ptr(act))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_fwd: pointers must be 16-byte aligned");
  GemmParams p{};
  p.a = A; p.b = B; p.b2 = B2; p.offsets = offsets; p.out = C; p.out2 = C2; p.act = act;
  p.G = G; p.R = R; p.K = K; p.N = N;
  p.mt_bound = (int)((R + kBM - 1) / kBM + G);
  const int cols_per_tile = B2 ? kBN / 2 : kBN;
  p.n_tiles = (int)((N + cols_per_tile - 1) / cols_per_tile);
  const unsigned grid = (unsigned)((int64_t)p.mt_bound * p.n_tiles);
  if (B2 && act) return launch<KIND_FWD, true, true>(p, grid, stream, "grouped_gemm_fwd(dual,swiglu)");
  if (B2) return launch<KIND_FWD, true, false>(p, grid, stream, "grouped_gemm_fwd(dual)");
  return launch<KIND_FWD, false, false>(p, grid, stream, "grouped_gemm_fwd");
}

extern "C" moe_status moe_grouped_gemm_dx(const moe_bf16* dC, const moe_bf16* B, const moe_bf16* dC2,
                                          const moe_bf16* B2, const int32_t* offsets, int32_t G,
                                          int64_t R, int64_t K, int64_t N, moe_bf16* dA,
                                          hipStream_t stream) {
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dx: need 1 <= G <= 256");
  if (R < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: bad size");
  if (K % 64 || N % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dx: K and N must be multiples of 64");
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dx: R >= 2^31");
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: offsets is NULL");
  if ((dC2 == nullptr) != (B2 == nullptr))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: dC2 and B2 must both be set or both NULL");
  if (R == 0) return MOE_SUCCESS;
  if (!dC || !B || !dA) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: NULL pointer");
  if (bad_ptr(dC) || bad_ptr(B) || bad_ptr(dC2) || bad_ptr(B2) || bad_ptr(dA))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: pointers must be 16-byte aligned");
  GemmParams p{};
  p.a = dC; p.a2 = dC2; p.b = B; p.b2 = B2; p.offsets = offsets; p.out = dA;
  p.G = G; p.R = R; p.K = K; p.N = N;
  p.mt_bound = (int)((R + kBM - 1) / kBM + G);
  p.n_tiles = (int)((K + kBN - 1) / kBN);
  const unsigned grid = (unsigned)((int64_t)p.mt_bound * p.n_tiles);
  if (dC2) return launch<KIND_DX, true, false>(p, grid, stream, "grouped_gemm_dx(dual)");
  return launch<KIND_DX, false, false>(p, grid, stream, "grouped_gemm_dx");
}

extern "C" moe_status moe_grouped_gemm_dw(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                                          const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                          int64_t N, float* dB, float* dB2, hipStream_t stream) {
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dw: need 1 <= G <= 256");
  if (R < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dw: bad size");
  if (K % 64 || N % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dw: K and N must be multiples of 64");
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dw: R >= 2^31");
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dw: offsets is NULL");
  if ((dC2 == nullptr) != (dB2 == nullptr))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dw: dC2 and dB2 must both be set or both NULL");
  if (!dB || (R > 0 && (!A || !dC)))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dw: NULL pointer");
  if (bad_ptr(A) || bad_ptr(dC) || bad_ptr(dC2) || bad_ptr(dB) || bad_ptr(dB2))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dw: pointers must be 16-byte aligned");
  GemmParams p{};
  p.a = A; p.b = dC; p.b2 = dC2; p.offsets = offsets; p.out = dB; p.out2 = dB2;
  p.G = G; p.R = R; p.K = K; p.N = N;
  p.m_tiles = (int)((K + kBM - 1) / kBM);
  const int cols_per_tile = dC2 ? kBN / 2 : kBN;
  p.n_tiles = (int)((N + cols_per_tile - 1) / cols_per_tile);
  const unsigned grid = (unsigned)((int64_t)G * p.m_tiles * p.n_tiles);
  if (dC2) return launch<KIND_DW, true, false>(p, grid, stream, "grouped_gemm_dw(dual)");
  return launch<KIND_DW, false, false>(p, grid, stream, "grouped_gemm_dw");
}
