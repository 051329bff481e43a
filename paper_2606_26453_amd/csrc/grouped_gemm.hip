// Grouped GEMMs over ragged expert row groups on gfx950 bf16 MFMA (fp32 accumulation).
//
// One kernel template serves the three products of the layer:
//   FWD  C[r, n]      = sum_c A[r, c]  * B[g][c, n]      rows r of group g (ragged), c < K
//   DX   dA[r, kk]    = sum_c dC[r, c] * B[g][kk, c]     rows r of group g (ragged), c < N (or 2N)
//   DW   dB[g][m, n]  = sum_r A[r, m]  * dC[r, n]        r over group g (ragged contraction)
// DW is the paper's dW1_e = X_e^T G_e (section 5.4, Appendix H).
//
// Work decomposition.  A workgroup owns a 256 x 256 output tile and walks the contraction 32 at a
// time through a ring of LDS slots.  Both operand tiles reach LDS through buffer loads that write
// LDS directly (16 bytes per lane, no register staging); ragged contraction rows beyond a group
// fall outside the buffer resource and read as zero.  An operand whose contraction is contiguous in
// memory (the routed rows, dX's weights) is read into MFMA layout with ds_read_b128; an operand
// whose contraction index is its memory row (the weights in FWD, both operands in DW) is kept in
// LDS with its rows intact and read with the transposing ds_read_b64_tr_b16, since the matrix
// cores take both operands contraction-contiguous per lane.
//
// MFMA operand roles: the N-side operand is the MFMA "A" (32 MFMA rows = 32 output columns) and
// the M-side operand the MFMA "B", so each lane's accumulator holds one output row and runs of
// 4 consecutive output columns, stored as 8-byte (bf16) or 16-byte (fp32) vectors.
//
// Dual mode (FWD gate/up, DW gate/up): the N side of a tile is split into column groups fed from
// two sources at the same output columns; each wave's 128 N-columns are 64 from each source, so the
// accumulators for the same (row, column) of both products sit in the same lane, which is what
// the fused SwiGLU epilogue needs.  DX dual mode appends the second pair to the contraction.
#include <type_traits>

#include "common.h"

namespace moe {
namespace {

constexpr int TN = 256;      // output tile columns (N side)
constexpr int BK = 32;       // contraction elements per pipeline stage

// Two LDS tile layouts, chosen so that DMA stores are plain 1 KiB runs and every fragment read
// of 8 (ds_read_b128) or 16 (ds_read_b64_tr_b16) lanes touches distinct banks:
//  - direct operand (contraction contiguous in memory, e.g. the routed rows): [256 rows][4 chunks
//    of 8 elements], chunk c of row r at r*64 + 16*(c ^ ((r >> 2) & 3)) (16 consecutive rows of one
//    chunk fill all 64 banks);
//  - mn operand (contraction is the memory row, e.g. a [K,N] weight): 4 groups of 64 columns,
//    each [32 contraction rows][8 chunks], chunk c of row k at group*4096 + k*128 +
//    16*(c ^ 2*(k & 3)).
__device__ __forceinline__ int swz_d(int r) { return (r >> 2) & 3; }
__device__ __forceinline__ int swz_t(int k) { return (k & 3) << 1; }

// FWD: C = A.B per group; DX: dA = dC.B^T per group; DW: dB[g] = A_g^T.dC_g from row-major
// operands (contraction = rows, read with transposing LDS reads); DWT: the same dB[g] from
// contraction-major copies A^T [K, ld], dC^T [N, ld] in which each group's rows form a contiguous
// segment zero-padded to 32 (both operands then read directly).
enum { KIND_FWD = 0, KIND_DX = 1, KIND_DW = 2, KIND_DWT = 3 };

struct GemmParams {
  const uint16_t* a;   // M side: FWD A [R,K]; DX dC [R,N]; DW A [R,K]
  const uint16_t* a2;  // DX: dC2
  const uint16_t* b;   // N side: FWD B [G,K,N]; DX B [G,K,N]; DW dC [R,N]
  const uint16_t* b2;  // FWD B2; DX B2; DW dC2
  const int32_t* offsets;
  void* out;           // FWD C; DX dA (dH_gate with the SwiGLU-backward epilogue); DW dB
  void* out2;          // FWD C2; DX dH_up with the SwiGLU-backward epilogue; DW dB2
  uint16_t* act;       // FWD SwiGLU output
  const uint16_t* hg;  // DX SwiGLU-backward epilogue: H_gate [R,K]
  const uint16_t* hu;  //                               H_up [R,K]
  int G;
  int64_t R, K, N;
  int mt_bound;        // FWD/DX: upper bound on the number of row tiles
  int m_tiles;         // DW: tiles over K
  int n_tiles;         // tiles over the output columns
  int64_t ld_t;        // DWT: row length of the contraction-major operands
  int* split_cnt;      // persistent kernels: split the last partial round's tiles (NULL: no split);
  float* split_part;   //   arrival counters (zero at launch) and fp32 partial tiles, one per unit
  int split_max;       //   at most this many contraction pieces per tail tile
  int split_slots;     //   workgroups resident at once (one-workgroup-per-tile kernels)
  int split_min_steps; //   contraction steps (of BK) a piece must have at least
  const int32_t* gather;   // FWD: row r of A is row gather[r] of a [gather_rows, K] source (NULL: A itself)
  int64_t gather_rows;
  const float* a_scale;    // FP8 products: per-row scale of the row operand [R]
  const float* w_scale;    //               per-output-column scale of the weight [G, K]
  const uint8_t* a_mx;     // MX products: E8M0 block scales of the row operand [C/128][R][4]
  const uint8_t* w_mx;     //              ... of the weight's rows [C/128][G*K][4] (DWT: of dC^T's rows)
  const uint8_t* w_mx2;    //              DWT dual: of dC2^T's rows
  int64_t mx_a_step, mx_w_step;   //       bytes from one 128-element group of scales to the next
  int* tile_queue;         // DW, persistent: 8 tile-claim counters, one per XCD (zero at launch)
  int* comb_cnt;           // FWD single output, fused combine: arrival counters [T, n_tiles] (zero
                           //   at launch); NULL: no combine
  const float* comb_w;     //   routing weights [T, k]
  const int32_t* comb_ros; //   row_of_slot [T * k]
  const int32_t* comb_tor; //   token_of_row [R]
  const uint16_t* comb_add;//   added to every Y row (shared FFN output) [T, N], or NULL
  uint16_t* comb_y;        //   Y [T, N]
  int comb_k;
};

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource (four scalar dwords) over [base, base + bytes): reads at offsets >= bytes
// return zero, which zero-fills the rows past a ragged group's end.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, int64_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const int n = bytes <= 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : (int)bytes);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((a >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane(n);
  r[3] = 0x00020000;
  return r;
}

// The same over [base, base + bytes) with bytes already in [0, 2^31).
__device__ __forceinline__ i32x4 make_rsrc32(const void* base, int bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((a >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane(bytes);
  r[3] = 0x00020000;
  return r;
}

// One 16-byte-per-lane buffer load written straight to LDS at lds_addr + 16*lane.  Issued as
// inline assembly so the compiler does not serialise later LDS reads behind it; completion is
// tracked explicitly with vmcnt waits (loads retire in order).
__device__ __forceinline__ void dma16(i32x4 rsrc, int voff, int lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(lds_addr)
               : "memory", "m0");
}

// The same with 4 bytes per lane (lds_addr + 4*lane).
__device__ __forceinline__ void dma4(i32x4 rsrc, int voff, int lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dword %0, %1, 0 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(lds_addr)
               : "memory", "m0");
}

// Cache-policy bit of buffer accesses: agent-scope coherent (sc1), i.e. written through to / read
// past the per-XCD L2s, which are not coherent with each other.
constexpr int CP_SC1 = 16;

template <int N>
__device__ __forceinline__ void wait_vm() {
  // s_waitcnt vmcnt(N) with the other counters left unconstrained
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ bf16x8 lds_read16(const char* p) { return *reinterpret_cast<const bf16x8*>(p); }

// Two transposing 8-byte LDS reads -> one MFMA operand (see the mn layout above).
__device__ __forceinline__ bf16x8 lds_read_tr(const char* p) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const lds_i16x4* q = (const lds_i16x4*)(const __attribute__((address_space(3))) char*)p;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_i16x4*>(q));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_i16x4*>(
      (const lds_i16x4*)((const __attribute__((address_space(3))) char*)p + 4 * 128)));
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  const i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// Logical tile index of block `bid` (< n): blocks go round-robin to the 8 XCDs, so give XCD x
// the contiguous logical range it would otherwise see interleaved with the other seven.
__device__ __forceinline__ int xcd_remap(int bid, int n) {
  const int q = n >> 3, r = n & 7, x = bid & 7, l = bid >> 3;
  return x * q + (x < r ? x : r) + l;
}

// Logical index within an (mt x nt) grid -> (m, n), walking bands of BW = 4 column tiles so that
// 32 consecutive tiles form an 8 x 4 block (B column panels reused 8x, A row panels 4x in the XCD's
// L2).  Measured against bands of 8 (4 x 8 blocks) and of 2, 3, 5 and 16: 1.1-1.8% shorter
// layer steps on the Mixtral, fine-grained and Zipf-skewed configs (dX gate/up -5% at the first).
__device__ __forceinline__ void band_order(int id, int mtiles, int ntiles, int& m, int& n) {
  constexpr int BW = 4;
  const int full = ntiles / BW;
  const int span = mtiles * BW;
  if (id < full * span) {
    const int band = id / span, rem = id - band * span;
    m = rem / BW;
    n = band * BW + rem % BW;
  } else {
    const int rem = id - full * span, w = ntiles - full * BW;
    m = rem / w;
    n = full * BW + rem % w;
  }
}

// One workgroup computes a TM x 256 output tile with WAVES_M x WAVES_N wavefronts through an
// NSTAGE-deep LDS ring; WPE workgroups share a CU (2 when the ring is small enough).  PERSIST: the
// workgroup loops over tiles (grid = CU slots) instead of computing one tile (grid = tiles).  OUT16:
// dW results are rounded to bf16 (as the paper's kernel stores them) instead of stored as fp32.
//
// F8 (dX kind only): both operands are E4M3 bytes; a stage then holds 64 contraction elements in the
// same 64-byte rows, and one v_mfma_scale_f32_32x32x64_f8f6f4 per block consumes the two 16-byte
// fragments a bf16 stage feeds to two 32x32x16 MFMAs.  The epilogue applies the fp32 row and
// column scales before rounding to bf16.  MX (with F8): the scales are instead powers of two, one
// per 32 contraction elements of every row of either operand, stored with each row's four scales
// of a 128-element group in one 4-byte word and the words of consecutive rows side by side; each
// stage carries its two blocks' scale bytes (one 4-byte LDS DMA load per wavefront, 256 contiguous
// bytes: waves 0-3 the words of the 256 tile rows, waves 4-7 those of the 256 weight rows, each
// word serving two stages), and the matrix core applies them inside the product (the epilogue only
// rounds).
template <int KIND, bool DUAL, bool ACT, int TM, int WAVES_M, int WAVES_N, int NSTAGE, bool PINGPONG, int WPE,
          bool PERSIST, bool OUT16, bool GATHER, bool F8, bool MX>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N, WPE) void grouped_gemm_kernel(GemmParams p) {
  // F8 && DUAL: one weight whose output channels interleave gate and up by 128 (tile columns
  // 0..127 gate, 128..255 up), stored as two outputs (+ SwiGLU with ACT) like the fwd dual product.
  // F8 && ACT && !DUAL: the dX-down product with the SwiGLU backward in its epilogue, applied to
  // the scaled, bf16-rounded dA exactly as in the bf16 product.
  static_assert(!F8 || KIND == KIND_DX || (KIND == KIND_DWT && MX),
                "FP8 operands: the dX-shaped products (and, with MX scales along the tokens, dW)");
  static_assert(!MX || (F8 && PINGPONG && WAVES_M * WAVES_N == 8 && TM == 256),
                "MX scales: the FP8 product's 8-wavefront ping-pong schedule");
  constexpr int ES = F8 ? 1 : 2;              // bytes per operand element
  constexpr int BKE = F8 ? 2 * BK : BK;       // contraction elements per stage (64-byte rows)
  constexpr int NWAVE = WAVES_M * WAVES_N;
  constexpr int OPND_M = TM * BK * 2;         // bytes of the M-side tile of one stage
  constexpr int OPND_N = TN * BK * 2;         // bytes of the N-side tile of one stage (16 KiB)
  constexpr int STAGE = OPND_M + OPND_N;      // M side at +0, N side at +OPND_M
  constexpr int DPW_M = TM / 16 / NWAVE;      // 1 KiB DMA loads per wave per stage, M side
  constexpr int DPW_N = TN / 16 / NWAVE;      // ... N side
  constexpr int DPW_T = DPW_M + DPW_N;
  constexpr int OPS = DPW_T + (MX ? 1 : 0);   // DMA loads per wave per stage (MX: + the scales)
  constexpr bool FSCALE = F8 && !MX;          // fp32 row/column scales applied in the epilogue
  constexpr bool FUSE_COMBINE = KIND == KIND_FWD && !DUAL && !ACT && !GATHER;   // may fuse the combine
  static_assert(DPW_M * NWAVE * 16 == TM && DPW_N * NWAVE * 16 == TN, "DMA split");
  constexpr int WTM = TM / WAVES_M;           // per-wave tile rows
  constexpr int WTN = TN / WAVES_N;           // per-wave tile columns
  constexpr int MB = WTM / 32;                // 32x32 MFMA blocks per wave along rows
  constexpr int NB = WTN / 32;                // ... and along columns
  constexpr bool M_T = (KIND == KIND_DW);     // M-side operand stored contraction-major
  constexpr bool N_T = (KIND == KIND_FWD || KIND == KIND_DW);   // N side stored contraction-major
  constexpr bool IS_DW = (KIND == KIND_DW || KIND == KIND_DWT); // weight gradient: groups own the
                                                                // contraction, outputs are dB[g]
  // persistent fp32 dW (single-group schedule): the next tile's first stages are issued before
  // this tile's epilogue, which then stages its results through the other half of the ring
  // (measured: dW gate/up 1.1% shorter on the Mixtral-shaped and long-batch layers, dW down 0.6%
  // longer; with bf16 results the extra live state made the epilogue spill, and the paper's dW1
  // shape ran 10% longer, so bf16 results keep the whole ring)
  constexpr bool EARLY = PERSIST && KIND == KIND_DW && !OUT16;

  __shared__ __attribute__((aligned(16))) char lds[NSTAGE * STAGE];
  // MX: per stage, the scale words of the 256 tile rows (bytes 0..1023) and of the 256 weight rows
  // (1024..2047); word of row r: 4*r, byte 2*(step & 1) + half is the scale of that half
  constexpr int SC_STAGE = 2048;
  __shared__ __attribute__((aligned(16))) char lds_sc[MX ? NSTAGE * SC_STAGE : 16];
  __shared__ int s_scan[256];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  // ---------------- persistent tile scheduler ----------------------------------------------------
  // The grid holds one workgroup per CU slot (or fewer, when there are fewer tiles); workgroup b
  // walks the dispatch indices b, b + gridDim.x, ...  gridDim.x is a multiple of 8 whenever it is
  // the CU count, so every index a workgroup takes belongs to the XCD it runs on.  The group
  // offsets, the tile prefix over groups (fwd/dX) and the group order (dW) are built once per
  // workgroup in LDS.
  __shared__ int s_off[257];
  __shared__ int s_pp[257];   // DWT: padded segment starts (exclusive prefix of ceil32(rows_g))
  for (int i = tid; i <= p.G; i += 64 * NWAVE) s_off[i] = p.offsets[i];   // G + 1 may exceed the threads
  int ntiles_all, mtotal = 0;
  if constexpr (KIND == KIND_DWT) {
    __syncthreads();
    // segments padded to 32 rows (128 with MX scales: each segment then starts a scale word)
    constexpr int PADM = MX ? 127 : 31;
    if (tid < 256) s_pp[tid + 1] = tid < p.G ? ((s_off[tid + 1] - s_off[tid] + PADM) & ~PADM) : 0;
    if (tid == 0) s_pp[0] = 0;
    __syncthreads();
    for (int off = 1; off < p.G; off <<= 1) {   // entries past G are zero
      const int add = (tid < 256 && tid >= off) ? s_pp[tid + 1 - off] : 0;
      __syncthreads();
      if (tid < 256) s_pp[tid + 1] += add;
      __syncthreads();
    }
  }
  if constexpr (IS_DW) {
    // Largest groups first (their tiles run longest).
    int kg = 0;
    if (tid < p.G) kg = p.offsets[tid + 1] - p.offsets[tid];
    if (tid < 256) s_scan[tid] = kg;
    __syncthreads();
    int rank = 0;
    if (tid < p.G)
      for (int h = 0; h < p.G; ++h) {
        const int kh = s_scan[h];
        rank += (kh > kg) || (kh == kg && h < tid);
      }
    __syncthreads();
    if (tid < p.G) s_scan[rank] = tid;
    __syncthreads();
    ntiles_all = p.G * p.m_tiles * p.n_tiles;
  } else {
    int cnt = 0;
    if (tid < p.G) cnt = (p.offsets[tid + 1] - p.offsets[tid] + TM - 1) / TM;
    if (tid < 256) s_scan[tid] = cnt;
    __syncthreads();
    for (int off = 1; off < p.G; off <<= 1) {   // entries past G are zero
      const int add = (tid < 256 && tid >= off) ? s_scan[tid - off] : 0;
      __syncthreads();
      if (tid < 256) s_scan[tid] += add;
      __syncthreads();
    }
    mtotal = s_scan[p.G - 1];
    ntiles_all = mtotal * p.n_tiles;
  }
  // dispatch index -> (group, row tile, column tile, row range).  FWD/DX: output rows of the
  // tile; DW: the group's contraction rows.  Uniform over the workgroup (FWD/DX use a barrier).
  auto map_tile = [&](int it, int& g, int& mt, int& nt, int& row_lo, int& row_hi) {
    if constexpr (IS_DW) {
      // When a group's tile count divides by 8, each XCD takes one contiguous eighth of every
      // group (in band order), so the long tiles of a hot group spread over all XCDs while each
      // XCD's L2 still sees neighbouring tiles.
      const int per_g = p.m_tiles * p.n_tiles;
      int slot, within;
      if ((per_g & 7) == 0) {
        const int c = per_g >> 3, x = it & 7, l = it >> 3;
        slot = l / c;
        within = x * c + (l - slot * c);
      } else {
        slot = it / per_g;
        within = it - slot * per_g;
      }
      g = s_scan[slot];
      band_order(within, p.m_tiles, p.n_tiles, mt, nt);
      if constexpr (KIND == KIND_DWT) {   // the group's padded segment of the contraction-major copies
        row_lo = s_pp[g];
        row_hi = s_pp[g + 1];
      } else {
        row_lo = s_off[g];
        row_hi = s_off[g + 1];
      }
    } else if ((p.n_tiles & 7) == 0 && p.n_tiles >= 32) {
      // Expert-major order for wide outputs: the groups one after the other, each group's tiles
      // shared out over the 8 XCDs by column (XCD x = dispatch index mod 8 takes column tiles
      // x*c .. x*c+c-1, c = n_tiles/8 >= 4, walked in bands), so the XCDs work on one group at a
      // time: its rows stay in the caches while its weight streams once.  Measured at config 1
      // against the order below: fwd gate/up (112 column tiles) 3446 -> 3246 us, dX down with the
      // fused SwiGLU backward (56) 1932 -> 1816 us; with 16 column tiles (c = 2) it lost 1-2%, so
      // narrower outputs keep the band order over all groups.
      g = __syncthreads_count(tid < p.G && s_scan[tid] * p.n_tiles <= it);
      const int base_rt = g > 0 ? s_scan[g - 1] : 0;
      const int pl = it - base_rt * p.n_tiles;
      const int c = p.n_tiles >> 3;
      int m, n;
      band_order(pl >> 3, s_scan[g] - base_rt, c, m, n);
      mt = m;
      nt = (pl & 7) * c + n;
      row_lo = s_off[g] + mt * TM;
      row_hi = s_off[g + 1];
    } else {
      int mt_glob;
      band_order(xcd_remap(it, ntiles_all), mtotal, p.n_tiles, mt_glob, nt);
      g = __syncthreads_count(tid < p.G && s_scan[tid] <= mt_glob);
      mt = mt_glob - (g > 0 ? s_scan[g - 1] : 0);
      row_lo = s_off[g] + mt * TM;
      row_hi = s_off[g + 1];
    }
    // values derived through LDS are uniform by construction; say so to the compiler so that
    // buffer resources and LDS DMA addresses stay in scalar registers
    g = __builtin_amdgcn_readfirstlane(g);
    mt = __builtin_amdgcn_readfirstlane(mt);
    nt = __builtin_amdgcn_readfirstlane(nt);
    row_lo = __builtin_amdgcn_readfirstlane(row_lo);
    row_hi = __builtin_amdgcn_readfirstlane(row_hi);
  };

  // ---------------- DMA descriptors ------------------------------------------------------------
  // Each stage stages 256 x 32 of both operands in 16 DMA loads of 1 KiB per operand; wave w
  // issues loads I = DPW*w .. DPW*w + DPW-1.  Direct side: load I covers rows 16I .. 16I+15 (lane
  // -> row 16I + lane/4, chunk (lane&3) ^ swz_d(row) = (lane&3) ^ swz_d(lane/4)).  mn side: load I
  // covers column group I/4, contraction rows 8(I%4) .. +7 (lane -> row 8(I%4) + lane/8, chunk
  // (lane&7) ^ swz_t(row)).
  const int lds0 = (int)(size_t)(const __attribute__((address_space(3))) char*)lds;

  const char* m_src = nullptr;    // M side: base of the contraction window at c = 0
  const char* m_src2 = nullptr;   // DX dual: second half of the contraction
  int64_t m_ld = 0;               // elements per memory row
  int m_voff[DPW_M];
  const char* n_src = nullptr;    // N side
  const char* n_src2 = nullptr;
  int64_t n_ld = 0;
  int n_voff[DPW_N];
  int64_t c_len = 0;              // contraction extent
  int nsteps = 0;
  int c_len32 = 0, m_row_bytes = 0, n_row_bytes = 0;   // the same sizes in 32 bits
  int tile_rows = TM;             // FWD/DX: output rows of the tile that are rows of its group
  const char* sc_src = nullptr;   // MX: this wave's scale words (tile rows or weight rows), group 0
  int sc_voff = 0;
  int64_t sc_step = 0;            //     bytes between consecutive 128-element groups
  auto setup = [&](int g, int mt, int nt, int64_t row_lo, int64_t row_hi) {
    tile_rows = (int)(row_hi - row_lo < TM ? row_hi - row_lo : TM);
    // lane-dependent terms are recomputed per tile rather than hoisted out of the tile loop and
    // kept live (in registers the main loop needs) across it
    int lane = threadIdx.x & 63;
    if constexpr (PERSIST) asm volatile("" : "+v"(lane));
    // M side
    if constexpr (KIND == KIND_DWT) {
      // A^T [K, ld_t]: tile rows = dB rows mt*TM .. (clamped to K), contraction = the group's
      // padded segment starting at column row_lo
      m_ld = p.ld_t;
      const int64_t rows_valid = p.K - (int64_t)mt * TM;   // > 0
      m_src = reinterpret_cast<const char*>(p.a) + ((int64_t)mt * TM * m_ld + row_lo) * ES;
#pragma unroll
      for (int i = 0; i < DPW_M; ++i) {
        int64_t r = 16 * (DPW_M * wave + i) + (lane >> 2);
        if (r > rows_valid - 1) r = rows_valid - 1;
        const int c = (lane & 3) ^ swz_d(lane >> 2);
        m_voff[i] = (int)(r * m_ld * ES + 16 * c);
      }
    } else if constexpr (!M_T) {
      m_ld = (KIND == KIND_FWD) ? p.K : p.N;
      const int64_t rows_valid = row_hi - row_lo;   // > 0
      if constexpr (GATHER) {
        // gathered rows: each lane's row of the source, read through the row list (the rows of
        // a ragged group's end clamp to its last row, as below)
        m_src = reinterpret_cast<const char*>(p.a);
#pragma unroll
        for (int i = 0; i < DPW_M; ++i) {
          int64_t r = 16 * (DPW_M * wave + i) + (lane >> 2);
          if (r > rows_valid - 1) r = rows_valid - 1;
          const int64_t src = p.gather[row_lo + r];
          const int c = (lane & 3) ^ swz_d(lane >> 2);
          m_voff[i] = (int)((src * m_ld + 8 * c) * 2);
        }
      } else {
        m_src = reinterpret_cast<const char*>(p.a) + row_lo * m_ld * ES;
        if constexpr (KIND == KIND_DX && DUAL && !F8) m_src2 = reinterpret_cast<const char*>(p.a2) + row_lo * m_ld * ES;
#pragma unroll
        for (int i = 0; i < DPW_M; ++i) {
          int64_t r = 16 * (DPW_M * wave + i) + (lane >> 2);
          if (r > rows_valid - 1) r = rows_valid - 1;
          const int c = (lane & 3) ^ swz_d(lane >> 2);
          m_voff[i] = (int)(r * m_ld * ES + 16 * c);
        }
      }
    } else {
      m_ld = p.K;
      const int grp = (DPW_M * wave) / 4;
      int64_t col0 = (int64_t)mt * TM + 64 * grp;
      if (col0 > p.K - 64) col0 = p.K - 64;
      m_src = reinterpret_cast<const char*>(p.a + row_lo * m_ld + col0);
#pragma unroll
      for (int i = 0; i < DPW_M; ++i) {
        const int k = 8 * ((DPW_M * wave + i) & 3) + (lane >> 3);
        const int c = (lane & 7) ^ swz_t(k);
        m_voff[i] = (int)((k * m_ld + 8 * c) * 2);
      }
    }
    // N side
    if constexpr (KIND == KIND_DWT) {
      // dC^T [N, ld_t]: tile row r is output column nt*TN + r, or in dual mode column
      // nt*TN/2 + 64*(r/128) + r%64 of dC^T (r%128 < 64) or of dC2^T (r%128 >= 64), so that each
      // wave's accumulator halves hold the two outputs at the same columns; this wave's 16*DPW_N
      // rows lie in one 64-row half (one source)
      n_ld = p.ld_t;
      const int r0w = 16 * DPW_N * wave;
      const uint16_t* src = p.b;
      if constexpr (DUAL) {
        if ((r0w & 127) >= 64) src = p.b2;
      }
      n_src = reinterpret_cast<const char*>(src) + row_lo * ES;
#pragma unroll
      for (int i = 0; i < DPW_N; ++i) {
        const int r = 16 * (DPW_N * wave + i) + (lane >> 2);
        int64_t col = DUAL ? (int64_t)nt * (TN / 2) + 64 * (r >> 7) + (r & 63) : (int64_t)nt * TN + r;
        if (col > p.N - 1) col = p.N - 1;
        const int c = (lane & 3) ^ swz_d(lane >> 2);
        n_voff[i] = (int)(col * n_ld * ES + 16 * c);
      }
    } else if constexpr (!N_T) {
      // DX: B[g][kk, c]; the tile's output columns kk = nt*TN + row, clamped
      n_ld = p.N;
      n_src = reinterpret_cast<const char*>(p.b) + (int64_t)g * p.K * p.N * ES;
      if constexpr (DUAL) n_src2 = reinterpret_cast<const char*>(p.b2) + (int64_t)g * p.K * p.N * ES;
#pragma unroll
      for (int i = 0; i < DPW_N; ++i) {
        int64_t kk = (int64_t)nt * TN + 16 * (DPW_N * wave + i) + (lane >> 2);
        if (kk > p.K - 1) kk = p.K - 1;
        const int c = (lane & 3) ^ swz_d(lane >> 2);
        n_voff[i] = (int)(kk * p.N * ES + 16 * c);
      }
    } else {
      // this wave's column group: in dual mode groups 0,2 come from the first source and 1,3 from
      // the second, at the same output columns
      n_ld = p.N;
      const int grp = (DPW_N * wave) / 4;
      int64_t col0;
      const uint16_t* src = p.b;
      if constexpr (DUAL) {
        col0 = (int64_t)nt * (TN / 2) + 64 * (grp >> 1);
        if (grp & 1) src = p.b2;
      } else {
        col0 = (int64_t)nt * TN + 64 * grp;
      }
      if (col0 > p.N - 64) col0 = p.N - 64;
      const int64_t rowbase = (KIND == KIND_FWD) ? (int64_t)g * p.K : row_lo;
      n_src = reinterpret_cast<const char*>(src + rowbase * p.N + col0);
#pragma unroll
      for (int i = 0; i < DPW_N; ++i) {
        const int k = 8 * ((DPW_N * wave + i) & 3) + (lane >> 3);
        const int c = (lane & 7) ^ swz_t(k);
        n_voff[i] = (int)((k * n_ld + 8 * c) * 2);
      }
    }

    if constexpr (MX && KIND == KIND_DWT) {
      // dW: the contraction is the group's padded token segment, starting at column row_lo (a
      // multiple of 128: scale word row_lo / 128).  waves 0-3: rows mt*TM + 64*wave + lane of A^T;
      // waves 4-7: the rows of dC^T (dual: dC^T or dC2^T, one source per wave) that tile rows
      // 64*(wave-4) + lane map to, as for the operand loads; all clamped to the last row
      const int r = 64 * (wave & 3) + lane;
      const int64_t grp0 = row_lo >> 7;
      if (wave < 4) {
        int64_t rr = (int64_t)mt * TM + r;
        if (rr > p.K - 1) rr = p.K - 1;
        sc_src = reinterpret_cast<const char*>(p.a_mx) + grp0 * p.mx_a_step;
        sc_voff = (int)(rr * 4);
        sc_step = p.mx_a_step;
      } else {
        const uint8_t* base = p.w_mx;
        int64_t col;
        if constexpr (DUAL) {
          col = (int64_t)nt * (TN / 2) + 64 * (r >> 7) + (r & 63);
          if ((r & 127) >= 64) base = p.w_mx2;
        } else {
          col = (int64_t)nt * TN + r;
        }
        if (col > p.N - 1) col = p.N - 1;
        sc_src = reinterpret_cast<const char*>(base) + grp0 * p.mx_w_step;
        sc_voff = (int)(col * 4);
        sc_step = p.mx_w_step;
      }
    } else if constexpr (MX) {
      // waves 0-3: tile rows 64*wave + lane (clamped to the group, like the row loads); waves 4-7:
      // weight rows (output columns) nt*TN + 64*(wave-4) + lane, clamped to the last
      const int r = 64 * (wave & 3) + lane;
      if (wave < 4) {
        int64_t rr = r;
        if (rr > row_hi - row_lo - 1) rr = row_hi - row_lo - 1;
        sc_src = reinterpret_cast<const char*>(p.a_mx) + row_lo * 4;
        sc_voff = (int)(rr * 4);
        sc_step = p.mx_a_step;
      } else {
        int64_t kk = (int64_t)nt * TN + r;
        if (kk > p.K - 1) kk = p.K - 1;
        sc_src = reinterpret_cast<const char*>(p.w_mx) + (int64_t)g * p.K * 4;
        sc_voff = (int)(kk * 4);
        sc_step = p.mx_w_step;
      }
    }
    // contraction extent
    if constexpr (KIND == KIND_FWD) c_len = p.K;
    else if constexpr (KIND == KIND_DX) c_len = (DUAL && !F8) ? 2 * p.N : p.N;
    else c_len = row_hi - row_lo;
    nsteps = (int)((c_len + BKE - 1) / BKE);
    c_len32 = (int)c_len;
    m_row_bytes = (int)(m_ld * 2);
    n_row_bytes = (int)(n_ld * 2);
  };

  // buffer resources of step s for the M and N operands
  int s_base = 0;   // first contraction step of the tile's range (a piece of a split tile)
  // Branch-free: the step's window is selected with scalar selects (a step past the end gets an
  // empty window), and every size is 32-bit (a 32-row slice of a transposed operand is < 2 GiB).
  auto rsrc_m = [&](int s) {
    const int sa = s + s_base;
    const bool live = s < nsteps;
    if constexpr (!M_T) {
      int64_t cc = (int64_t)sa * BKE;
      const char* base = m_src;
      if constexpr (KIND == KIND_DX && DUAL && !F8) {
        const bool second = cc >= p.N;
        base = second ? m_src2 : m_src;
        cc = second ? cc - p.N : cc;
      }
      int bytes = 0x7fffffff;
      // gathered rows: the window ends with the source, so a row index past it reads zeros
      if constexpr (GATHER) bytes = (int)((p.gather_rows * m_ld - cc) * 2);
      return make_rsrc32(base + cc * ES, live ? bytes : 0);
    } else {
      const int left = c_len32 - sa * BK;
      const int rows = left < BK ? left : BK;
      return make_rsrc32(m_src + (int64_t)sa * (BK * 2) * m_ld, live ? rows * m_row_bytes : 0);
    }
  };
  auto rsrc_n = [&](int s) {
    const int sa = s + s_base;
    const bool live = s < nsteps;
    if constexpr (!N_T) {
      int64_t cc = (int64_t)sa * BKE;
      const char* base = n_src;
      if constexpr (DUAL && KIND == KIND_DX && !F8) {
        const bool second = cc >= p.N;
        base = second ? n_src2 : n_src;
        cc = second ? cc - p.N : cc;
      }
      return make_rsrc32(base + cc * ES, live ? 0x7fffffff : 0);
    } else {
      const int left = c_len32 - sa * BK;
      const int rows = left < BK ? left : BK;
      return make_rsrc32(n_src + (int64_t)sa * (BK * 2) * n_ld, live ? rows * n_row_bytes : 0);
    }
  };
  // load d (0 .. DPW_T-1) of this wave for a step whose slot starts at LDS byte slot_lds
  auto dma_one = [&](int d, const i32x4& rm, const i32x4& rn, int slot_lds) {
    if (d < DPW_M) dma16(rm, m_voff[d], slot_lds + (DPW_M * wave + d) * 1024);
    else dma16(rn, n_voff[d - DPW_M], slot_lds + OPND_M + (DPW_N * wave + d - DPW_M) * 1024);
  };
  auto slot_of = [&](int s) { return s % NSTAGE; };
  // MX: this wave's scale load of step s: the 4-byte word holding the scales of steps s & ~1 and
  // s | 1 (a step past the end reads zeros, like the operands)
  const int lds_sc0 = (int)(size_t)(const __attribute__((address_space(3))) char*)lds_sc;
  auto dma_sc = [&](int s) {
    const int sa = s + s_base;
    const i32x4 rs = make_rsrc32(sc_src + (int64_t)(sa >> 1) * sc_step, s < nsteps ? 0x7fffffff : 0);
    dma4(rs, sc_voff, lds_sc0 + slot_of(s) * SC_STAGE + wave * 256);
  };
  auto issue = [&](int s) {
    const int slot_lds = lds0 + slot_of(s) * STAGE;
    const i32x4 rm = rsrc_m(s), rn = rsrc_n(s);
#pragma unroll
    for (int d = 0; d < DPW_T; ++d) dma_one(d, rm, rn, slot_lds);
    if constexpr (MX) dma_sc(s);
  };

  // ---------------- fragment reads ---------------------------------------------------------------
  // direct side: rows R0 + 32j + lane%32, chunk 2ks + lane/32
  // mn side (transposing reads): lane group G = lane/16, j16 = lane%16 reads contraction row
  //   16ks + 8(G>>1) + j16/4 (+4 for the second read), columns 32j + 16(G&1) + 4(j16&3) .. +3
  const int l32 = lane & 31, fh = lane >> 5;
  const int G16 = lane >> 4, j16 = lane & 15, kq = j16 >> 2, cq = j16 & 3;
  auto d_addr = [&](int R0, int ks) {
    return (R0 + l32) * 64 + (((2 * ks + fh) ^ swz_d(l32)) << 4);
  };
  auto t_addr = [&](int grp0, int jodd) {
    return grp0 * 4096 + (8 * (G16 >> 1) + kq) * 128 +
           (((4 * jodd + 2 * (G16 & 1) + (cq >> 1)) ^ (2 * kq)) << 4) + (cq & 1) * 8;
  };
  // byte offsets within a stage (M side at 0, N side at OPND_M), per ks (direct) or j parity (mn)
  const int m_a0 = M_T ? t_addr(wm * WTM / 64, 0) : d_addr(wm * WTM, 0);
  const int m_a1 = M_T ? t_addr(wm * WTM / 64, 1) : d_addr(wm * WTM, 1);
  const int n_a0 = OPND_M + (N_T ? t_addr(wn * WTN / 64, 0) : d_addr(wn * WTN, 0));
  const int n_a1 = OPND_M + (N_T ? t_addr(wn * WTN / 64, 1) : d_addr(wn * WTN, 1));

  f32x16 acc[MB][NB];
  auto zero_acc = [&]() {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[i][j] = f32x16{};
  };

  // fragment sets: 0/1 hold the first K-half of alternating stages, 2 the second K-half
  bf16x8 fa[3][NB], fb[3][MB];   // N-side (MFMA A) and M-side (MFMA B) fragments
  auto load_frags = [&](int set, int slot, int ks) {
    const char* st = lds + slot * STAGE;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if constexpr (N_T)
        fa[set][j] = lds_read_tr(st + ((j & 1) ? n_a1 : n_a0) + (j >> 1) * 4096 + ks * 2048);
      else
        fa[set][j] = lds_read16(st + (ks ? n_a1 : n_a0) + j * 2048);
    }
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      if constexpr (M_T)
        fb[set][i] = lds_read_tr(st + ((i & 1) ? m_a1 : m_a0) + (i >> 1) * 4096 + ks * 2048);
      else
        fb[set][i] = lds_read16(st + (ks ? m_a1 : m_a0) + i * 2048);
    }
  };
  // MFMAs m0 .. m1-1 of the MB x NB block grid (row-major order) with fragment set `set`
  auto mfmas = [&](int set, int m0, int m1) {
#pragma unroll
    for (int m = m0; m < m1; ++m)
      acc[m / NB][m % NB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[set][m % NB], fb[set][m / NB],
                                                                   acc[m / NB][m % NB], 0, 0, 0);
  };
  // FP8: one 32x32x64 MFMA per block from the concatenated 16-byte fragments of sets 0 and 1: lane
  // half h holds bytes 16h..16h+15 and 32+16h..32+16h+15 of the stage's row, which the instruction
  // takes as its contraction elements in the same order (its first 16 bytes of either half are
  // elements 0..31, the second 16 elements 32..63).  So its two scale blocks are the contraction's
  // own 32-element blocks 2*step and 2*step + 1, and lane half h supplies block h's scale of its row.
  int sc_m[MB], sc_n[NB];   // MX: this lane's scale bytes for the current stage
  auto read_scales = [&](int s) {
    if constexpr (MX) {
      const char* b = lds_sc + slot_of(s) * SC_STAGE + 2 * ((s + s_base) & 1) + fh;
#pragma unroll
      for (int i = 0; i < MB; ++i) sc_m[i] = *reinterpret_cast<const uint8_t*>(b + 4 * (wm * WTM + 32 * i + l32));
#pragma unroll
      for (int j = 0; j < NB; ++j)
        sc_n[j] = *reinterpret_cast<const uint8_t*>(b + 1024 + 4 * (wn * WTN + 32 * j + l32));
    }
  };
  auto mfmas_f8 = [&]() {
#pragma unroll
    for (int m = 0; m < MB * NB; ++m) {
      const i32x4 a0 = __builtin_bit_cast(i32x4, fa[0][m % NB]), a1 = __builtin_bit_cast(i32x4, fa[1][m % NB]);
      const i32x4 b0 = __builtin_bit_cast(i32x4, fb[0][m / NB]), b1 = __builtin_bit_cast(i32x4, fb[1][m / NB]);
      const i32x8 a8 = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
      const i32x8 b8 = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
      // operand formats 0 (E4M3) for both; without MX the block scales are 127 (2^0), leaving the
      // products unscaled
      if constexpr (MX)
        acc[m / NB][m % NB] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            a8, b8, acc[m / NB][m % NB], 0, 0, 0, sc_n[m % NB], 0, sc_m[m / NB]);
      else
        acc[m / NB][m % NB] =
            __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, acc[m / NB][m % NB], 0, 0, 0, 127, 0, 127);
    }
  };
  // the same, with the DPW_T refill loads of step `s` spread evenly between the MFMAs so the
  // vector-memory and LDS-write work of the refill overlaps the matrix cores
  auto mfmas_refill = [&](int set, int s) {
    const int slot_lds = lds0 + slot_of(s) * STAGE;
    const i32x4 rm = rsrc_m(s), rn = rsrc_n(s);
    constexpr int NM = MB * NB;
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      acc[m / NB][m % NB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[set][m % NB], fb[set][m / NB],
                                                                   acc[m / NB][m % NB], 0, 0, 0);
#pragma unroll
      for (int d = (m * DPW_T) / NM; d < ((m + 1) * DPW_T) / NM; ++d) dma_one(d, rm, rn, slot_lds);
      if (((m + 1) * DPW_T) / NM > (m * DPW_T) / NM) __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---------------- pipelined main loop ---------------------------------------------------------
  // Per stage s (two K-halves of 16):
  //   a. read the second half of stage s into set 2
  //   b. first MFMAs of the first half (set s&1)
  //   c. wait for this wave's loads of stage s+1 (two later stages may stay in flight); barrier:
  //      stage s+1 is now visible to all, and every read of stage s has completed
  //   d. read the first half of stage s+1 into set (s+1)&1
  //   e. remaining MFMAs of the first half, then the second half (set 2) with the refill of stage
  //      s's slot by stage s+4 spread between them
  // so the reads issued in (d) have ~3/4 of a stage of MFMAs to land before they are used.  Refills
  // past the last stage use an empty buffer resource (no memory access; the slot fills with
  // zeros), which keeps the wait counts the same on every iteration; the loop runs an even number
  // of stages, a trailing all-zero stage adding nothing.
  constexpr int MFMA_HALF = MB * NB;
  // the first stages of a tile are issued by prefill(), possibly while the previous tile's
  // results are still being stored
  constexpr int PREFILL = PINGPONG ? NSTAGE - 1 : NSTAGE;
  auto prefill = [&]() {
    if (nsteps > 0) {
#pragma unroll
      for (int s = 0; s < PREFILL; ++s) issue(s);
    }
  };
  auto main_loop = [&]() {
  if constexpr (!PINGPONG) {
    constexpr int MFMA_HALF = MB * NB;
    constexpr int SPLIT = MFMA_HALF / 2;
    auto stage_body = [&](int s, int cur) {
      const int slot = slot_of(s);
      load_frags(2, slot, 1);
      mfmas(cur, 0, SPLIT);
      __builtin_amdgcn_sched_barrier(0);
      wait_vm<(NSTAGE - 2) * DPW_T>();
      __syncthreads();
      load_frags(cur ^ 1, slot_of(s + 1), 0);   // unused after the last stage
      mfmas(cur, SPLIT, MFMA_HALF);
      // interleave the next stage's fragment reads with these MFMAs (two LDS reads, one MFMA)
      // rather than issuing all reads first: the matrix core keeps busy while the LDS queue
      // drains (measured: 1320-1360 -> 1185-1270 cycles per step on the fwd and dW products)
#pragma unroll
      for (int q = 0; q < (MB + NB) * (N_T ? 2 : 1) / 2; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // DS reads
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
      }
      __builtin_amdgcn_sched_barrier(0);
      mfmas_refill(2, s + NSTAGE);
    };
    if (nsteps > 0) {
      wait_vm<(NSTAGE - 1) * DPW_T>();
      __syncthreads();
      load_frags(0, 0, 0);
    }
    for (int s = 0; s < nsteps; s += 2) {
      stage_body(s, 0);
      stage_body(s + 1, 1);
    }
    wait_vm<0>();
  } else {
    // Ping-pong (8 wavefronts, two per SIMD): wave group 0 (tile rows 0..127) and group 1 (rows
    // 128..255) alternate every half stage between a compute phase (all MFMAs of one stage) and a
    // memory phase (all fragment reads of the next stage + this group's DMA of stage s+3), so one
    // wavefront of each SIMD feeds the matrix core while the other waits on LDS and memory.  Every
    // half stage ends with one barrier; group 1 runs half a stage behind (one extra barrier at the
    // start, one for group 0 at the end).  Before each barrier every wave waits until at most two
    // of its DMA stages are in flight: stage t is read (group 0 first) only after the barrier that
    // follows both groups' waits for t, and stage s+3 refills the slot of stage s-1, whose reads
    // both groups completed before the previous barrier.
    static_assert(NWAVE == 8 && WAVES_N == 2 && TM == 256, "ping-pong needs the 4x2 wave layout");
    const int grp = wave >> 2;
    static_assert(NSTAGE == 4, "ping-pong refill distance assumes a 4-slot ring");
    // A tile with at most 128 rows (the last tile of a group) gives group 1 no output rows: it
    // then skips its MFMAs (its fragment reads and share of the DMA stay, keeping the schedule and
    // the registers as they are), so each SIMD's matrix core serves group 0 alone and the step
    // costs about a compute phase plus a memory phase instead of two compute phases.  (The
    // single-group schedule cannot gain this way: its four wavefronts sit on four SIMDs.)
    static_assert(!PINGPONG || KIND == KIND_DX || KIND == KIND_DWT, "row-tile kinds");
    const bool live = (grp == 0) || (KIND == KIND_DWT) || (tile_rows > 128);   // uniform
    auto memory_phase = [&](int s) {
      const int slot = slot_of(s);
      load_frags(0, slot, 0);
      load_frags(1, slot, 1);
      read_scales(s);
      const int slot_lds = lds0 + slot_of(s + 3) * STAGE;
      const i32x4 rm = rsrc_m(s + 3), rn = rsrc_n(s + 3);
#pragma unroll
      for (int d = 0; d < DPW_T; ++d) dma_one(d, rm, rn, slot_lds);
      if constexpr (MX) dma_sc(s + 3);
    };
    auto half_end = [&]() {
      __builtin_amdgcn_sched_barrier(0);
      wait_vm<(NSTAGE - 2) * OPS>();
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
    };
    if (nsteps > 0) {
      wait_vm<(NSTAGE - 2) * OPS>();
      __syncthreads();
      if (grp == 1) half_end();
      for (int s = 0; s < nsteps; ++s) {
        memory_phase(s);
        half_end();
        if (live) {
          if constexpr (F8) {
            mfmas_f8();
          } else {
            mfmas(0, 0, MFMA_HALF);
            mfmas(1, 0, MFMA_HALF);
          }
        }
        half_end();
      }
      if (grp == 0) half_end();
    }
    wait_vm<0>();
  }
  };

  // ---------------- epilogue ------------------------------------------------------------------
  // lane holds output row (wm*WTM + 32*i + lane%32) and columns wn*WTN + 32*j + 8*q + 4*(lane/32) + 0..3
  auto epilogue = [&](int g, int mt, int nt, int64_t row_lo, int64_t row_hi) {
  int tid = threadIdx.x;   // recomputed per tile, as in setup()
  if constexpr (PERSIST) asm volatile("" : "+v"(tid));
  const int lane = tid & 63, l32 = lane & 31, fh = lane >> 5;
  const int col_in = 4 * fh;
  // EARLY: the tile is staged through the ring's upper half (slots 2 and 3) one row half at a
  // time, while the next tile's first two stages load into slots 0 and 1
  constexpr int RH = EARLY ? 2 : 1, TMP = TM / RH;
  char* const stg = lds + (EARLY ? 2 * STAGE : 0);
  if constexpr (IS_DW && !OUT16) {
    // fp32 results leave through LDS too, in two passes of 256 rows x 128 columns (128 KiB, the
    // ring; EARLY: each pass once per 128-row half, 64 KiB in the ring's upper half): pass h holds
    // column blocks 2h and 2h+1 of every wavefront (dual: pass 0 the gate
    // output's 128 columns of the tile, pass 1 the up output's).  Tile row t, 16-byte chunk c (4
    // columns) sits at t*512 + 16*(c ^ (t & 31)), conflict-free for both the accumulator-ordered
    // writes and the row-ordered reads.  Read back, every store instruction covers 4 rows x 256
    // contiguous bytes instead of the accumulator layout's 32 rows x 32 bytes, which a CU drains
    // 2-3x faster (256 KiB per tile).
    static_assert(NB == 4 && TMP * 512 <= (EARLY ? 2 : NSTAGE) * STAGE, "passes of 128 columns through the ring");
    constexpr int PER_WAVE = 2 * (TMP / 4) / NWAVE;   // store instructions per wave and pass
    constexpr int BATCH = 8;
    static_assert(PER_WAVE % BATCH == 0, "batches of LDS reads");
    const int64_t obase = (int64_t)g * p.K * p.N;
    for (int rh = 0; rh < RH; ++rh)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      __syncthreads();   // first pass: every wave is done with the ring; then: the last pass's reads are done
      if (!EARLY || wm == rh) {   // uniform per wavefront
#pragma unroll
      for (int i = 0; i < MB; ++i) {
        char* trow = stg + (wm * WTM - rh * TMP + 32 * i + l32) * 512;   // (t & 31) == l32
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int j = 2 * h + jj;
            const int c = wn * 16 + jj * 8 + 2 * q + fh;
            const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            *reinterpret_cast<f32x4*>(trow + 16 * (c ^ l32)) = v;
          }
      }
      }
      __syncthreads();
      // instruction s of wave w: tile rows 4*(w + NWAVE*(s/2)) + lane/16, chunks 16*(s%2) + lane%16.
      // Segment s%2 (64 columns) is output columns nseg[s%2] + 0..63: dual, nt*128 + 64*(s%2) (the
      // LDS chunk c is column nt*128 + 4c); otherwise nt*256 + 128*(s%2) + 64h.  K and N are
      // multiples of 64, so a row quad and a segment lie entirely inside or outside the output
      // (uniform tests).
      float* out = static_cast<float*>((DUAL && h == 1) ? p.out2 : p.out) + obase;
      const int64_t nseg0 = DUAL ? (int64_t)nt * (TN / 2) : (int64_t)nt * TN + 64 * h;
      constexpr int SEG1 = DUAL ? 64 : 128;
      const bool seg_in[2] = {nseg0 < p.N, nseg0 + SEG1 < p.N};
      const int rows_left = (int)(p.K - (int64_t)mt * TM - rh * TMP);   // > 0 for the first row half
      float* base = out + ((int64_t)mt * TM + rh * TMP + 4 * wave) * p.N + nseg0 + ((lane >> 4) * p.N + 4 * (lane & 15));
#pragma unroll
      for (int b = 0; b < PER_WAVE; b += BATCH) {
        f32x4 v[BATCH];
#pragma unroll
        for (int e = 0; e < BATCH; ++e) {
          const int s = b + e;
          const int t = 4 * (wave + NWAVE * (s >> 1)) + (lane >> 4);
          const int c = 16 * (s & 1) + (lane & 15);
          v[e] = *reinterpret_cast<const f32x4*>(stg + t * 512 + 16 * (c ^ (t & 31)));
        }
        // the whole batch of LDS reads is issued before the first store waits for its data
#pragma unroll
        for (int e = 0; e < BATCH; ++e) asm volatile("" : "+v"(v[e]));
#pragma unroll
        for (int e = 0; e < BATCH; ++e) {
          const int s = b + e;
          const int dr = 4 * NWAVE * (s >> 1);   // rows past the wave's first quad
          if (4 * wave + dr < rows_left && seg_in[s & 1])
            *reinterpret_cast<f32x4*>(base + (int64_t)dr * p.N + SEG1 * (s & 1)) = v[e];
        }
      }
    }
  } else {
    // bf16 results leave through LDS.  The accumulators, rounded to bf16, go to an LDS copy of the
    // tile (tile row t, 16-byte chunk c = 8 columns, at t*512 + 16*(c ^ (t & 31))); then each thread
    // moves whole chunks, so a wavefront's global accesses cover two (dual: four) contiguous row
    // segments instead of 16 bytes in each of 32 rows.  Dual mode keeps the gate columns of a row in
    // chunks 0..15 and the up columns in chunks 16..31.
    static_assert(TMP * TN * 2 <= (EARLY ? 2 : NSTAGE) * STAGE, "a row half (EARLY) or the bf16 tile fits");
    // the dual fwd and dW products have two outputs side by side in their tile; the dual dX
    // product sums both contractions into one output
    constexpr bool SPLIT = DUAL && (KIND != KIND_DX || F8);       // two outputs side by side in the tile
    constexpr bool ACC_SPLIT = DUAL && (KIND != KIND_DX);         // ... within each wave's columns
    // output rows of the tile: fwd/dX the permuted rows row_lo .. row_hi-1; dW rows mt*TM .. of
    // dB[g] (at most K)
    int64_t obase = 0;
    if constexpr (IS_DW) {
      obase = (int64_t)g * p.K * p.N;
      row_lo = (int64_t)mt * TM;
      row_hi = p.K;
    }
    for (int rh = 0; rh < RH; ++rh) {
    __syncthreads();   // every wave is done with the ring (EARLY, second row half: with the first's reads)
    const int64_t row_lo_p = row_lo + rh * TMP;   // first row of this pass
    if (!EARLY || wm == rh) {   // uniform per wavefront
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      char* trow = stg + (wm * WTM - rh * TMP + 32 * i + l32) * 512;   // (t & 31) == l32
#pragma unroll
      for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          int c;
          if constexpr (ACC_SPLIT) c = (j >= NB / 2 ? 16 : 0) + (wn * (WTN / 2) + 32 * (j % (NB / 2)) + 8 * q) / 8;
          else c = (wn * WTN + 32 * j + 8 * q) / 8;
          uint2 v;
          if constexpr (FSCALE) {
            // fp32 row and column scales; rows past the group and columns past the output (not
            // stored) read clamped scales
            int64_t r = row_lo + wm * WTM + 32 * i + l32;
            if (r > row_hi - 1) r = row_hi - 1;
            int64_t n = (int64_t)nt * TN + wn * WTN + 32 * j + 8 * q + col_in;
            if (n > p.K - 4) n = p.K - 4;
            const float sr = p.a_scale[r];
            const f32x4 sc = *reinterpret_cast<const f32x4*>(p.w_scale + (int64_t)g * p.K + n);
            v.x = pack_bf16(acc[i][j][4 * q] * sr * sc[0], acc[i][j][4 * q + 1] * sr * sc[1]);
            v.y = pack_bf16(acc[i][j][4 * q + 2] * sr * sc[2], acc[i][j][4 * q + 3] * sr * sc[3]);
          } else {
            v.x = pack_bf16(acc[i][j][4 * q], acc[i][j][4 * q + 1]);
            v.y = pack_bf16(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
          }
          *reinterpret_cast<uint2*>(trow + 16 * (c ^ l32) + 8 * fh) = v;
        }
    }
    }
    __syncthreads();
    constexpr int NT = 64 * NWAVE;
    auto chunk = [&](int t, int c) { return *reinterpret_cast<const u32x4*>(stg + t * 512 + 16 * (c ^ (t & 31))); };
    if constexpr (SPLIT) {
      // FWD gate/up and FP8 interleaved gate/up (+ SwiGLU): thread -> gate chunk c and up chunk 16 + c of rows t, t + NT/16, ...
      const int c = tid & 15;
      // width of each output (the FP8 interleaved gate/up product is dX-shaped: its 2F output
      // columns are p.K)
      const int64_t Wo = (F8 && KIND == KIND_DX) ? p.K / 2 : p.N;
      const int64_t n = (int64_t)nt * (TN / 2) + 8 * c;
      if (n < Wo) {
        uint16_t* c1 = static_cast<uint16_t*>(p.out) + obase + n;
        uint16_t* c2 = static_cast<uint16_t*>(p.out2) + obase + n;
        // passes of NT/16 rows, UB passes' LDS reads issued ahead of their stores
        constexpr int RPP = NT / 16, PASSES = TMP / RPP, UB = 4;
        static_assert(PASSES % UB == 0, "batches of passes");
#pragma unroll
        for (int b = 0; b < PASSES; b += UB) {
          if (row_lo_p + b * RPP >= row_hi) break;   // uniform: no row of the batch is an output row
          u32x4 vg[UB], vu[UB];
#pragma unroll
          for (int u = 0; u < UB; ++u) {
            const int t = (tid >> 4) + (b + u) * RPP;
            vg[u] = chunk(t, c);
            vu[u] = chunk(t, 16 + c);
          }
#pragma unroll
          for (int u = 0; u < UB; ++u) asm volatile("" : "+v"(vg[u]), "+v"(vu[u]));
#pragma unroll
          for (int u = 0; u < UB; ++u) {
            const int64_t r = row_lo_p + (tid >> 4) + (b + u) * RPP;
            if (r < row_hi) {
              if constexpr (IS_DW) {   // bf16 weight gradients: not read again in the step
                __builtin_nontemporal_store(vg[u], reinterpret_cast<u32x4*>(c1 + r * Wo));
                __builtin_nontemporal_store(vu[u], reinterpret_cast<u32x4*>(c2 + r * Wo));
              } else {
                *reinterpret_cast<u32x4*>(c1 + r * Wo) = vg[u];
                *reinterpret_cast<u32x4*>(c2 + r * Wo) = vu[u];
              }
              if constexpr (ACT) {
                u32x4 va;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  va[e] = pack_bf16(silu_f32(bf16_lo(vg[u][e])) * bf16_lo(vu[u][e]),
                                    silu_f32(bf16_hi(vg[u][e])) * bf16_hi(vu[u][e]));
                *reinterpret_cast<u32x4*>(p.act + r * Wo + n) = va;
              }
            }
          }
        }
      }
    } else {
      // thread -> chunk c of rows t, t + NT/32, ...
      const int64_t W = (KIND == KIND_DX) ? p.K : p.N;   // output row length
      const int c = tid & 31;
      const int64_t n = (int64_t)nt * TN + 8 * c;
      if (n < W) {
        if constexpr (KIND == KIND_DX && ACT) {
          // SwiGLU backward on the bf16-rounded dA (what moe_swiglu_bwd would read back); the
          // H_gate/H_up chunks of U rows are loaded ahead of their use (rows clamped in range), as
          // streaming loads: H is read this once in the step (1.7% shorter than plain loads)
          constexpr int RPP = NT / 32, U = (TMP / RPP) < 4 ? (TMP / RPP) : 4;
          uint16_t* og = static_cast<uint16_t*>(p.out) + n;
          uint16_t* ou = static_cast<uint16_t*>(p.out2) + n;
          for (int t0 = tid >> 5; t0 < TMP; t0 += U * RPP) {
            if (row_lo_p + t0 >= row_hi) break;
            u32x4 gv[U], uv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
              int64_t r = row_lo_p + t0 + u * RPP;
              if (r > row_hi - 1) r = row_hi - 1;
              gv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p.hg + r * W + n));
              uv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p.hu + r * W + n));
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
              const int t = t0 + u * RPP;
              const int64_t r = row_lo_p + t;
              if (r < row_hi) {
                const u32x4 dv = chunk(t, c);
                u32x4 vg, vu;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  float a0, a1, b0, b1;
                  swiglu_bwd1(bf16_lo(gv[u][e]), bf16_lo(uv[u][e]), bf16_lo(dv[e]), a0, b0);
                  swiglu_bwd1(bf16_hi(gv[u][e]), bf16_hi(uv[u][e]), bf16_hi(dv[e]), a1, b1);
                  vg[e] = pack_bf16(a0, a1);
                  vu[e] = pack_bf16(b0, b1);
                }
                *reinterpret_cast<u32x4*>(og + r * W) = vg;
                *reinterpret_cast<u32x4*>(ou + r * W) = vu;
              }
            }
          }
        } else {
          uint16_t* dst = static_cast<uint16_t*>(p.out) + obase + n;
          constexpr int RPP = NT / 32, PASSES = TMP / RPP, UB = 8;
          static_assert(PASSES % UB == 0, "batches of passes");
          // fused combine: the rows are stored agent-coherent (sc1: through to memory), since the
          // tile that completes a token's combine may run on another XCD
          auto store_rows = [&](auto coherent) {
            const __amdgpu_buffer_rsrc_t ys = __builtin_amdgcn_make_buffer_rsrc(dst + row_lo_p * W, 0, TMP * (int)W * 2,
                                                                                0x00020000);
#pragma unroll
            for (int b = 0; b < PASSES; b += UB) {
              if (row_lo_p + b * RPP >= row_hi) break;   // uniform
              u32x4 v[UB];
#pragma unroll
              for (int u = 0; u < UB; ++u) v[u] = chunk((tid >> 5) + (b + u) * RPP, c);
#pragma unroll
              for (int u = 0; u < UB; ++u) asm volatile("" : "+v"(v[u]));
#pragma unroll
              for (int u = 0; u < UB; ++u) {
                const int t = (tid >> 5) + (b + u) * RPP;
                const int64_t r = row_lo_p + t;
                if (r < row_hi) {
                  if constexpr (decltype(coherent)::value)
                    __builtin_amdgcn_raw_buffer_store_b128(v[u], ys, (int)(t * W * 2), 0, CP_SC1);
                  else if constexpr (IS_DW)   // bf16 weight gradients: not read again in the step
                    __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(dst + r * W));
                  else
                    *reinterpret_cast<u32x4*>(dst + r * W) = v[u];
                }
              }
            }
          };
          if (FUSE_COMBINE && p.comb_cnt != nullptr) store_rows(std::true_type{});
          else store_rows(std::false_type{});
        }
      }
      if constexpr (FUSE_COMBINE) {
        if (p.comb_cnt != nullptr) {   // uniform
          // The weighted combine (section 5.4's step E) fused: once this tile's Y_perm rows have
          // all been stored, each of its rows counts one arrival for its (token, column tile); the
          // tile whose arrival brings a pair's count to k sums that token's k rows of these 256
          // columns in slot order (read agent-coherent), adds the shared output and stores Y --
          // the arithmetic of moe_unpermute_combine, so Y is bitwise the two-call result.  No
          // tile waits for another.
          __shared__ int s_last[TM];
          __shared__ int s_nlast;
          wait_vm<0>();
          if (tid == 0) s_nlast = 0;
          __syncthreads();
          for (int t = tid; t < TM; t += NT) {
            const int64_t r = row_lo + t;
            if (r < row_hi) {
              const int tok = p.comb_tor[r];
              const int old = __hip_atomic_fetch_add(p.comb_cnt + (int64_t)tok * p.n_tiles + nt, 1,
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              if (old == p.comb_k - 1) s_last[atomicAdd(&s_nlast, 1)] = tok;
            }
          }
          __syncthreads();
          const int nl = s_nlast;
          if (n < W) {
            const __amdgpu_buffer_rsrc_t yp =
                __builtin_amdgcn_make_buffer_rsrc(static_cast<uint16_t*>(p.out), 0, (int)(p.R * W * 2), 0x00020000);
            for (int i = tid >> 5; i < nl; i += NT / 32) {
              const int64_t tok = s_last[i];
              float acc[8];
#pragma unroll
              for (int e = 0; e < 8; ++e) acc[e] = 0.f;
              for (int j = 0; j < p.comb_k; ++j) {
                const int64_t rj = p.comb_ros[tok * p.comb_k + j];
                const float wj = p.comb_w[tok * p.comb_k + j];
                const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                              yp, (int)((rj * W + n) * 2), 0, CP_SC1));
                float f[8];
                unpack8(v, f);
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[e] += wj * f[e];
              }
              if (p.comb_add) {
                float f[8];
                unpack8(*reinterpret_cast<const u32x4*>(p.comb_add + tok * W + n), f);
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[e] += f[e];
              }
              *reinterpret_cast<u32x4*>(p.comb_y + tok * W + n) = pack8(acc);
            }
          }
        }
      }
    }
    }   // row halves
  }
  };

  // ---------------- tile loop -----------------------------------------------------------------
  // Given a split workspace, only the full rounds of tiles (a round: one tile per resident
  // workgroup) run this way; the tiles of the last, partial round are split along the
  // contraction (below).
  int normal_end = ntiles_all, tail_first = ntiles_all, S = 1;
  {
    if (p.split_part != nullptr) {
      const int slots = PERSIST ? (int)gridDim.x : p.split_slots;
      const int full = (ntiles_all / slots) * slots;
      const int tail = ntiles_all - full;
      if (tail > 0) {
        // pieces of a tile: as many as the idle slots allow, at most split_max, and each at least
        // split_min_steps long (short pieces cost more in partial-tile traffic than they save)
        int64_t clen;
        if constexpr (KIND == KIND_FWD) clen = p.K;
        else if constexpr (IS_DW) clen = (KIND == KIND_DW && p.G == 1) ? s_off[1] - s_off[0] : 0;   // one group
        else clen = (DUAL && !F8) ? 2 * p.N : p.N;
        const int csteps = (int)((clen + BKE - 1) / BKE);
        int sp = slots / tail;
        if (sp > p.split_max) sp = p.split_max;
        if (sp > csteps / p.split_min_steps) sp = csteps / p.split_min_steps;
        if (sp > 1) {
          S = sp;
          normal_end = full;
          tail_first = full;
        }
      }
    }
  }
  int it = blockIdx.x;
  int g, mt, nt, row_lo, row_hi;
  if (it < normal_end) {   // uniform over the workgroup
    map_tile(it, g, mt, nt, row_lo, row_hi);
    setup(g, mt, nt, row_lo, row_hi);
    zero_acc();
    prefill();
    if constexpr (!PERSIST) {
      // one tile per workgroup; the hardware dispatcher hands the next tile to whichever CU frees
      main_loop();
      epilogue(g, mt, nt, row_lo, row_hi);
      return;
    }
    // dW: tiles differ in length with their group's size, so instead of walking a fixed list the
    // workgroup claims its next tile from its XCD's queue (dispatch indices x, x + 8, ... in claim
    // order after the grid's own first round), issuing the claim as this tile's main loop starts
    // so that its round trip is hidden.  dX walks b, b + gridDim.x, ...
    __shared__ int s_next;
    for (;;) {
      int claim = 0;
      if constexpr (IS_DW) {
        if (tid == 0)
          claim = __hip_atomic_fetch_add(p.tile_queue + (blockIdx.x & 7), 1, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
      }
      main_loop();
      if constexpr (IS_DW) {
        // the claim's result is first needed here (kept opaque until now, so that nothing derived
        // from it, and hence no wait for it, is placed before the main loop)
        asm volatile("" : "+v"(claim));
        if (tid == 0) {
          const int x = blockIdx.x & 7;
          s_next = 8 * (claim + (((int)gridDim.x - x + 7) >> 3)) + x;
        }
      }
      int next = it + (int)gridDim.x;
      int g2 = 0, mt2 = 0, nt2 = 0, lo2 = 0, hi2 = 0;
      if constexpr (EARLY) {
        // The next tile's first two stages load into slots 0 and 1 while this tile's epilogue
        // stages its results through slots 2 and 3; its stages 2 and 3 follow the epilogue.  The
        // epilogue's stores then sit between stages 1 and 2 in the in-order vector-memory count,
        // so the main loop's count-based waits still cover every stage they wait for.
        static_assert(NSTAGE == 4 && PREFILL == 4 && WTM == TM / 2, "two slots each way, one row half per wave row");
        __syncthreads();   // s_next is visible, and every wave is done with this tile's stages
        next = __builtin_amdgcn_readfirstlane(s_next);
        const bool more = next < normal_end;   // uniform
        if (more) {
          map_tile(next, g2, mt2, nt2, lo2, hi2);
          setup(g2, mt2, nt2, lo2, hi2);
          if (nsteps > 0) {
            issue(0);
            issue(1);
          }
        }
        epilogue(g, mt, nt, row_lo, row_hi);
        if (!more) break;
        __syncthreads();   // every staged chunk has been read
        if (nsteps > 0) {
          issue(2);
          issue(3);
        }
      } else {
        epilogue(g, mt, nt, row_lo, row_hi);   // stages the tile through the ring (barriers first)
        if constexpr (IS_DW) next = __builtin_amdgcn_readfirstlane(s_next);
        const bool more = next < normal_end;   // uniform
        if (more) {
          __syncthreads();   // every staged chunk has been read
          map_tile(next, g2, mt2, nt2, lo2, hi2);
          setup(g2, mt2, nt2, lo2, hi2);
          prefill();
        }
        if (!more) break;
      }
      it = next;
      g = g2; mt = mt2; nt = nt2; row_lo = lo2; row_hi = hi2;
      zero_acc();
    }
  }

  // ---------------- split tail ------------------------------------------------------------------
  // Unit u (one per workgroup: a persistent workgroup after its full rounds, else one of the
  // workgroups past the full rounds' tiles, which the dispatcher starts as the last round's CUs
  // free) computes piece q = u % S of tail tile u / S: contraction steps [q*n/S, (q+1)*n/S).  It
  // stores its fp32 partial tile to the workspace and counts itself in; the last of the S pieces
  // to arrive adds the S partials in piece order (a fixed order: the result does not depend on
  // which piece arrives last) and runs the tile's epilogue.  Nothing waits for another workgroup.
  {
    __shared__ int s_arrived;
    const int units = (ntiles_all - tail_first) * S;
    const int u = PERSIST ? (int)blockIdx.x : (int)blockIdx.x - tail_first;
    if (S > 1 && u >= 0 && u < units) {
      const int tl = u / S, q = u - tl * S;
      __syncthreads();   // the ring and the staging area are free (the last normal tile is done)
      map_tile(tail_first + tl, g, mt, nt, row_lo, row_hi);
      setup(g, mt, nt, row_lo, row_hi);
      const int total = nsteps;
      const int sb = (int)((int64_t)total * q / S), se = (int)((int64_t)total * (q + 1) / S);
      s_base = sb;
      nsteps = se - sb;
      zero_acc();
      prefill();
      main_loop();
      constexpr int NT = 64 * NWAVE;
      constexpr int SLOT = NT * 4;   // floats per float4 slot across the workgroup
      auto part_of = [&](int unit) { return p.split_part + (int64_t)unit * (TM * TN); };
      // The partials cross XCDs (separate L2s).  They are written and read with agent-coherent
      // (sc1) buffer accesses, which write through / bypass the non-coherent caches, so the only
      // ordering needed is: every store of the piece has completed (vmcnt 0, then the barrier)
      // before the piece is counted, and the reads start after the count was seen.  A device-scope
      // fence would do the same by writing back and invalidating the whole L2 of the XCD, which
      // measured 3-4% slower on the whole product.
      constexpr int SC1 = CP_SC1;
      auto off_of = [&](int i, int j, int q4) { return (((i * NB + j) * 4 + q4) * SLOT + tid * 4) * 4; };
      {
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(part_of(u), 0, TM * TN * 4, 0x00020000);
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
              const f32x4 v = {acc[i][j][4 * q4], acc[i][j][4 * q4 + 1], acc[i][j][4 * q4 + 2], acc[i][j][4 * q4 + 3]};
              __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs, off_of(i, j, q4), 0, SC1);
            }
      }
      wait_vm<0>();
      __syncthreads();
      if (tid == 0)
        s_arrived = __hip_atomic_fetch_add(p.split_cnt + tl, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __syncthreads();
      if (s_arrived == S - 1) {   // uniform: this workgroup completes the tile
        zero_acc();
        for (int r = 0; r < S; ++r) {
          const __amdgpu_buffer_rsrc_t rs =
              __builtin_amdgcn_make_buffer_rsrc(part_of(tl * S + r), 0, TM * TN * 4, 0x00020000);
#pragma unroll
          for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j)
#pragma unroll
              for (int q4 = 0; q4 < 4; ++q4) {
                const f32x4 v =
                    __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off_of(i, j, q4), 0, SC1));
                acc[i][j][4 * q4] += v[0];
                acc[i][j][4 * q4 + 1] += v[1];
                acc[i][j][4 * q4 + 2] += v[2];
                acc[i][j][4 * q4 + 3] += v[3];
              }
        }
        epilogue(g, mt, nt, row_lo, row_hi);
      }
    }
  }
}

// Tile shape and schedule per product, chosen by measurement on the Mixtral-shaped layer: every
// product uses 256x256 tiles with a 4-slot ring (128-row tiles, which would pad ragged groups
// less, measured 10-20% slower: they need 1.5x the LDS and DMA traffic per MFMA).  dX (both
// operands read 16 bytes per lane) runs 8 wavefronts in the ping-pong schedule (the single-group
// schedule below measured 6-8% slower for it); fwd and dW, whose transposing LDS reads make a
// memory phase longer than a compute phase, run 4 wavefronts (one per SIMD, 128x128 each) in the
// single-group schedule.  dX walks its tiles persistently (1-3% faster than one workgroup per
// tile); fwd keeps one workgroup per tile (a persistent fwd, walking or claiming its tiles,
// measured 1% and more slower: it spills registers around its epilogue).  dW, whose tiles differ
// in length with the group sizes, runs one workgroup per tile, which the hardware dispatcher
// balances (a static walk of the largest-first order measured 7% slower on the Zipf-skewed
// layer), or, given claim counters, as a persistent grid whose workgroups claim their tiles
// (launch<..., QUEUE>): 2-13% faster than one per tile.
template <int KIND> struct Cfg {
  static constexpr bool PP = (KIND == KIND_DX || KIND == KIND_DWT);   // both operands read directly
  static constexpr int TM = 256;
  static constexpr int WM = PP ? 4 : 2, WN = 2;
  static constexpr int NS = 4;
  static constexpr int WPE = 1;
  static constexpr bool PERSIST = (KIND == KIND_DX);
};

// Split-tail workspace: 256 arrival counters, then one fp32 256x256 partial tile per unit (at most
// one unit per resident workgroup, i.e. per CU, which attach_split bounds by 256).
constexpr int SPLIT_UNITS = 256, SPLIT_MAX = 8, SPLIT_MIN_STEPS = 64;
constexpr size_t SPLIT_CNT_BYTES = SPLIT_UNITS * sizeof(int);
constexpr size_t SPLIT_BYTES = SPLIT_CNT_BYTES + (size_t)SPLIT_UNITS * 256 * TN * sizeof(float);

// QUEUE (dW): a persistent grid whose workgroups claim tiles from p.tile_queue.
template <int KIND, bool DUAL, bool ACT, bool OUT16 = false, bool GATHER = false, bool F8 = false,
          bool QUEUE = false, bool MX = false>
moe_status launch(const GemmParams& p, int64_t tiles_bound, hipStream_t stream, const char* name) {
  if (tiles_bound == 0) return MOE_SUCCESS;
  if (tiles_bound >= ((int64_t)1 << 31) - SPLIT_UNITS) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: too many tiles", name);
  static_assert(!QUEUE || KIND == KIND_DW || KIND == KIND_DWT, "tile queues: the dW products");
  using C = Cfg<KIND>;
  constexpr bool PERSIST = C::PERSIST || QUEUE;
  // persistent grid: one workgroup per CU slot (a multiple of 8, one share per XCD), or one per
  // tile when there are fewer tiles; otherwise one workgroup per (bound on the) tile count
  unsigned grid = (unsigned)tiles_bound;
  if constexpr (PERSIST) {
    unsigned slots = (unsigned)device_cu_count() * C::WPE;
    if (slots > 8) slots &= ~7u;
    if (grid > slots) {
      grid = slots;
    } else if (p.split_part != nullptr) {
      // fewer tiles than slots: every slot runs when the contraction is long enough for the tiles
      // to be split into pieces (single-group dW: the group's rows; dX: N or 2N)
      const int64_t clen = (KIND == KIND_DW) ? (p.G == 1 ? p.R : 0) : ((DUAL && !F8) ? 2 * p.N : p.N);
      if (clen / (F8 ? 2 * BK : BK) >= 2 * SPLIT_MIN_STEPS) grid = slots;
    }
  } else if (p.split_part != nullptr) {
    grid += SPLIT_UNITS;   // the split units run past the full rounds' tiles (idle ones exit)
  }
  static_assert(!GATHER || KIND == KIND_FWD, "gathered rows feed the forward product only");
  grouped_gemm_kernel<KIND, DUAL, ACT, C::TM, C::WM, C::WN, C::NS, C::PP, C::WPE, PERSIST, OUT16, GATHER, F8, MX>
      <<<grid, 64 * C::WM * C::WN, 0, stream>>>(p);
  return check_launch(name);
}

bool bad_ptr(const void* q) { return q != nullptr && !aligned16(q); }


__global__ void zero_i32_kernel(int* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// Attach a split workspace to p (zeroing its counters on `stream`); NULL leaves p unsplit.
moe_status attach_split(GemmParams& p, void* ws, size_t ws_bytes, const char* fn, hipStream_t stream) {
  if (ws == nullptr) return MOE_SUCCESS;
  if (ws_bytes < SPLIT_BYTES || !aligned16(ws))
    return fail(MOE_ERROR_WORKSPACE, "%s: a 16-byte aligned workspace of %zu bytes is needed", fn, SPLIT_BYTES);
  const int cus = device_cu_count();
  if (cus > SPLIT_UNITS) return MOE_SUCCESS;   // more slots than partial tiles: no split
  p.split_cnt = static_cast<int*>(ws);
  p.split_slots = cus;   // one workgroup per CU (the LDS ring admits no second)
  p.split_part = reinterpret_cast<float*>(static_cast<char*>(ws) + SPLIT_CNT_BYTES);
  p.split_max = SPLIT_MAX;
  p.split_min_steps = SPLIT_MIN_STEPS;
  zero_i32_kernel<<<1, SPLIT_UNITS, 0, stream>>>(p.split_cnt, SPLIT_UNITS);
  return check_launch(fn);
}

}  // namespace
}  // namespace moe

using namespace moe;

namespace moe {
namespace {
// The combine fused into the single-output forward product (moe_grouped_gemm_fwd_combine).
struct FusedCombine {
  int* cnt;
  const float* w;
  const int32_t* row_of_slot;
  const int32_t* token_of_row;
  const moe_bf16* add;
  moe_bf16* y;
  int64_t T;
  int k;
};

moe_status grouped_gemm_fwd_impl(const moe_bf16* A, const moe_bf16* B, const moe_bf16* B2, const int32_t* offsets,
                                 int32_t G, int64_t R, int64_t K, int64_t N, moe_bf16* C, moe_bf16* C2,
                                 moe_bf16* act, void* ws, size_t ws_bytes, hipStream_t stream,
                                 const int32_t* gather = nullptr, int64_t gather_rows = 0,
                                 const FusedCombine* fc = nullptr) {
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
  p.gather = gather; p.gather_rows = gather_rows;
  constexpr int TM = Cfg<KIND_FWD>::TM;
  p.mt_bound = (int)((R + TM - 1) / TM + G);
  const int cols_per_tile = B2 ? TN / 2 : TN;
  p.n_tiles = (int)((N + cols_per_tile - 1) / cols_per_tile);
  const int64_t tiles = (int64_t)p.mt_bound * p.n_tiles;   // upper bound; exact count on device
  const moe_status st = attach_split(p, ws, ws_bytes, "moe_grouped_gemm_fwd", stream);
  if (st != MOE_SUCCESS) return st;
  if (fc) {
    p.comb_cnt = fc->cnt; p.comb_w = fc->w; p.comb_ros = fc->row_of_slot; p.comb_tor = fc->token_of_row;
    p.comb_add = fc->add; p.comb_y = fc->y; p.comb_k = fc->k;
    const int64_t ncnt = fc->T * p.n_tiles;
    zero_i32_kernel<<<(unsigned)((ncnt + 255) / 256), 256, 0, stream>>>(fc->cnt, (int)ncnt);
    const moe_status zs = check_launch("moe_grouped_gemm_fwd_combine");
    if (zs != MOE_SUCCESS) return zs;
    return launch<KIND_FWD, false, false>(p, tiles, stream, "grouped_gemm_fwd(combine)");
  }
  if (gather) {
    if (B2 && act) return launch<KIND_FWD, true, true, false, true>(p, tiles, stream, "grouped_gemm_fwd(gather,dual,swiglu)");
    if (B2) return launch<KIND_FWD, true, false, false, true>(p, tiles, stream, "grouped_gemm_fwd(gather,dual)");
    return launch<KIND_FWD, false, false, false, true>(p, tiles, stream, "grouped_gemm_fwd(gather)");
  }
  if (B2 && act) return launch<KIND_FWD, true, true>(p, tiles, stream, "grouped_gemm_fwd(dual,swiglu)");
  if (B2) return launch<KIND_FWD, true, false>(p, tiles, stream, "grouped_gemm_fwd(dual)");
  return launch<KIND_FWD, false, false>(p, tiles, stream, "grouped_gemm_fwd");
}
}  // namespace
}  // namespace moe

extern "C" moe_status moe_grouped_gemm_fwd(const moe_bf16* A, const moe_bf16* B, const moe_bf16* B2,
                                           const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                           int64_t N, moe_bf16* C, moe_bf16* C2, moe_bf16* act,
                                           hipStream_t stream) {
  return grouped_gemm_fwd_impl(A, B, B2, offsets, G, R, K, N, C, C2, act, nullptr, 0, stream);
}

extern "C" size_t moe_grouped_gemm_fwd_combine_workspace_bytes(int64_t T, int64_t N) {
  return T <= 0 || N <= 0 ? 0 : (size_t)T * (size_t)((N + TN - 1) / TN) * sizeof(int);
}

extern "C" moe_status moe_grouped_gemm_fwd_combine(const moe_bf16* A, const moe_bf16* B, const int32_t* offsets,
                                                   int32_t G, int64_t R, int64_t K, int64_t N, const float* topk_w,
                                                   const int32_t* row_of_slot, const int32_t* token_of_row,
                                                   int64_t T, int32_t k, const moe_bf16* add, moe_bf16* y_perm,
                                                   moe_bf16* y, void* count_workspace, size_t count_workspace_bytes,
                                                   void* split_workspace, size_t split_workspace_bytes,
                                                   hipStream_t stream) {
  const char* fn = "moe_grouped_gemm_fwd_combine";
  if (T < 0 || k < 1 || R != T * (int64_t)k)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: need k >= 1 and R == T * k", fn);
  if (R * N * 2 >= ((int64_t)1 << 31) || T * ((N + TN - 1) / TN) >= ((int64_t)1 << 31))
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: Y_perm must be < 2 GiB", fn);
  if (R == 0) return MOE_SUCCESS;
  if (!topk_w || !row_of_slot || !token_of_row || !y || !count_workspace)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (bad_ptr(add) || bad_ptr(y) || (reinterpret_cast<uintptr_t>(count_workspace) & 3))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: add and y must be 16-byte, the counters 4-byte aligned", fn);
  if (count_workspace_bytes < moe_grouped_gemm_fwd_combine_workspace_bytes(T, N))
    return fail(MOE_ERROR_WORKSPACE, "%s: the counters need %zu bytes", fn,
                moe_grouped_gemm_fwd_combine_workspace_bytes(T, N));
  const FusedCombine fc{static_cast<int*>(count_workspace), topk_w, row_of_slot, token_of_row, add, y, T, k};
  return grouped_gemm_fwd_impl(A, B, nullptr, offsets, G, R, K, N, y_perm, nullptr, nullptr, split_workspace,
                               split_workspace_bytes, stream, nullptr, 0, &fc);
}

extern "C" moe_status moe_grouped_gemm_fwd_gather(const moe_bf16* X, int64_t T, const int32_t* row_src,
                                                  const moe_bf16* B, const moe_bf16* B2, const int32_t* offsets,
                                                  int32_t G, int64_t R, int64_t K, int64_t N, moe_bf16* C,
                                                  moe_bf16* C2, moe_bf16* act, void* workspace,
                                                  size_t workspace_bytes, hipStream_t stream) {
  const char* fn = "moe_grouped_gemm_fwd_gather";
  if (T < 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (R > 0 && (!row_src || T == 0)) return fail(MOE_ERROR_INVALID_VALUE, "%s: row_src is NULL or T == 0", fn);
  if (T * K * 2 >= ((int64_t)1 << 31))
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: the source X must be < 2 GiB", fn);
  return grouped_gemm_fwd_impl(X, B, B2, offsets, G, R, K, N, C, C2, act, workspace, workspace_bytes, stream,
                               row_src, T);
}

extern "C" moe_status moe_grouped_gemm_fwd_split(const moe_bf16* A, const moe_bf16* B, const moe_bf16* B2,
                                                 const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                                 int64_t N, moe_bf16* C, moe_bf16* C2, moe_bf16* act,
                                                 void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!workspace) return fail(MOE_ERROR_WORKSPACE, "moe_grouped_gemm_fwd_split: workspace is NULL");
  return grouped_gemm_fwd_impl(A, B, B2, offsets, G, R, K, N, C, C2, act, workspace, workspace_bytes, stream);
}

namespace moe {
namespace {
moe_status grouped_gemm_dx_impl(const moe_bf16* dC, const moe_bf16* B, const moe_bf16* dC2, const moe_bf16* B2,
                                const int32_t* offsets, int32_t G, int64_t R, int64_t K, int64_t N, moe_bf16* dA,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dx: need 1 <= G <= 256");
  if (R < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: bad size");
  if (K % 64 || N % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dx: K and N must be multiples of 64");
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dx: R >= 2^31");
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: offsets is NULL");
  if ((dC2 == nullptr) != (B2 == nullptr))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: dC2 and B2 must both be set or both NULL");
  if (K * N * 2 >= ((int64_t)1 << 31))
    return fail(MOE_ERROR_NOT_SUPPORTED, "moe_grouped_gemm_dx: one group's B must be < 2 GiB");
  if (R == 0) return MOE_SUCCESS;
  if (!dC || !B || !dA) return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: NULL pointer");
  if (bad_ptr(dC) || bad_ptr(B) || bad_ptr(dC2) || bad_ptr(B2) || bad_ptr(dA))
    return fail(MOE_ERROR_INVALID_VALUE, "moe_grouped_gemm_dx: pointers must be 16-byte aligned");
  GemmParams p{};
  p.a = dC; p.a2 = dC2; p.b = B; p.b2 = B2; p.offsets = offsets; p.out = dA;
  p.G = G; p.R = R; p.K = K; p.N = N;
  constexpr int TM = Cfg<KIND_DX>::TM;
  p.mt_bound = (int)((R + TM - 1) / TM + G);
  p.n_tiles = (int)((K + TN - 1) / TN);
  const int64_t tiles = (int64_t)p.mt_bound * p.n_tiles;   // upper bound; exact count on device
  const moe_status st = attach_split(p, ws, ws_bytes, "moe_grouped_gemm_dx", stream);
  if (st != MOE_SUCCESS) return st;
  if (dC2) return launch<KIND_DX, true, false>(p, tiles, stream, "grouped_gemm_dx(dual)");
  return launch<KIND_DX, false, false>(p, tiles, stream, "grouped_gemm_dx");
}
}  // namespace
}  // namespace moe

extern "C" moe_status moe_grouped_gemm_dx(const moe_bf16* dC, const moe_bf16* B, const moe_bf16* dC2,
                                          const moe_bf16* B2, const int32_t* offsets, int32_t G,
                                          int64_t R, int64_t K, int64_t N, moe_bf16* dA,
                                          hipStream_t stream) {
  return grouped_gemm_dx_impl(dC, B, dC2, B2, offsets, G, R, K, N, dA, nullptr, 0, stream);
}

extern "C" size_t moe_grouped_gemm_split_workspace_bytes(void) { return SPLIT_BYTES; }

namespace moe {
namespace {
// The E4M3 products, all dX-shaped (rows of A against rows of Wt[g], both read along the
// contraction Kc; Nout output columns): plain, the interleaved gate/up pair (+ SwiGLU), and the
// dX-down product with the SwiGLU backward in its epilogue.  Scales: fp32 per row / per output
// channel, or (mx) E8M0 bytes per 32 contraction elements of every row of either operand.
enum F8Op { F8_PLAIN, F8_GATE_UP, F8_SWIGLU_BWD };

template <bool MX>
moe_status f8_product(const char* fn, F8Op op, const uint8_t* A, const void* a_scale, const uint8_t* Wt,
                      const void* w_scale, const int32_t* offsets, int32_t G, int64_t R, int64_t Kc, int64_t Nout,
                      moe_bf16* out, moe_bf16* out2, moe_bf16* act, const moe_bf16* hg, const moe_bf16* hu,
                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: need 1 <= G <= 256", fn);
  if (R < 0 || Kc <= 0 || Nout <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (op == F8_GATE_UP) {
    if (Kc % 64 || Nout % 256) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K must be a multiple of 64, F of 128", fn);
  } else if (Kc % 64 || Nout % 64) {
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K and N must be multiples of 64", fn);
  }
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: R >= 2^31", fn);
  if (Nout * Kc >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: one group's weight must be < 2 GiB", fn);
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "%s: offsets is NULL", fn);
  if (R == 0) return MOE_SUCCESS;
  if (!A || !a_scale || !Wt || !w_scale || !out) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if ((op == F8_GATE_UP && !out2) || (op == F8_SWIGLU_BWD && (!out2 || !hg || !hu)))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (bad_ptr(A) || bad_ptr(Wt) || bad_ptr(out) || bad_ptr(out2) || bad_ptr(act) || bad_ptr(hg) || bad_ptr(hu))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: operand and output pointers must be 16-byte aligned", fn);
  if ((reinterpret_cast<uintptr_t>(a_scale) & 3) || (MX ? (reinterpret_cast<uintptr_t>(w_scale) & 3) : bad_ptr(w_scale)))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: a_scale must be 4-byte, w_scale %s aligned", fn, MX ? "4-byte" : "16-byte");
  GemmParams p{};
  p.a = reinterpret_cast<const uint16_t*>(A);
  p.b = reinterpret_cast<const uint16_t*>(Wt);
  p.offsets = offsets; p.out = out; p.out2 = out2; p.act = act; p.hg = hg; p.hu = hu;
  if constexpr (MX) {
    p.a_mx = static_cast<const uint8_t*>(a_scale);
    p.w_mx = static_cast<const uint8_t*>(w_scale);
    p.mx_a_step = R * 4;
    p.mx_w_step = (int64_t)G * Nout * 4;
  } else {
    p.a_scale = static_cast<const float*>(a_scale);
    p.w_scale = static_cast<const float*>(w_scale);
  }
  p.G = G; p.R = R; p.K = Nout; p.N = Kc;
  constexpr int TM = Cfg<KIND_DX>::TM;
  p.mt_bound = (int)((R + TM - 1) / TM + G);
  p.n_tiles = (int)((Nout + TN - 1) / TN);
  const int64_t tiles = (int64_t)p.mt_bound * p.n_tiles;
  const moe_status st = attach_split(p, workspace, workspace_bytes, fn, stream);
  if (st != MOE_SUCCESS) return st;
  if (op == F8_GATE_UP) {
    if (act) return launch<KIND_DX, true, true, false, false, true, false, MX>(p, tiles, stream, fn);
    return launch<KIND_DX, true, false, false, false, true, false, MX>(p, tiles, stream, fn);
  }
  if (op == F8_SWIGLU_BWD) return launch<KIND_DX, false, true, false, false, true, false, MX>(p, tiles, stream, fn);
  return launch<KIND_DX, false, false, false, false, true, false, MX>(p, tiles, stream, fn);
}
}  // namespace
}  // namespace moe

extern "C" int64_t moe_mx_scale_bytes(int64_t rows, int64_t C) {
  return rows <= 0 || C <= 0 ? 0 : (C + 127) / 128 * rows * 4;
}

extern "C" moe_status moe_grouped_gemm_fwd_fp8_gate_up(const uint8_t* A, const float* a_scale, const uint8_t* Wt,
                                                       const float* w_scale, const int32_t* offsets, int32_t G,
                                                       int64_t R, int64_t K, int64_t F, moe_bf16* h_gate,
                                                       moe_bf16* h_up, moe_bf16* act, void* workspace,
                                                       size_t workspace_bytes, hipStream_t stream) {
  return f8_product<false>("moe_grouped_gemm_fwd_fp8_gate_up", F8_GATE_UP, A, a_scale, Wt, w_scale, offsets, G, R, K,
                           2 * F, h_gate, h_up, act, nullptr, nullptr, workspace, workspace_bytes, stream);
}

extern "C" moe_status moe_grouped_gemm_fwd_fp8(const uint8_t* A, const float* a_scale, const uint8_t* Wt,
                                               const float* w_scale, const int32_t* offsets, int32_t G, int64_t R,
                                               int64_t K, int64_t N, moe_bf16* C, void* workspace,
                                               size_t workspace_bytes, hipStream_t stream) {
  return f8_product<false>("moe_grouped_gemm_fwd_fp8", F8_PLAIN, A, a_scale, Wt, w_scale, offsets, G, R, K, N, C,
                           nullptr, nullptr, nullptr, nullptr, workspace, workspace_bytes, stream);
}

extern "C" moe_status moe_grouped_gemm_dx_swiglu_bwd_fp8(const uint8_t* A, const float* a_scale, const uint8_t* Wt,
                                                          const float* w_scale, const int32_t* offsets, int32_t G,
                                                          int64_t R, int64_t K, int64_t N, const moe_bf16* h_gate,
                                                          const moe_bf16* h_up, moe_bf16* dh_gate, moe_bf16* dh_up,
                                                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return f8_product<false>("moe_grouped_gemm_dx_swiglu_bwd_fp8", F8_SWIGLU_BWD, A, a_scale, Wt, w_scale, offsets, G,
                           R, K, N, dh_gate, dh_up, nullptr, h_gate, h_up, workspace, workspace_bytes, stream);
}

extern "C" moe_status moe_grouped_gemm_fwd_mx_gate_up(const uint8_t* A, const uint8_t* a_scale, const uint8_t* Wt,
                                                     const uint8_t* w_scale, const int32_t* offsets, int32_t G,
                                                     int64_t R, int64_t K, int64_t F, moe_bf16* h_gate, moe_bf16* h_up,
                                                     moe_bf16* act, void* workspace, size_t workspace_bytes,
                                                     hipStream_t stream) {
  return f8_product<true>("moe_grouped_gemm_fwd_mx_gate_up", F8_GATE_UP, A, a_scale, Wt, w_scale, offsets, G, R, K,
                          2 * F, h_gate, h_up, act, nullptr, nullptr, workspace, workspace_bytes, stream);
}

extern "C" moe_status moe_grouped_gemm_fwd_mx(const uint8_t* A, const uint8_t* a_scale, const uint8_t* Wt,
                                             const uint8_t* w_scale, const int32_t* offsets, int32_t G, int64_t R,
                                             int64_t K, int64_t N, moe_bf16* C, void* workspace,
                                             size_t workspace_bytes, hipStream_t stream) {
  return f8_product<true>("moe_grouped_gemm_fwd_mx", F8_PLAIN, A, a_scale, Wt, w_scale, offsets, G, R, K, N, C,
                          nullptr, nullptr, nullptr, nullptr, workspace, workspace_bytes, stream);
}

extern "C" moe_status moe_grouped_gemm_dx_swiglu_bwd_mx(const uint8_t* A, const uint8_t* a_scale, const uint8_t* Wt,
                                                        const uint8_t* w_scale, const int32_t* offsets, int32_t G,
                                                        int64_t R, int64_t K, int64_t N, const moe_bf16* h_gate,
                                                        const moe_bf16* h_up, moe_bf16* dh_gate, moe_bf16* dh_up,
                                                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return f8_product<true>("moe_grouped_gemm_dx_swiglu_bwd_mx", F8_SWIGLU_BWD, A, a_scale, Wt, w_scale, offsets, G, R,
                          K, N, dh_gate, dh_up, nullptr, h_gate, h_up, workspace, workspace_bytes, stream);
}

extern "C" moe_status moe_grouped_gemm_dx_split(const moe_bf16* dC, const moe_bf16* B, const moe_bf16* dC2,
                                                const moe_bf16* B2, const int32_t* offsets, int32_t G,
                                                int64_t R, int64_t K, int64_t N, moe_bf16* dA, void* workspace,
                                                size_t workspace_bytes, hipStream_t stream) {
  if (!workspace) return fail(MOE_ERROR_WORKSPACE, "moe_grouped_gemm_dx_split: workspace is NULL");
  return grouped_gemm_dx_impl(dC, B, dC2, B2, offsets, G, R, K, N, dA, workspace, workspace_bytes, stream);
}

namespace moe {
namespace {
moe_status grouped_gemm_dx_swiglu_bwd_impl(const moe_bf16* dC, const moe_bf16* B, const int32_t* offsets, int32_t G,
                                           int64_t R, int64_t K, int64_t N, const moe_bf16* h_gate,
                                           const moe_bf16* h_up, moe_bf16* dh_gate, moe_bf16* dh_up, void* ws,
                                           size_t ws_bytes, hipStream_t stream) {
  const char* fn = "moe_grouped_gemm_dx_swiglu_bwd";
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: need 1 <= G <= 256", fn);
  if (R < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (K % 64 || N % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K and N must be multiples of 64", fn);
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: R >= 2^31", fn);
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "%s: offsets is NULL", fn);
  if (K * N * 2 >= ((int64_t)1 << 31))
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: one group's B must be < 2 GiB", fn);
  if (R == 0) return MOE_SUCCESS;
  if (!dC || !B || !h_gate || !h_up || !dh_gate || !dh_up)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (bad_ptr(dC) || bad_ptr(B) || bad_ptr(h_gate) || bad_ptr(h_up) || bad_ptr(dh_gate) || bad_ptr(dh_up))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: pointers must be 16-byte aligned", fn);
  GemmParams p{};
  p.a = dC; p.b = B; p.offsets = offsets; p.out = dh_gate; p.out2 = dh_up; p.hg = h_gate; p.hu = h_up;
  p.G = G; p.R = R; p.K = K; p.N = N;
  constexpr int TM = Cfg<KIND_DX>::TM;
  p.mt_bound = (int)((R + TM - 1) / TM + G);
  p.n_tiles = (int)((K + TN - 1) / TN);
  const int64_t tiles = (int64_t)p.mt_bound * p.n_tiles;   // upper bound; exact count on device
  const moe_status st = attach_split(p, ws, ws_bytes, fn, stream);
  if (st != MOE_SUCCESS) return st;
  return launch<KIND_DX, false, true>(p, tiles, stream, "grouped_gemm_dx(swiglu_bwd)");
}
}  // namespace
}  // namespace moe

extern "C" moe_status moe_grouped_gemm_dx_swiglu_bwd(const moe_bf16* dC, const moe_bf16* B,
                                                      const int32_t* offsets, int32_t G, int64_t R,
                                                      int64_t K, int64_t N, const moe_bf16* h_gate,
                                                      const moe_bf16* h_up, moe_bf16* dh_gate,
                                                      moe_bf16* dh_up, hipStream_t stream) {
  return grouped_gemm_dx_swiglu_bwd_impl(dC, B, offsets, G, R, K, N, h_gate, h_up, dh_gate, dh_up, nullptr, 0,
                                         stream);
}

extern "C" moe_status moe_grouped_gemm_dx_swiglu_bwd_split(const moe_bf16* dC, const moe_bf16* B,
                                                            const int32_t* offsets, int32_t G, int64_t R,
                                                            int64_t K, int64_t N, const moe_bf16* h_gate,
                                                            const moe_bf16* h_up, moe_bf16* dh_gate,
                                                            moe_bf16* dh_up, void* workspace,
                                                            size_t workspace_bytes, hipStream_t stream) {
  if (!workspace) return fail(MOE_ERROR_WORKSPACE, "moe_grouped_gemm_dx_swiglu_bwd_split: workspace is NULL");
  return grouped_gemm_dx_swiglu_bwd_impl(dC, B, offsets, G, R, K, N, h_gate, h_up, dh_gate, dh_up, workspace,
                                         workspace_bytes, stream);
}

namespace moe {
namespace {
moe_status grouped_gemm_dw_impl(const char* fn, bool out16, const moe_bf16* A, const moe_bf16* dC,
                                const moe_bf16* dC2, const int32_t* offsets, int32_t G, int64_t R,
                                int64_t K, int64_t N, void* dB, void* dB2, int32_t* counters,
                                bool persistent, hipStream_t stream, void* ws = nullptr, size_t ws_bytes = 0) {
  if (persistent && (counters == nullptr || (reinterpret_cast<uintptr_t>(counters) & 3u)))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: counters must be 8 int32 of device memory", fn);
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: need 1 <= G <= 256", fn);
  if (R < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (K % 64 || N % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K and N must be multiples of 64", fn);
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: R >= 2^31", fn);
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "%s: offsets is NULL", fn);
  if ((dC2 == nullptr) != (dB2 == nullptr))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: dC2 and dB2 must both be set or both NULL", fn);
  if (!dB || (R > 0 && (!A || !dC))) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (bad_ptr(A) || bad_ptr(dC) || bad_ptr(dC2) || bad_ptr(dB) || bad_ptr(dB2))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: pointers must be 16-byte aligned", fn);
  GemmParams p{};
  p.a = A; p.b = dC; p.b2 = dC2; p.offsets = offsets; p.out = dB; p.out2 = dB2;
  p.G = G; p.R = R; p.K = K; p.N = N;
  p.m_tiles = (int)((K + Cfg<KIND_DW>::TM - 1) / Cfg<KIND_DW>::TM);
  const int cols_per_tile = dC2 ? TN / 2 : TN;
  p.n_tiles = (int)((N + cols_per_tile - 1) / cols_per_tile);
  const int64_t tiles = (int64_t)G * p.m_tiles * p.n_tiles;
  if (ws != nullptr && (ws_bytes < SPLIT_BYTES || !aligned16(ws)))   // before any launch
    return fail(MOE_ERROR_WORKSPACE, "%s: a 16-byte aligned workspace of %zu bytes is needed", fn, SPLIT_BYTES);
  if (persistent && tiles > 0) {
    p.tile_queue = counters;
    zero_i32_kernel<<<1, 64, 0, stream>>>(counters, 8);
    if (G == 1) {   // one group: the last round's tiles may be split along the contraction
      const moe_status st = attach_split(p, ws, ws_bytes, fn, stream);
      if (st != MOE_SUCCESS) return st;
    }
    if (out16) {
      if (dC2) return launch<KIND_DW, true, false, true, false, false, true>(p, tiles, stream, "grouped_gemm_dw_bf16(dual, persistent)");
      return launch<KIND_DW, false, false, true, false, false, true>(p, tiles, stream, "grouped_gemm_dw_bf16(persistent)");
    }
    if (dC2) return launch<KIND_DW, true, false, false, false, false, true>(p, tiles, stream, "grouped_gemm_dw(dual, persistent)");
    return launch<KIND_DW, false, false, false, false, false, true>(p, tiles, stream, "grouped_gemm_dw(persistent)");
  }
  if (out16) {
    if (dC2) return launch<KIND_DW, true, false, true>(p, tiles, stream, "grouped_gemm_dw_bf16(dual)");
    return launch<KIND_DW, false, false, true>(p, tiles, stream, "grouped_gemm_dw_bf16");
  }
  if (dC2) return launch<KIND_DW, true, false>(p, tiles, stream, "grouped_gemm_dw(dual)");
  return launch<KIND_DW, false, false>(p, tiles, stream, "grouped_gemm_dw");
}
}  // namespace
}  // namespace moe

extern "C" moe_status moe_grouped_gemm_dw_t(const moe_bf16* At, const moe_bf16* dCt, const moe_bf16* dC2t,
                                            const int32_t* offsets, int32_t G, int64_t R, int64_t K, int64_t N,
                                            int64_t ld, void* dB, void* dB2, int32_t out_bf16,
                                            hipStream_t stream) {
  const char* fn = "moe_grouped_gemm_dw_t";
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: need 1 <= G <= 256", fn);
  if (R < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (K % 64 || N % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K and N must be multiples of 64", fn);
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: R >= 2^31", fn);
  const int64_t bound = ((R + 31) & ~(int64_t)31) + 32 * (int64_t)G;
  if (ld < bound || ld % 64)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: ld must be a multiple of 64 and >= %lld", fn, (long long)bound);
  if ((K > N ? K : N) * ld * 2 >= ((int64_t)1 << 31))
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: operands of 2 GiB or more", fn);
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "%s: offsets is NULL", fn);
  if ((dC2t == nullptr) != (dB2 == nullptr))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: dC2t and dB2 must both be set or both NULL", fn);
  if (!dB || !At || !dCt) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (bad_ptr(At) || bad_ptr(dCt) || bad_ptr(dC2t) || bad_ptr(dB) || bad_ptr(dB2))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: pointers must be 16-byte aligned", fn);
  GemmParams p{};
  p.a = At; p.b = dCt; p.b2 = dC2t; p.offsets = offsets; p.out = dB; p.out2 = dB2;
  p.G = G; p.R = R; p.K = K; p.N = N; p.ld_t = ld;
  p.m_tiles = (int)((K + Cfg<KIND_DWT>::TM - 1) / Cfg<KIND_DWT>::TM);
  const int cols_per_tile = dC2t ? TN / 2 : TN;
  p.n_tiles = (int)((N + cols_per_tile - 1) / cols_per_tile);
  const int64_t tiles = (int64_t)G * p.m_tiles * p.n_tiles;
  if (out_bf16) {
    if (dC2t) return launch<KIND_DWT, true, false, true>(p, tiles, stream, "grouped_gemm_dw_t_bf16(dual)");
    return launch<KIND_DWT, false, false, true>(p, tiles, stream, "grouped_gemm_dw_t_bf16");
  }
  if (dC2t) return launch<KIND_DWT, true, false>(p, tiles, stream, "grouped_gemm_dw_t(dual)");
  return launch<KIND_DWT, false, false>(p, tiles, stream, "grouped_gemm_dw_t");
}

extern "C" moe_status moe_grouped_gemm_dw_mx(const uint8_t* At, const uint8_t* a_scale, const uint8_t* dCt,
                                             const uint8_t* c_scale, const uint8_t* dC2t, const uint8_t* c2_scale,
                                             const int32_t* offsets, int32_t G, int64_t R, int64_t K, int64_t N,
                                             int64_t ld, void* dB, void* dB2, int32_t out_bf16, int32_t* counters,
                                             hipStream_t stream) {
  const char* fn = "moe_grouped_gemm_dw_mx";
  if (reinterpret_cast<uintptr_t>(counters) & 3u)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: counters must be 8 int32 of device memory", fn);
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: need 1 <= G <= 256", fn);
  if (R < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (K % 64 || N % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K and N must be multiples of 64", fn);
  if (R >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: R >= 2^31", fn);
  const int64_t bound = moe_mx_tokens_cols_bound(R, G);
  if (ld < bound || ld % 128)
    return fail(MOE_ERROR_INVALID_VALUE, "%s: ld must be a multiple of 128 and >= %lld", fn, (long long)bound);
  if ((K > N ? K : N) * ld >= ((int64_t)1 << 31))
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: operands of 2 GiB or more", fn);
  if (!offsets) return fail(MOE_ERROR_INVALID_VALUE, "%s: offsets is NULL", fn);
  if ((dC2t == nullptr) != (dB2 == nullptr) || (dC2t == nullptr) != (c2_scale == nullptr))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: dC2t, c2_scale and dB2 must all be set or all NULL", fn);
  if (!dB || !At || !dCt || !a_scale || !c_scale) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (bad_ptr(At) || bad_ptr(dCt) || bad_ptr(dC2t) || bad_ptr(dB) || bad_ptr(dB2) ||
      ((reinterpret_cast<uintptr_t>(a_scale) | reinterpret_cast<uintptr_t>(c_scale) |
        reinterpret_cast<uintptr_t>(c2_scale)) & 3))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: operands and outputs must be 16-byte, scales 4-byte aligned", fn);
  GemmParams p{};
  p.a = reinterpret_cast<const uint16_t*>(At);
  p.b = reinterpret_cast<const uint16_t*>(dCt);
  p.b2 = reinterpret_cast<const uint16_t*>(dC2t);
  p.a_mx = a_scale; p.w_mx = c_scale; p.w_mx2 = c2_scale;
  p.mx_a_step = K * 4;
  p.mx_w_step = N * 4;
  p.offsets = offsets; p.out = dB; p.out2 = dB2;
  p.G = G; p.R = R; p.K = K; p.N = N; p.ld_t = ld;
  p.m_tiles = (int)((K + Cfg<KIND_DWT>::TM - 1) / Cfg<KIND_DWT>::TM);
  const int cols_per_tile = dC2t ? TN / 2 : TN;
  p.n_tiles = (int)((N + cols_per_tile - 1) / cols_per_tile);
  const int64_t tiles = (int64_t)G * p.m_tiles * p.n_tiles;
  if (counters != nullptr && tiles > 0) {   // persistent grid claiming its tiles, as the bf16 dW
    p.tile_queue = counters;
    zero_i32_kernel<<<1, 64, 0, stream>>>(counters, 8);
    if (out_bf16) {
      if (dC2t) return launch<KIND_DWT, true, false, true, false, true, true, true>(p, tiles, stream, fn);
      return launch<KIND_DWT, false, false, true, false, true, true, true>(p, tiles, stream, fn);
    }
    if (dC2t) return launch<KIND_DWT, true, false, false, false, true, true, true>(p, tiles, stream, fn);
    return launch<KIND_DWT, false, false, false, false, true, true, true>(p, tiles, stream, fn);
  }
  if (out_bf16) {
    if (dC2t) return launch<KIND_DWT, true, false, true, false, true, false, true>(p, tiles, stream, fn);
    return launch<KIND_DWT, false, false, true, false, true, false, true>(p, tiles, stream, fn);
  }
  if (dC2t) return launch<KIND_DWT, true, false, false, false, true, false, true>(p, tiles, stream, fn);
  return launch<KIND_DWT, false, false, false, false, true, false, true>(p, tiles, stream, fn);
}

extern "C" moe_status moe_grouped_gemm_dw(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                                          const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                          int64_t N, float* dB, float* dB2, hipStream_t stream) {
  return grouped_gemm_dw_impl("moe_grouped_gemm_dw", false, A, dC, dC2, offsets, G, R, K, N, dB, dB2, nullptr,
                              false, stream);
}

extern "C" moe_status moe_grouped_gemm_dw_persistent(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                                                     const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                                     int64_t N, float* dB, float* dB2, int32_t* counters,
                                                     hipStream_t stream) {
  return grouped_gemm_dw_impl("moe_grouped_gemm_dw_persistent", false, A, dC, dC2, offsets, G, R, K, N, dB, dB2,
                              counters, true, stream);
}

extern "C" moe_status moe_grouped_gemm_dw_split(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                                                const int32_t* offsets, int32_t G, int64_t R, int64_t K, int64_t N,
                                                float* dB, float* dB2, int32_t* counters, void* workspace,
                                                size_t workspace_bytes, hipStream_t stream) {
  return grouped_gemm_dw_impl("moe_grouped_gemm_dw_split", false, A, dC, dC2, offsets, G, R, K, N, dB, dB2,
                              counters, true, stream, workspace, workspace_bytes);
}

extern "C" moe_status moe_grouped_gemm_dw_bf16(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                                               const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                               int64_t N, moe_bf16* dB, moe_bf16* dB2, hipStream_t stream) {
  return grouped_gemm_dw_impl("moe_grouped_gemm_dw_bf16", true, A, dC, dC2, offsets, G, R, K, N, dB, dB2, nullptr,
                              false, stream);
}

extern "C" moe_status moe_grouped_gemm_dw_bf16_persistent(const moe_bf16* A, const moe_bf16* dC,
                                                          const moe_bf16* dC2, const int32_t* offsets, int32_t G,
                                                          int64_t R, int64_t K, int64_t N, moe_bf16* dB,
                                                          moe_bf16* dB2, int32_t* counters, hipStream_t stream) {
  return grouped_gemm_dw_impl("moe_grouped_gemm_dw_bf16_persistent", true, A, dC, dC2, offsets, G, R, K, N, dB,
                              dB2, counters, true, stream);
}
