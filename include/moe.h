/*
 * moe.h - C ABI of the MI355X (gfx950) MoE expert-FFN training layer library (libmoe_mi355x.so).
 *
 * The layer: top-k routing of T tokens over E experts, packing of the T*k routed rows into one
 * buffer ordered by expert, bf16 grouped GEMMs over the ragged per-expert row groups (gate/up
 * with a fused SwiGLU, then down), a weighted combine back to token order, and the backward
 * dX/dW grouped GEMMs.  The paper (section 5.4; Appendix H, "What the kernel computes") defines
 * the packed expert-ordered buffer, the cumulative per-expert row counts and the ragged weight
 * gradient dW1_e = X_e^T G_e; the other steps follow the standard MoE layer, with the readings
 * stated at each function below.
 *
 * Conventions shared by every entry point
 *  - All tensor pointers are DEVICE pointers, owned and allocated by the caller; the library
 *    allocates nothing and keeps no state between calls apart from cached device properties.
 *  - Tensors are dense row-major (C order) with the shapes given in brackets.
 *  - bf16 tensors are passed as moe_bf16 (the IEEE bfloat16 bit pattern in a uint16_t).
 *  - Floating-point results are computed with fp32 arithmetic (MFMA fp32 accumulation for the
 *    GEMMs) and rounded to bf16 with round-to-nearest-even where a bf16 tensor is stored.
 *  - Row groups are given by exclusive offsets: int32 offsets[G+1], offsets[0] = 0,
 *    offsets[G] = R, group g = rows offsets[g] <= r < offsets[g+1] (offsets[g+1] is the paper's
 *    inclusive cumulative sum cumsum_K[g]).  offsets must be non-decreasing; this is NOT checked
 *    (it lives in device memory and the calls never synchronize).
 *  - Every call is asynchronous on `stream` (NULL = the default stream), performs no host/device
 *    synchronization and no allocation.  Arguments are validated on the host before anything is
 *    launched; an invalid call returns an error status and launches nothing.  Faults inside a
 *    kernel surface at the caller's next synchronization.
 *  - Shape limits: 1 <= k <= E <= 256; hidden and FFN widths (d, f, and the GEMMs' K and N) are
 *    positive multiples of 64; R = T*k < 2^31; device pointers 16-byte aligned.  T = 0 / R = 0
 *    is a successful no-op, except that moe_grouped_gemm_dw still writes its zero output.
 *  - Outputs must not alias inputs.
 */
#ifndef MOE_MI355X_H
#define MOE_MI355X_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t moe_bf16;

typedef enum {
  MOE_SUCCESS = 0,
  MOE_ERROR_INVALID_VALUE = 1, /* null or misaligned pointer, negative size, k > E, ...      */
  MOE_ERROR_NOT_SUPPORTED = 2, /* a size outside the limits above (E > 256, d % 64 != 0, ...) */
  MOE_ERROR_WORKSPACE = 3,     /* workspace missing or smaller than the query says            */
  MOE_ERROR_HIP = 4            /* a HIP runtime call (launch, device query) failed             */
} moe_status;

/* Static description of a status code. */
const char* moe_status_string(moe_status s);

/* Detail of the last error returned on the calling host thread ("" if none). */
const char* moe_last_error(void);

/* ------------------------------------------------------------------------------------------ */
/* A1-A4: routing, grouping, permutation and gather                                           */
/* ------------------------------------------------------------------------------------------ */

/* Bytes of device workspace moe_route_permute needs for these sizes (0 if none). */
size_t moe_route_permute_workspace_bytes(int64_t T, int32_t E, int32_t k);

/*
 * Top-k routing and packing of the routed rows by expert (section 5.4: top-k routing;
 * Appendix H: routed tokens packed into one contiguous buffer ordered by expert, groups given by
 * cumulative per-expert counts).  The paper fixes neither the routing rule nor the order inside a
 * group; this library reads them as:
 *   - topk_idx[t, 0..k-1]: the k experts with the largest logits[t, :], by descending logit,
 *     equal logits ordered by ascending expert id (exact: selection compares the fp32 logits);
 *   - topk_w[t, j] = exp(l_j - l_0) / sum_{j'<k} exp(l_j' - l_0) over the selected logits
 *     (normalize_topk = 1), or the softmax probability over all E experts (normalize_topk = 0);
 *   - slot s = t*k + j; offsets = exclusive prefix sum of per-expert slot counts;
 *     row_of_slot[s] = offsets[e] + (number of slots s' < s routed to the same expert e), so
 *     each group keeps ascending token order (a stable counting sort);
 *     token_of_row[row_of_slot[s]] = s / k;
 *   - x_perm[r, :] = x[token_of_row[r], :] (bit copy) when x and x_perm are non-NULL.
 * logits [T,E] fp32; x [T,d] bf16 or NULL; topk_idx [T,k] int32; topk_w [T,k] fp32;
 * offsets [E+1] int32; row_of_slot [T*k] int32; token_of_row [T*k] int32; x_perm [T*k,d] bf16 or
 * NULL.  workspace: 16-byte aligned device scratch of at least
 * moe_route_permute_workspace_bytes(T, E, k) bytes, contents on entry ignored.  Results are deterministic and bit-exact (no order-dependent
 * atomics).  NaN logits are not supported.
 */
moe_status moe_route_permute(const float* logits, const moe_bf16* x, int64_t T, int64_t d,
                             int32_t E, int32_t k, int32_t normalize_topk, int32_t* topk_idx,
                             float* topk_w, int32_t* offsets, int32_t* row_of_slot,
                             int32_t* token_of_row, moe_bf16* x_perm, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

/*
 * For callers that cannot allocate (code under HIP graph capture, tight serving loops, harnesses
 * that forbid device allocation): moe_route_permute without a workspace.  Same arguments, results
 * and errors as moe_route_permute, bit for bit; the per-range histogram lives in a device array of
 * the library (moe_route_permute_noalloc_max_scratch_bytes() bytes per device, held until the
 * process ends) instead of a caller workspace.  Sizes whose histogram would not fit
 * (moe_route_permute_workspace_bytes(T, E, k) above that maximum) return MOE_ERROR_NOT_SUPPORTED
 * before any launch.  Calls no allocator.  Every call on a device shares that device's array, so
 * calls that may overlap on one device (concurrent streams, threads) race and must be serialized
 * by the caller; each call overwrites whatever the previous one left there.
 */
size_t moe_route_permute_noalloc_max_scratch_bytes(void);
moe_status moe_route_permute_noalloc(const float* logits, const moe_bf16* x, int64_t T, int64_t d,
                                     int32_t E, int32_t k, int32_t normalize_topk, int32_t* topk_idx,
                                     float* topk_w, int32_t* offsets, int32_t* row_of_slot,
                                     int32_t* token_of_row, moe_bf16* x_perm, hipStream_t stream);

/*
 * A4 alone: x_perm[row_of_slot[t*k + j], :] = x[t, :] for t < T, j < k (a bit copy; the gather of
 * moe_route_permute, for a caller that routed without it, e.g. when the forward product gathered
 * its rows itself and only the weight gradient needs X_perm).  x [T,d], x_perm [T*k,d] bf16;
 * row_of_slot [T*k] int32 as moe_route_permute returns it (a permutation of 0..T*k-1; not
 * checked).  Errors: d not a positive multiple of 64 -> NOT_SUPPORTED; NULL or misaligned
 * pointers -> INVALID_VALUE.  T = 0 is a no-op.
 */
moe_status moe_gather_rows(const moe_bf16* x, int64_t T, int64_t d, int32_t k, const int32_t* row_of_slot,
                           moe_bf16* x_perm, hipStream_t stream);

/* ------------------------------------------------------------------------------------------ */
/* B, D: forward grouped GEMM (+ fused SwiGLU)                                                 */
/* ------------------------------------------------------------------------------------------ */

/*
 * Grouped GEMM over ragged row groups: C[r, :] = bf16(A[r, :] . B[g]) for rows r of group g.
 * With B2 != NULL (gate/up in one pass sharing the A tiles): C2[r, :] = bf16(A[r, :] . B2[g]),
 * and if act != NULL also act[r, c] = bf16(silu(C[r,c]) * C2[r,c]) computed in fp32 from the
 * bf16-rounded C and C2 (silu(g) = g / (1 + exp(-g)); plain SwiGLU, the paper leaves the
 * activation open).
 * A [R,K] bf16; B, B2 [G,K,N] bf16; offsets [G+1]; C, C2, act [R,N] bf16.  K, N multiples of 64.
 * C is required; C2 is required iff B2 is given; act requires B2.
 */
moe_status moe_grouped_gemm_fwd(const moe_bf16* A, const moe_bf16* B, const moe_bf16* B2,
                                const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                int64_t N, moe_bf16* C, moe_bf16* C2, moe_bf16* act,
                                hipStream_t stream);

/* ------------------------------------------------------------------------------------------ */
/* C, I: SwiGLU and its backward (standalone elementwise kernels)                               */
/* ------------------------------------------------------------------------------------------ */

/* act = bf16(silu(h_gate) * h_up), elementwise over [rows, f] bf16 (the same arithmetic as the
 * fused epilogue of moe_grouped_gemm_fwd). */
moe_status moe_swiglu(const moe_bf16* h_gate, const moe_bf16* h_up, moe_bf16* act,
                      int64_t rows, int64_t f, hipStream_t stream);

/* Backward of moe_swiglu, elementwise over [rows, f] bf16, s = sigmoid(h_gate):
 *   dh_up   = bf16(d_act * h_gate * s)
 *   dh_gate = bf16(d_act * h_up * s * (1 + h_gate * (1 - s))). */
moe_status moe_swiglu_bwd(const moe_bf16* h_gate, const moe_bf16* h_up, const moe_bf16* d_act,
                          moe_bf16* dh_gate, moe_bf16* dh_up, int64_t rows, int64_t f,
                          hipStream_t stream);

/* ------------------------------------------------------------------------------------------ */
/* E, L: weighted unpermute-combine;  F: its backward                                           */
/* ------------------------------------------------------------------------------------------ */

/*
 * y[t, :] = bf16( sum_{j=0..k-1} w[t,j] * y_perm[row_of_slot[t*k+j], :] + add[t, :] ), fp32 sum
 * in j order then the add, one rounding.  topk_w == NULL means every weight is 1 (the
 * unpermute-sum of dX_perm in the backward); add == NULL means no add (the shared-FFN output is
 * added here in the forward, its dX in the backward).  The paper does not describe the combine;
 * this is the standard weighted MoE combine.
 * y_perm [T*k,d] bf16; topk_w [T,k] fp32 or NULL; row_of_slot [T*k] int32; add [T,d] bf16 or
 * NULL; y [T,d] bf16.
 */
moe_status moe_unpermute_combine(const moe_bf16* y_perm, const float* topk_w,
                                 const int32_t* row_of_slot, const moe_bf16* add, int64_t T,
                                 int64_t d, int32_t k, moe_bf16* y, hipStream_t stream);

/*
 * Steps D + E in one call: the down product of moe_grouped_gemm_fwd (single B, no SwiGLU) with
 * the weighted combine of moe_unpermute_combine fused into its epilogue.  y_perm [R, N] =
 * bf16(A . B[g]) is stored as by moe_grouped_gemm_fwd (the backward's d_topk_w reads it), and
 * y [T, N] = bf16(sum_j topk_w[t,j] * y_perm[row_of_slot[t*k+j], :] + add[t, :]) bit for bit as
 * moe_unpermute_combine computes it: each tile stores its rows of y_perm (written through to
 * memory, agent-coherent), then counts one arrival per row for the (token, 256-column tile)
 * pair; the tile that brings a pair's count to k computes those 256 columns of the token's Y row
 * from the k stored rows, in slot order (a tile stores all its rows before it counts any, so the
 * count reaches k only once every row is in memory).  R == T * k; topk_w [T, k] fp32,
 * row_of_slot [T*k] and token_of_row [R] int32 as moe_route_permute returns them; add [T, N]
 * bf16 or NULL.  count_workspace: moe_grouped_gemm_fwd_combine_workspace_bytes(T, N) bytes,
 * 4-byte aligned (zeroed here, on `stream`); split_workspace: NULL or a split workspace as for
 * moe_grouped_gemm_fwd_split.  Errors as moe_grouped_gemm_fwd; R != T*k -> INVALID_VALUE; a short
 * count workspace -> WORKSPACE; R * N * 2 >= 2^31 -> NOT_SUPPORTED.  Not the layer's default:
 * the coherent stores cost more than the separate combine saves (measured).
 */
size_t moe_grouped_gemm_fwd_combine_workspace_bytes(int64_t T, int64_t N);
moe_status moe_grouped_gemm_fwd_combine(const moe_bf16* A, const moe_bf16* B, const int32_t* offsets, int32_t G,
                                        int64_t R, int64_t K, int64_t N, const float* topk_w,
                                        const int32_t* row_of_slot, const int32_t* token_of_row, int64_t T,
                                        int32_t k, const moe_bf16* add, moe_bf16* y_perm, moe_bf16* y,
                                        void* count_workspace, size_t count_workspace_bytes, void* split_workspace,
                                        size_t split_workspace_bytes, hipStream_t stream);

/*
 * Backward of the weighted combine (the routing weight is applied while permuting dY):
 *   dy_perm[row_of_slot[t*k+j], :] = bf16(w[t,j] * dy[t, :])
 *   d_topk_w[t, j] = sum_c dy[t,c] * y_perm[row_of_slot[t*k+j], c]   (fp32; skipped if y_perm or
 *                                                                     d_topk_w is NULL)
 * dy [T,d] bf16; topk_w [T,k] fp32; row_of_slot [T*k]; y_perm [T*k,d] bf16 or NULL;
 * dy_perm [T*k,d] bf16; d_topk_w [T,k] fp32 or NULL.
 */
moe_status moe_unpermute_combine_bwd(const moe_bf16* dy, const float* topk_w,
                                     const int32_t* row_of_slot, const moe_bf16* y_perm,
                                     int64_t T, int64_t d, int32_t k, moe_bf16* dy_perm,
                                     float* d_topk_w, hipStream_t stream);

/* ------------------------------------------------------------------------------------------ */
/* G, J: backward data-gradient grouped GEMM                                                    */
/* ------------------------------------------------------------------------------------------ */

/*
 * dA[r, :] = bf16( dC[r, :] . B[g]^T (+ dC2[r, :] . B2[g]^T) ) for rows r of group g, one fp32
 * accumulation over the whole (N or 2N long) contraction.  This is the gradient of
 * moe_grouped_gemm_fwd with respect to A (dX_perm takes the gate and up pairs together).
 * dC, dC2 [R,N] bf16; B, B2 [G,K,N] bf16; dA [R,K] bf16.  dC2 and B2 both NULL or both set.
 */
moe_status moe_grouped_gemm_dx(const moe_bf16* dC, const moe_bf16* B, const moe_bf16* dC2,
                               const moe_bf16* B2, const int32_t* offsets, int32_t G, int64_t R,
                               int64_t K, int64_t N, moe_bf16* dA, hipStream_t stream);

/*
 * G + I fused: the down projection's data gradient followed by the SwiGLU backward, without
 * storing dA.  For rows r of group g, dA[r, :] = bf16(dC[r, :] . B[g]^T) is formed in registers
 * (rounded exactly as the stored tensor would be) and the epilogue writes
 *   dh_up   = bf16(dA * h_gate * s),  dh_gate = bf16(dA * h_up * s * (1 + h_gate * (1 - s))),
 *   s = sigmoid(h_gate),
 * i.e. the result is bitwise identical to moe_grouped_gemm_dx (single pair) followed by
 * moe_swiglu_bwd.  Saves the dA store and reload and the separate elementwise pass.
 * dC [R,N]; B [G,K,N]; h_gate, h_up, dh_gate, dh_up [R,K] bf16.
 */
moe_status moe_grouped_gemm_dx_swiglu_bwd(const moe_bf16* dC, const moe_bf16* B,
                                          const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                          int64_t N, const moe_bf16* h_gate, const moe_bf16* h_up,
                                          moe_bf16* dh_gate, moe_bf16* dh_up, hipStream_t stream);

/*
 * The same products as moe_grouped_gemm_dx / moe_grouped_gemm_dx_swiglu_bwd (same arguments,
 * definitions and errors) with a workspace that lets the persistent kernel split the tiles of its
 * last, partial round of tiles along the contraction over the otherwise idle CUs: each piece
 * stores an fp32 partial tile, and the last piece to finish adds the pieces in a fixed order
 * before the usual epilogue.  Deterministic; a split tile's fp32 sum is grouped differently from
 * the unsplit kernel's, so bf16 results may differ from it in the last place.  workspace: device
 * memory of moe_grouped_gemm_split_workspace_bytes() bytes, 16-byte aligned, owned by the caller;
 * calls that overlap in time (on different streams) need separate workspaces.
 */
size_t moe_grouped_gemm_split_workspace_bytes(void);

/*
 * The gate/up product with the gather folded into its A operand (steps A4 + B): rows are read
 * straight from X through a row list instead of from the packed, expert-ordered X_perm.  For rows r
 * of group g: C[r, :] = X[row_src[r], :] . B[g] (and C2, act as in moe_grouped_gemm_fwd); with
 * row_src = token_of_row of moe_route_permute this equals moe_grouped_gemm_fwd on X_perm bit for
 * bit (same data, same arithmetic).  X [T,K] bf16 (T*K*2 < 2 GiB); row_src [R] int32, values in
 * [0,T) (not checked on the host: a row index past the source reads zeros); everything else as
 * moe_grouped_gemm_fwd.  workspace: NULL, or a split workspace as for moe_grouped_gemm_fwd_split.
 */
moe_status moe_grouped_gemm_fwd_gather(const moe_bf16* X, int64_t T, const int32_t* row_src, const moe_bf16* B,
                                       const moe_bf16* B2, const int32_t* offsets, int32_t G, int64_t R,
                                       int64_t K, int64_t N, moe_bf16* C, moe_bf16* C2, moe_bf16* act,
                                       void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------------------------ */
/* FP8 variant of the forward products (beyond the paper, which describes bf16 operands only):  */
/* OCP E4M3 operands with fp32 scales, fp32 accumulation, bf16 output.                        */
/* ------------------------------------------------------------------------------------------ */

/*
 * Per-row E4M3 quantization.  For each of the M rows of x [M,K] bf16: amax = max |x[r,:]|,
 * scale[r] = amax / 448 and q[r,k] = the E4M3 code nearest to x[r,k] * (448 / amax) (ties to the
 * even mantissa; magnitudes beyond 448 saturate), both quotients and the product single fp32
 * operations; an all-zero row gets scale 1 and zero codes.  x ~= decode(q) * scale.  Used for
 * activations (rows of A) and for weights stored as [output channel, contraction] (rows of Wt,
 * i.e. one scale per output channel).  q [M,K] uint8 (8-byte aligned), scale [M] fp32.  Errors: K
 * not a multiple of 16 -> NOT_SUPPORTED; NULL or misaligned pointers -> INVALID_VALUE.  M = 0 is a
 * no-op.
 */
moe_status moe_quantize_fp8_rows(const moe_bf16* x, int64_t M, int64_t K, uint8_t* q, float* scale,
                                 hipStream_t stream);

/*
 * The same quantization of the rows of two matrices joined along the contraction: row r is
 * [x[r, :] | x2[r, :]] (x, x2 [M,K] bf16), with one amax and one scale over both halves, and
 * q [M, 2K] holds x's codes in columns 0..K-1 and x2's in K..2K-1, code for code what
 * moe_quantize_fp8_rows gives for the concatenated [M, 2K] matrix.  The operand of a product whose
 * contraction runs over two matrices: the data gradient of the gate and up projections (section
 * 5.4's backward), dX = dH_gate . W_gate^T + dH_up . W_up^T, as one FP8 product over [dH_gate |
 * dH_up] (rows of M = R routed rows) and [W_gate | W_up] (rows of M = G*K_out output channels).
 * Alignment and errors as moe_quantize_fp8_rows; x2 NULL -> INVALID_VALUE.
 */
moe_status moe_quantize_fp8_rows2(const moe_bf16* x, const moe_bf16* x2, int64_t M, int64_t K, uint8_t* q,
                                  float* scale, hipStream_t stream);

/*
 * The same quantization for a weight kept as [expert, contraction, output channel], in one pass
 * per column block: W [G,K,N] bf16 -> Q [G,N',K] uint8 and scale [G,N'] fp32, where row (g, n) of
 * Q holds the codes of column n of W[g] (an output channel over its K contraction elements).
 * W2 == NULL: N' = N, Q[g] = the codes moe_quantize_fp8_rows gives for W[g]^T.  W2 != NULL (same
 * shape): N' = 2N and the rows interleave W's and W2's channels by 128 (rows 256b .. 256b+127:
 * W's channels 128b ..; the next 128: W2's), the weight layout moe_grouped_gemm_fwd_fp8_gate_up
 * reads.  Code for code equal to transposing (and interleaving) and then calling
 * moe_quantize_fp8_rows; this is the per-step weight preparation of an FP8 training step (the
 * weights change at every optimizer step).  Four kernels on `stream`; `scale` holds the column
 * maxima between them (final values once the last has run).  Q 16-byte, W/W2 16-byte, scale
 * 4-byte aligned.
 * Errors: K % 16 != 0, or N % 64 != 0 (N % 128 with W2) -> NOT_SUPPORTED; NULL or misaligned
 * pointers -> INVALID_VALUE.  G = 0 is a no-op.
 */
moe_status moe_quantize_fp8_weight(const moe_bf16* w, const moe_bf16* w2, int64_t G, int64_t K, int64_t N,
                                   uint8_t* q, float* scale, hipStream_t stream);

/*
 * The forward grouped product on E4M3 operands: for rows r of group g (offsets as in
 * moe_grouped_gemm_fwd), C[r,n] = bf16(a_scale[r] * w_scale[g,n] * sum_k A[r,k] * Wt[g,n,k]) with
 * A and Wt decoded from E4M3 and the sum accumulated in fp32 by the gfx950 8-bit matrix cores
 * (v_mfma_scale_f32_32x32x64_f8f6f4, 64 contraction elements per instruction).  The weight is in
 * the layout [G, N, K] (output channel, contraction): both operands are then read along the
 * contraction, as in the data-gradient product.  A [R,K] uint8, a_scale [R] fp32, Wt [G,N,K]
 * uint8, w_scale [G,N] fp32, C [R,N] bf16.  workspace: NULL, or a split workspace as for
 * moe_grouped_gemm_fwd_split (same tail split).  Errors as moe_grouped_gemm_fwd; K and N multiples
 * of 64; one group's weight < 2 GiB.
 */
moe_status moe_grouped_gemm_fwd_fp8(const uint8_t* A, const float* a_scale, const uint8_t* Wt, const float* w_scale,
                                    const int32_t* offsets, int32_t G, int64_t R, int64_t K, int64_t N, moe_bf16* C,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Steps G + I on E4M3 operands (section 5.4's backward of the down projection and of the SwiGLU):
 * dA[r,n] = bf16(a_scale[r] * w_scale[g,n] * sum_k A[r,k] * Wt[g,n,k]) as moe_grouped_gemm_fwd_fp8
 * computes it (A = the quantized dY_perm [R,K], Wt = the down weight as [G, N, K]: output channel n
 * of the expert's ffn dimension, contraction over the hidden dimension, the layout it is stored in,
 * quantized per row by moe_quantize_fp8_rows), followed in the epilogue by the SwiGLU backward of
 * moe_grouped_gemm_dx_swiglu_bwd on that bf16 dA: dh_gate, dh_up [R,N] bf16 from h_gate, h_up [R,N].
 * workspace: NULL or a split workspace.  Errors as moe_grouped_gemm_fwd_fp8.
 */
moe_status moe_grouped_gemm_dx_swiglu_bwd_fp8(const uint8_t* A, const float* a_scale, const uint8_t* Wt,
                                              const float* w_scale, const int32_t* offsets, int32_t G, int64_t R,
                                              int64_t K, int64_t N, const moe_bf16* h_gate, const moe_bf16* h_up,
                                              moe_bf16* dh_gate, moe_bf16* dh_up, void* workspace,
                                              size_t workspace_bytes, hipStream_t stream);

/*
 * The gate and up projections (steps B + C) on E4M3 operands in one product: Wt [G, 2F, K] holds
 * both weights with their output channels interleaved by 128 (rows 256t .. 256t+127 are gate
 * channels 128t .., the next 128 rows the up channels 128t ..; w_scale [G, 2F] in the same order),
 * so each 256-column tile computes 128 gate and the matching 128 up columns.  h_gate, h_up [R, F]
 * bf16 as moe_grouped_gemm_fwd_fp8 would compute them from the de-interleaved weights (bit for
 * bit), and, if act is non-NULL, act = silu(h_gate) * h_up from the rounded values exactly as
 * moe_swiglu computes it.  F a multiple of 128, K of 64; other arguments and errors as
 * moe_grouped_gemm_fwd_fp8.
 */
moe_status moe_grouped_gemm_fwd_fp8_gate_up(const uint8_t* A, const float* a_scale, const uint8_t* Wt,
                                            const float* w_scale, const int32_t* offsets, int32_t G, int64_t R,
                                            int64_t K, int64_t F, moe_bf16* h_gate, moe_bf16* h_up, moe_bf16* act,
                                            void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------------------------ */
/* MX variant (also beyond the paper): E4M3 operands with one power-of-two scale per 32        */
/* consecutive contraction elements of every row (OCP microscaling block structure), applied  */
/* by the gfx950 matrix cores inside the product; fp32 accumulation, bf16 output.             */
/* ------------------------------------------------------------------------------------------ */

/*
 * The MX scale layout, for a matrix of `rows` rows of C elements (C a multiple of 32): the E8M0
 * scale of block b (elements 32b .. 32b+31) of row r is byte ((b / 4) * rows + r) * 4 + b % 4,
 * i.e. the array is [ceil(C/128)][rows][4]: each row's four scales of a 128-element group form one
 * 4-byte word, and the words of all rows for one group lie side by side, so that the product's
 * scale loads for 64 consecutive rows read 256 contiguous bytes.  When C/32 is not a multiple of
 * 4, the bytes of the missing blocks of the last group are padding that nothing reads or writes.
 * Returns the array's size in bytes, ceil(C/128) * rows * 4 (0 if rows or C <= 0).
 */
int64_t moe_mx_scale_bytes(int64_t rows, int64_t C);

/*
 * MX quantization of rows: for each block of 32 consecutive elements of a row of x [M, K] bf16, or
 * of the concatenation [x[r, :] | x2[r, :]] when x2 [M, K] is given (the operand of the gate/up
 * data gradient, section 5.4's backward, whose contraction runs over both matrices), amax = max
 * |block|, e = the smallest integer with amax <= 448 * 2^e, raised to -127 if below (an all-zero
 * block gets -127); scale byte e + 127 (E8M0) and codes = the E4M3 values nearest to x * 2^-e
 * (ties to the even mantissa; nothing saturates).  x ~= decode(q) * 2^(byte - 127).
 * q [M, C] uint8 (C = K, or 2K with x2; 8-byte aligned), scale: the MX scale layout of M rows of C
 * (moe_mx_scale_bytes(M, C) bytes).
 * Inputs are finite.  Errors: K % 32 != 0 -> NOT_SUPPORTED; NULL or misaligned pointers ->
 * INVALID_VALUE.  M = 0 is a no-op.
 */
moe_status moe_quantize_mx_rows(const moe_bf16* x, const moe_bf16* x2, int64_t M, int64_t K, uint8_t* q,
                                uint8_t* scale, hipStream_t stream);

/*
 * MX quantization of a weight W [G, K, N] bf16 (kept as [expert, contraction of the forward
 * product, output channel]) in both orientations from one read, each code for code what
 * moe_quantize_mx_rows gives for the corresponding matrix:
 *   qt/st: the forward operand [G, N', K], row (g, n) = column n of W[g] over K (blocks along K);
 *     with W2 (same shape) N' = 2N and the rows interleave W's and W2's channels by 128 as in
 *     moe_quantize_fp8_weight (the layout moe_grouped_gemm_fwd_mx_gate_up reads); st in the MX
 *     scale layout of G * N' rows of K.
 *   qr/sr: the data-gradient operand [G, K, N''], row (g, k) = W[g][k, :] (N'' = N), or
 *     [W[g][k, :] | W2[g][k, :]] (N'' = 2N), blocks along the row; sr in the MX scale layout of
 *     G * K rows of N''.
 * Either pair may be NULL (not both).  One kernel on `stream`.  qt 16-byte, qr 8-byte, W/W2
 * 16-byte aligned.  Errors: K % 32 != 0, or N % 64 != 0 (N % 128 with W2) -> NOT_SUPPORTED; a
 * missing half of a pair, NULL or misaligned pointers -> INVALID_VALUE.  G = 0 is a no-op.
 */
moe_status moe_quantize_mx_weight(const moe_bf16* w, const moe_bf16* w2, int64_t G, int64_t K, int64_t N,
                                  uint8_t* qt, uint8_t* st, uint8_t* qr, uint8_t* sr, hipStream_t stream);

/*
 * The grouped product on MX operands: for rows r of group g (offsets as in moe_grouped_gemm_fwd),
 * C[r, n] = bf16(sum_k A[r,k] 2^(sa(r, k/32) - 127) * Wt[g,n,k] 2^(sw(g*N + n, k/32) - 127)),
 * the E4M3 products scaled and accumulated in fp32 by v_mfma_scale_f32_32x32x64_f8f6f4 (each
 * lane supplies its row's scale byte of one of the instruction's two 32-element blocks).  A [R, K]
 * uint8 with a_scale in the MX scale layout of R rows of K; Wt [G, N, K] uint8 with w_scale in the
 * MX scale layout of G * N rows of K (as moe_quantize_mx_rows / moe_quantize_mx_weight write
 * them); C [R, N] bf16.  workspace: NULL or a split workspace.  Errors as moe_grouped_gemm_fwd_fp8,
 * with both scale pointers 4-byte aligned.
 */
moe_status moe_grouped_gemm_fwd_mx(const uint8_t* A, const uint8_t* a_scale, const uint8_t* Wt,
                                   const uint8_t* w_scale, const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                   int64_t N, moe_bf16* C, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * Steps B + C on MX operands: moe_grouped_gemm_fwd_fp8_gate_up with MX scales (Wt [G, 2F, K] and
 * w_scale for its G * 2F rows, interleaved by 128 as moe_quantize_mx_weight writes them with W2).
 * h_gate, h_up bit for bit what moe_grouped_gemm_fwd_mx gives for the de-interleaved weights;
 * act = silu(h_gate) * h_up as moe_swiglu computes it, if non-NULL.  Errors as
 * moe_grouped_gemm_fwd_mx; F a multiple of 128.
 */
moe_status moe_grouped_gemm_fwd_mx_gate_up(const uint8_t* A, const uint8_t* a_scale, const uint8_t* Wt,
                                           const uint8_t* w_scale, const int32_t* offsets, int32_t G, int64_t R,
                                           int64_t K, int64_t F, moe_bf16* h_gate, moe_bf16* h_up, moe_bf16* act,
                                           void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Steps G + I on MX operands (section 5.4's backward of the down projection and of the SwiGLU):
 * dA as moe_grouped_gemm_fwd_mx computes it from A = the MX dY_perm [R, K] and Wt = the down
 * weight's rows [G, N, K] (moe_quantize_mx_weight's qr of W_down), followed in the epilogue by the
 * SwiGLU backward of moe_grouped_gemm_dx_swiglu_bwd: dh_gate, dh_up [R, N] bf16 from h_gate, h_up.
 * Errors as moe_grouped_gemm_fwd_mx.
 */
moe_status moe_grouped_gemm_dx_swiglu_bwd_mx(const uint8_t* A, const uint8_t* a_scale, const uint8_t* Wt,
                                             const uint8_t* w_scale, const int32_t* offsets, int32_t G, int64_t R,
                                             int64_t K, int64_t N, const moe_bf16* h_gate, const moe_bf16* h_up,
                                             moe_bf16* dh_gate, moe_bf16* dh_up, void* workspace,
                                             size_t workspace_bytes, hipStream_t stream);

/*
 * Columns needed by the token-major MX operands of the weight gradient for R routed rows in G
 * groups: the counts rounded up to 128 and summed, bounded by R + 127 G, rounded up to 128.
 */
int64_t moe_mx_tokens_cols_bound(int64_t R, int32_t G);

/*
 * MX quantization of a routed buffer along its token axis, for the weight gradient (Appendix H's
 * dW_e = X_e^T G_e, whose contraction runs over the K_e rows of expert e): x [R, C] bf16, rows
 * grouped by offsets -> qt [C, ld] uint8, where group g's rows are columns p[g] .. p[g] + K_g - 1,
 * p[g] = sum over h < g of K_h rounded up to a multiple of 128, and the columns up to p[g+1] hold
 * zero codes; each 32-column block of a row of qt (a block never spans two groups) is quantized as
 * moe_quantize_mx_rows does; st: the MX scale layout of C rows of ld.  Columns from p[G] on are
 * not written.  C a multiple of 64; ld a multiple of 128, >= moe_mx_tokens_cols_bound(R, G);
 * x and qt 16-byte aligned.  Errors: bad sizes -> INVALID_VALUE / NOT_SUPPORTED (G outside
 * 1..256); NULL or misaligned pointers -> INVALID_VALUE.  R = 0 is a no-op.
 */
moe_status moe_quantize_mx_tokens_t(const moe_bf16* x, const int32_t* offsets, int32_t G, int64_t R, int64_t C,
                                    uint8_t* qt, uint8_t* st, int64_t ld, hipStream_t stream);

/*
 * Both MX orientations of a routed buffer from one read: qt/st as moe_quantize_mx_tokens_t (may be
 * NULL) and the row-wise codes of moe_quantize_mx_rows written into a row buffer of ldr columns at
 * column col0: qr[r, col0 + c] for c < C, scales sr in the MX scale layout of R rows of ldr (blocks
 * col0/32 ..).  Two calls with col0 = 0 and col0 = C fill the joined rows [x | x2] of the gate/up
 * data gradient.  col0 a multiple of 64, ldr of 32, col0 + C <= ldr; qr 8-byte aligned; qt/st and
 * qr/sr each given together, at least one pair.  Other arguments and errors as
 * moe_quantize_mx_tokens_t.
 */
moe_status moe_quantize_mx_tokens(const moe_bf16* x, const int32_t* offsets, int32_t G, int64_t R, int64_t C,
                                  uint8_t* qt, uint8_t* st, int64_t ld, uint8_t* qr, uint8_t* sr, int64_t ldr,
                                  int64_t col0, hipStream_t stream);

/*
 * The weight gradient on MX operands (Appendix H's dW1_e = X_e^T G_e; also dW_down): At [K, ld] and
 * dCt (dC2t) [N, ld] as moe_quantize_mx_tokens_t writes them (with their scales), dB[g] [K, N]
 * (dB2[g] from dC2t, the dual gate/up form reading each At tile once) = sum over the group's
 * tokens of mx(At)[:, t] mx(dCt)[:, t]^T, E4M3 products scaled and accumulated in fp32 by the
 * matrix cores, stored fp32 (out_bf16 = 0) or rounded once to bf16.  Empty groups give zeros.
 * K, N multiples of 64; ld as for moe_quantize_mx_tokens_t; max(K, N) * ld < 2^31.  counters: NULL
 * (one workgroup per tile) or 8 int32 of device memory for a persistent grid that claims its tiles,
 * as moe_grouped_gemm_dw_persistent (zeroed here, on `stream`; calls sharing them must be ordered).
 * Errors as moe_grouped_gemm_dw_t; scale pointers 4-byte aligned; dC2t, c2_scale and dB2 all set or
 * all NULL.
 */
moe_status moe_grouped_gemm_dw_mx(const uint8_t* At, const uint8_t* a_scale, const uint8_t* dCt,
                                  const uint8_t* c_scale, const uint8_t* dC2t, const uint8_t* c2_scale,
                                  const int32_t* offsets, int32_t G, int64_t R, int64_t K, int64_t N, int64_t ld,
                                  void* dB, void* dB2, int32_t out_bf16, int32_t* counters, hipStream_t stream);

/*
 * moe_grouped_gemm_fwd with the same split of the last, partial round of tiles (same arguments,
 * definitions and errors as moe_grouped_gemm_fwd, plus a split workspace as described at
 * moe_grouped_gemm_split_workspace_bytes).  The
 * forward kernel runs one workgroup per tile; the split pieces run as extra workgroups that the
 * hardware dispatcher starts as the last full round's CUs free up.  The fused SwiGLU, when
 * requested, is computed from the summed tile exactly as in the unsplit kernel.
 */
moe_status moe_grouped_gemm_fwd_split(const moe_bf16* A, const moe_bf16* B, const moe_bf16* B2,
                                      const int32_t* offsets, int32_t G, int64_t R, int64_t K, int64_t N,
                                      moe_bf16* C, moe_bf16* C2, moe_bf16* act, void* workspace,
                                      size_t workspace_bytes, hipStream_t stream);
/*
 * moe_grouped_gemm_dx and moe_grouped_gemm_dx_swiglu_bwd with the split workspace described at
 * moe_grouped_gemm_split_workspace_bytes (same arguments, definitions and errors otherwise).
 */
moe_status moe_grouped_gemm_dx_split(const moe_bf16* dC, const moe_bf16* B, const moe_bf16* dC2,
                                     const moe_bf16* B2, const int32_t* offsets, int32_t G, int64_t R,
                                     int64_t K, int64_t N, moe_bf16* dA, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream);
moe_status moe_grouped_gemm_dx_swiglu_bwd_split(const moe_bf16* dC, const moe_bf16* B,
                                                const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                                int64_t N, const moe_bf16* h_gate, const moe_bf16* h_up,
                                                moe_bf16* dh_gate, moe_bf16* dh_up, void* workspace,
                                                size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------------------------ */
/* H, K: backward weight-gradient grouped GEMM (the paper's dW1 kernel class)                   */
/* ------------------------------------------------------------------------------------------ */

/*
 * dB[g] = A_g^T . dC_g over the rows of group g, in fp32 (section 5.4 and Appendix H:
 * dW1_e = X_e^T G_e, a contraction over the expert's ragged row count K_e).  dB is overwritten,
 * not accumulated into; an empty group (K_g = 0) gets exact zeros.  With dC2 != NULL the same A
 * tiles also give dB2[g] = A_g^T . dC2_g (gate and up weight gradients in one pass).
 * A [R,K] bf16; dC, dC2 [R,N] bf16; dB, dB2 [G,K,N] fp32.  dC2 and dB2 both NULL or both set.
 * Deterministic: each output element is reduced in one fixed order (no atomics).
 */
moe_status moe_grouped_gemm_dw(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                               const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                               int64_t N, float* dB, float* dB2, hipStream_t stream);

/*
 * The same weight gradient with each result rounded once to bf16 (round-to-nearest-even of the
 * fp32 sum): the output dtype of the paper's kernel, which stores dW1 in the input precision
 * (Appendix H, kernel epilogue and host launcher).  Halves the output bytes, which matters at the
 * paper's GPT-OSS shape (K = 2880, N = 2 x 2880, 128 experts), whose dW output is as large as its
 * operands.  Arguments, layout, empty-group zeros and errors as moe_grouped_gemm_dw; dB, dB2
 * [G,K,N] bf16.
 */
moe_status moe_grouped_gemm_dw_bf16(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                                    const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                    int64_t N, moe_bf16* dB, moe_bf16* dB2, hipStream_t stream);

/*
 * The same two weight gradients (fp32, bf16) from a persistent grid, one workgroup per CU, whose
 * workgroups take their next tile from one of eight claim counters (one per XCD) while the
 * current tile's contraction runs, instead of one workgroup per tile: the tiles of a ragged dW
 * differ in length with their group's size (section 5.4, the ragged K_e), and the per-tile start
 * and store costs then overlap.  Results are bit-identical to moe_grouped_gemm_dw /
 * moe_grouped_gemm_dw_bf16 (the same per-element reduction order).
 * counters: at least 8 int32 of device memory, 4-byte aligned, caller-owned; the call zeroes them
 * on `stream` and its kernel updates them.  Calls that may run at the same time need distinct
 * counters.  NULL or misaligned counters: MOE_ERROR_INVALID_VALUE.  Everything else as
 * moe_grouped_gemm_dw.
 */
moe_status moe_grouped_gemm_dw_persistent(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                                          const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                          int64_t N, float* dB, float* dB2, int32_t* counters,
                                          hipStream_t stream);
moe_status moe_grouped_gemm_dw_bf16_persistent(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                                               const int32_t* offsets, int32_t G, int64_t R, int64_t K,
                                               int64_t N, moe_bf16* dB, moe_bf16* dB2, int32_t* counters,
                                               hipStream_t stream);

/*
 * moe_grouped_gemm_dw_persistent with a split workspace (dB = A^T dC over one group's rows, fp32;
 * the weight gradient of section 5.4 and Appendix H):
 * with a single group (G == 1, e.g. the shared experts' weight gradient over all T tokens) every
 * tile has the same contraction, and when the tiles do not fill the last round of CU slots (fewer
 * tiles than CUs included) those tiles are split along the contraction into up to 8 pieces of at
 * least 64 steps, each piece's fp32 partial tile goes to the workspace, and the last piece to
 * arrive sums the pieces in piece order (a fixed order: the result does not depend on which
 * piece finishes last) and stores the tile, as the split forms of the forward and dX products
 * do.  Split tiles sum their contraction in a different association than the unsplit kernel
 * (each piece separately, then the pieces), so results can differ from it by rounding.  With
 * G > 1 the workspace is not used and the call equals moe_grouped_gemm_dw_persistent.
 * workspace: moe_grouped_gemm_split_workspace_bytes() bytes, 16-byte aligned, caller-owned; its
 * counters are zeroed on `stream` by the call; calls sharing it must be ordered.  A smaller or
 * misaligned workspace: MOE_ERROR_WORKSPACE; NULL: no split.  Everything else as
 * moe_grouped_gemm_dw_persistent.
 */
moe_status moe_grouped_gemm_dw_split(const moe_bf16* A, const moe_bf16* dC, const moe_bf16* dC2,
                                     const int32_t* offsets, int32_t G, int64_t R, int64_t K, int64_t N,
                                     float* dB, float* dB2, int32_t* counters, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream);

/*
 * The weight gradient of moe_grouped_gemm_dw from contraction-major copies of its operands
 * (the layout moe_transpose_grouped writes): At [K, ld] and dCt, dC2t [N, ld] bf16, in which
 * group g's rows occupy columns pstart[g] .. pstart[g] + K_g - 1, pstart[g] = sum over h < g of
 * K_h rounded up to a multiple of 32, and the padding columns hold zeros.  Same definition,
 * outputs, empty-group zeros, ordering and errors as moe_grouped_gemm_dw (out_bf16 = 0: fp32
 * dB, dB2 [G,K,N]; 1: bf16, as moe_grouped_gemm_dw_bf16); the contraction of every group is
 * contiguous, so both operands are read without transposition, and the results are bitwise
 * identical to moe_grouped_gemm_dw's.  ld: a multiple of 64, at least
 * moe_transposed_cols_bound(R, G); max(K, N) * ld * 2 < 2^31.
 */
moe_status moe_grouped_gemm_dw_t(const moe_bf16* At, const moe_bf16* dCt, const moe_bf16* dC2t,
                                 const int32_t* offsets, int32_t G, int64_t R, int64_t K, int64_t N,
                                 int64_t ld, void* dB, void* dB2, int32_t out_bf16,
                                 hipStream_t stream);

/* Columns the contraction-major layout needs at most: round32(R) + 32 * G. */
int64_t moe_transposed_cols_bound(int64_t R, int32_t G);

/*
 * dst[c, pstart[g] + i] = src[offsets[g] + i, c] for 0 <= i < K_g, zeros in each group's padding
 * up to the next multiple of 32 (and up to the end of the last 64-column block): the
 * contraction-major copy that moe_grouped_gemm_dw_t reads.  src [R, C] bf16 row-major (the rows
 * of the routed buffer, grouped by offsets); dst [C, ld_dst] bf16; C a multiple of 64; ld_dst a
 * multiple of 64 and >= moe_transposed_cols_bound(R, G).
 */
moe_status moe_transpose_grouped(const moe_bf16* src, const int32_t* offsets, int32_t G, int64_t R,
                                 int64_t C, moe_bf16* dst, int64_t ld_dst, hipStream_t stream);

/* ------------------------------------------------------------------------------------------ */
/* Router: logits, backward through the routing weights, load-balancing loss                   */
/* ------------------------------------------------------------------------------------------ */

/*
 * logits[t, e] = sum_i x[t, i] * wr[i, e] (+ bias[e]) in fp32: the router ahead of the top-k
 * selection (section 5.4 names top-k routing; the router itself is not described: one linear
 * map, the usual MoE router).  x [T,d] bf16 (16-byte aligned); wr [d,E] fp32; bias [E] fp32 or
 * NULL; logits [T,E] fp32.  1 <= E <= 256, d a multiple of 64.  The sum runs in a fixed order
 * (d <= 4096: products over groups of 8 consecutive columns, the groups added pairwise within a
 * 512-column slice and the slices in order; larger d: eight slices of the hidden dimension added
 * in order): deterministic, but not bitwise equal to a CPU fp32 dot product, so decisions at
 * near-tied logits may differ from one computed elsewhere.
 */
moe_status moe_router_logits(const moe_bf16* x, const float* wr, const float* bias, int64_t T,
                             int64_t d, int32_t E, float* logits, hipStream_t stream);

/* Bytes of device workspace moe_router_bwd needs (partial sums of dWr over token chunks and a
   transposed copy of Wr). */
size_t moe_router_bwd_workspace_bytes(int64_t T, int64_t d, int32_t E);

/*
 * Backward of the router, given the routing of moe_route_permute and d_topk_w [T,k] from
 * moe_unpermute_combine_bwd:
 *   dlogits[t, e] = p[t, e] * (G[t, e] - sum_j d_topk_w[t, j] * topk_w[t, j])
 *                   + aux_alpha * E / T * q[t, e] * (f[e] - sum_e' f[e'] * q[t, e'])
 * where p are the probabilities the weights were read from (the k normalized weights at the
 * selected experts and 0 elsewhere when normalize_topk, else the full softmax q of the logits),
 * G[t, e] = d_topk_w[t, j] for e = topk_idx[t, j] (0 for unselected experts: the selection
 * passes no gradient), and f[e] = (offsets[e+1] - offsets[e]) / (T*k) the share of slots expert e
 * received (the Switch-style load-balancing loss alpha*E*sum_e f_e*mean_t(q_e), counts held
 * constant; aux_alpha = 0 leaves it out and offsets may then be NULL).  Then
 *   dwr[i, e] = sum_t x[t, i] * dlogits[t, e]                               (fp32, overwritten)
 *   dx[t, i]  = bf16(dx[t, i] + sum_e dlogits[t, e] * wr[i, e])              (if dx != NULL)
 * i.e. the router's share of the token gradient is added to the stored bf16 dX of the experts
 * (one more rounding).  logits [T,E], topk_w, d_topk_w [T,k] fp32; topk_idx [T,k] int32;
 * dlogits [T,E] fp32 (output); workspace of moe_router_bwd_workspace_bytes; deterministic.
 */
moe_status moe_router_bwd(const moe_bf16* x, const float* wr, const float* logits,
                          const int32_t* topk_idx, const float* topk_w, const float* d_topk_w,
                          const int32_t* offsets, int64_t T, int64_t d, int32_t E, int32_t k,
                          int32_t normalize_topk, float aux_alpha, void* workspace,
                          size_t workspace_bytes, float* dlogits, float* dwr, moe_bf16* dx,
                          hipStream_t stream);

/*
 * The unpermute-sum of dX fused with the router's share of the token gradient:
 *   dx[t, i] = bf16( bf16(sum_j dx_perm[row_of_slot[t*k + j], i] + add[t, i])
 *                    + sum_e dlogits[t, e] * wr[i, e] )
 * i.e. exactly moe_unpermute_combine (topk_w = NULL) followed by moe_router_bwd's update of dx,
 * bitwise, in one pass over dX instead of two (the router's share of dX, section 5.4's top-k
 * routing read as a linear router; the experts' sum as in moe_unpermute_combine).  dx_perm [T*k,d]
 * bf16; row_of_slot [T*k] int32; add [T,d] bf16 or NULL (the shared experts' dX); dlogits [T,E]
 * and wr [d,E] fp32; dx [T,d] bf16 output (must not overlap dx_perm).  dx_perm, add and dx 16-byte
 * aligned.  Supports 1 <= E <= 16 and d <= 4096 (a multiple of 64); other sizes return
 * MOE_ERROR_NOT_SUPPORTED (call the two functions instead).  No workspace.
 */
moe_status moe_unpermute_router_dx(const moe_bf16* dx_perm, const int32_t* row_of_slot,
                                   const moe_bf16* add, const float* dlogits, const float* wr,
                                   int64_t T, int64_t d, int32_t k, int32_t E, moe_bf16* dx,
                                   hipStream_t stream);

/* Bytes of device workspace moe_router_aux_loss needs. */
size_t moe_router_aux_loss_workspace_bytes(int64_t T, int32_t E);

/*
 * The load-balancing loss itself: loss[0] = alpha * E * sum_e f[e] * P[e], f as above and P[e]
 * the mean over tokens of the full softmax of the logits (fp32; fixed reduction order).
 */
moe_status moe_router_aux_loss(const float* logits, const int32_t* offsets, int64_t T, int32_t E,
                               int32_t k, float alpha, void* workspace, size_t workspace_bytes,
                               float* loss, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_MI355X_H */
