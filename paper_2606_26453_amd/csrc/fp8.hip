// Per-row quantization of bf16 rows to OCP E4M3 with an fp32 scale per row (the operand format of
// the FP8 grouped product): amax = max |x[r, :]|, scale[r] = amax / 448, and each element becomes
// the E4M3 code nearest to x * (448 / amax), ties to the even mantissa (the scaled magnitudes
// exceed 448 by at most a rounding of the product, which rounds back to 448); an all-zero row gets
// scale 1 and zero codes.  The quotients and the product are single fp32 operations (IEEE round to
// nearest), so the codes are a function of the inputs alone.
#include "common.h"

namespace moe {
namespace {

// E4M3 (OCP e4m3fn) codes of four fp32 values, packed low byte first, by gfx950's conversion
// instruction (v_cvt_pk_fp8_f32, two values each): round to nearest, ties to the even mantissa, 3
// mantissa bits in the normal range (2^-6 and up) and multiples of 2^-9 below it.  Every input here
// has |y| <= 448 up to one rounding of its scaling product (which rounds back to 448).
__device__ __forceinline__ uint32_t e4m3_pack4(float a, float b, float c, float d) {
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c, d, lo, true);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// One workgroup (256 threads) per row; each thread handles 8 elements (16 bytes) at a time.  With
// a second source x2 the row is the concatenation [x[r, :] | x2[r, :]] (one amax and one scale
// over both, x's codes first): the operand of a product whose contraction runs over two matrices.
__global__ __launch_bounds__(256) void quantize_fp8_rows_kernel(const u32x4* __restrict__ x,
                                                                const u32x4* __restrict__ x2, int64_t K8,
                                                                uint2* __restrict__ q, float* __restrict__ scale) {
  __shared__ float s_max[4];
  const int64_t r = blockIdx.x;
  const int nsrc = x2 ? 2 : 1;
  float m = 0.0f;
  for (int h = 0; h < nsrc; ++h) {
    const u32x4* row = (h ? x2 : x) + r * K8;
    for (int64_t c = threadIdx.x; c < K8; c += 256) {
      const u32x4 v = row[c];
#pragma unroll
      for (int e = 0; e < 4; ++e) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[e])), fabsf(bf16_hi(v[e]))));
    }
  }
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) s_max[threadIdx.x >> 6] = m;
  __syncthreads();
  const float amax = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
  const bool nz = amax > 0.0f;
  const float inv = nz ? __fdiv_rn(448.0f, amax) : 1.0f;
  if (threadIdx.x == 0) scale[r] = nz ? __fdiv_rn(amax, 448.0f) : 1.0f;
  for (int h = 0; h < nsrc; ++h) {
    const u32x4* row = (h ? x2 : x) + r * K8;
    uint2* qrow = q + r * (nsrc * K8) + h * K8;
    for (int64_t c = threadIdx.x; c < K8; c += 256) {
      const u32x4 v = row[c];
      uint32_t w[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        w[hh] = e4m3_pack4(__fmul_rn(bf16_lo(v[2 * hh]), inv), __fmul_rn(bf16_hi(v[2 * hh]), inv),
                           __fmul_rn(bf16_lo(v[2 * hh + 1]), inv), __fmul_rn(bf16_hi(v[2 * hh + 1]), inv));
      }
      qrow[c] = make_uint2(w[0], w[1]);
    }
  }
}

// The same quantization applied to the columns of a weight W [G, K, N] (column n of expert g: one
// output channel, its K elements the contraction), written transposed: row (g, n) of Q [G, N', K]
// holds column n's codes and scale [G, N'] its scale.  With a second weight W2 of the same shape
// the output interleaves the two by IL = 128 channels: output row 2*IL*b + i (i < IL) is W's
// channel IL*b + i and row 2*IL*b + IL + i is W2's.  Code for code and scale for scale this is
// quantize_fp8_rows_kernel on the transposed (and interleaved) weight: the same amax, quotients
// and products.  Three passes, each spread over (64-column block, expert, matrix, K block)
// workgroups so that long contractions still fill the chip: the column amax (partial maxima of K
// blocks combined with an integer atomic max on the fp32 bits, which orders non-negative floats
// like their values; kept in `scale`), the codes, then scale = amax / 448.  Thread t of a
// workgroup handles 8-column chunk t % 8 of row (quad) t / 8, so that a wavefront's 16-byte loads
// cover 8 whole 128-byte row segments.
constexpr int QC_IL = 128;   // gate/up interleave (channels)
constexpr int QC_CW = 64;    // columns per workgroup
constexpr int QC_KA = 2048;  // rows per workgroup, amax pass
constexpr int QC_KQ = 1024;  // rows per workgroup, code pass (8 blocks of 128)

__device__ __forceinline__ int64_t qc_out_row(int64_t n, bool dual, bool second) {
  if (!dual) return n;
  return (n / QC_IL) * 2 * QC_IL + (second ? QC_IL : 0) + n % QC_IL;
}

__global__ __launch_bounds__(256) void fill_f32_kernel(float* p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

// pass 1: blockIdx.z = matrix * kblocks + kb
__global__ __launch_bounds__(256) void amax_cols_kernel(const uint16_t* __restrict__ w, const uint16_t* __restrict__ w2,
                                                        int64_t K, int64_t N, int64_t n_out, int kblocks,
                                                        float* __restrict__ amax) {
  __shared__ float s_part[32][QC_CW];
  const int t = threadIdx.x, c = t & 7, rq = t >> 3;
  const bool second = (int)blockIdx.z >= kblocks;
  const int64_t kb = blockIdx.z - (second ? kblocks : 0);
  const int64_t g = blockIdx.y, n0 = (int64_t)blockIdx.x * QC_CW;
  const uint16_t* src = (second ? w2 : w) + g * K * N + n0 + 8 * c;
  const int64_t k_end = (kb + 1) * QC_KA < K ? (kb + 1) * QC_KA : K;
  float m[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) m[i] = 0.0f;
#pragma unroll 4
  for (int64_t k = kb * QC_KA + rq; k < k_end; k += 32) {
    const u32x4 v = ld_stream(reinterpret_cast<const u32x4*>(src + k * N));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      m[2 * e] = fmaxf(m[2 * e], fabsf(bf16_lo(v[e])));
      m[2 * e + 1] = fmaxf(m[2 * e + 1], fabsf(bf16_hi(v[e])));
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) s_part[rq][8 * c + i] = m[i];
  __syncthreads();
  if (t < QC_CW) {
    float a = 0.0f;
    for (int r = 0; r < 32; ++r) a = fmaxf(a, s_part[r][t]);
    // fmaxf drops NaNs as the row quantizer's reduction does, so a >= 0 here
    atomicMax(reinterpret_cast<unsigned*>(amax) + g * n_out + qc_out_row(n0 + t, w2 != nullptr, second),
              __float_as_uint(a));
  }
}

// pass 2: the codes of K block kb (QC_KQ rows) of 64 columns, written transposed 128 rows at a time
__global__ __launch_bounds__(256) void quantize_cols_kernel(const uint16_t* __restrict__ w,
                                                            const uint16_t* __restrict__ w2, int64_t K, int64_t N,
                                                            int64_t n_out, int kblocks, const float* __restrict__ amax,
                                                            uint8_t* __restrict__ q) {
  constexpr int TS = 132;   // LDS row stride (bytes) of the transposed 64-column x 128-row block
  __shared__ __attribute__((aligned(16))) uint8_t s_t[QC_CW * TS];
  const int t = threadIdx.x, c = t & 7, rq = t >> 3;
  const bool second = (int)blockIdx.z >= kblocks;
  const int64_t kb = blockIdx.z - (second ? kblocks : 0);
  const int64_t g = blockIdx.y, n0 = (int64_t)blockIdx.x * QC_CW;
  const bool dual = w2 != nullptr;
  const uint16_t* src = (second ? w2 : w) + g * K * N + n0 + 8 * c;
  float inv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float a = amax[g * n_out + qc_out_row(n0 + 8 * c + i, dual, second)];
    inv[i] = a > 0.0f ? __fdiv_rn(448.0f, a) : 1.0f;
  }
  const int64_t k_beg = kb * QC_KQ, k_end = (kb + 1) * QC_KQ < K ? (kb + 1) * QC_KQ : K;
  for (int64_t k0 = k_beg; k0 < k_end; k0 += 128) {
    uint32_t packed[8];
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t k = k0 + 4 * rq + u;
      v[u] = u32x4{0u, 0u, 0u, 0u};
      if (k < k_end) v[u] = ld_stream(reinterpret_cast<const u32x4*>(src + k * N));
    }
    // column 2e (2e+1) of the chunk: its four rows' codes, row u in byte u
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      packed[2 * e] = e4m3_pack4(__fmul_rn(bf16_lo(v[0][e]), inv[2 * e]), __fmul_rn(bf16_lo(v[1][e]), inv[2 * e]),
                                 __fmul_rn(bf16_lo(v[2][e]), inv[2 * e]), __fmul_rn(bf16_lo(v[3][e]), inv[2 * e]));
      packed[2 * e + 1] =
          e4m3_pack4(__fmul_rn(bf16_hi(v[0][e]), inv[2 * e + 1]), __fmul_rn(bf16_hi(v[1][e]), inv[2 * e + 1]),
                     __fmul_rn(bf16_hi(v[2][e]), inv[2 * e + 1]), __fmul_rn(bf16_hi(v[3][e]), inv[2 * e + 1]));
    }
    __syncthreads();   // the previous block's codes have been written out
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<uint32_t*>(s_t + (8 * c + i) * TS + 4 * rq) = packed[i];
    __syncthreads();
    // write out: thread -> column j = t / 4, 32 bytes at k0 + 32 * (t % 4)
    const int j = t >> 2, seg = t & 3;
    const int64_t kk = k0 + 32 * seg;
    uint32_t o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = *reinterpret_cast<const uint32_t*>(s_t + j * TS + 32 * seg + 4 * i);
    uint8_t* dst = q + (g * n_out + qc_out_row(n0 + j, dual, second)) * K + kk;
    if (kk < k_end) *reinterpret_cast<u32x4*>(dst) = u32x4{o[0], o[1], o[2], o[3]};
    if (kk + 16 < k_end) *reinterpret_cast<u32x4*>(dst + 16) = u32x4{o[4], o[5], o[6], o[7]};
  }
}

// pass 3: amax -> scale
__global__ __launch_bounds__(256) void scale_from_amax_kernel(float* __restrict__ s, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) {
    const float a = s[i];
    s[i] = a > 0.0f ? __fdiv_rn(a, 448.0f) : 1.0f;
  }
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status moe_quantize_fp8_weight(const moe_bf16* w, const moe_bf16* w2, int64_t G, int64_t K,
                                              int64_t N, uint8_t* q, float* scale, hipStream_t stream) {
  const char* fn = "moe_quantize_fp8_weight";
  if (G < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  const int nmul = w2 ? QC_IL : QC_CW;
  if (K % 16 || N % nmul)
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K must be a multiple of 16 and N of %d", fn, nmul);
  const int64_t nmat = w2 ? 2 : 1;
  const int64_t ka = (K + QC_KA - 1) / QC_KA, kq = (K + QC_KQ - 1) / QC_KQ;
  if (G > 65535 || N / QC_CW > 0x7fffffff || nmat * kq > 65535)
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: too many experts, columns or rows", fn);
  if (G == 0) return MOE_SUCCESS;
  if (!w || !q || !scale) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (!aligned16(w) || (w2 && !aligned16(w2)) || !aligned16(q) || (reinterpret_cast<uintptr_t>(scale) & 3))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: w, w2 and q must be 16-byte, scale 4-byte aligned", fn);
  const int64_t n_out = nmat * N, ns = G * n_out;
  const uint16_t* a = w;
  const uint16_t* b = w2;
  fill_f32_kernel<<<(unsigned)((ns + 255) / 256), 256, 0, stream>>>(scale, ns, 0.0f);
  amax_cols_kernel<<<dim3((unsigned)(N / QC_CW), (unsigned)G, (unsigned)(nmat * ka)), 256, 0, stream>>>(
      a, b, K, N, n_out, (int)ka, scale);
  quantize_cols_kernel<<<dim3((unsigned)(N / QC_CW), (unsigned)G, (unsigned)(nmat * kq)), 256, 0, stream>>>(
      a, b, K, N, n_out, (int)kq, scale, q);
  scale_from_amax_kernel<<<(unsigned)((ns + 255) / 256), 256, 0, stream>>>(scale, ns);
  return check_launch("quantize_cols_kernel");
}

namespace moe {
namespace {
moe_status quantize_rows_impl(const char* fn, const moe_bf16* x, const moe_bf16* x2, int64_t M, int64_t K,
                              uint8_t* q, float* scale, hipStream_t stream) {
  if (M < 0 || K <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (K % 16) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K must be a multiple of 16", fn);
  if (M >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: M >= 2^31", fn);
  if (M == 0) return MOE_SUCCESS;
  if (!x || !q || !scale) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (!aligned16(x) || (x2 && !aligned16(x2)) || (reinterpret_cast<uintptr_t>(q) & 7) ||
      (reinterpret_cast<uintptr_t>(scale) & 3))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: x (and x2) must be 16-byte, q 8-byte, scale 4-byte aligned", fn);
  quantize_fp8_rows_kernel<<<(unsigned)M, 256, 0, stream>>>(reinterpret_cast<const u32x4*>(x),
                                                             reinterpret_cast<const u32x4*>(x2), K / 8,
                                                             reinterpret_cast<uint2*>(q), scale);
  return check_launch("quantize_fp8_rows_kernel");
}
}  // namespace
}  // namespace moe

extern "C" moe_status moe_quantize_fp8_rows(const moe_bf16* x, int64_t M, int64_t K, uint8_t* q, float* scale,
                                            hipStream_t stream) {
  return quantize_rows_impl("moe_quantize_fp8_rows", x, nullptr, M, K, q, scale, stream);
}

extern "C" moe_status moe_quantize_fp8_rows2(const moe_bf16* x, const moe_bf16* x2, int64_t M, int64_t K,
                                             uint8_t* q, float* scale, hipStream_t stream) {
  if (!x2) return fail(MOE_ERROR_INVALID_VALUE, "moe_quantize_fp8_rows2: x2 is NULL");
  return quantize_rows_impl("moe_quantize_fp8_rows2", x, x2, M, K, q, scale, stream);
}

// ---------------------------------------------------------------------------------------------
// MX quantization: E4M3 codes with one power-of-two scale per 32 consecutive elements of a row,
// stored as an E8M0 byte (value 2^(byte - 127)).  The block's exponent is the smallest e with
// amax <= 448 * 2^e (no element saturates), at least -127 (all-zero blocks get byte 0); the codes
// round x * 2^-e, an exact scaling, to the nearest E4M3 value (ties to the even mantissa).
// ---------------------------------------------------------------------------------------------
namespace moe {
namespace {

// amax = (1 + m / 2^23) * 2^(E - 127) for a biased exponent E >= 1, and 448 * 2^e = 1.75 * 2^(e + 8):
// e = E - 135 when the significand is at most 1.75 (m <= 0x600000), else E - 134.  A zero or
// subnormal amax (E = 0) gives at most -134, raised to -127.  The byte is e + 127.
__device__ __forceinline__ uint32_t mx_scale_byte(float amax) {
  const uint32_t b = __float_as_uint(amax);   // amax >= 0
  const int byte = (int)(b >> 23) - 8 + ((b & 0x7FFFFFu) > 0x600000u ? 1 : 0);
  return byte < 0 ? 0u : (uint32_t)byte;
}

// 2^-e for byte = e + 127: the biased exponent 127 - e = 254 - byte, 7 .. 254 for the bytes that
// finite bf16 inputs produce (0 .. 247)
__device__ __forceinline__ float mx_inv_scale(uint32_t byte) { return __uint_as_float((254u - byte) << 23); }

// the codes of a, b, c, d times an MX block's inverse scale (a power of two: the products are exact)
__device__ __forceinline__ uint32_t e4m3_pack4(float a, float b, float c, float d, float inv) {
  return e4m3_pack4(a * inv, b * inv, c * inv, d * inv);
}

// Scale byte of block b of row r in the MX scale layout of a matrix with `rows` rows: the four
// scales of a row's 128-element group form one 4-byte word, and the words of all rows for one group
// lie side by side (what the product's scale loads read, 256 contiguous bytes per wavefront).
__device__ __forceinline__ int64_t mx_scale_at(int64_t r, int64_t b, int64_t rows) {
  return ((b >> 2) * rows + r) * 4 + (b & 3);
}

// Rows: workgroup (row r, chunk block cb) covers 8-element chunks cb*256 .. cb*256+255 of row r of
// the [M, C] matrix (C = K, or 2K for the concatenation [x | x2]); four neighbouring lanes hold a
// 32-element block and combine their maxima by lane exchange.
__global__ __launch_bounds__(256) void quantize_mx_rows_kernel(const u32x4* __restrict__ x, const u32x4* __restrict__ x2,
                                                               int64_t K8, int cpr, int64_t M, uint2* __restrict__ q,
                                                               uint8_t* __restrict__ s) {
  const int64_t C8 = x2 ? 2 * K8 : K8;
  const int64_t r = blockIdx.x / cpr;
  const int64_t c8 = (int64_t)(blockIdx.x - r * cpr) * 256 + threadIdx.x;
  const bool live = c8 < C8;   // whole blocks: C8 is a multiple of 4
  u32x4 v = {0u, 0u, 0u, 0u};
  if (live) v = (c8 < K8) ? x[r * K8 + c8] : x2[r * K8 + c8 - K8];
  float m = 0.0f;
#pragma unroll
  for (int e = 0; e < 4; ++e) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[e])), fabsf(bf16_hi(v[e]))));
  m = fmaxf(m, __shfl_xor(m, 1));
  m = fmaxf(m, __shfl_xor(m, 2));
  const uint32_t byte = mx_scale_byte(m);
  const float inv = mx_inv_scale(byte);
  if (live) {
    q[r * C8 + c8] = make_uint2(e4m3_pack4(bf16_lo(v[0]), bf16_hi(v[0]), bf16_lo(v[1]), bf16_hi(v[1]), inv),
                                e4m3_pack4(bf16_lo(v[2]), bf16_hi(v[2]), bf16_lo(v[3]), bf16_hi(v[3]), inv));
    if ((c8 & 3) == 0) s[mx_scale_at(r, c8 >> 2, M)] = (uint8_t)byte;
  }
}

// A 128 x CW bf16 tile staged row-major in LDS with its 16-byte chunks (8 columns) permuted per
// 32-row block: element (k, n) sits at k*CW + (n ^ 16*(k/32)), so that the lanes of a wavefront
// reading 16 columns in each of the four blocks (below) cover four disjoint 32-byte spans of a
// row, i.e. distinct banks.
template <int CW = 64>
__device__ __forceinline__ int mx_tile_at(int k, int n) { return k * CW + (n ^ ((k >> 5) << 4)); }

// From that tile: the MX codes of column n over rows 32*kb .. 32*kb + 31 (one block), packed 4 to
// a word in o[8]; returns the block's scale byte.
template <int CW = 64>
__device__ __forceinline__ uint32_t mx_tile_col_block(const uint16_t* s_w, int n, int kb, uint32_t o[8]) {
  float v[32];
  float m = 0.0f;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    v[i] = __uint_as_float((uint32_t)s_w[mx_tile_at<CW>(32 * kb + i, n)] << 16);
    m = fmaxf(m, fabsf(v[i]));
  }
  const uint32_t byte = mx_scale_byte(m);
  const float inv = mx_inv_scale(byte);
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = e4m3_pack4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3], inv);
  return byte;
}

// Weights, both orientations from one read.  Workgroup (column block n0 = CW*bx, row block
// k0 = 128*by, matrix/expert bz) stages the 128 x CW tile of W[g] (or W2[g]) in LDS (CW = 128
// when N allows: each output row segment is then a whole 128-byte line, written by one workgroup):
//   rows (qr, sr): row (g, k) of the [G, K, nmat*N] matrix [W[g] | W2[g]], blocks of 32 columns;
//     thread t: column chunk t%(CW/8) of rows k0 + t/(CW/8) + (256/(CW/8))*u, lanes t^1, t^2
//     share its block;
//   columns (qt, st): row (g, n') of [G, N', K] = column n of W[g] (or W2[g], interleaved by 128
//     as in the fp32-scale weight layout), blocks of 32 rows; thread t: columns t/4 + 64j, rows
//     k0 + 32*(t%4) .. +31, 32 contiguous bytes of row n' (the four lanes of a column write its
//     128 bytes of the row).
// Scales in the MX scale layout of each output (rows G*K for qr, G*N' for qt).
template <int CW>
__global__ __launch_bounds__(256) void quantize_mx_weight_kernel(const uint16_t* __restrict__ w,
                                                                 const uint16_t* __restrict__ w2, int64_t G, int64_t K,
                                                                 int64_t N, uint8_t* __restrict__ qt,
                                                                 uint8_t* __restrict__ st, uint8_t* __restrict__ qr,
                                                                 uint8_t* __restrict__ sr) {
  constexpr int CPR = CW / 8, RP = 256 / CPR;   // chunks per tile row, rows per pass
  __shared__ __attribute__((aligned(16))) uint16_t s_w[128 * CW];
  const int t = threadIdx.x;
  const int nmat = w2 ? 2 : 1;
  const int64_t g = blockIdx.z / nmat;
  const bool second = (int)(blockIdx.z - g * nmat) == 1;
  const int64_t n0 = (int64_t)blockIdx.x * CW, k0 = (int64_t)blockIdx.y * 128;
  const uint16_t* src = (second ? w2 : w) + g * K * N + n0;
  const int c8 = t % CPR, rq = t / CPR;
#pragma unroll
  for (int u = 0; u < 128 / RP; ++u) {
    const int kl = rq + RP * u;
    const int64_t k = k0 + kl;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (k < K) v = *reinterpret_cast<const u32x4*>(src + k * N + 8 * c8);
    *reinterpret_cast<u32x4*>(s_w + mx_tile_at<CW>(kl, 8 * c8)) = v;
    if (qr != nullptr) {
      float m = 0.0f;
#pragma unroll
      for (int e = 0; e < 4; ++e) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[e])), fabsf(bf16_hi(v[e]))));
      m = fmaxf(m, __shfl_xor(m, 1));
      m = fmaxf(m, __shfl_xor(m, 2));
      const uint32_t byte = mx_scale_byte(m);
      const float inv = mx_inv_scale(byte);
      if (k < K) {
        const int64_t row = g * K + k, col = (second ? N : 0) + n0 + 8 * c8;
        *reinterpret_cast<uint2*>(qr + row * (nmat * N) + col) =
            make_uint2(e4m3_pack4(bf16_lo(v[0]), bf16_hi(v[0]), bf16_lo(v[1]), bf16_hi(v[1]), inv),
                       e4m3_pack4(bf16_lo(v[2]), bf16_hi(v[2]), bf16_lo(v[3]), bf16_hi(v[3]), inv));
        if ((c8 & 3) == 0) sr[mx_scale_at(row, col >> 5, G * K)] = (uint8_t)byte;
      }
    }
  }
  if (qt == nullptr) return;   // uniform
  __syncthreads();
  // thread -> columns n = t/4 + 64j, block kb = t%4: the four lanes of a column hold its 128
  // contiguous bytes of the output row, so a wavefront's stores touch 16 rows instead of 64
  const int kb = t & 3;
  if (k0 + 32 * kb >= K) return;   // K is a multiple of 32: the block is whole or absent
#pragma unroll
  for (int j = 0; j < CW / 64; ++j) {
    const int n = (t >> 2) + 64 * j;
    uint32_t o[8];
    const uint32_t byte = mx_tile_col_block<CW>(s_w, n, kb, o);
    const int64_t row = g * (nmat * N) + qc_out_row(n0 + n, w2 != nullptr, second);
    uint8_t* dst = qt + row * K + k0 + 32 * kb;
    *reinterpret_cast<u32x4*>(dst) = u32x4{o[0], o[1], o[2], o[3]};
    *reinterpret_cast<u32x4*>(dst + 16) = u32x4{o[4], o[5], o[6], o[7]};
    st[mx_scale_at(row, (k0 >> 5) + kb, G * nmat * N)] = (uint8_t)byte;
  }
}

// Token-major operands of the weight gradient: x [R, C] bf16, rows grouped by offsets -> qt [C, ld]
// codes with group g's K_g rows as columns p[g] .. p[g] + K_g - 1, p the prefix of the counts
// rounded up to 128 (no 32-element block spans two groups, and each group starts a 128-element
// scale word), zero codes in each group's padding; scales in the MX layout of C rows of ld.
// Workgroup (CW-column block n0 = CW*bx of x, CW = 128 when the widths allow, else 64; 128-column
// block j0 = 128*by of qt) stages the 128 source rows that land in columns j0 .. j0+127 (zeros past
// the group's end) and quantizes them
// column by column as the weight kernel's transposed half does; blocks past p[G] are left alone.
// With qr, the same read also gives the row-wise codes (every source row lies in exactly one such
// tile): row r's blocks of 32 columns go to qr[r, col0 + c] (rows of ldr bytes, e.g. one half of
// the joined rows [dH_gate | dH_up]) with scales in the MX layout of R rows of ldr.
template <int CW>
__global__ __launch_bounds__(256) void quantize_mx_tokens_t_kernel(const uint16_t* __restrict__ x,
                                                                   const int32_t* __restrict__ offsets, int G,
                                                                   int64_t R, int64_t C, int64_t ld,
                                                                   uint8_t* __restrict__ qt, uint8_t* __restrict__ st,
                                                                   uint8_t* __restrict__ qr, uint8_t* __restrict__ sr,
                                                                   int64_t ldr, int64_t col0) {
  constexpr int CPR = CW / 8, RP = 256 / CPR;   // chunks per tile row, rows per pass
  __shared__ int s_o[257];
  __shared__ int s_p[257];
  __shared__ __attribute__((aligned(16))) uint16_t s_w[128 * CW];
  const int t = threadIdx.x;
  for (int i = t; i <= G; i += 256) s_o[i] = offsets[i];
  __syncthreads();
  s_p[t + 1] = t < G ? ((s_o[t + 1] - s_o[t] + 127) & ~127) : 0;
  if (t == 0) s_p[0] = 0;
  __syncthreads();
  for (int off = 1; off < G; off <<= 1) {   // inclusive scan of the rounded counts
    const int add = t >= off ? s_p[t + 1 - off] : 0;
    __syncthreads();
    s_p[t + 1] += add;
    __syncthreads();
  }
  const int64_t j0 = (int64_t)blockIdx.y * 128;
  if (j0 >= s_p[G]) return;   // uniform
  const int g = __syncthreads_count(t < G && s_p[t + 1] <= j0);   // the group holding j0 .. j0+127
  const int64_t src0 = s_o[g] + (j0 - s_p[g]), src_end = s_o[g + 1];
  const int64_t n0 = (int64_t)blockIdx.x * CW;
  const int c8 = t % CPR, rq = t / CPR;
#pragma unroll
  for (int u = 0; u < 128 / RP; ++u) {
    const int kl = rq + RP * u;
    const int64_t r = src0 + kl;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r < src_end) v = *reinterpret_cast<const u32x4*>(x + r * C + n0 + 8 * c8);
    *reinterpret_cast<u32x4*>(s_w + mx_tile_at<CW>(kl, 8 * c8)) = v;
    if (qr != nullptr) {   // uniform; lanes t^1, t^2 share the block (same row)
      float m = 0.0f;
#pragma unroll
      for (int e = 0; e < 4; ++e) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[e])), fabsf(bf16_hi(v[e]))));
      m = fmaxf(m, __shfl_xor(m, 1));
      m = fmaxf(m, __shfl_xor(m, 2));
      const uint32_t byte = mx_scale_byte(m);
      const float inv = mx_inv_scale(byte);
      if (r < src_end) {
        const int64_t col = col0 + n0 + 8 * c8;
        *reinterpret_cast<uint2*>(qr + r * ldr + col) =
            make_uint2(e4m3_pack4(bf16_lo(v[0]), bf16_hi(v[0]), bf16_lo(v[1]), bf16_hi(v[1]), inv),
                       e4m3_pack4(bf16_lo(v[2]), bf16_hi(v[2]), bf16_lo(v[3]), bf16_hi(v[3]), inv));
        if ((c8 & 3) == 0) sr[mx_scale_at(r, col >> 5, R)] = (uint8_t)byte;
      }
    }
  }
  if (qt == nullptr) return;   // uniform
  __syncthreads();
  const int kb = t & 3;   // columns t/4 + 64j, as in the weight kernel
#pragma unroll
  for (int j = 0; j < CW / 64; ++j) {
    const int n = (t >> 2) + 64 * j;
    uint32_t o[8];
    const uint32_t byte = mx_tile_col_block<CW>(s_w, n, kb, o);
    uint8_t* dst = qt + (n0 + n) * ld + j0 + 32 * kb;
    *reinterpret_cast<u32x4*>(dst) = u32x4{o[0], o[1], o[2], o[3]};
    *reinterpret_cast<u32x4*>(dst + 16) = u32x4{o[4], o[5], o[6], o[7]};
    st[mx_scale_at(n0 + n, (j0 >> 5) + kb, C)] = (uint8_t)byte;
  }
}

}  // namespace
}  // namespace moe

extern "C" int64_t moe_mx_tokens_cols_bound(int64_t R, int32_t G) {
  return R < 0 || G < 1 ? 0 : (R + 127 * (int64_t)G + 127) / 128 * 128;
}

namespace moe {
namespace {
moe_status quantize_mx_tokens_impl(const char* fn, const moe_bf16* x, const int32_t* offsets, int32_t G, int64_t R,
                                   int64_t C, uint8_t* qt, uint8_t* st, int64_t ld, uint8_t* qr, uint8_t* sr,
                                   int64_t ldr, int64_t col0, hipStream_t stream) {
  if (G < 1 || G > 256) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: need 1 <= G <= 256", fn);
  if (R < 0 || C <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (C % 64) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: C must be a multiple of 64", fn);
  if (ld % 128 || ld < moe_mx_tokens_cols_bound(R, G))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: ld must be a multiple of 128 and >= %lld", fn,
                (long long)moe_mx_tokens_cols_bound(R, G));
  if (ld / 128 > 65535 || C / 64 > 0x7fffffff) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: too many columns", fn);
  if ((qt == nullptr) != (st == nullptr) || (qr == nullptr) != (sr == nullptr) || (!qt && !qr))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: give qt with st and/or qr with sr", fn);
  if (qr && (col0 < 0 || col0 % 64 || ldr % 32 || col0 + C > ldr))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: need col0 a multiple of 64, ldr of 32, col0 + C <= ldr", fn);
  if (!offsets || (R > 0 && !x)) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if ((x && !aligned16(x)) || (qt && !aligned16(qt)) || (reinterpret_cast<uintptr_t>(qr) & 7))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: x and qt must be 16-byte, qr 8-byte aligned", fn);
  if (R == 0) return MOE_SUCCESS;
  // 128-column tiles when the width allows (each row-code segment a whole 128-byte line)
  if (C % 128 == 0 && col0 % 128 == 0)
    quantize_mx_tokens_t_kernel<128><<<dim3((unsigned)(C / 128), (unsigned)(ld / 128)), 256, 0, stream>>>(
        x, offsets, G, R, C, ld, qt, st, qr, sr, ldr, col0);
  else
    quantize_mx_tokens_t_kernel<64><<<dim3((unsigned)(C / 64), (unsigned)(ld / 128)), 256, 0, stream>>>(
        x, offsets, G, R, C, ld, qt, st, qr, sr, ldr, col0);
  return check_launch("quantize_mx_tokens_t_kernel");
}
}  // namespace
}  // namespace moe

extern "C" moe_status moe_quantize_mx_tokens_t(const moe_bf16* x, const int32_t* offsets, int32_t G, int64_t R,
                                               int64_t C, uint8_t* qt, uint8_t* st, int64_t ld, hipStream_t stream) {
  if (!qt || !st) return fail(MOE_ERROR_INVALID_VALUE, "moe_quantize_mx_tokens_t: NULL pointer");
  return quantize_mx_tokens_impl("moe_quantize_mx_tokens_t", x, offsets, G, R, C, qt, st, ld, nullptr, nullptr, 0,
                                 0, stream);
}

extern "C" moe_status moe_quantize_mx_tokens(const moe_bf16* x, const int32_t* offsets, int32_t G, int64_t R,
                                             int64_t C, uint8_t* qt, uint8_t* st, int64_t ld, uint8_t* qr,
                                             uint8_t* sr, int64_t ldr, int64_t col0, hipStream_t stream) {
  return quantize_mx_tokens_impl("moe_quantize_mx_tokens", x, offsets, G, R, C, qt, st, ld, qr, sr, ldr, col0,
                                 stream);
}

extern "C" moe_status moe_quantize_mx_rows(const moe_bf16* x, const moe_bf16* x2, int64_t M, int64_t K, uint8_t* q,
                                           uint8_t* scale, hipStream_t stream) {
  const char* fn = "moe_quantize_mx_rows";
  if (M < 0 || K <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  if (K % 32) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K must be a multiple of 32", fn);
  const int64_t C8 = (x2 ? 2 : 1) * K / 8;
  const int64_t cpr = (C8 + 255) / 256;
  if (M * cpr >= ((int64_t)1 << 31)) return fail(MOE_ERROR_NOT_SUPPORTED, "%s: too many rows", fn);
  if (M == 0) return MOE_SUCCESS;
  if (!x || !q || !scale) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (!aligned16(x) || (x2 && !aligned16(x2)) || (reinterpret_cast<uintptr_t>(q) & 7))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: x (and x2) must be 16-byte, q 8-byte aligned", fn);
  quantize_mx_rows_kernel<<<(unsigned)(M * cpr), 256, 0, stream>>>(
      reinterpret_cast<const u32x4*>(x), reinterpret_cast<const u32x4*>(x2), K / 8, (int)cpr, M,
      reinterpret_cast<uint2*>(q), scale);
  return check_launch("quantize_mx_rows_kernel");
}

extern "C" moe_status moe_quantize_mx_weight(const moe_bf16* w, const moe_bf16* w2, int64_t G, int64_t K, int64_t N,
                                             uint8_t* qt, uint8_t* st, uint8_t* qr, uint8_t* sr, hipStream_t stream) {
  const char* fn = "moe_quantize_mx_weight";
  if (G < 0 || K <= 0 || N <= 0) return fail(MOE_ERROR_INVALID_VALUE, "%s: bad size", fn);
  const int nmul = w2 ? QC_IL : 64;
  if (K % 32 || N % nmul)
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: K must be a multiple of 32 and N of %d", fn, nmul);
  const int64_t nmat = w2 ? 2 : 1;
  if (G * nmat > 65535 || (K + 127) / 128 > 65535 || N / 64 > 0x7fffffff)
    return fail(MOE_ERROR_NOT_SUPPORTED, "%s: too many experts, rows or columns", fn);
  if ((qt == nullptr) != (st == nullptr) || (qr == nullptr) != (sr == nullptr) || (!qt && !qr))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: give qt with st and/or qr with sr", fn);
  if (G == 0) return MOE_SUCCESS;
  if (!w) return fail(MOE_ERROR_INVALID_VALUE, "%s: NULL pointer", fn);
  if (!aligned16(w) || (w2 && !aligned16(w2)) || (qt && !aligned16(qt)) || (reinterpret_cast<uintptr_t>(qr) & 7))
    return fail(MOE_ERROR_INVALID_VALUE, "%s: w, w2 and qt must be 16-byte, qr 8-byte aligned", fn);
  if (N % 128 == 0)
    quantize_mx_weight_kernel<128><<<dim3((unsigned)(N / 128), (unsigned)((K + 127) / 128), (unsigned)(G * nmat)),
                                     256, 0, stream>>>(w, w2, G, K, N, qt, st, qr, sr);
  else
    quantize_mx_weight_kernel<64><<<dim3((unsigned)(N / 64), (unsigned)((K + 127) / 128), (unsigned)(G * nmat)),
                                    256, 0, stream>>>(w, w2, G, K, N, qt, st, qr, sr);
  return check_launch("quantize_mx_weight_kernel");
}
