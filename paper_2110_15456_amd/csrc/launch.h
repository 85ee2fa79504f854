// launch.h -- internal launchers behind the C ABI (host side).  Arguments are
// validated by the callers in api.cpp; these functions only pick a kernel
// specialisation and launch it on the given stream.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fastbfp {

// Rounding modes, numerically equal to bfp_round_t.
enum { kNearest = 0, kStochastic = 1, kTruncate = 2 };

// Chunk-plane formats of an m-bit tensor (the layout of include/fastbfp.h).
// A plane holds one chunk of every value, with the value's sign, in one of
// three encodings:
//   kPlaneFP6: FP6 E2M3 codes of +-chunk/2 (chunks up to 15; 12 bytes per 16
//              values);
//   kPlaneFP4: FP4 E2M1 codes of +-chunk/2 (chunks up to 3; 8 bytes);
//   kPlaneLo2: a 2-bit chunk as the FP6 E2M3 codes of +-chunk/8 (subnormal
//              codes: only the sign and the two low bits of a field can be
//              set), with the zero bits squeezed out (8 bytes, see lo2_pack).
// m = 1, 2: one FP4 plane (q).  m = 3, 4: one FP6 plane (q).  m = 5, 6: an FP6
// plane of q >> 2 and a Lo2 plane of q & 3.  m = 7, 8: FP6 planes of q >> 4 and
// q & 15.
enum { kPlaneFP6 = 0, kPlaneFP4 = 1, kPlaneLo2 = 2 };
__host__ __device__ constexpr int plane_kind(int m, int p) {
  return p == 0 ? (m <= 2 ? kPlaneFP4 : kPlaneFP6) : (m <= 6 ? kPlaneLo2 : kPlaneFP6);
}
__host__ __device__ constexpr bool plane0_fp4(int m) { return m <= 2; }
// Bits of the lower chunk of a two-chunk magnitude (the upper chunk's weight
// is 2^low_chunk_bits): 2 for m = 5, 6; 4 for m = 7, 8.
__host__ __device__ constexpr int low_chunk_bits(int m) { return m <= 6 ? 2 : 4; }
// Bytes per group of g values in plane p.
__host__ __device__ constexpr int plane_group_bytes(int g, int m, int p) {
  return plane_kind(m, p) == kPlaneFP6 ? 3 * g / 4 : g / 2;
}

// Packed storage (section V-D; include/fastbfp.h): groups of 16, m even, m/2
// planes of 3-bit fields (a 2-bit chunk with the value's sign), 6 bytes per
// group and plane; exponents as a 32-bit E_max word, then 3 bits per group in
// 24-byte blocks of 64 groups.
constexpr int kPackedGroup = 16;
constexpr int kPackedPlaneGroupBytes = 6;
__host__ __device__ constexpr int64_t packed_exp_bytes(int64_t ngroups) { return 4 + 24 * ((ngroups + 63) / 64); }
hipError_t launch_quantize_packed(const float* x, int64_t rows, int64_t len, int m, int mode, uint64_t seed,
                                  uint8_t* mant, uint8_t* exps, uint32_t* status, hipStream_t s);
hipError_t launch_dequantize_packed(const uint8_t* mant, const uint8_t* exps, int64_t rows, int64_t len, int m,
                                    float* y, hipStream_t s);

hipError_t launch_quantize_rows(const float* x, int64_t rows, int64_t len, int g, int m, int mode, uint64_t seed,
                                uint8_t* mant, uint8_t* exps, uint32_t* status, hipStream_t s);
// Groups down the columns of x[R][C], written transposed (rows = C, len = R);
// with nbatch > 1, of each of the matrices x[nbatch][R][C], slice b's output
// rows following slice b - 1's.
hipError_t launch_quantize_cols(const float* x, int64_t R, int64_t C, int g, int m, int mode, uint64_t seed,
                                uint8_t* mant, uint8_t* exps, uint32_t* status, hipStream_t s, int64_t nbatch = 1);
// Workgroups launch_quantize_cols / launch_quantize_rows start (the caller
// keeps them below 2^31).
int64_t quantize_cols_blocks(int64_t R, int64_t C, int g, int64_t nbatch);
int64_t quantize_rows_blocks(int64_t rows, int64_t len, int g);
// Adaptive precision (Algorithm 1, Eq. 2): quantize at m = 4 into mant4/exps,
// optionally write the low-chunk-discarded 2-bit mantissas to mant2, and set
// sums[0] = sum |BFP(X,4) - BFP(X,2)|, sums[1] = sum |BFP(X,2)| (sums holds
// 2 + 2 * adaptive_parts(...) doubles; the rest is workspace).
// Partial-sum pairs the adaptive kernel writes (one per workgroup).
int64_t adaptive_parts(int64_t R, int64_t C, int group_axis, int g);
hipError_t launch_quantize_adaptive(const float* x, int64_t R, int64_t C, int group_axis, int g, int mode,
                                    uint64_t seed, uint8_t* mant4, uint8_t* mant2, uint8_t* exps, double* sums,
                                    uint32_t* status, hipStream_t s);
// Capacity, in doubles, of the device scratch array that holds the partial
// pairs of the allocation-free adaptive converter (2 MiB per GPU).
constexpr int64_t kAdaptiveScratchDoubles = int64_t(1) << 18;
// launch_quantize_adaptive without a caller workspace: sums holds the two
// result doubles only; the partials use the library's device scratch array
// (the caller checks 2 * adaptive_parts(...) <= kAdaptiveScratchDoubles).
// Calls that overlap on one GPU share that array and race.
hipError_t launch_quantize_adaptive_static(const float* x, int64_t R, int64_t C, int group_axis, int g, int mode,
                                           uint64_t seed, uint8_t* mant4, uint8_t* mant2, uint8_t* exps,
                                           double* sums, uint32_t* status, hipStream_t s);
// Both groupings (g = 16) of x[R][C] from one read: mr/er along rows (seed_r),
// mc/ec along columns (seed_c), in the layout of quantize.
hipError_t launch_quantize_dual(const float* x, int64_t R, int64_t C, int m, int mode, uint64_t seed_r,
                                uint64_t seed_c, uint8_t* mr, uint8_t* er, uint8_t* mc, uint8_t* ec,
                                uint32_t* status, hipStream_t s);
// w_out = w + alpha * dw (two FP32 roundings), then both groupings of w_out as
// launch_quantize_dual.  w_out may be w.
hipError_t launch_weight_update(const float* w, const float* dw, float alpha, float* w_out, int64_t R, int64_t C,
                                int m, int mode, uint64_t seed_r, uint64_t seed_c, uint8_t* mr, uint8_t* er,
                                uint8_t* mc, uint8_t* ec, uint32_t* status, hipStream_t s);
hipError_t launch_dequantize(const uint8_t* mant, const uint8_t* exps, int64_t rows, int64_t len, int g, int m,
                             float* y, hipStream_t s);
// a_m / b_m: the stored operands' widths (they fix the plane formats and
// plane stride); na / nb: chunk planes read (1 or 2); g: 16 or 32.
// scale_log2 = 4 - m_a - m_b.  tile: -1 chosen from the shape, 0 the default
// tile of the operand formats, 1..4 256x128 / 256x64 / 128x64 / 128x128 (one
// chunk plane per operand and g = 16 only; the caller checks).
hipError_t launch_gemm_mx(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int na, const uint8_t* b_mant,
                          const uint8_t* b_exp, int b_m, int nb, int64_t M, int64_t N, int64_t K, int g,
                          int scale_log2, float* C, int64_t ldc, int tile, hipStream_t s);
// bfp_gemm with the output converted in the epilogue: groups of 16 along each
// row of C at c_m bits (rounding mode and Philox seed as for quantize).
hipError_t launch_gemm_mx_bfp(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int na, const uint8_t* b_mant,
                              const uint8_t* b_exp, int b_m, int nb, int64_t M, int64_t N, int64_t K, int g,
                              int scale_log2,
                              int c_m, int mode, uint64_t seed, uint8_t* c_mant, uint8_t* c_exp, uint32_t* status,
                              hipStream_t s);
// The general BFP GEMM (gemm_general.hip): any m_a <= a_m and m_b <= b_m, g in
// {4, 8, 16, 32, 64} (K a multiple of g and of 16).  With P non-null it writes
// the int32 group partials P[K/g][M][N] instead of C.
// Re-encoding of a stored tensor (chunk planes with groups of g, or packed)
// into the chunk-plane layout at m_use bits that the block-scaled kernel reads:
// len_out = len * 16/g for g < 16 (one group per zero-padded 16-value unit),
// else len; groups of g_out = 16 (g <= 16) or 32 (g >= 32).
void repack_shape(int64_t len, int g, int64_t* len_out, int* g_out);
hipError_t launch_repack(const uint8_t* mant, const uint8_t* exps, int64_t rows, int64_t len, int g, int m, int m_use,
                         bool packed, uint8_t* out_mant, uint8_t* out_exps, hipStream_t s);
hipError_t launch_gemm_general(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int m_a, const uint8_t* b_mant,
                               const uint8_t* b_exp, int b_m, int m_b, int64_t M, int64_t N, int64_t K, int g,
                               float* C, int64_t ldc, int32_t* P, hipStream_t s, bool packed = false);

}  // namespace fastbfp
