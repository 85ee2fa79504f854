/*
 * fastbfp.h -- C ABI of the MI355X (gfx950) block-floating-point hot path of
 * FAST (Zhang, McDanel, Kung, "FAST: DNN Training Under Variable Precision
 * Block Floating Point with Stochastic Rounding", HPCA 2022).
 *
 * Two operations sit behind this boundary:
 *   bfp_quantize  FP32 -> BFP conversion (section III-A; converter of
 *                 section V-C): one shared exponent per group of g values,
 *                 sign-magnitude mantissas of m bits, nearest, stochastic or
 *                 truncating rounding.
 *   bfp_gemm      the variable-precision BFP dot product / GEMM (section III-B,
 *                 fMAC of section V-B): per-group integer dot products, one
 *                 exponent addition per group pair, FP32 accumulation across
 *                 groups, and a pass count that grows with the mantissa widths.
 *
 * Conventions shared by every entry point
 *   - Pointers named x, y, C, P, mant, exp, status_word are DEVICE pointers
 *     (hipMalloc'd or torch CUDA tensors); pointers to size_t outputs are HOST
 *     pointers.  The caller owns every buffer; the library allocates nothing
 *     and keeps no state besides a per-device properties cache.
 *   - stream is a hipStream_t passed as void* (NULL = the default stream).
 *     Calls enqueue work on it and return without synchronising.
 *   - Every argument and shape check happens on the host before any launch;
 *     a failed check returns a non-zero bfp_status_t and enqueues nothing.
 *     A failed launch returns BFP_E_HIP.
 *   - All entry points are thread-safe.
 *
 * BFP tensor layout (rows x len values, groups of g consecutive values along
 * len; g in {4, 8, 16, 32, 64}; len a multiple of g and of 16)
 *   exp  : uint8 [rows][len/g]   shared exponent E = the largest FP32 biased
 *          exponent field in the group (0 for a group of zeros/subnormals).
 *          One unit in the last place of the group is 2^(E - 127 - (m-1)).
 *   mant : chunk planes.  A magnitude q in [0, 2^m - 1] is stored as one
 *          chunk (m <= 4: q itself) or two (m = 5, 6: hi = q >> 2, which has
 *          m - 2 bits, and lo = q & 3; m = 7, 8: hi = q >> 4, which has m - 4
 *          bits, and lo = q & 15).  Plane c holds chunk c of every value with
 *          the value's sign, in one of three encodings:
 *            FP4 E2M1 codes of +-chunk/2 (4 bits: the sign, then the chunk
 *              itself in the three low bits) -- m = 1, 2;
 *            FP6 E2M3 codes of +-chunk/2 (6 bits; every integer 0..15 halved
 *              is exact) -- m = 3, 4, the hi plane of m = 5..8 and the lo
 *              plane of m = 7, 8;
 *            Lo2 -- the lo plane of m = 5, 6: per 16 values, the 96 bits of
 *              their FP6 E2M3 codes of +-chunk/8 (subnormal codes: only a
 *              field's sign and two lowest bits can be set), as the three
 *              little-endian dwords T0, T1, T2, stored as the two dwords
 *              T0 | (T1 >> 1) and T2 (T1's possible bits shifted down by one
 *              fall exactly on T0's always-zero bits).
 *          FP4 and FP6 codes are packed little-endian, w bits per value
 *          (value t of a group at bits w*t .. w*t + w - 1; w = 4 or 6).  A
 *          group takes B_c = g/2 (FP4, Lo2) or 3g/4 (FP6) bytes in plane c:
 *            plane 0, row r, group G at byte offset (r * (len/g) + G) * B_0,
 *            plane 1 at rows * (len/g) * B_0 + (r * (len/g) + G) * B_1.
 *          The planes are laid out in 16-value units: a group of 32 or 64 is
 *          two or four consecutive units, and a unit holds 4 groups of 4 or 2
 *          of 8 (their codes in the unit's order).  A Lo2 plane is defined per
 *          unit only.
 *          A zero chunk is stored as code 0 (no sign).
 *          This is the paper's chunk-plane storage (section V-D): each plane
 *          holds one chunk of every value with its sign, the upper chunk's
 *          weight is the lower chunk's times 2^(bits of the lower chunk), and
 *          a 2-bit chunk with its sign takes the paper's 3 bits (a Lo2 plane
 *          packs 16 of them in 6 of its 8 bytes); the chunk widths are those
 *          gfx950's block-scaled MFMA consumes at its full FP6/FP4 rate.
 *          Bits per value at g = 16, exponent included: 4.5 (m <= 2), 6.5
 *          (m = 3, 4), 10.5 (m = 5, 6), 12.5 (m = 7, 8).
 */
#ifndef FASTBFP_H
#define FASTBFP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FASTBFP_ABI_VERSION 7

typedef enum {
  BFP_ROUND_NEAREST = 0,    /* add half an LSB, then truncate (ties away from zero) */
  BFP_ROUND_STOCHASTIC = 1, /* add an 8-bit Philox noise byte below the LSB, then truncate */
  BFP_ROUND_TRUNCATE = 2    /* drop the low-order bits (the converter without noise) */
} bfp_round_t;

typedef enum {
  BFP_OK = 0,
  BFP_E_ARG = 1,         /* null pointer, negative size, bad enum value */
  BFP_E_SHAPE = 2,       /* g does not divide the grouped axis, K mismatch, ldc < N */
  BFP_E_UNSUPPORTED = 3, /* a valid but unimplemented combination (e.g. g not in {16,32}) */
  BFP_E_PRECISION = 4,   /* m outside 1..8, or a GEMM precision the stored planes cannot give */
  BFP_E_HIP = 5          /* the HIP runtime reported an error at launch */
} bfp_status_t;

/* ABI version of the loaded library (FASTBFP_ABI_VERSION it was built with). */
int bfp_abi_version(void);

/* Static, NUL-terminated description of a status code. */
const char* bfp_status_str(int status);

/* Number of chunk planes for an m-bit magnitude: 1 if m <= 4, 2 if
 * 5 <= m <= 8, 0 if m is outside 1..8. */
int bfp_chunks(int m_bits);

/* Host-side sizes of the two BFP arrays for a rows x len tensor.
 * Returns BFP_E_ARG for null outputs or negative sizes, BFP_E_SHAPE if len is
 * not a multiple of g and of 16, BFP_E_UNSUPPORTED for g not in
 * {4, 8, 16, 32, 64}, BFP_E_PRECISION for m outside 1..8. */
int bfp_quantized_sizes(int64_t rows, int64_t len, int g, int m_bits, size_t* mant_bytes, size_t* exp_bytes);

/*
 * bfp_quantize -- FP32 -> BFP (section III-A, steps (a)-(d); converter of
 * section V-C).
 *   x           : FP32 [R][C], row-major, contiguous.
 *   group_axis  : 1 -> groups of g consecutive values along each row; the
 *                 output tensor has rows = R, len = C.
 *                 0 -> groups of g consecutive values down each column; the
 *                 output is written with the group axis last, i.e. rows = C,
 *                 len = R (transpose-on-quantize: every GEMM operand is then
 *                 K-contiguous, which serves the transposed operands of the
 *                 backward GEMMs of section II-B).
 *   g           : 4, 8, 16, 32 or 64; the grouped axis must be a multiple of g
 *                 and of 16 (BFP_E_SHAPE otherwise).
 *   m_bits      : magnitude width 1..8 (a sign bit is kept besides).
 *   round_mode  : bfp_round_t.
 *   seed        : stochastic rounding only.  The noise byte of output value t
 *                 of group gid (gid = the flat index into exp) is byte (t mod 4)
 *                 of word ((t div 4) mod 4) of Philox4x32-10 with key =
 *                 (seed mod 2^32, seed div 2^32) and counter = (gid mod 2^32,
 *                 gid div 2^32, t div 16, 0) (Salmon et al., SC'11), so it does
 *                 not depend on the launch shape.  The magnitude is then
 *                 floor(a + U/256), a being the magnitude in units of the LSB.
 *   mant, exp   : outputs in the layout above, sized by bfp_quantized_sizes.
 *   status_word : optional device uint32; bit 0 is OR-ed in if any input was
 *                 Inf or NaN (a precondition violation: those groups' outputs
 *                 are unspecified).  May be NULL.
 * Subnormal inputs are flushed to zero.  A group maximum that rounds up to
 * 2^m saturates at 2^m - 1.
 */
int bfp_quantize(const float* x, int64_t R, int64_t C, int group_axis, int g, int m_bits, int round_mode,
                 uint64_t seed, uint8_t* mant, uint8_t* exp, uint32_t* status_word, void* stream);

/*
 * bfp_quantize_nd -- bfp_quantize of an N-dimensional tensor grouped along any
 * one axis (section III-A; the backward GEMMs of section II-B group their
 * operands along other axes than the forward ones).
 *   x           : FP32, contiguous row-major with ndim dimensions shape[0..ndim)
 *                 (host array of ndim >= 1 sizes, each >= 0).
 *   group_axis  : 0 <= group_axis < ndim; shape[group_axis] is a multiple of g
 *                 and of 16 (BFP_E_SHAPE otherwise).
 *   Output      : the BFP tensor with the group axis innermost: rows = the
 *                 product of the other sizes in their order (the row of index
 *                 (i_0, .., i_{a-1}, i_{a+1}, .., i_{n-1}) is that index in
 *                 row-major order), len = shape[group_axis]; the layout and
 *                 the noise addressing (gid = row * len/g + group) as
 *                 bfp_quantize.  The last axis is bfp_quantize with group_axis
 *                 1 and R = the product of the others; axis 0 of a 2-D tensor
 *                 is group_axis 0.
 *   The rest    : as bfp_quantize.  BFP_E_UNSUPPORTED if a size product
 *                 exceeds 2^62 or the launch would exceed 2^31 workgroups.
 */
int bfp_quantize_nd(const float* x, int ndim, const int64_t* shape, int group_axis, int g, int m_bits, int round_mode,
                    uint64_t seed, uint8_t* mant, uint8_t* exp, uint32_t* status_word, void* stream);

/*
 * bfp_dequantize -- BFP -> FP32: y[r][k] = +-q * 2^(E - 127 - (m-1)), the value
 * the BFP element stands for (section III-A).  Exact whenever the result is a
 * normal FP32 number.  y is FP32 [rows][len].
 */
int bfp_dequantize(const uint8_t* mant, const uint8_t* exp, int64_t rows, int64_t len, int g, int m_bits, float* y,
                   void* stream);

/*
 * bfp_gemm -- C[M][N] = A[M][K] * B[N][K]^T for BFP operands grouped along K
 * (section III-B and the fMAC of section V-B):
 *   C[i][j] = sum over groups G of P_G * 2^(ea + eb - 254 - (m_a-1) - (m_b-1)),
 *   P_G     = sum_{k in G} qa[i][k] * qb[j][k]   (exact integer products).
 * The products are exact; the cross-group sum is accumulated in FP32.
 *   a_mant/a_exp : A stored with a_m_bits (rows M, len K); likewise B (rows N).
 *   m_a, m_b     : the precisions the product is taken at, 1 .. the stored
 *                  width (BFP_E_PRECISION otherwise): each magnitude is
 *                  truncated to its top m_a (m_b) bits, the paper's discard of
 *                  low-order bits (section V-D).  The width of a two-chunk
 *                  operand's upper chunk (m - 2 for m = 5, 6; m - 4 for
 *                  m = 7, 8) simply skips the low chunk plane.
 *   Passes: one block-scaled MFMA per chunk-plane pair and group pair, the
 *   counterpart of the paper's (m_a/2)(m_b/2) fMAC rounds -- except that an
 *   operand split at 2 bits (m = 5, 6) puts both of its chunks in one
 *   32-value MFMA block, so it adds no pass of its own: (6,6) takes 2 MFMAs
 *   per group of 16, (6, m <= 4) 1.
 *   g            : 4, 8, 16, 32 or 64 (both operands); K a multiple of g and
 *                  of 16.  Groups of 16 and 32 at the stored width or with a
 *                  low chunk plane dropped run on the block-scaled MFMA
 *                  kernel (a group of 32 fills a whole MFMA block; a group of
 *                  16 leaves half of it zero, except for operands split at 2
 *                  bits).  Every other case -- groups of 4, 8 or 64, or a
 *                  precision that is not a chunk boundary -- runs on a
 *                  general kernel: int8 MFMA on the decoded, truncated
 *                  magnitudes of one group at a time, each exact integer
 *                  group partial scaled exactly by its power of two and added
 *                  in FP32 (same result contract, far lower throughput;
 *                  bfp_gemm_ws runs these cases on the block-scaled kernel
 *                  with a caller workspace).
 *   C            : FP32 with row stride ldc >= N (elements).
 *   Size limits  : M, N < 2^31, K <= 11184784 (256 rows of 12 bytes per 16
 *                  values stay below 2^31 bytes: the kernels address operand
 *                  tiles with 32-bit offsets), and
 *                  ceil(M / 128) * ceil(N / 64) < 2^31 (on the general
 *                  kernel also ceil(M / 32) * ceil(N / 32) < 2^31);
 *                  otherwise BFP_E_UNSUPPORTED.
 * Preconditions for the stated accuracy: every group exponent E is at most 250,
 * and every scaled group sum, partial sum and |C| stays in the FP32 normal range.
 */
int bfp_gemm(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant, const uint8_t* b_exp,
             int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, float* C, int64_t ldc,
             void* stream);

/*
 * bfp_repack -- re-encodes a stored BFP tensor into the chunk-plane layout at
 * m_use bits with groups of 16 or 32, the form the block-scaled GEMM kernel
 * reads.  The values are those the stored tensor stands for at m_use bits:
 * every magnitude truncated to its top m_use bits (the paper's discard of
 * low-order bits, section V-D), the exponents unchanged.
 *   mant, exp   : the source, rows x len with groups of g in the chunk-plane
 *                 layout (packed = 0; g in {4, 8, 16, 32, 64}), or in the
 *                 packed storage (packed = 1; g must be 16), stored with
 *                 m_bits (1..8).
 *   m_use       : 1 .. m_bits (BFP_E_PRECISION otherwise).
 *   out_mant, out_exp : the result, sized by bfp_repack_sizes: rows x len_out
 *                 with groups of g_out, m_use bits, where
 *                   g = 4, 8     : len_out = len * 16/g, g_out = 16 -- group G
 *                                  becomes 16-value unit G: its g values,
 *                                  then 16 - g zeros, with the group's
 *                                  exponent;
 *                   g = 16, 32   : len_out = len, g_out = g;
 *                   g = 64       : len_out = len, g_out = 32 -- both halves of
 *                                  a group take its exponent.
 *                 A product of two tensors repacked from the same g sums the
 *                 same exact per-group terms T_G as the stored tensors at
 *                 (m_a, m_b): the padding zeros meet zeros, and the two halves
 *                 of a group of 64 add up to its integer dot product.
 * Pointers: mant and out_mant 4-byte aligned, exp too when packed.
 */
int bfp_repack_sizes(int64_t rows, int64_t len, int g, int m_use, size_t* mant_bytes, size_t* exp_bytes,
                     int64_t* len_out, int* g_out);
int bfp_repack(const uint8_t* mant, const uint8_t* exp, int64_t rows, int64_t len, int g, int m_bits, int packed,
               int m_use, uint8_t* out_mant, uint8_t* out_exp, void* stream);

/*
 * bfp_gemm_ws -- bfp_gemm (the same product and result contract, section
 * III-B) with a caller workspace, so that every case runs on the block-scaled
 * MFMA kernel: an operand the kernel cannot read as stored -- a group size of
 * 4, 8 or 64, a precision that is not a chunk boundary, or packed storage
 * (packed = 1: both operands in the packed storage, g = 16) -- is first
 * re-encoded into the workspace by bfp_repack at (m_a, m_b), and the kernel
 * then runs on K_out = len_out with groups of g_out.  Products bfp_gemm
 * already runs on that kernel need no workspace.  bfp_gemm itself keeps
 * running the other cases on its general kernel, allocation- and
 * workspace-free, at a far lower rate.
 *   workspace   : device memory of at least bfp_gemm_ws_size bytes (may be
 *                 NULL when that is 0), 256-byte aligned; its contents on
 *                 entry do not matter and are overwritten.  Calls that share
 *                 a workspace must not overlap.
 *   Size limits : as bfp_gemm, with K_out in place of K (BFP_E_UNSUPPORTED).
 *   BFP_E_ARG   : also for a workspace below the required size.
 */
int bfp_gemm_ws_size(int a_m_bits, int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, int packed,
                     size_t* bytes);
int bfp_gemm_ws(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant, const uint8_t* b_exp,
                int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, int packed, float* C,
                int64_t ldc, void* workspace, size_t workspace_bytes, void* stream);

/*
 * bfp_gemm_tiled -- bfp_gemm (the same product, section III-B) with the C tile
 * that one workgroup computes chosen by the caller instead of from the shape:
 *   tile = -1 : chosen from M and N, exactly as bfp_gemm does;
 *   tile =  0 : the operand formats' default tile (256 x 256 for one chunk
 *               plane per operand);
 *   tile =  1, 2, 3, 4 : 256 x 128, 256 x 64, 128 x 64, 128 x 128 -- only for
 *               one chunk plane per operand (m_a, m_b <= 4) with g = 16, else
 *               BFP_E_UNSUPPORTED.
 * A product that bfp_gemm runs on its general kernel takes only tile = -1
 * (BFP_E_UNSUPPORTED otherwise).
 * For one-chunk, g = 16 products bfp_gemm picks 128 x 64 when N <= 64;
 * 256 x 128 when A's plane holds FP4 codes (A stored with m = 1, 2, 5 or 6);
 * otherwise 256 x 256, or 128 x 128 when N <= 128; and it steps down to a
 * smaller tile while fewer than 192 tiles would leave CUs idle.  Every tile
 * computes the same products, per-group scales and per-output accumulation
 * order, so results do not depend on the tile.  Any other tile value returns
 * BFP_E_ARG.  For tests and tuning.
 */
int bfp_gemm_tiled(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant,
                   const uint8_t* b_exp, int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b,
                   float* C, int64_t ldc, int tile, void* stream);

/*
 * bfp_gemm_bfp -- bfp_gemm with its output converted to BFP in the epilogue,
 * from the FP32 results, by the converter of section V-C (the paper's
 * converter sits at the output of the systolic array, section V-A): C is
 * written as a BFP tensor of rows = M, len = N with groups of 16 along each
 * row (the K axis of a GEMM that consumes C as its left operand) at c_m_bits,
 * in the layout of bfp_quantize.  The result is exactly bfp_quantize(C, group
 * axis 1, g = 16, c_m_bits, round_mode, seed) of the FP32 C that bfp_gemm
 * computes: the same values, the same noise addressing (gid = the index into
 * c_exp), without writing or re-reading FP32 C.
 *   Operands and precisions : as bfp_gemm, for the products bfp_gemm runs
 *                 on its block-scaled kernel only (groups of 16 or 32, each
 *                 operand at its stored width or without its low chunk plane;
 *                 BFP_E_UNSUPPORTED otherwise); the output is grouped by 16.
 *   c_m_bits    : 1..8.  round_mode, seed, status_word : as bfp_quantize.
 *   c_mant, c_exp : outputs sized by bfp_quantized_sizes(M, N, 16, c_m_bits).
 * N must be a multiple of 16 (BFP_E_SHAPE otherwise).  The workgroup tile
 * follows bfp_gemm's choice from the shape (bfp_gemm_tiled), except that an
 * A in FP4 codes is tiled like one in FP6 codes.
 */
int bfp_gemm_bfp(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant, const uint8_t* b_exp,
                 int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, int c_m_bits, int round_mode,
                 uint64_t seed, uint8_t* c_mant, uint8_t* c_exp, uint32_t* status_word, void* stream);

/*
 * bfp_gemm_group_partials -- the exact integer group dot products
 *   P[G][i][j] = sum_{k in G} qa'[i][k] * qb'[j][k]
 * (parts M and A of section III-B), qa' and qb' being the magnitudes at m_a and
 * m_b bits with their signs, computed with int8 MFMA on the decoded
 * magnitudes (an 8-bit magnitude as two 4-bit chunks combined in integers).
 * P is int32 [K/g][M][N].  Meant for verification: it writes K/g times more
 * output than bfp_gemm.  Same operand, group-size and precision rules as
 * bfp_gemm (the exponents do not enter P, so only the mantissa planes are
 * passed).
 */
int bfp_gemm_group_partials(const uint8_t* a_mant, int a_m_bits, const uint8_t* b_mant, int b_m_bits, int64_t M,
                            int64_t N, int64_t K, int g, int m_a, int m_b, int32_t* P, void* stream);

/*
 * Packed storage -- the paper's memory layout for variable-precision BFP
 * (section V-D): every magnitude split into 2-bit chunks, each stored with the
 * value's sign in 3 bits, the chunks of one position of all values in a group
 * together, and a 3-bit shared exponent, so that a group of g = 16 takes
 * e + 16 * ceil(m/2) * 3 bits (3.1875 bits per value at m = 2, 6.1875 at
 * m = 4, with e = 3).  This is a storage form: bfp_gemm_packed reads it on the
 * general kernel, or after bfp_repack on the block-scaled kernel (bfp_gemm_ws).
 *   Groups      : 16 consecutive values along each row (len a multiple of 16).
 *   Exponents   : a 3-bit exponent cannot hold an FP32 exponent field, so it is
 *                 read as an offset above one base per tensor: exp starts with
 *                 a little-endian uint32 holding E_max, the largest FP32
 *                 exponent field in the tensor; the base is
 *                 B = max(E_max - 7, 0); group gid (= row * len/16 + group)
 *                 has the shared exponent E = max(its largest exponent field,
 *                 B), stored as e = E - B in bits 3 gid .. 3 gid + 2 of the
 *                 little-endian bit stream that follows the word (padded to
 *                 24 bytes per 64 groups).  A group whose largest exponent is
 *                 below B is quantized at B: its small values lose low bits.
 *   Mantissas   : NP = ceil(m/2) planes, plane c (most significant first)
 *                 holding chunk c of every magnitude q, (q >> 2 (NP-1-c)) & 3,
 *                 as a 3-bit field: the chunk in bits 0-1, the value's sign in
 *                 bit 2 when the chunk is nonzero (a zero chunk is stored as
 *                 0).  A group's 16 fields are the 48 bits of 6 bytes (value t
 *                 at bits 3t .. 3t+2, little-endian); plane c, group gid at
 *                 byte offset (c * ngroups + gid) * 6, ngroups = rows * len/16.
 *   Values      : one LSB of group gid is 2^(E - 127 - (m-1)) as in the chunk-
 *                 plane layout; a tensor of Inf/NaN-free inputs whose groups
 *                 all have exponents within 7 of E_max converts to the same
 *                 (q, E) as bfp_quantize.
 */

/* Host-side sizes of a packed rows x len tensor: mant_bytes = ceil(m/2) * 6 *
 * ngroups, exp_bytes = 4 + 24 * ceil(ngroups / 64).  So with ngroups a multiple
 * of 64 the tensor takes (51/16, 99/16, ...) bits per value plus the 32-bit
 * E_max word.  BFP_E_ARG for null outputs or negative sizes, BFP_E_SHAPE if
 * len is not a multiple of 16, BFP_E_PRECISION for m outside 1..8,
 * BFP_E_UNSUPPORTED for 2^56 groups or more. */
int bfp_packed_sizes(int64_t rows, int64_t len, int m_bits, size_t* mant_bytes, size_t* exp_bytes);

/*
 * bfp_quantize_packed -- FP32 [R][C] -> packed BFP with groups of 16 along
 * each row (section III-A steps (a)-(d), with the shared exponent raised to
 * the tensor base; section V-D storage).
 *   x           : FP32 [R][C], row-major, contiguous, 16-byte aligned; C a
 *                 multiple of 16.
 *   m_bits, round_mode, seed, status_word : as bfp_quantize (the same noise
 *                 addressing: gid = row * C/16 + group).
 *   mant, exp   : outputs sized by bfp_packed_sizes, 4-byte aligned.
 * Three launches on the stream: the E_max word is cleared, reduced over x,
 * then the groups are converted.
 */
int bfp_quantize_packed(const float* x, int64_t R, int64_t C, int m_bits, int round_mode, uint64_t seed,
                        uint8_t* mant, uint8_t* exp, uint32_t* status_word, void* stream);

/* bfp_dequantize_packed -- packed BFP -> FP32 [rows][len]: y = +-q *
 * 2^(E - 127 - (m-1)) (section III-A), exact whenever the result is a normal
 * FP32 number.  y 16-byte aligned; mant, exp 4-byte aligned. */
int bfp_dequantize_packed(const uint8_t* mant, const uint8_t* exp, int64_t rows, int64_t len, int m_bits, float* y,
                          void* stream);

/*
 * bfp_gemm_packed -- bfp_gemm (section III-B) on operands in packed storage:
 * A [M][K] stored with a_m_bits, B [N][K] with b_m_bits, each with its own
 * base; m_a, m_b as bfp_gemm (1 .. the stored width: the magnitude truncated to
 * its top bits, section V-D).  Runs on the general kernel: per group the
 * chunk fields are unpacked to signed magnitudes, the exact integer group dot
 * product P_G taken on int8 MFMA, scaled by 2^(ea + eb - 254 - (m_a-1) -
 * (m_b-1)) and added in FP32.  C FP32 with row stride ldc >= N.  Size limits:
 * as bfp_gemm, and ceil(M/32) * ceil(N/32) < 2^31.  exp pointers 4-byte
 * aligned.  Allocation- and workspace-free; bfp_gemm_ws with packed = 1 runs
 * the same product on the block-scaled kernel (operands unpacked into a
 * caller workspace).
 */
int bfp_gemm_packed(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant,
                    const uint8_t* b_exp, int b_m_bits, int64_t M, int64_t N, int64_t K, int m_a, int m_b, float* C,
                    int64_t ldc, void* stream);

/*
 * bfp_quantize_dual -- both groupings of one FP32 matrix from a single read:
 * the row grouping (group_axis 1: rows = R, len = C) into mant_r/exp_r with
 * seed_r, and the column grouping (group_axis 0: rows = C, len = R) into
 * mant_c/exp_c with seed_c, each byte for byte what bfp_quantize writes for
 * that axis and seed.  A training step needs both of some tensors: the
 * activations and the output gradient enter one GEMM along their feature axis
 * and the weight-gradient GEMM along the token axis (section II-B), which the
 * paper serves by entering the systolic array from another side (section V-A).
 *   x           : FP32 [R][C], row-major, contiguous, 16-byte aligned.
 *   R, C        : multiples of 16 (BFP_E_SHAPE otherwise), C < 2^22.
 *   g           : 16 (BFP_E_UNSUPPORTED otherwise).
 *   m_bits, round_mode, status_word : as bfp_quantize (one width and rounding
 *                 rule for both outputs).
 *   outputs     : sized by bfp_quantized_sizes(R, C, 16, m_bits) (either).
 */
int bfp_quantize_dual(const float* x, int64_t R, int64_t C, int g, int m_bits, int round_mode, uint64_t seed_r,
                      uint64_t seed_c, uint8_t* mant_r, uint8_t* exp_r, uint8_t* mant_c, uint8_t* exp_c,
                      uint32_t* status_word, void* stream);

/*
 * bfp_weight_update -- the end of a training step (sections V-A and the
 * training workflow): the weight gradient is added to the weights and the
 * updated weights are converted to BFP for the next step, in one pass:
 *   w_out[r][c] = w[r][c] + alpha * dw[r][c]
 * in FP32 with the product and the sum each rounded to nearest (no fused
 * multiply-add; alpha = 1 is the paper's plain sum, alpha = -learning rate an
 * SGD step on a raw gradient), then both groupings of w_out as
 * bfp_quantize_dual.  Subnormal inputs, products and sums are read as, and
 * flushed to, zero of the same sign.  w_out may be w (in place); dw must not
 * overlap w_out.
 *   w, dw, w_out : FP32 [R][C], row-major, contiguous, 16-byte aligned.
 *   The rest     : as bfp_quantize_dual.
 */
int bfp_weight_update(const float* w, const float* dw, float alpha, float* w_out, int64_t R, int64_t C, int g,
                      int m_bits, int round_mode, uint64_t seed_r, uint64_t seed_c, uint8_t* mant_r, uint8_t* exp_r,
                      uint8_t* mant_c, uint8_t* exp_c, uint32_t* status_word, void* stream);

/*
 * bfp_quantize_adaptive -- the converter and improvement block of the adaptive
 * scheme (Algorithm 1, Eq. 2, section V-C; section V-D for the chunk discard),
 * in one pass over x: BFP(X, 4) is written as by bfp_quantize with m_bits = 4;
 * BFP(X, 2) is that tensor with the low 2-bit chunk of every mantissa
 * discarded (same shared exponents: value +-(q >> 2) * 2^(E - 128)); and
 *   sums[0] = sum_n |BFP(X_n, 4) - BFP(X_n, 2)|,  sums[1] = sum_n |BFP(X_n, 2)|,
 * so that r(X) = sums[0] / sums[1] (Eq. 2).
 *   x, R, C, group_axis, round_mode, seed, status_word : as bfp_quantize.
 *   g           : 16 or 32 (BFP_E_UNSUPPORTED otherwise).
 *   mant4, exp  : the m = 4 tensor (layout of bfp_quantize, m_bits = 4).
 *   mant2       : optional (may be NULL): the m = 2 tensor's mantissas (layout
 *                 of bfp_quantize, m_bits = 2: one plane of 4-bit codes, two
 *                 thirds of mant4's size); it shares exp.  Either tensor can be handed to
 *                 bfp_gemm (m_bits 4 or 2) without converting again.
 *   sums        : device doubles, bfp_adaptive_sums_len(R, C, group_axis, g)
 *                 of them (8-byte aligned): sums[0] and sums[1] receive the two
 *                 sums, the rest is the workspace of their per-workgroup
 *                 partials.  The partials are added in a fixed order, so the
 *                 result is the same on every run.
 */
int bfp_quantize_adaptive(const float* x, int64_t R, int64_t C, int group_axis, int g, int round_mode, uint64_t seed,
                          uint8_t* mant4, uint8_t* mant2, uint8_t* exp, double* sums, uint32_t* status_word,
                          void* stream);

/*
 * bfp_quantize_adaptive_noalloc -- bfp_quantize_adaptive for callers that
 * cannot allocate device memory or pass a workspace (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * outputs, computed by the same kernels, but the per-workgroup partial sums
 * live in a device array inside the library (2 MiB per GPU, reserved when the
 * library is loaded and held until the process ends) instead of in sums[2..].
 * The call allocates nothing.
 *   sums        : device doubles, at least 2 (8-byte aligned): sums[0] and
 *                 sums[1] as bfp_quantize_adaptive.
 *   The rest    : as bfp_quantize_adaptive.
 * Limit: bfp_adaptive_parts(R, C, group_axis, g) <=
 * bfp_adaptive_noalloc_max_parts() (131072: 2^26 groups along rows, e.g.
 * 2^30 values at g = 16); larger shapes return BFP_E_UNSUPPORTED.
 * Every call on one GPU uses that GPU's one array: calls that overlap on the
 * same GPU (different streams, or threads) race and give wrong sums; the
 * caller must order them.  Each call writes every partial it reads, so no
 * state carries over between calls.
 */
int bfp_quantize_adaptive_noalloc(const float* x, int64_t R, int64_t C, int group_axis, int g, int round_mode,
                                  uint64_t seed, uint8_t* mant4, uint8_t* mant2, uint8_t* exp, double* sums,
                                  uint32_t* status_word, void* stream);

/* The number of per-workgroup partial pairs the adaptive converter produces
 * for this shape (-1 if group_axis or g is invalid), and the most that
 * bfp_quantize_adaptive_noalloc can hold. */
int64_t bfp_adaptive_parts(int64_t R, int64_t C, int group_axis, int g);
int64_t bfp_adaptive_noalloc_max_parts(void);

/*
 * bfp_adaptive_sums_len -- the number of doubles bfp_quantize_adaptive needs
 * at `sums` for this shape (at least 2); -1 if group_axis or g is invalid.
 */
int64_t bfp_adaptive_sums_len(int64_t R, int64_t C, int group_axis, int g);

/*
 * bfp_adaptive_threshold -- Eq. 1: epsilon(l, i) = alpha - beta * i / I -
 * beta * l / L for iteration i of I and layer l of L (the paper uses alpha =
 * 0.6, beta = 0.3).  Host arithmetic; returns NaN if I or L is not positive.
 */
double bfp_adaptive_threshold(double alpha, double beta, int64_t i, int64_t I, int64_t l, int64_t L);

/*
 * bfp_adaptive_mantissa -- Algorithm 1's choice for one tensor: 2 if
 * r(X) = num / den < eps, else 4 (r = 0 when den = 0: an all-zero tensor gains
 * nothing from 4 bits).  Host arithmetic on the two sums read back from
 * bfp_quantize_adaptive.
 */
int bfp_adaptive_mantissa(double num, double den, double eps);

#ifdef __cplusplus
}
#endif

#endif /* FASTBFP_H */
