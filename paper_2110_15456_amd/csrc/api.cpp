// api.cpp -- the C ABI declared in include/fastbfp.h: argument validation on
// the host, then a launch on the caller's stream.  No exception, allocation or
// synchronisation happens here.
#include <hip/hip_runtime.h>

#include "../../include/fastbfp.h"
#include "launch.h"

namespace {

bool group_supported(int g) { return g == 4 || g == 8 || g == 16 || g == 32 || g == 64; }

// Rows hold whole 16-value units (the plane layout's unit): with g = 4 or 8
// the grouped length must be a multiple of 16 as well as of g.
bool length_ok(int64_t len, int g) { return len % g == 0 && len % 16 == 0; }

// Largest K the GEMM accepts: 256 * (K / 16) * 12 < 2^31.
constexpr int64_t kMaxK = ((int64_t(1) << 31) / (256 * 12) - 1) * 16;

int check_tensor(int64_t rows, int64_t len, int g, int m) {
  if (rows < 0 || len < 0) return BFP_E_ARG;
  if (m < 1 || m > 8) return BFP_E_PRECISION;
  if (g <= 0) return BFP_E_ARG;
  if (!group_supported(g)) return BFP_E_UNSUPPORTED;
  if (!length_ok(len, g)) return BFP_E_SHAPE;
  return BFP_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Planes the GEMM reads for an operand stored at m_stored and used at m_use:
// every stored plane, or only the high plane when the low chunk (2 bits for
// m = 5, 6; 4 for m = 7, 8) is dropped.
int planes_used(int m_stored, int m_use) {
  if (m_use == m_stored) return m_stored > 4 ? 2 : 1;
  if (m_stored > 4 && m_use == m_stored - fastbfp::low_chunk_bits(m_stored)) return 1;
  return 0;
}

int status_of(hipError_t e) { return e == hipSuccess ? BFP_OK : BFP_E_HIP; }

// True when the block-scaled kernel (gemm_mx.h) takes the product: groups of
// 16 or 32 and each operand at its stored width or with its low chunk plane
// dropped; everything else runs on the general kernel (gemm_general.hip).
bool fast_path(int a_m, int b_m, int g, int m_a, int m_b) {
  return (g == 16 || g == 32) && planes_used(a_m, m_a) != 0 && planes_used(b_m, m_b) != 0;
}

// The shape and precision rules of a GEMM (no pointers).
int check_gemm_shape(int a_m, int b_m, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b);

int check_gemm(const uint8_t* a_mant, int a_m, const uint8_t* b_mant, int b_m, int64_t M, int64_t N, int64_t K, int g,
               int m_a, int m_b) {
  if (M < 0 || N < 0 || K < 0) return BFP_E_ARG;
  if ((M > 0 && K > 0 && !a_mant) || (N > 0 && K > 0 && !b_mant)) return BFP_E_ARG;
  const int st = check_gemm_shape(a_m, b_m, M, N, K, g, m_a, m_b);
  if (st != BFP_OK) return st;
  if (!aligned(a_mant, 4) || !aligned(b_mant, 4)) return BFP_E_ARG;
  return BFP_OK;
}

int check_gemm_shape(int a_m, int b_m, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b) {
  if (M < 0 || N < 0 || K < 0) return BFP_E_ARG;
  if (a_m < 1 || a_m > 8 || b_m < 1 || b_m > 8) return BFP_E_PRECISION;
  if (g <= 0) return BFP_E_ARG;
  if (!group_supported(g)) return BFP_E_UNSUPPORTED;
  if (!length_ok(K, g)) return BFP_E_SHAPE;
  if (m_a < 1 || m_a > a_m || m_b < 1 || m_b > b_m) return BFP_E_PRECISION;
  // The kernels address a tile's operand rows through 32-bit buffer offsets:
  // 256 rows of an FP6 plane (12 bytes per 16 values) must span less than
  // 2^31 bytes (offsets at 2^31 and above are the zero-reading sentinel of
  // groups past K), and the workgroup count of the smallest tile (128 x 64)
  // must fit in 31 bits.
  if (M > 0x7fffffff || N > 0x7fffffff || K > kMaxK) return BFP_E_UNSUPPORTED;
  if (((M + 127) / 128) * ((N + 63) / 64) > 0x7fffffff) return BFP_E_UNSUPPORTED;
  return BFP_OK;
}

// The general kernel launches one 64-lane workgroup per 32 x 32 tile of C.
bool general_grid_ok(int64_t M, int64_t N) { return ((M + 31) / 32) * ((N + 31) / 32) <= 0x7fffffff; }

// Packed tensors: groups of 16 along rows, m in 1..8, fewer than 2^56 groups.
int check_packed(int64_t rows, int64_t len, int m) {
  if (rows < 0 || len < 0) return BFP_E_ARG;
  if (m < 1 || m > 8) return BFP_E_PRECISION;
  if (len % fastbfp::kPackedGroup != 0) return BFP_E_SHAPE;
  if (rows > 0 && len / fastbfp::kPackedGroup > (int64_t(1) << 56) / rows) return BFP_E_UNSUPPORTED;
  return BFP_OK;
}

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

// How bfp_gemm_ws runs a product: which operands it repacks into the layout
// of the block-scaled kernel, the K and group size that kernel then sees, and
// the workspace the repacked operands take (A's mantissas and exponents, then
// B's, each 256-byte aligned).
struct WsPlan {
  bool rep_a, rep_b;
  int64_t k_out;
  int g_out;
  size_t a_mant, a_exp, b_mant, b_exp, bytes;
};

int ws_plan(int a_m, int b_m, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, int packed, WsPlan* p) {
  if (packed != 0 && packed != 1) return BFP_E_ARG;
  if (packed && g != 16) return BFP_E_UNSUPPORTED;
  const bool native = g == 16 || g == 32;
  p->rep_a = packed || !native || planes_used(a_m, m_a) == 0;
  p->rep_b = packed || !native || planes_used(b_m, m_b) == 0;
  fastbfp::repack_shape(K, g, &p->k_out, &p->g_out);
  if (p->k_out > kMaxK) return BFP_E_UNSUPPORTED;
  // the repack kernel: one thread per output 16-value unit, 256 per workgroup
  if ((p->rep_a && (M * (p->k_out / 16) + 255) / 256 > 0x7fffffff) ||
      (p->rep_b && (N * (p->k_out / 16) + 255) / 256 > 0x7fffffff))
    return BFP_E_UNSUPPORTED;
  p->a_mant = p->a_exp = p->b_mant = p->b_exp = 0;
  if (p->rep_a && bfp_quantized_sizes(M, p->k_out, p->g_out, m_a, &p->a_mant, &p->a_exp) != BFP_OK)
    return BFP_E_UNSUPPORTED;
  if (p->rep_b && bfp_quantized_sizes(N, p->k_out, p->g_out, m_b, &p->b_mant, &p->b_exp) != BFP_OK)
    return BFP_E_UNSUPPORTED;
  p->bytes = align256(p->a_mant) + align256(p->a_exp) + align256(p->b_mant) + align256(p->b_exp);
  return BFP_OK;
}

int check_dual(const float* x, int64_t R, int64_t C, int g, int m_bits, int round_mode, const uint8_t* mr,
               const uint8_t* er, const uint8_t* mc, const uint8_t* ec, const uint32_t* status_word) {
  if (round_mode < BFP_ROUND_NEAREST || round_mode > BFP_ROUND_TRUNCATE) return BFP_E_ARG;
  int st = check_tensor(R, C, g, m_bits);
  if (st != BFP_OK) return st;
  if (g != 16) return BFP_E_UNSUPPORTED;
  if (R % 16 != 0) return BFP_E_SHAPE;
  if (C >= (int64_t(1) << 22)) return BFP_E_UNSUPPORTED;
  if (((R + 63) / 64) * ((C + 63) / 64) > 0x7fffffff) return BFP_E_UNSUPPORTED;  // 64 x 64 tiles in an int
  if (R == 0 || C == 0) return BFP_OK;
  if (!x || !mr || !er || !mc || !ec) return BFP_E_ARG;
  if (!aligned(x, 16) || !aligned(mr, 4) || !aligned(mc, 4) || !aligned(status_word, 4)) return BFP_E_ARG;
  return BFP_OK;
}

}  // namespace

extern "C" {

int bfp_abi_version(void) { return FASTBFP_ABI_VERSION; }

const char* bfp_status_str(int status) {
  switch (status) {
    case BFP_OK: return "ok";
    case BFP_E_ARG: return "invalid argument (null or misaligned pointer, negative size, bad enum)";
    case BFP_E_SHAPE: return "shape mismatch (the grouped axis must be a multiple of g and of 16; K and ldc must "
                             "agree)";
    case BFP_E_UNSUPPORTED: return "unsupported configuration (group size, size limit, or an entry point that takes "
                                   "fewer group sizes or precisions)";
    case BFP_E_PRECISION: return "unsupported precision (m in 1..8; a GEMM precision between 1 and the stored width)";
    case BFP_E_HIP: return "HIP runtime error at launch";
    default: return "unknown status";
  }
}

int bfp_chunks(int m_bits) { return (m_bits < 1 || m_bits > 8) ? 0 : (m_bits > 4 ? 2 : 1); }

int bfp_quantized_sizes(int64_t rows, int64_t len, int g, int m_bits, size_t* mant_bytes, size_t* exp_bytes) {
  if (!mant_bytes || !exp_bytes) return BFP_E_ARG;
  const int st = check_tensor(rows, len, g, m_bits);
  if (st != BFP_OK) return st;
  size_t per_group = 0;
  for (int p = 0; p < bfp_chunks(m_bits); ++p) per_group += (size_t)fastbfp::plane_group_bytes(g, m_bits, p);
  *mant_bytes = per_group * (size_t)rows * (size_t)(len / g);
  *exp_bytes = (size_t)rows * (size_t)(len / g);
  return BFP_OK;
}

int bfp_quantize(const float* x, int64_t R, int64_t C, int group_axis, int g, int m_bits, int round_mode,
                 uint64_t seed, uint8_t* mant, uint8_t* exp, uint32_t* status_word, void* stream) {
  if (group_axis != 0 && group_axis != 1) return BFP_E_ARG;
  if (round_mode < BFP_ROUND_NEAREST || round_mode > BFP_ROUND_TRUNCATE) return BFP_E_ARG;
  const int64_t rows = group_axis == 1 ? R : C, len = group_axis == 1 ? C : R;
  const int st = check_tensor(rows, len, g, m_bits);
  if (st != BFP_OK) return st;
  if (R == 0 || C == 0) return BFP_OK;
  if (!x || !mant || !exp) return BFP_E_ARG;
  if (!aligned(x, group_axis == 1 ? 16 : 4) || !aligned(mant, 4) || !aligned(status_word, 4)) return BFP_E_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (group_axis == 1) {
    if (fastbfp::quantize_rows_blocks(R, C, g) > 0x7fffffff) return BFP_E_UNSUPPORTED;
    return status_of(fastbfp::launch_quantize_rows(x, R, C, g, m_bits, round_mode, seed, mant, exp, status_word, s));
  }
  if (fastbfp::quantize_cols_blocks(R, C, g, 1) > 0x7fffffff) return BFP_E_UNSUPPORTED;
  return status_of(fastbfp::launch_quantize_cols(x, R, C, g, m_bits, round_mode, seed, mant, exp, status_word, s));
}

int bfp_quantize_nd(const float* x, int ndim, const int64_t* shape, int group_axis, int g, int m_bits, int round_mode,
                    uint64_t seed, uint8_t* mant, uint8_t* exp, uint32_t* status_word, void* stream) {
  if (ndim < 1 || !shape || group_axis < 0 || group_axis >= ndim) return BFP_E_ARG;
  if (round_mode < BFP_ROUND_NEAREST || round_mode > BFP_ROUND_TRUNCATE) return BFP_E_ARG;
  // outer axes x group axis x inner axes; the output rows are the outer and
  // inner indices in order
  int64_t outer = 1, inner = 1;
  const int64_t L = shape[group_axis];
  for (int d = 0; d < ndim; ++d) {
    if (shape[d] < 0) return BFP_E_ARG;
    if (d == group_axis) continue;
    int64_t& acc = d < group_axis ? outer : inner;
    if (shape[d] != 0 && acc > (int64_t(1) << 62) / shape[d]) return BFP_E_UNSUPPORTED;
    acc *= shape[d];
  }
  if (inner != 0 && outer > (int64_t(1) << 62) / inner) return BFP_E_UNSUPPORTED;
  const int st = check_tensor(outer * inner, L, g, m_bits);
  if (st != BFP_OK) return st;
  if (outer == 0 || inner == 0 || L == 0) return BFP_OK;
  if (!x || !mant || !exp) return BFP_E_ARG;
  if (!aligned(x, inner == 1 ? 16 : 4) || !aligned(mant, 4) || !aligned(status_word, 4)) return BFP_E_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (inner == 1) {
    if (fastbfp::quantize_rows_blocks(outer, L, g) > 0x7fffffff) return BFP_E_UNSUPPORTED;
    return status_of(fastbfp::launch_quantize_rows(x, outer, L, g, m_bits, round_mode, seed, mant, exp, status_word, s));
  }
  if (fastbfp::quantize_cols_blocks(L, inner, g, outer) > 0x7fffffff) return BFP_E_UNSUPPORTED;
  return status_of(
      fastbfp::launch_quantize_cols(x, L, inner, g, m_bits, round_mode, seed, mant, exp, status_word, s, outer));
}

int bfp_dequantize(const uint8_t* mant, const uint8_t* exp, int64_t rows, int64_t len, int g, int m_bits, float* y,
                   void* stream) {
  const int st = check_tensor(rows, len, g, m_bits);
  if (st != BFP_OK) return st;
  if (rows == 0 || len == 0) return BFP_OK;
  if (!mant || !exp || !y) return BFP_E_ARG;
  if (!aligned(mant, 4) || !aligned(y, 16)) return BFP_E_ARG;
  return status_of(fastbfp::launch_dequantize(mant, exp, rows, len, g, m_bits, y, static_cast<hipStream_t>(stream)));
}

int bfp_gemm_tiled(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant,
                   const uint8_t* b_exp, int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b,
                   float* C, int64_t ldc, int tile, void* stream) {
  int st = check_gemm(a_mant, a_m_bits, b_mant, b_m_bits, M, N, K, g, m_a, m_b);
  if (st != BFP_OK) return st;
  if (ldc < N) return BFP_E_SHAPE;
  if (tile < -1 || tile > 4) return BFP_E_ARG;
  const bool fast = fast_path(a_m_bits, b_m_bits, g, m_a, m_b);
  if (!fast && tile >= 0) return BFP_E_UNSUPPORTED;
  if (!fast && !general_grid_ok(M, N)) return BFP_E_UNSUPPORTED;
  const int na = planes_used(a_m_bits, m_a), nb = planes_used(b_m_bits, m_b);
  if (tile > 0 && (g != 16 || na != 1 || nb != 1)) return BFP_E_UNSUPPORTED;
  if (M == 0 || N == 0) return BFP_OK;
  if (!C || (K > 0 && (!a_exp || !b_exp))) return BFP_E_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!fast)
    return status_of(fastbfp::launch_gemm_general(a_mant, a_exp, a_m_bits, m_a, b_mant, b_exp, b_m_bits, m_b, M, N, K,
                                                  g, C, ldc, nullptr, s));
  return status_of(fastbfp::launch_gemm_mx(a_mant, a_exp, a_m_bits, na, b_mant, b_exp, b_m_bits, nb, M, N, K, g,
                                           4 - m_a - m_b, C, ldc, tile, s));
}

int bfp_gemm(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant, const uint8_t* b_exp,
             int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, float* C, int64_t ldc,
             void* stream) {
  return bfp_gemm_tiled(a_mant, a_exp, a_m_bits, b_mant, b_exp, b_m_bits, M, N, K, g, m_a, m_b, C, ldc, -1, stream);
}

int bfp_gemm_bfp(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant, const uint8_t* b_exp,
                 int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, int c_m_bits, int round_mode,
                 uint64_t seed, uint8_t* c_mant, uint8_t* c_exp, uint32_t* status_word, void* stream) {
  int st = check_gemm(a_mant, a_m_bits, b_mant, b_m_bits, M, N, K, g, m_a, m_b);
  if (st != BFP_OK) return st;
  if (!fast_path(a_m_bits, b_m_bits, g, m_a, m_b)) return BFP_E_UNSUPPORTED;
  if (round_mode < BFP_ROUND_NEAREST || round_mode > BFP_ROUND_TRUNCATE) return BFP_E_ARG;
  st = check_tensor(M, N, 16, c_m_bits);
  if (st != BFP_OK) return st;
  if (M == 0 || N == 0) return BFP_OK;
  if (!c_mant || !c_exp || (K > 0 && (!a_exp || !b_exp))) return BFP_E_ARG;
  if (!aligned(c_mant, 4) || !aligned(status_word, 4)) return BFP_E_ARG;
  const int na = planes_used(a_m_bits, m_a), nb = planes_used(b_m_bits, m_b);
  return status_of(fastbfp::launch_gemm_mx_bfp(a_mant, a_exp, a_m_bits, na, b_mant, b_exp, b_m_bits, nb, M, N, K, g,
                                               4 - m_a - m_b, c_m_bits, round_mode, seed, c_mant, c_exp, status_word,
                                               static_cast<hipStream_t>(stream)));
}

int bfp_gemm_group_partials(const uint8_t* a_mant, int a_m_bits, const uint8_t* b_mant, int b_m_bits, int64_t M,
                            int64_t N, int64_t K, int g, int m_a, int m_b, int32_t* P, void* stream) {
  int st = check_gemm(a_mant, a_m_bits, b_mant, b_m_bits, M, N, K, g, m_a, m_b);
  if (st != BFP_OK) return st;
  if (!general_grid_ok(M, N)) return BFP_E_UNSUPPORTED;
  if (M == 0 || N == 0 || K == 0) return BFP_OK;
  if (!P) return BFP_E_ARG;
  // the group partials need no exponents: the decoder reads only mantissas
  return status_of(fastbfp::launch_gemm_general(a_mant, nullptr, a_m_bits, m_a, b_mant, nullptr, b_m_bits, m_b, M, N,
                                                K, g, nullptr, N, P, static_cast<hipStream_t>(stream)));
}

int bfp_packed_sizes(int64_t rows, int64_t len, int m_bits, size_t* mant_bytes, size_t* exp_bytes) {
  if (!mant_bytes || !exp_bytes) return BFP_E_ARG;
  const int st = check_packed(rows, len, m_bits);
  if (st != BFP_OK) return st;
  const int64_t ngroups = rows * (len / fastbfp::kPackedGroup);
  *mant_bytes = (size_t)((m_bits + 1) / 2) * fastbfp::kPackedPlaneGroupBytes * (size_t)ngroups;
  *exp_bytes = (size_t)fastbfp::packed_exp_bytes(ngroups);
  return BFP_OK;
}

int bfp_quantize_packed(const float* x, int64_t R, int64_t C, int m_bits, int round_mode, uint64_t seed,
                        uint8_t* mant, uint8_t* exp, uint32_t* status_word, void* stream) {
  if (round_mode < BFP_ROUND_NEAREST || round_mode > BFP_ROUND_TRUNCATE) return BFP_E_ARG;
  const int st = check_packed(R, C, m_bits);
  if (st != BFP_OK) return st;
  if (R == 0 || C == 0) return BFP_OK;
  if (!x || !mant || !exp) return BFP_E_ARG;
  if (!aligned(x, 16) || !aligned(mant, 4) || !aligned(exp, 4) || !aligned(status_word, 4)) return BFP_E_ARG;
  if ((R * (C / 16) + 255) / 256 > 0x7fffffff) return BFP_E_UNSUPPORTED;  // 256 groups per workgroup
  return status_of(fastbfp::launch_quantize_packed(x, R, C, m_bits, round_mode, seed, mant, exp, status_word,
                                                   static_cast<hipStream_t>(stream)));
}

int bfp_dequantize_packed(const uint8_t* mant, const uint8_t* exp, int64_t rows, int64_t len, int m_bits, float* y,
                          void* stream) {
  const int st = check_packed(rows, len, m_bits);
  if (st != BFP_OK) return st;
  if (rows == 0 || len == 0) return BFP_OK;
  if (!mant || !exp || !y) return BFP_E_ARG;
  if (!aligned(mant, 4) || !aligned(exp, 4) || !aligned(y, 16)) return BFP_E_ARG;
  if ((rows * (len / 16) + 255) / 256 > 0x7fffffff) return BFP_E_UNSUPPORTED;
  return status_of(
      fastbfp::launch_dequantize_packed(mant, exp, rows, len, m_bits, y, static_cast<hipStream_t>(stream)));
}

int bfp_gemm_packed(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant,
                    const uint8_t* b_exp, int b_m_bits, int64_t M, int64_t N, int64_t K, int m_a, int m_b, float* C,
                    int64_t ldc, void* stream) {
  int st = check_gemm(a_mant, a_m_bits, b_mant, b_m_bits, M, N, K, fastbfp::kPackedGroup, m_a, m_b);
  if (st != BFP_OK) return st;
  if (ldc < N) return BFP_E_SHAPE;
  if (!general_grid_ok(M, N)) return BFP_E_UNSUPPORTED;
  if (M == 0 || N == 0) return BFP_OK;
  if (!C || !a_exp || !b_exp) return BFP_E_ARG;
  if (!aligned(a_exp, 4) || !aligned(b_exp, 4)) return BFP_E_ARG;
  return status_of(fastbfp::launch_gemm_general(a_mant, a_exp, a_m_bits, m_a, b_mant, b_exp, b_m_bits, m_b, M, N, K,
                                                fastbfp::kPackedGroup, C, ldc, nullptr,
                                                static_cast<hipStream_t>(stream), true));
}

int bfp_repack_sizes(int64_t rows, int64_t len, int g, int m_use, size_t* mant_bytes, size_t* exp_bytes,
                     int64_t* len_out, int* g_out) {
  if (!mant_bytes || !exp_bytes || !len_out || !g_out) return BFP_E_ARG;
  const int st = check_tensor(rows, len, g, m_use);
  if (st != BFP_OK) return st;
  int64_t lo;
  int go;
  fastbfp::repack_shape(len, g, &lo, &go);
  if (rows > 0 && lo / 16 > (int64_t(1) << 56) / rows) return BFP_E_UNSUPPORTED;
  *len_out = lo;
  *g_out = go;
  return bfp_quantized_sizes(rows, lo, go, m_use, mant_bytes, exp_bytes);
}

int bfp_repack(const uint8_t* mant, const uint8_t* exp, int64_t rows, int64_t len, int g, int m_bits, int packed,
               int m_use, uint8_t* out_mant, uint8_t* out_exp, void* stream) {
  if (packed != 0 && packed != 1) return BFP_E_ARG;
  if (packed && g != 16) return BFP_E_UNSUPPORTED;
  int st = packed ? check_packed(rows, len, m_bits) : check_tensor(rows, len, g, m_bits);
  if (st != BFP_OK) return st;
  if (m_use < 1 || m_use > m_bits) return BFP_E_PRECISION;
  size_t mb, eb;
  int64_t lo;
  int go;
  st = bfp_repack_sizes(rows, len, g, m_use, &mb, &eb, &lo, &go);
  if (st != BFP_OK) return st;
  if (rows == 0 || len == 0) return BFP_OK;
  if (!mant || !exp || !out_mant || !out_exp) return BFP_E_ARG;
  if (!aligned(mant, 4) || !aligned(out_mant, 4) || (packed && !aligned(exp, 4))) return BFP_E_ARG;
  if ((rows * (lo / 16) + 255) / 256 > 0x7fffffff) return BFP_E_UNSUPPORTED;
  return status_of(fastbfp::launch_repack(mant, exp, rows, len, g, m_bits, m_use, packed != 0, out_mant, out_exp,
                                          static_cast<hipStream_t>(stream)));
}

int bfp_gemm_ws_size(int a_m_bits, int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, int packed,
                     size_t* bytes) {
  if (!bytes) return BFP_E_ARG;
  int st = check_gemm_shape(a_m_bits, b_m_bits, M, N, K, g, m_a, m_b);
  if (st != BFP_OK) return st;
  WsPlan p;
  st = ws_plan(a_m_bits, b_m_bits, M, N, K, g, m_a, m_b, packed, &p);
  if (st != BFP_OK) return st;
  *bytes = p.bytes;
  return BFP_OK;
}

int bfp_gemm_ws(const uint8_t* a_mant, const uint8_t* a_exp, int a_m_bits, const uint8_t* b_mant, const uint8_t* b_exp,
                int b_m_bits, int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, int packed, float* C,
                int64_t ldc, void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_gemm(a_mant, a_m_bits, b_mant, b_m_bits, M, N, K, g, m_a, m_b);
  if (st != BFP_OK) return st;
  if (ldc < N) return BFP_E_SHAPE;
  WsPlan p;
  st = ws_plan(a_m_bits, b_m_bits, M, N, K, g, m_a, m_b, packed, &p);
  if (st != BFP_OK) return st;
  if (M == 0 || N == 0) return BFP_OK;
  if (!C || (K > 0 && (!a_exp || !b_exp))) return BFP_E_ARG;
  if (packed && (!aligned(a_exp, 4) || !aligned(b_exp, 4))) return BFP_E_ARG;
  if (p.bytes > 0 && (!workspace || workspace_bytes < p.bytes || !aligned(workspace, 256))) return BFP_E_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  const uint8_t *am = a_mant, *ae = a_exp, *bm = b_mant, *be = b_exp;
  int a_m = a_m_bits, b_m = b_m_bits;
  // (with K = 0 nothing is repacked or read: the kernel writes zeros)
  if (p.rep_a) {
    a_m = m_a;
    if (K > 0) {
      uint8_t *om = ws, *oe = ws + align256(p.a_mant);
      st = status_of(fastbfp::launch_repack(a_mant, a_exp, M, K, g, a_m_bits, m_a, packed != 0, om, oe, s));
      if (st != BFP_OK) return st;
      am = om, ae = oe;
    }
  }
  if (p.rep_b) {
    b_m = m_b;
    if (K > 0) {
      uint8_t *om = ws + align256(p.a_mant) + align256(p.a_exp), *oe = om + align256(p.b_mant);
      st = status_of(fastbfp::launch_repack(b_mant, b_exp, N, K, g, b_m_bits, m_b, packed != 0, om, oe, s));
      if (st != BFP_OK) return st;
      bm = om, be = oe;
    }
  }
  return status_of(fastbfp::launch_gemm_mx(am, ae, a_m, planes_used(a_m, m_a), bm, be, b_m, planes_used(b_m, m_b), M,
                                           N, p.k_out, p.g_out, 4 - m_a - m_b, C, ldc, -1, s));
}

int bfp_quantize_dual(const float* x, int64_t R, int64_t C, int g, int m_bits, int round_mode, uint64_t seed_r,
                      uint64_t seed_c, uint8_t* mant_r, uint8_t* exp_r, uint8_t* mant_c, uint8_t* exp_c,
                      uint32_t* status_word, void* stream) {
  const int st = check_dual(x, R, C, g, m_bits, round_mode, mant_r, exp_r, mant_c, exp_c, status_word);
  if (st != BFP_OK || R == 0 || C == 0) return st;
  return status_of(fastbfp::launch_quantize_dual(x, R, C, m_bits, round_mode, seed_r, seed_c, mant_r, exp_r, mant_c,
                                                 exp_c, status_word, static_cast<hipStream_t>(stream)));
}

int bfp_weight_update(const float* w, const float* dw, float alpha, float* w_out, int64_t R, int64_t C, int g,
                      int m_bits, int round_mode, uint64_t seed_r, uint64_t seed_c, uint8_t* mant_r, uint8_t* exp_r,
                      uint8_t* mant_c, uint8_t* exp_c, uint32_t* status_word, void* stream) {
  const int st = check_dual(w, R, C, g, m_bits, round_mode, mant_r, exp_r, mant_c, exp_c, status_word);
  if (st != BFP_OK || R == 0 || C == 0) return st;
  if (!dw || !w_out || !aligned(dw, 16) || !aligned(w_out, 16)) return BFP_E_ARG;
  const size_t bytes = (size_t)R * (size_t)C * 4;
  const uintptr_t d0 = reinterpret_cast<uintptr_t>(dw), o0 = reinterpret_cast<uintptr_t>(w_out);
  if (d0 < o0 + bytes && o0 < d0 + bytes) return BFP_E_ARG;  // dw overlaps w_out
  return status_of(fastbfp::launch_weight_update(w, dw, alpha, w_out, R, C, m_bits, round_mode, seed_r, seed_c, mant_r,
                                                 exp_r, mant_c, exp_c, status_word,
                                                 static_cast<hipStream_t>(stream)));
}

int bfp_quantize_adaptive(const float* x, int64_t R, int64_t C, int group_axis, int g, int round_mode, uint64_t seed,
                          uint8_t* mant4, uint8_t* mant2, uint8_t* exp, double* sums, uint32_t* status_word,
                          void* stream) {
  if (group_axis != 0 && group_axis != 1) return BFP_E_ARG;
  if (round_mode < BFP_ROUND_NEAREST || round_mode > BFP_ROUND_TRUNCATE) return BFP_E_ARG;
  const int64_t rows = group_axis == 1 ? R : C, len = group_axis == 1 ? C : R;
  const int st = check_tensor(rows, len, g, 4);
  if (st != BFP_OK) return st;
  if (g != 16 && g != 32) return BFP_E_UNSUPPORTED;
  if (!sums || !aligned(sums, 8)) return BFP_E_ARG;
  if (R != 0 && C != 0) {
    if (!x || !mant4 || !exp) return BFP_E_ARG;
    if (!aligned(x, group_axis == 1 ? 16 : 4) || !aligned(mant4, 4) || !aligned(mant2, 4) ||
        !aligned(status_word, 4))
      return BFP_E_ARG;
  }
  return status_of(fastbfp::launch_quantize_adaptive(x, R, C, group_axis, g, round_mode, seed, mant4, mant2, exp, sums,
                                                     status_word, static_cast<hipStream_t>(stream)));
}

int bfp_quantize_adaptive_noalloc(const float* x, int64_t R, int64_t C, int group_axis, int g, int round_mode,
                                  uint64_t seed, uint8_t* mant4, uint8_t* mant2, uint8_t* exp, double* sums,
                                  uint32_t* status_word, void* stream) {
  if (group_axis != 0 && group_axis != 1) return BFP_E_ARG;
  if (round_mode < BFP_ROUND_NEAREST || round_mode > BFP_ROUND_TRUNCATE) return BFP_E_ARG;
  const int64_t rows = group_axis == 1 ? R : C, len = group_axis == 1 ? C : R;
  const int st = check_tensor(rows, len, g, 4);
  if (st != BFP_OK) return st;
  if (g != 16 && g != 32) return BFP_E_UNSUPPORTED;
  if (!sums || !aligned(sums, 8)) return BFP_E_ARG;
  if (2 * fastbfp::adaptive_parts(R, C, group_axis, g) > fastbfp::kAdaptiveScratchDoubles) return BFP_E_UNSUPPORTED;
  if (R != 0 && C != 0) {
    if (!x || !mant4 || !exp) return BFP_E_ARG;
    if (!aligned(x, group_axis == 1 ? 16 : 4) || !aligned(mant4, 4) || !aligned(mant2, 4) ||
        !aligned(status_word, 4))
      return BFP_E_ARG;
  }
  return status_of(fastbfp::launch_quantize_adaptive_static(x, R, C, group_axis, g, round_mode, seed, mant4, mant2,
                                                            exp, sums, status_word,
                                                            static_cast<hipStream_t>(stream)));
}

int64_t bfp_adaptive_noalloc_max_parts(void) { return fastbfp::kAdaptiveScratchDoubles / 2; }

int64_t bfp_adaptive_parts(int64_t R, int64_t C, int group_axis, int g) {
  if ((group_axis != 0 && group_axis != 1) || (g != 16 && g != 32) || R < 0 || C < 0) return -1;
  if ((group_axis == 1 ? C : R) % g != 0) return -1;
  return fastbfp::adaptive_parts(R, C, group_axis, g);
}

int64_t bfp_adaptive_sums_len(int64_t R, int64_t C, int group_axis, int g) {
  if ((group_axis != 0 && group_axis != 1) || (g != 16 && g != 32) || R < 0 || C < 0) return -1;
  if ((group_axis == 1 ? C : R) % g != 0) return -1;
  return 2 + 2 * fastbfp::adaptive_parts(R, C, group_axis, g);
}

double bfp_adaptive_threshold(double alpha, double beta, int64_t i, int64_t I, int64_t l, int64_t L) {
  if (I <= 0 || L <= 0) return __builtin_nan("");
  return alpha - beta * (double)i / (double)I - beta * (double)l / (double)L;
}

int bfp_adaptive_mantissa(double num, double den, double eps) {
  const double r = den > 0.0 ? num / den : 0.0;
  return r < eps ? 2 : 4;
}

}  // extern "C"
