// gemm_mx.hip -- dispatch of the BFP GEMM (kernel in gemm_mx.h) over the
// group size and the operand formats: chunk planes read per operand (1 or 2)
// and whether the first plane holds FP4 codes.  Each group size and
// plane-count pair is instantiated in its own file
// (gemm_mx_{11,12,21,22}[_g32].hip) so that they compile in parallel.
#include "gemm_mx.h"

namespace fastbfp {

FASTBFP_MX_DECLARE(1, 1, 0, 0, 16)
FASTBFP_MX_DECLARE(1, 1, 0, 1, 16)
FASTBFP_MX_DECLARE(1, 1, 1, 0, 16)
FASTBFP_MX_DECLARE(1, 1, 1, 1, 16)
FASTBFP_MX_DECLARE(1, 2, 0, 0, 16)
FASTBFP_MX_DECLARE(1, 2, 0, 1, 16)
FASTBFP_MX_DECLARE(1, 2, 1, 0, 16)
FASTBFP_MX_DECLARE(1, 2, 1, 1, 16)
FASTBFP_MX_DECLARE(2, 1, 0, 0, 16)
FASTBFP_MX_DECLARE(2, 1, 0, 1, 16)
FASTBFP_MX_DECLARE(2, 1, 1, 0, 16)
FASTBFP_MX_DECLARE(2, 1, 1, 1, 16)
FASTBFP_MX_DECLARE(2, 2, 0, 0, 16)
FASTBFP_MX_DECLARE(2, 2, 0, 1, 16)
FASTBFP_MX_DECLARE(2, 2, 1, 0, 16)
FASTBFP_MX_DECLARE(2, 2, 1, 1, 16)
FASTBFP_MX_DECLARE(1, 1, 0, 0, 32)
FASTBFP_MX_DECLARE(1, 1, 0, 1, 32)
FASTBFP_MX_DECLARE(1, 1, 1, 0, 32)
FASTBFP_MX_DECLARE(1, 1, 1, 1, 32)
FASTBFP_MX_DECLARE(1, 2, 0, 0, 32)
FASTBFP_MX_DECLARE(1, 2, 0, 1, 32)
FASTBFP_MX_DECLARE(1, 2, 1, 0, 32)
FASTBFP_MX_DECLARE(1, 2, 1, 1, 32)
FASTBFP_MX_DECLARE(2, 1, 0, 0, 32)
FASTBFP_MX_DECLARE(2, 1, 0, 1, 32)
FASTBFP_MX_DECLARE(2, 1, 1, 0, 32)
FASTBFP_MX_DECLARE(2, 1, 1, 1, 32)
FASTBFP_MX_DECLARE(2, 2, 0, 0, 32)
FASTBFP_MX_DECLARE(2, 2, 0, 1, 32)
FASTBFP_MX_DECLARE(2, 2, 1, 0, 32)
FASTBFP_MX_DECLARE(2, 2, 1, 1, 32)

template <int NA, int NB, int G>
static hipError_t launch_fmt(int fa, int fb, const uint8_t* a_mant, const uint8_t* a_exp, int64_t a_ps,
                             const uint8_t* b_mant, const uint8_t* b_exp, int64_t b_ps, int M, int N, int ng,
                             float scale, float* C, int64_t ldc, const OutBFP* qo, hipStream_t s) {
  if (!fa && !fb) return launch_mx_t<NA, NB, 0, 0, G>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, qo, s);
  if (!fa) return launch_mx_t<NA, NB, 0, 1, G>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, qo, s);
  if (!fb) return launch_mx_t<NA, NB, 1, 0, G>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, qo, s);
  return launch_mx_t<NA, NB, 1, 1, G>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, qo, s);
}

// a_m / b_m: the stored operands' widths (they fix the plane formats and the
// plane stride); na / nb: planes read; g: the group size.
template <int G>
static hipError_t launch_gemm_g(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int na, const uint8_t* b_mant,
                                const uint8_t* b_exp, int b_m, int nb, int64_t M, int64_t N, int64_t K, int scale_log2,
                                float* C, int64_t ldc, const OutBFP* qo, hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  const int ng = (int)(K / 16);  // 16-value halves per row (the plane layout's unit)
  const int64_t a_ps = M * (K / G) * plane_group_bytes(G, a_m, 0), b_ps = N * (K / G) * plane_group_bytes(G, b_m, 0);
  const int fa = plane0_fp4(a_m), fb = plane0_fp4(b_m);
  const float scale = ldexpf(1.0f, scale_log2);
  const int m = (int)M, n = (int)N;
  if (na == 1 && nb == 1)
    return launch_fmt<1, 1, G>(fa, fb, a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, m, n, ng, scale, C, ldc, qo, s);
  if (na == 1 && nb == 2)
    return launch_fmt<1, 2, G>(fa, fb, a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, m, n, ng, scale, C, ldc, qo, s);
  if (na == 2 && nb == 1)
    return launch_fmt<2, 1, G>(fa, fb, a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, m, n, ng, scale, C, ldc, qo, s);
  return launch_fmt<2, 2, G>(fa, fb, a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, m, n, ng, scale, C, ldc, qo, s);
}

static hipError_t launch_gemm_any(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int na, const uint8_t* b_mant,
                                  const uint8_t* b_exp, int b_m, int nb, int64_t M, int64_t N, int64_t K, int g,
                                  int scale_log2, float* C, int64_t ldc, const OutBFP* qo, hipStream_t s) {
  if (g == 32)
    return launch_gemm_g<32>(a_mant, a_exp, a_m, na, b_mant, b_exp, b_m, nb, M, N, K, scale_log2, C, ldc, qo, s);
  return launch_gemm_g<16>(a_mant, a_exp, a_m, na, b_mant, b_exp, b_m, nb, M, N, K, scale_log2, C, ldc, qo, s);
}

hipError_t launch_gemm_mx(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int na, const uint8_t* b_mant,
                          const uint8_t* b_exp, int b_m, int nb, int64_t M, int64_t N, int64_t K, int g,
                          int scale_log2, float* C, int64_t ldc, hipStream_t s) {
  return launch_gemm_any(a_mant, a_exp, a_m, na, b_mant, b_exp, b_m, nb, M, N, K, g, scale_log2, C, ldc, nullptr, s);
}

hipError_t launch_gemm_mx_bfp(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int na, const uint8_t* b_mant,
                              const uint8_t* b_exp, int b_m, int nb, int64_t M, int64_t N, int64_t K, int g,
                              int scale_log2, int c_m, int mode, uint64_t seed, uint8_t* c_mant, uint8_t* c_exp,
                              uint32_t* status, hipStream_t s) {
  const OutBFP qo{c_mant,     c_mant + M * (N / 16) * plane_group_bytes(16, c_m, 0), c_exp, status, c_m, mode,
                  plane0_fp4(c_m), (uint32_t)seed, (uint32_t)(seed >> 32)};
  return launch_gemm_any(a_mant, a_exp, a_m, na, b_mant, b_exp, b_m, nb, M, N, K, g, scale_log2, nullptr, N, &qo, s);
}

}  // namespace fastbfp
