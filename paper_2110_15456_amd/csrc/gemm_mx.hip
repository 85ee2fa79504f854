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

#define FASTBFP_MX11_TILES_DECLARE(FA, FB)      \
  FASTBFP_MX11_TILE_DECLARE(256, 128, FA, FB)   \
  FASTBFP_MX11_TILE_DECLARE(256, 64, FA, FB)    \
  FASTBFP_MX11_TILE_DECLARE(128, 64, FA, FB)    \
  FASTBFP_MX11_TILE_DECLARE(128, 128, FA, FB)
FASTBFP_MX11_TILES_DECLARE(0, 0)
FASTBFP_MX11_TILES_DECLARE(0, 1)
FASTBFP_MX11_TILES_DECLARE(1, 0)
FASTBFP_MX11_TILES_DECLARE(1, 1)

// Tile of the one-chunk, groups-of-16, FP32-output GEMM (0..4: 256x256,
// 256x128, 256x64, 128x64, 128x128), from measurements on MI355X over the
// transformer, FFN-step and ResNet-18 im2col shapes:
//  * N <= 64: 128x64 (a wider tile is mostly padding; 256x64 was never the
//    fastest);
//  * A in FP4 codes: 256x128 (5-11% faster than 256x256 on the transformer
//    shapes: its two LDS stages take 60-76 KB, so two workgroups share a CU);
//  * A in FP6 codes: 256x256 (a 256x128 tile still takes 92-108 KB of LDS, one
//    workgroup per CU, and ran 30-40% slower; 128x128, two per CU, 15-35%
//    slower), but 128x128 for N <= 128 or when 256x256 tiles are too few;
//  * too few: fewer than 192 tiles leave over a quarter of the 256 CUs idle;
//    then the next smaller tile, down to 128x64.
// With C converted to BFP in the epilogue (converted), A in FP4 codes gets
// the FP6 rule: there the 256x128 tile was the slower one (ffn_up (2,2) to
// m = 2: 0.71 ms against 0.60-0.63 ms on 256x256).
static int gemm_mx11_tile(int64_t M, int64_t N, int fa, bool converted) {
  constexpr int64_t MIN_TILES = 192;
  auto tiles = [&](int bm, int bn) { return ((M + bm - 1) / bm) * ((N + bn - 1) / bn); };
  if (N <= 64) return 3;
  if (fa && !converted) return tiles(256, 128) >= MIN_TILES ? 1 : 3;
  if (N > 128 && tiles(256, 256) >= MIN_TILES) return 0;
  return tiles(128, 128) >= MIN_TILES ? 4 : 3;
}

template <int FA, int FB>
static hipError_t launch_11_tile(int t, const uint8_t* a_mant, const uint8_t* a_exp, const uint8_t* b_mant,
                                 const uint8_t* b_exp, int M, int N, int ng, float scale, float* C, int64_t ldc,
                                 const OutBFP* qo, hipStream_t s) {
  if (t == 1) return launch_mx_11_tile<256, 128, FA, FB>(a_mant, a_exp, b_mant, b_exp, M, N, ng, scale, C, ldc, qo, s);
  if (t == 2) return launch_mx_11_tile<256, 64, FA, FB>(a_mant, a_exp, b_mant, b_exp, M, N, ng, scale, C, ldc, qo, s);
  if (t == 4) return launch_mx_11_tile<128, 128, FA, FB>(a_mant, a_exp, b_mant, b_exp, M, N, ng, scale, C, ldc, qo, s);
  return launch_mx_11_tile<128, 64, FA, FB>(a_mant, a_exp, b_mant, b_exp, M, N, ng, scale, C, ldc, qo, s);
}

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
                                float* C, int64_t ldc, const OutBFP* qo, int tile, hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  const int ng = (int)(K / 16);  // 16-value halves per row (the plane layout's unit)
  const int64_t a_ps = M * (K / G) * plane_group_bytes(G, a_m, 0), b_ps = N * (K / G) * plane_group_bytes(G, b_m, 0);
  // the kernels' FA / FB: one plane read, FP4 codes; two, split at 2 bits
  const int fa = na == 1 ? plane0_fp4(a_m) : a_m <= 6, fb = nb == 1 ? plane0_fp4(b_m) : b_m <= 6;
  const float scale = ldexpf(1.0f, scale_log2);
  const int m = (int)M, n = (int)N;
  if (G == 16 && na == 1 && nb == 1) {
    const int t = tile >= 0 ? tile : gemm_mx11_tile(M, N, fa, qo != nullptr);
    if (t != 0) {
      if (!fa && !fb) return launch_11_tile<0, 0>(t, a_mant, a_exp, b_mant, b_exp, m, n, ng, scale, C, ldc, qo, s);
      if (!fa) return launch_11_tile<0, 1>(t, a_mant, a_exp, b_mant, b_exp, m, n, ng, scale, C, ldc, qo, s);
      if (!fb) return launch_11_tile<1, 0>(t, a_mant, a_exp, b_mant, b_exp, m, n, ng, scale, C, ldc, qo, s);
      return launch_11_tile<1, 1>(t, a_mant, a_exp, b_mant, b_exp, m, n, ng, scale, C, ldc, qo, s);
    }
  }
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
                                  int scale_log2, float* C, int64_t ldc, const OutBFP* qo, int tile,
                                  hipStream_t s) {
  if (g == 32)
    return launch_gemm_g<32>(a_mant, a_exp, a_m, na, b_mant, b_exp, b_m, nb, M, N, K, scale_log2, C, ldc, qo, 0, s);
  return launch_gemm_g<16>(a_mant, a_exp, a_m, na, b_mant, b_exp, b_m, nb, M, N, K, scale_log2, C, ldc, qo, tile, s);
}

hipError_t launch_gemm_mx(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int na, const uint8_t* b_mant,
                          const uint8_t* b_exp, int b_m, int nb, int64_t M, int64_t N, int64_t K, int g,
                          int scale_log2, float* C, int64_t ldc, int tile, hipStream_t s) {
  return launch_gemm_any(a_mant, a_exp, a_m, na, b_mant, b_exp, b_m, nb, M, N, K, g, scale_log2, C, ldc, nullptr, tile,
                         s);
}

hipError_t launch_gemm_mx_bfp(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int na, const uint8_t* b_mant,
                              const uint8_t* b_exp, int b_m, int nb, int64_t M, int64_t N, int64_t K, int g,
                              int scale_log2, int c_m, int mode, uint64_t seed, uint8_t* c_mant, uint8_t* c_exp,
                              uint32_t* status, hipStream_t s) {
  const OutBFP qo{c_mant, c_mant + M * (N / 16) * plane_group_bytes(16, c_m, 0), c_exp, status, c_m, mode,
                  c_m <= 4 ? plane0_fp4(c_m) : c_m <= 6, (uint32_t)seed, (uint32_t)(seed >> 32)};
  return launch_gemm_any(a_mant, a_exp, a_m, na, b_mant, b_exp, b_m, nb, M, N, K, g, scale_log2, nullptr, N, &qo, -1, s);
}

}  // namespace fastbfp
