// gemm_i8.hip -- exact integer BFP group partials on int8 MFMA (parts M and A
// of the group dot product, section III-B), for verification.
//
// P[G][i][j] = sum_{k in G} qa'[i][k] * qb'[j][k].  Each 16-value sub-block of
// a group is one v_mfma_i32_32x32x16_i8.  The FP6/FP4 chunk codes are decoded to
// signed int8 chunks (|chunk| <= 15), one MFMA pass is issued per chunk-plane
// pair (ca, cb), and the passes are combined exactly in int32 as
// sum 2^(4 (sa + sb)) * P_{ca,cb}, sa and sb being the chunks' significance --
// the pass structure of the paper's variable-precision fMAC (section V-B)
// with 4-bit instead of 2-bit chunks.
#include "bfp_device.h"
#include "launch.h"

namespace fastbfp {

// Eight consecutive codes starting at value v0 of a group (v0 % 8 == 0)
// decoded to int8 and packed little-endian into 64 bits: FP6 codes (6 bytes)
// or, with fp4, FP4 codes (4 bytes: the sign bit above the chunk).
__device__ __forceinline__ long decode8(const uint8_t* __restrict__ grp, int v0, bool valid, bool fp4) {
  if (!valid) return 0;
  const int w = fp4 ? 4 : 6;
  const uint8_t* p = grp + (v0 * w) / 8;
  uint64_t bits = 0;
  for (int k = 0; k < w; ++k) bits |= (uint64_t)p[k] << (8 * k);
  uint64_t out = 0;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    int c;
    if (fp4) {
      const uint32_t nib = (uint32_t)(bits >> (4 * t)) & 0xFu;
      c = (nib & 8u) ? -(int)(nib & 7u) : (int)(nib & 7u);
    } else {
      c = e2m3_half_decode((uint32_t)(bits >> (6 * t)) & 0x3Fu);
    }
    out |= (uint64_t)(uint8_t)(int8_t)c << (8 * t);
  }
  return (long)out;
}

// One wave computes a 32x32 tile of P for one group.
// a4 / b4: plane 0 of A / B holds FP4 codes; a_ps / b_ps: plane 0's size.
template <int G>
__global__ __launch_bounds__(64) void k_group_partials(const uint8_t* __restrict__ a_mant, int64_t a_ps, int na,
                                                       int a4, const uint8_t* __restrict__ b_mant, int64_t b_ps,
                                                       int nb, int b4, int M, int N, int ng,
                                                       int32_t* __restrict__ P) {
  const int lane = threadIdx.x;
  const int col0 = blockIdx.x * 32, row0 = blockIdx.y * 32, grp = blockIdx.z;
  const int ar = row0 + (lane & 31), bc = col0 + (lane & 31), half = lane >> 5;
  v16i total = {};
  for (int ca = 0; ca < na; ++ca)
    for (int cb = 0; cb < nb; ++cb) {
      v16i part = {};
      const bool fa = ca == 0 && a4, fb = cb == 0 && b4;
      const int gba = fa ? G / 2 : G * 3 / 4, gbb = fb ? G / 2 : G * 3 / 4;  // bytes per group in the plane
      const uint8_t* ga = a_mant + ca * a_ps + ((int64_t)ar * ng + grp) * gba;
      const uint8_t* gb = b_mant + cb * b_ps + ((int64_t)bc * ng + grp) * gbb;
#pragma unroll
      for (int sb = 0; sb < G / 16; ++sb) {
        const long av = decode8(ga, 16 * sb + 8 * half, ar < M, fa);
        const long bv = decode8(gb, 16 * sb + 8 * half, bc < N, fb);
        part = __builtin_amdgcn_mfma_i32_32x32x16_i8(av, bv, part, 0, 0, 0);
      }
      const int shift = 4 * ((na - 1 - ca) + (nb - 1 - cb));
#pragma unroll
      for (int r = 0; r < 16; ++r) total[r] += part[r] << shift;
    }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int row = row0 + (r / 4) * 8 + half * 4 + (r % 4), col = col0 + (lane & 31);
    if (row < M && col < N) P[((int64_t)grp * M + row) * N + col] = total[r];
  }
}

hipError_t launch_group_partials(const uint8_t* a_mant, int a_m, int na, const uint8_t* b_mant, int b_m, int nb,
                                 int64_t M, int64_t N, int64_t K, int g, int32_t* P, hipStream_t s) {
  if (M == 0 || N == 0 || K == 0) return hipSuccess;
  const int ng = (int)(K / g);
  const int64_t a_ps = M * ng * plane_group_bytes(g, a_m, 0), b_ps = N * ng * plane_group_bytes(g, b_m, 0);
  const int a4 = plane0_fp4(a_m), b4 = plane0_fp4(b_m);
  const dim3 grid((unsigned)((N + 31) / 32), (unsigned)((M + 31) / 32), (unsigned)ng);
  if (g == 16)
    hipLaunchKernelGGL((k_group_partials<16>), grid, dim3(64), 0, s, a_mant, a_ps, na, a4, b_mant, b_ps, nb, b4,
                       (int)M, (int)N, ng, P);
  else
    hipLaunchKernelGGL((k_group_partials<32>), grid, dim3(64), 0, s, a_mant, a_ps, na, a4, b_mant, b_ps, nb, b4,
                       (int)M, (int)N, ng, P);
  return hipGetLastError();
}

}  // namespace fastbfp
