// gemm_i8.hip -- exact integer BFP group partials on int8 MFMA (parts M and A
// of the group dot product, section III-B), for verification.
//
// P[G][i][j] = sum_{k in G} qa'[i][k] * qb'[j][k].  Each 16-value sub-block of
// a group is one v_mfma_i32_32x32x16_i8.  The FP6 chunk codes are decoded to
// signed int8 chunks (|chunk| <= 15), one MFMA pass is issued per chunk-plane
// pair (ca, cb), and the passes are combined exactly in int32 as
// sum 2^(4 (sa + sb)) * P_{ca,cb}, sa and sb being the chunks' significance --
// the pass structure of the paper's variable-precision fMAC (section V-B)
// with 4-bit instead of 2-bit chunks.
#include "bfp_device.h"
#include "launch.h"

namespace fastbfp {

// Eight consecutive FP6 codes starting at value v0 of a group (v0 % 8 == 0)
// decoded to int8 and packed little-endian into 64 bits.
__device__ __forceinline__ long decode8(const uint8_t* __restrict__ grp, int v0, bool valid) {
  if (!valid) return 0;
  const uint8_t* p = grp + (v0 * 6) / 8;  // 6 bytes hold the 8 codes
  uint64_t bits = 0;
#pragma unroll
  for (int k = 0; k < 6; ++k) bits |= (uint64_t)p[k] << (8 * k);
  uint64_t out = 0;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const int c = e2m3_half_decode((uint32_t)(bits >> (6 * t)) & 0x3Fu);
    out |= (uint64_t)(uint8_t)(int8_t)c << (8 * t);
  }
  return (long)out;
}

// One wave computes a 32x32 tile of P for one group.
template <int G>
__global__ __launch_bounds__(64) void k_group_partials(const uint8_t* __restrict__ a_mant, int64_t a_ps, int na,
                                                       const uint8_t* __restrict__ b_mant, int64_t b_ps, int nb,
                                                       int M, int N, int ng, int32_t* __restrict__ P) {
  const int lane = threadIdx.x;
  const int col0 = blockIdx.x * 32, row0 = blockIdx.y * 32, grp = blockIdx.z;
  const int ar = row0 + (lane & 31), bc = col0 + (lane & 31), half = lane >> 5;
  constexpr int GB = G * 3 / 4;  // bytes per group per plane
  v16i total = {};
  for (int ca = 0; ca < na; ++ca)
    for (int cb = 0; cb < nb; ++cb) {
      v16i part = {};
      const uint8_t* ga = a_mant + ca * a_ps + ((int64_t)ar * ng + grp) * GB;
      const uint8_t* gb = b_mant + cb * b_ps + ((int64_t)bc * ng + grp) * GB;
#pragma unroll
      for (int sb = 0; sb < G / 16; ++sb) {
        const long av = decode8(ga, 16 * sb + 8 * half, ar < M);
        const long bv = decode8(gb, 16 * sb + 8 * half, bc < N);
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

hipError_t launch_group_partials(const uint8_t* a_mant, int a_planes, int na, const uint8_t* b_mant, int b_planes,
                                 int nb, int64_t M, int64_t N, int64_t K, int g, int32_t* P, hipStream_t s) {
  (void)a_planes;
  (void)b_planes;
  if (M == 0 || N == 0 || K == 0) return hipSuccess;
  const int ng = (int)(K / g);
  const int64_t a_ps = M * K * 3 / 4, b_ps = N * K * 3 / 4;
  const dim3 grid((unsigned)((N + 31) / 32), (unsigned)((M + 31) / 32), (unsigned)ng);
  if (g == 16)
    hipLaunchKernelGGL((k_group_partials<16>), grid, dim3(64), 0, s, a_mant, a_ps, na, b_mant, b_ps, nb, (int)M,
                       (int)N, ng, P);
  else
    hipLaunchKernelGGL((k_group_partials<32>), grid, dim3(64), 0, s, a_mant, a_ps, na, b_mant, b_ps, nb, (int)M,
                       (int)N, ng, P);
  return hipGetLastError();
}

}  // namespace fastbfp
