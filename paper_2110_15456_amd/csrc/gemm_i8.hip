// gemm_i8.hip -- exact integer BFP group partials on int8 MFMA (parts M and A
// of the group dot product, section III-B), for verification.
//
// P[G][i][j] = sum_{k in G} qa'[i][k] * qb'[j][k].  Each 16-value sub-block of
// a group is one v_mfma_i32_32x32x16_i8.  The chunk codes are decoded to
// signed int8 chunks (|chunk| <= 15), one MFMA pass is issued per chunk-plane
// pair (ca, cb), and the passes are combined exactly in int32 as
// sum 2^(wa sa + wb sb) * P_{ca,cb}, sa and sb being the chunks' significance
// and w the bits of an operand's lower chunk (2 for m = 5, 6; 4 for m = 7, 8)
// -- the pass structure of the paper's variable-precision fMAC (section V-B).
#include "bfp_device.h"
#include "launch.h"

namespace fastbfp {

// Eight consecutive codes starting at value v0 of a group (v0 % 8 == 0)
// decoded to int8 chunks and packed little-endian into 64 bits, from a plane
// of kind pk (launch.h): FP6 codes of +-c/2 (6 bytes), FP4 codes (4 bytes:
// the sign bit above the chunk), or a Lo2 plane (the 8 bytes of the value's
// 16-value half, unpacked to FP6 codes of +-c/8).
__device__ __forceinline__ long decode8(const uint8_t* __restrict__ grp, int v0, bool valid, int pk) {
  if (!valid) return 0;
  uint64_t bits = 0;
  int t0 = 0;  // field of value v0 in the decoded bit string
  if (pk == kPlaneLo2) {
    const uint32_t* h = reinterpret_cast<const uint32_t*>(grp + (v0 / 16) * 8);
    uint32_t c0, c1, c2;
    lo2_unpack(h[0], h[1], c0, c1, c2);
    const int bit = 6 * (v0 % 16);  // 0 or 48
    const uint64_t lo = (uint64_t)c0 | ((uint64_t)c1 << 32);
    bits = bit == 0 ? lo : ((lo >> 48) | ((uint64_t)c2 << 16));
  } else {
    const int w = pk == kPlaneFP4 ? 4 : 6;
    const uint8_t* p = grp + (v0 * w) / 8;
    for (int k = 0; k < w; ++k) bits |= (uint64_t)p[k] << (8 * k);
  }
  uint64_t out = 0;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    int c;
    if (pk == kPlaneFP4) {
      const uint32_t nib = (uint32_t)(bits >> (4 * t)) & 0xFu;
      c = (nib & 8u) ? -(int)(nib & 7u) : (int)(nib & 7u);
    } else if (pk == kPlaneLo2) {
      c = e2m3_eighth_decode((uint32_t)(bits >> (6 * (t0 + t))) & 0x3Fu);
    } else {
      c = e2m3_half_decode((uint32_t)(bits >> (6 * t)) & 0x3Fu);
    }
    out |= (uint64_t)(uint8_t)(int8_t)c << (8 * t);
  }
  return (long)out;
}

// One wave computes a 32x32 tile of P for one group.
// a_m / b_m: the stored widths (plane formats and the weight of the upper
// chunk); a_ps / b_ps: plane 0's size; na / nb: planes read.
template <int G>
__global__ __launch_bounds__(64) void k_group_partials(const uint8_t* __restrict__ a_mant, int64_t a_ps, int na,
                                                       int a_m, const uint8_t* __restrict__ b_mant, int64_t b_ps,
                                                       int nb, int b_m, int M, int N, int ng,
                                                       int32_t* __restrict__ P) {
  const int lane = threadIdx.x;
  const int col0 = blockIdx.x * 32, row0 = blockIdx.y * 32, grp = blockIdx.z;
  const int ar = row0 + (lane & 31), bc = col0 + (lane & 31), half = lane >> 5;
  v16i total = {};
  for (int ca = 0; ca < na; ++ca)
    for (int cb = 0; cb < nb; ++cb) {
      v16i part = {};
      const int ka = plane_kind(a_m, ca), kb = plane_kind(b_m, cb);
      const int gba = plane_group_bytes(G, a_m, ca), gbb = plane_group_bytes(G, b_m, cb);  // bytes per group
      const uint8_t* ga = a_mant + ca * a_ps + ((int64_t)ar * ng + grp) * gba;
      const uint8_t* gb = b_mant + cb * b_ps + ((int64_t)bc * ng + grp) * gbb;
#pragma unroll
      for (int sb = 0; sb < G / 16; ++sb) {
        const long av = decode8(ga, 16 * sb + 8 * half, ar < M, ka);
        const long bv = decode8(gb, 16 * sb + 8 * half, bc < N, kb);
        part = __builtin_amdgcn_mfma_i32_32x32x16_i8(av, bv, part, 0, 0, 0);
      }
      // the upper chunk's weight: 2^2 (m = 5, 6) or 2^4 (m = 7, 8)
      const int shift = low_chunk_bits(a_m) * (na - 1 - ca) + low_chunk_bits(b_m) * (nb - 1 - cb);
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
  const dim3 grid((unsigned)((N + 31) / 32), (unsigned)((M + 31) / 32), (unsigned)ng);
  if (g == 16)
    hipLaunchKernelGGL((k_group_partials<16>), grid, dim3(64), 0, s, a_mant, a_ps, na, a_m, b_mant, b_ps, nb, b_m,
                       (int)M, (int)N, ng, P);
  else
    hipLaunchKernelGGL((k_group_partials<32>), grid, dim3(64), 0, s, a_mant, a_ps, na, a_m, b_mant, b_ps, nb, b_m,
                       (int)M, (int)N, ng, P);
  return hipGetLastError();
}

}  // namespace fastbfp
