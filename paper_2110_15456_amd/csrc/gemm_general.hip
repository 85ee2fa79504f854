// gemm_general.hip -- the BFP GEMM for every case the block-scaled kernel
// (gemm_mx.h) does not take, and the exact integer group partials: int8 MFMA
// on decoded magnitudes (section III-B parts M and A), one group at a time.
//
// Either operand may be taken at any precision m_use <= its stored m (the
// magnitude truncated to its top m_use bits, the paper's discard of low-order
// bits, section V-D), and the group size may be 4, 8, 16, 32 or 64 (the
// sensitivity study of section VI-C uses 8, 16 and 32).
//
// One wave computes a 32 x 32 tile of C.  Per group: the lanes decode their
// rows' and columns' codes to signed magnitudes, truncate them, and issue
// v_mfma_i32_32x32x16_i8 per 16 values of the group (a group of 4 or 8 is its
// 16-value unit with the other groups' values masked to zero), splitting an
// 8-bit magnitude into two 4-bit chunks combined in int32 as 16 P_hi + P_lo --
// the fMAC's pass structure (section V-B).  The group's exact integer partial
// P_G is then scaled by 2^(ea + eb - 254 - (m_a-1) - (m_b-1)) (an exact
// power-of-two scaling) and added to an FP32 accumulator: the fMAC's exponent
// addition and FP32 accumulation.  With WRITE_P the kernel writes P_G instead
// (bfp_gemm_group_partials).  The same kernel takes operands in the packed
// layout of packed.hip (bfp_gemm_packed).
#include "bfp_decode.h"

namespace fastbfp {

namespace {

// Eight int8 chunks packed little-endian: pass `pass` of `npass` (the whole
// magnitude when npass = 1; its upper or lower 4 bits, signed, when 2), with
// the values outside [lo, hi) of the 8 zeroed.
__device__ __forceinline__ long pack8(const int (&q)[8], int pass, int npass, int lo, int hi) {
  uint64_t out = 0;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const int a = q[t] < 0 ? -q[t] : q[t];
    int c = npass == 1 ? a : (pass == 0 ? a >> 4 : a & 15);
    if (q[t] < 0) c = -c;
    if (t < lo || t >= hi) c = 0;
    out |= (uint64_t)(uint8_t)(int8_t)c << (8 * t);
  }
  return (long)out;
}

typedef int v16i_t __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

// WRITE_P: write the int32 group partials P[G][M][N]; otherwise accumulate C.
template <bool WRITE_P>
__global__ __launch_bounds__(64) void k_gemm_general(Opnd A, Opnd B, int g, int tiles_n, int M, int N, float* C,
                                                     int64_t ldc, int32_t* P) {
  const int lane = threadIdx.x;
  const int tm = (int)(blockIdx.x / tiles_n), tn = (int)(blockIdx.x % tiles_n);
  const int row0 = tm * 32, col0 = tn * 32;
  const int ar = row0 + (lane & 31), bc = col0 + (lane & 31), half = lane >> 5;
  const int npa = A.m_use == 8 ? 2 : 1, npb = B.m_use == 8 ? 2 : 1;
  const int bias = 254 + (A.m_use - 1) + (B.m_use - 1);
  v16f acc = {};
  // groups of 4 or 8 share a 16-value unit: decode the unit once
  const int gpu = g < 16 ? 16 / g : 1;  // groups per decoded unit
  const int64_t nunits_loop = g < 16 ? A.units : A.ngr;
  for (int64_t it = 0; it < nunits_loop; ++it) {
    for (int sg = 0; sg < gpu; ++sg) {
      const int64_t G = it * gpu + sg;
      v16i_t total = {};
      for (int sb = 0; sb < (g < 16 ? 1 : g / 16); ++sb) {
        const int64_t unit = g < 16 ? it : G * (g / 16) + sb;
        int qa[8], qb[8];
        decode_q8(A, ar, unit, half, qa);
        decode_q8(B, bc, unit, half, qb);
        // values of this group among the lane's 8: positions [lo, hi) of the
        // lane's half of the unit
        int lo = 0, hi = 8;
        if (g < 16) {
          lo = max(0, sg * g - 8 * half);
          hi = min(8, (sg + 1) * g - 8 * half);
        }
        for (int pa = 0; pa < npa; ++pa)
          for (int pb = 0; pb < npb; ++pb) {
            const long av = pack8(qa, pa, npa, lo, hi), bv = pack8(qb, pb, npb, lo, hi);
            const v16i_t part = __builtin_amdgcn_mfma_i32_32x32x16_i8(av, bv, v16i_t{}, 0, 0, 0);
            const int shift = 4 * ((npa - 1 - pa) + (npb - 1 - pb));
#pragma unroll
            for (int r = 0; r < 16; ++r) total[r] += part[r] << shift;
          }
      }
      if constexpr (WRITE_P) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + (r / 4) * 8 + half * 4 + (r % 4), col = bc;
          if (row < M && col < N) P[(G * M + row) * N + col] = total[r];
        }
      } else {
        // the shared exponents: lane l holds row row0 + (l & 31)'s; element r
        // of every lane belongs to row (r / 4) * 8 + half * 4 + r % 4
        const int ea_mine = ar < M ? opnd_exponent(A, ar, G) : 0;
        const int eb = bc < N ? opnd_exponent(B, bc, G) : 0;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ea = __shfl(ea_mine, (r / 4) * 8 + half * 4 + (r % 4));
          acc[r] += ldexpf((float)total[r], ea + eb - bias);  // exact scaling, one FP32 rounding
        }
      }
    }
  }
  if constexpr (!WRITE_P) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = row0 + (r / 4) * 8 + half * 4 + (r % 4), col = bc;
      if (row < M && col < N) C[(int64_t)row * ldc + col] = acc[r];
    }
  }
}


}  // namespace

hipError_t launch_gemm_general(const uint8_t* a_mant, const uint8_t* a_exp, int a_m, int m_a, const uint8_t* b_mant,
                               const uint8_t* b_exp, int b_m, int m_b, int64_t M, int64_t N, int64_t K, int g,
                               float* C, int64_t ldc, int32_t* P, hipStream_t s, bool packed) {
  if (M == 0 || N == 0) return hipSuccess;
  const Opnd A = make_opnd(a_mant, a_exp, M, K, g, a_m, m_a, packed),
             B = make_opnd(b_mant, b_exp, N, K, g, b_m, m_b, packed);
  const int tiles_m = (int)((M + 31) / 32), tiles_n = (int)((N + 31) / 32);
  const dim3 grid((unsigned)((int64_t)tiles_m * tiles_n));
  if (P)
    hipLaunchKernelGGL(k_gemm_general<true>, grid, dim3(64), 0, s, A, B, g, tiles_n, (int)M, (int)N, C, ldc, P);
  else
    hipLaunchKernelGGL(k_gemm_general<false>, grid, dim3(64), 0, s, A, B, g, tiles_n, (int)M, (int)N, C, ldc, P);
  return hipGetLastError();
}

}  // namespace fastbfp
