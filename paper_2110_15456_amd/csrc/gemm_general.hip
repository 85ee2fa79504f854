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
#include "bfp_device.h"
#include "launch.h"

namespace fastbfp {

namespace {

// One operand as the decoder reads it: planes in 16-value units, or the
// packed layout (3-bit fields of 2-bit chunks, g = 16).
struct Opnd {
  const uint8_t* p0;    // plane 0 (packed: all ceil(m/2) planes, plane c at c * rows * units * 6)
  const uint8_t* p1;    // plane 1 (m > 4; unused when packed)
  const uint8_t* exps;  // [rows][len / g], or the packed exponent stream
  int64_t units;        // 16-value units per row (len / 16)
  int64_t ngr;          // groups per row (len / g)
  int rows, m, m_use;
  bool packed;
};

// Bytes of a 16-value unit of plane p of an m-bit tensor.
__device__ __forceinline__ int unit_bytes(int m, int p) { return plane_kind(m, p) == kPlaneFP6 ? 12 : 8; }

// The 8 chunks (signed) of values 8h .. 8h + 7 of the unit at u (a pointer to
// its first byte) in a plane of kind k.
__device__ __forceinline__ void decode_chunks(const uint8_t* u, int k, int h, int (&c)[8]) {
  const uint32_t* w = reinterpret_cast<const uint32_t*>(u);
  if (k == kPlaneFP4) {
    const uint32_t x = w[h];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint32_t nib = (x >> (4 * t)) & 0xFu;
      c[t] = (nib & 8u) ? -(int)(nib & 7u) : (int)(nib & 7u);
    }
    return;
  }
  uint32_t f[3];
  if (k == kPlaneLo2) {
    lo2_unpack(w[0], w[1], f[0], f[1], f[2]);
  } else {
    f[0] = w[0];
    f[1] = w[1];
    f[2] = w[2];
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const uint32_t code = fp6_field(f, 8 * h + t);
    c[t] = k == kPlaneLo2 ? e2m3_eighth_decode(code) : e2m3_half_decode(code);
  }
}

// Signed magnitudes of values 8h .. 8h + 7 of packed group idx: per plane the
// 24 bits of those values' 3-bit fields, chunk c of the magnitude weighted
// 4^(ceil(m/2) - 1 - c), the sign from any nonzero chunk.
__device__ __forceinline__ void decode_packed(const Opnd& o, int64_t idx, int h, int (&q)[8]) {
  const int64_t plane_bytes = (int64_t)o.rows * o.units * 6;
  int mag[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  uint32_t neg = 0;
  for (int c = 0; c < (o.m + 1) / 2; ++c) {
    const uint8_t* u = o.p0 + c * plane_bytes + idx * 6 + 3 * h;
    const uint32_t w = (uint32_t)u[0] | ((uint32_t)u[1] << 8) | ((uint32_t)u[2] << 16);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint32_t f = (w >> (3 * t)) & 7u;
      mag[t] = 4 * mag[t] + (int)(f & 3u);
      neg |= ((f >> 2) & 1u) << t;
    }
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) q[t] = ((neg >> t) & 1u) ? -mag[t] : mag[t];
}

// Signed magnitudes of values 8h .. 8h + 7 of 16-value unit `unit` of row
// `row`, truncated from m to m_use bits (zero past the last row).
__device__ __forceinline__ void decode_q8(const Opnd& o, int row, int64_t unit, int h, int (&q)[8]) {
#pragma unroll
  for (int t = 0; t < 8; ++t) q[t] = 0;
  if (row >= o.rows) return;
  const int64_t idx = (int64_t)row * o.units + unit;
  if (o.packed) {
    decode_packed(o, idx, h, q);
  } else {
    decode_chunks(o.p0 + idx * unit_bytes(o.m, 0), plane_kind(o.m, 0), h, q);
  }
  if (!o.packed && o.m > 4) {
    int lo[8];
    decode_chunks(o.p1 + idx * unit_bytes(o.m, 1), plane_kind(o.m, 1), h, lo);
    const int w = low_chunk_bits(o.m);
#pragma unroll
    for (int t = 0; t < 8; ++t) q[t] = q[t] * (1 << w) + lo[t];  // both chunks carry the value's sign
  }
  const int s = o.m - o.m_use;
#pragma unroll
  for (int t = 0; t < 8; ++t) q[t] = q[t] < 0 ? -((-q[t]) >> s) : (q[t] >> s);
}

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

// The shared exponent of group G of row `row`.
__device__ __forceinline__ int opnd_exponent(const Opnd& o, int row, int64_t G) {
  const int64_t gid = (int64_t)row * o.ngr + G;
  if (!o.packed) return (int)o.exps[gid];
  const uint32_t* w = reinterpret_cast<const uint32_t*>(o.exps);
  return (int)(packed_base(w[0]) + packed_exponent_offset(w, gid));
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

Opnd make_opnd(const uint8_t* mant, const uint8_t* exps, int64_t rows, int64_t K, int g, int m, int m_use,
               bool packed) {
  const int64_t units = K / 16;
  const int64_t p0_bytes = rows * units * (plane_kind(m, 0) == kPlaneFP6 ? 12 : 8);
  return Opnd{mant, packed ? nullptr : mant + p0_bytes, exps, units, K / g, (int)rows, m, m_use, packed};
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
