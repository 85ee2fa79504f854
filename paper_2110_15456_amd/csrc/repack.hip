// repack.hip -- re-encodes a stored BFP tensor into the chunk-plane layout that
// the block-scaled GEMM kernel (gemm_mx.h) reads, so that the products it does
// not take directly still run on it (bfp_gemm_ws):
//   * a precision below the stored width: each magnitude truncated to its top
//     m_use bits (the discard of low-order bits, section V-D) and stored as an
//     m_use-bit tensor, with the same exponents;
//   * groups of 4 or 8: each group becomes one 16-value unit holding its g
//     values and 16 - g zeros, with the group's exponent (the other operand
//     gets the same padding, so the zeros meet zeros and every product is the
//     group's own);
//   * groups of 64: two groups of 32 that share the group's exponent (the
//     sum of their exact products is the 64-value group's);
//   * the packed storage of section V-D: unpacked, each group at its stored
//     exponent E = base + e.
// The values stay exactly what the stored tensor stands for at m_use bits, so
// a GEMM on the repacked operands computes the same per-group terms T_G.
#include "bfp_decode.h"

namespace fastbfp {

namespace {

typedef uint32_t u2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u3_t __attribute__((ext_vector_type(3)));

// OR a 6-bit code into position t of 16 little-endian packed FP6 codes.
__device__ __forceinline__ void put6(uint32_t (&w)[3], int t, uint32_t code) {
  const int bit = 6 * t, wi = bit >> 5, sh = bit & 31;
  w[wi] |= code << sh;
  if (sh > 26) w[wi + 1] |= code >> (32 - sh);
}

// One thread per output 16-value unit: unit u of row r, idx = r * units_out + u.
// G: the source group size.
template <int G>
__global__ __launch_bounds__(256) void k_repack(Opnd src, int64_t units_out, int64_t total, int m_out,
                                                uint8_t* __restrict__ p0, uint8_t* __restrict__ p1,
                                                uint8_t* __restrict__ exps_out) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= total) return;
  const int row = (int)(idx / units_out);
  const int64_t u = idx % units_out;
  // source unit, source group, and (G < 16) the group's first value in its unit
  const int64_t src_unit = G < 16 ? (u * G) / 16 : u;
  const int64_t grp = G < 16 ? u : (u * 16) / G;
  const int first = G < 16 ? (int)((u * G) % 16) : 0;
  int a[8], b[8], s[16];
  decode_q8(src, row, src_unit, 0, a);
  decode_q8(src, row, src_unit, 1, b);
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    s[t] = a[t];
    s[8 + t] = b[t];
  }
  int q[16];
  if constexpr (G < 16) {
#pragma unroll
    for (int t = 0; t < 16; ++t) q[t] = 0;
#pragma unroll
    for (int k = 0; k < 16; k += G)
      if (first == k) {
#pragma unroll
        for (int t = 0; t < G; ++t) q[t] = s[k + t];
      }
  } else {
#pragma unroll
    for (int t = 0; t < 16; ++t) q[t] = s[t];
  }
  // planes of the m_out-bit tensor (launch.h): FP4 for m <= 2, FP6 for m <= 4,
  // FP6 of q >> 2 and Lo2 of q & 3 for m = 5, 6, FP6 of q >> 4 and q & 15 for m = 7, 8
  const int lo_bits = m_out <= 4 ? 0 : low_chunk_bits(m_out);
  uint32_t w0[3] = {0u, 0u, 0u}, w1[3] = {0u, 0u, 0u};
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    const uint32_t mag = (uint32_t)(q[t] < 0 ? -q[t] : q[t]), neg = q[t] < 0 ? 1u : 0u;
    const uint32_t hi = mag >> lo_bits, lo = mag & ((1u << lo_bits) - 1u);
    if (m_out <= 2) {
      w0[t >> 3] |= (hi ? (neg << 3) | hi : 0u) << (4 * (t & 7));
    } else {
      put6(w0, t, hi ? (neg << 5) | e2m3_half_code(hi) : 0u);
      if (m_out > 6) put6(w1, t, lo ? (neg << 5) | e2m3_half_code(lo) : 0u);
      else if (m_out > 4) put6(w1, t, lo ? (neg << 5) | lo : 0u);  // FP6 code of +-lo/8 (subnormal)
    }
  }
  if (m_out <= 2) {
    *reinterpret_cast<u2_t*>(p0 + idx * 8) = u2_t{w0[0], w0[1]};
  } else {
    *reinterpret_cast<u3_t*>(p0 + idx * 12) = u3_t{w0[0], w0[1], w0[2]};
    if (m_out > 6) {
      *reinterpret_cast<u3_t*>(p1 + idx * 12) = u3_t{w1[0], w1[1], w1[2]};
    } else if (m_out > 4) {
      const uint2 d = lo2_pack(w1[0], w1[1], w1[2]);
      *reinterpret_cast<u2_t*>(p1 + idx * 8) = u2_t{d.x, d.y};
    }
  }
  // exponents: one per output group of 16, or of 32 (source groups of 32 and 64)
  const int e = opnd_exponent(src, row, grp);
  if (G <= 16)
    exps_out[idx] = (uint8_t)e;
  else if ((u & 1) == 0)
    exps_out[idx / 2] = (uint8_t)e;
}

}  // namespace

void repack_shape(int64_t len, int g, int64_t* len_out, int* g_out) {
  *len_out = g < 16 ? len * (16 / g) : len;
  *g_out = g <= 16 ? 16 : 32;
}

hipError_t launch_repack(const uint8_t* mant, const uint8_t* exps, int64_t rows, int64_t len, int g, int m, int m_use,
                         bool packed, uint8_t* out_mant, uint8_t* out_exps, hipStream_t s) {
  int64_t len_out;
  int g_out;
  repack_shape(len, g, &len_out, &g_out);
  const int64_t units_out = len_out / 16, total = rows * units_out;
  if (total == 0) return hipSuccess;
  const Opnd src = make_opnd(mant, exps, rows, len, g, m, m_use, packed);
  uint8_t* p1 = out_mant + total * (plane_kind(m_use, 0) == kPlaneFP6 ? 12 : 8);
  const dim3 grid((unsigned)((total + 255) / 256));
  switch (g) {
    case 4: hipLaunchKernelGGL(k_repack<4>, grid, dim3(256), 0, s, src, units_out, total, m_use, out_mant, p1, out_exps);
      break;
    case 8: hipLaunchKernelGGL(k_repack<8>, grid, dim3(256), 0, s, src, units_out, total, m_use, out_mant, p1, out_exps);
      break;
    case 16: hipLaunchKernelGGL(k_repack<16>, grid, dim3(256), 0, s, src, units_out, total, m_use, out_mant, p1,
                                out_exps);
      break;
    case 32: hipLaunchKernelGGL(k_repack<32>, grid, dim3(256), 0, s, src, units_out, total, m_use, out_mant, p1,
                                out_exps);
      break;
    default: hipLaunchKernelGGL(k_repack<64>, grid, dim3(256), 0, s, src, units_out, total, m_use, out_mant, p1,
                                out_exps);
      break;
  }
  return hipGetLastError();
}

}  // namespace fastbfp
