// bfp_decode.h -- decoding a stored BFP operand back to signed integer
// magnitudes, for the kernels that do not read it as MFMA codes directly:
// the general GEMM kernel and the repack pass.  Handles the chunk-plane layout
// of include/fastbfp.h (any group size, planes in 16-value units) and the
// packed storage of section V-D, and truncates each magnitude from its stored
// m bits to its top m_use bits (the discard of low-order bits, section V-D).
#pragma once
#include "bfp_device.h"
#include "launch.h"

namespace fastbfp {

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

// The shared exponent of group G of row `row`.
__device__ __forceinline__ int opnd_exponent(const Opnd& o, int row, int64_t G) {
  const int64_t gid = (int64_t)row * o.ngr + G;
  if (!o.packed) return (int)o.exps[gid];
  const uint32_t* w = reinterpret_cast<const uint32_t*>(o.exps);
  return (int)(packed_base(w[0]) + packed_exponent_offset(w, gid));
}

// The decoder's view of a stored rows x K operand (host side).
inline Opnd make_opnd(const uint8_t* mant, const uint8_t* exps, int64_t rows, int64_t K, int g, int m, int m_use,
               bool packed) {
  const int64_t units = K / 16;
  const int64_t p0_bytes = rows * units * (plane_kind(m, 0) == kPlaneFP6 ? 12 : 8);
  return Opnd{mant, packed ? nullptr : mant + p0_bytes, exps, units, K / g, (int)rows, m, m_use, packed};
}

}  // namespace fastbfp
