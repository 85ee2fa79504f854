// bfp_device.h -- device helpers shared by the gfx950 BFP kernels:
// the Philox4x32-10 generator, the FP6 E2M3 chunk codec and small vector types.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fastbfp {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11, section 3): ten rounds of
// two 32x32->64 multiplications with the round key bumped by the Weyl
// increments between rounds.  The key is wave-uniform (the seed), so its
// schedule stays in scalar registers.
__device__ __forceinline__ uint4 philox4x32_10(uint4 ctr, uint32_t key0, uint32_t key1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint64_t prod0 = (uint64_t)0xD2511F53u * ctr.x;
    const uint64_t prod1 = (uint64_t)0xCD9E8D57u * ctr.z;
    ctr = make_uint4((uint32_t)(prod1 >> 32) ^ ctr.y ^ key0, (uint32_t)prod1,
                     (uint32_t)(prod0 >> 32) ^ ctr.w ^ key1, (uint32_t)prod0);
    key0 += 0x9E3779B9u;
    key1 += 0xBB67AE85u;
  }
  return ctr;
}

// FP6 E2M3 code (OCP MX: 1 sign, 2 exponent bits with bias 1, 3 mantissa
// bits) of c/2 for an integer chunk c in [0, 15], without the sign bit.
// Values below 1 are subnormal (code = 8 * value), [1,2) has code 8 * value,
// [2,4) has code 16 + 4 * (value - 2), [4,8) has code 24 + 2 * (value - 4).
// With value = c/2 these three pieces are 4c (c <= 3), 2c + 8 (4 <= c <= 7) and
// c + 16 (c >= 8), i.e. c + min(3c, c + 8, 16).
__device__ __forceinline__ uint32_t e2m3_half_code(uint32_t c) {
  return c + min(min(3u * c, c + 8u), 16u);
}

// Inverse of e2m3_half_code with the sign: returns +-c for a 6-bit code.
__device__ __forceinline__ int e2m3_half_decode(uint32_t code) {
  const uint32_t e = (code >> 3) & 3u, f = code & 7u;
  const uint32_t c = e ? (((8u + f) << e) >> 3) : (f >> 2);
  return (code & 0x20u) ? -(int)c : (int)c;
}

// A Lo2 chunk plane (a 2-bit chunk c with its sign, per value) holds, per 16
// values, the three dwords T0, T1, T2 of their packed FP6 E2M3 codes of
// +-c/8.  Such a code is subnormal: of its 6 bits only the two mantissa bits
// of the value (field bits 0, 1) and the sign (bit 5) can be set.  Across the
// 96 bits, T1's possible bits moved down by one fall exactly on T0's
// always-zero bits, so the 16 codes fit in two dwords:
//   D0 = T0 | (T1 >> 1),  D1 = T2
// and come back with three instructions.  kLo2M0 / kLo2M1 are the bits T0 /
// T1 can have set (T2's are D1 as stored).
constexpr uint32_t kLo2M0 = 0xE38E38E3u, kLo2M1 = 0x38E38E38u;
__device__ __forceinline__ uint2 lo2_pack(uint32_t t0, uint32_t t1, uint32_t t2) {
  return make_uint2(t0 | (t1 >> 1), t2);
}
__device__ __forceinline__ void lo2_unpack(uint32_t d0, uint32_t d1, uint32_t& t0, uint32_t& t1, uint32_t& t2) {
  t0 = d0 & kLo2M0;
  t1 = (d0 << 1) & kLo2M1;
  t2 = d1;
}
// +-c for a 6-bit FP6 E2M3 code of +-c/8 (c <= 7: a subnormal code).
__device__ __forceinline__ int e2m3_eighth_decode(uint32_t code) {
  return (code & 0x20u) ? -(int)(code & 7u) : (int)(code & 7u);
}

// 6-bit field t of a packed little-endian FP6 group held in dwords w[].
__device__ __forceinline__ uint32_t fp6_field(const uint32_t* w, int t) {
  const int bit = 6 * t, wi = bit >> 5, sh = bit & 31;
  uint32_t v = w[wi] >> sh;
  if (sh > 26) v |= w[wi + 1] << (32 - sh);
  return v & 0x3Fu;
}

// Packed exponents (section V-D reading): the tensor base max(E_max - 7, 0)
// from the stream's leading E_max word, and the 3-bit offset of group gid
// (bits 3 gid .. 3 gid + 2 of the dwords after it; a field crosses into the
// next dword only inside a 24-byte block of 64 groups).
__device__ __forceinline__ uint32_t packed_base(uint32_t emax) { return emax > 7u ? emax - 7u : 0u; }
__device__ __forceinline__ uint32_t packed_exponent_offset(const uint32_t* expw, int64_t gid) {
  const int64_t bit = 3 * gid;
  const int sh = (int)(bit % 32);
  uint32_t v = expw[1 + bit / 32] >> sh;
  if (sh > 29) v |= expw[2 + bit / 32] << (32 - sh);
  return v & 7u;
}

}  // namespace fastbfp
