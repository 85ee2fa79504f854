// bfp_quant.h -- the FP32 -> BFP group converter (section III-A steps
// (a)-(d); the converter of section V-C), shared by the quantize kernels and
// the GEMM epilogue that converts its output.
#pragma once
#include "bfp_device.h"
#include "launch.h"

namespace fastbfp {

// Signed chunk value as the float the FP6 converter takes: +-c * 0.5 (the
// E2M3 code of c/2), with a zero magnitude as +0.0 so that it packs as code 0.
// neg_half is -0.5 or +0.5 carrying the sign of the input value.
__device__ __forceinline__ float signed_half(uint32_t c, float neg_half) {
  return __builtin_fmaf((float)c, neg_half, 0.0f);  // 0 * -0.5 + 0 = +0
}

// Cache policy of the streaming accesses of the conversion kernels (every
// input element is read once and every output byte written once): nt, so the
// lines do not displace others in L2.  Measured on the row quantizer: 72-78%
// of HBM peak against 64-71% with the default policy.  Only for loads, and for
// stores whose wave writes whole contiguous lines: stores of scattered groups
// (the two-grouping conversion's 12-byte groups) rely on L2 to merge partial
// lines from neighbouring workgroups, and as nt stores ran 2-3x slower.
constexpr int kStreamPolicy = 2;
template <class T>
__device__ __forceinline__ void stream_store(T* p, T v) {
  __builtin_nontemporal_store(v, p);
}
template <class T>
__device__ __forceinline__ T stream_load(const T* p) {
  return __builtin_nontemporal_load(p);
}

typedef float v16f_t __attribute__((ext_vector_type(16)));
typedef uint32_t v6u_t __attribute__((ext_vector_type(6)));

// The gfx950 FP6 converter (32 FP32 values -> 32 packed E2M3 codes, scale
// 1), issued with an early-clobber result: its destination must not overlap
// its sources, which the compiler otherwise allows -- a destination placed a
// few registers into a source gave wrong codes (it overwrote inputs before
// they were read).
__device__ __forceinline__ v6u_t cvt_fp6_x32(v16f_t a, v16f_t b) {
  v6u_t r;
  asm("v_cvt_scalef32_2xpk16_fp6_f32 %0, %1, %2, 1.0" : "=&v"(r) : "v"(a), "v"(b));
  return r;
}

// Step (a): the shared exponent of a group of G values (their FP32 bit
// patterns at b[0..G)): the largest biased exponent field.
template <int G>
__device__ __forceinline__ uint32_t group_exponent(const uint32_t* b) {
  uint32_t E = 0;
#pragma unroll
  for (int t = 0; t < G; ++t) E = max(E, (b[t] >> 23) & 0xFFu);
  return E;
}

// The stochastic-rounding noise of group gid: byte t of noise[0..G/4) is
// value t's noise byte.  One Philox4x32-10 block per 16 values, with counter
// (gid lo, gid hi, t div 16, 0) and key (key0, key1) (a group of 4 or 8 uses
// the first G/4 words of its block).
template <int G>
__device__ __forceinline__ void group_noise(uint64_t gid, uint32_t key0, uint32_t key1, uint32_t* noise) {
#pragma unroll
  for (int blk = 0; blk < (G + 15) / 16; ++blk) {
    const uint4 r = philox4x32_10(make_uint4((uint32_t)gid, (uint32_t)(gid >> 32), (uint32_t)blk, 0u), key0, key1);
    noise[4 * blk] = r.x;
    if constexpr (G >= 8) noise[4 * blk + 1] = r.y;
    if constexpr (G >= 16) {
      noise[4 * blk + 2] = r.z;
      noise[4 * blk + 3] = r.w;
    }
  }
}

// Steps (b)-(d) for one value of bit pattern `bits`: its magnitude q in units
// of the group's LSB, rounded as MODE says and saturated at qmax.  `align` is
// 127 + (m - 1) - E, plus 1 for nearest and 8 for stochastic rounding (the
// ldexp then scales |x| to 2, 1 or 256 times its magnitude in LSBs, exactly);
// the noise byte is byte t mod 4 of noise word `nw` (t: the value's position).
// Subnormals read as zero: by the FP32 flush mode of the including file
// (FTZ), or explicitly.
template <int MODE, bool FTZ>
__device__ __forceinline__ uint32_t value_magnitude(uint32_t bits, int align, uint32_t nw, int t, uint32_t qmax) {
  const uint32_t abits = (FTZ || ((bits >> 23) & 0xFFu)) ? (bits & 0x7FFFFFFFu) : 0u;
  const float mag = __builtin_ldexpf(__uint_as_float(abits), align);
  const uint32_t fl = (uint32_t)mag;  // truncating conversion: floor
  uint32_t q;
  if (MODE == kNearest) {
    q = (fl + 1u) >> 1;  // half an LSB added
  } else if (MODE == kTruncate) {
    q = fl;
  } else {
    // (c) add the noise byte below the LSB, (d) truncate.
    q = (fl + ((nw >> (8 * (t & 3))) & 0xFFu)) >> 8;
  }
  return min(q, qmax);  // a group maximum that rounds up to 2^m saturates
}
// The align argument of value_magnitude.
template <int MODE>
__device__ __forceinline__ int magnitude_align(uint32_t m, uint32_t E) {
  return 127 + (int)m - 1 - (int)E + (MODE == kNearest ? 1 : MODE == kStochastic ? 8 : 0);
}

// Quantize NG consecutive groups (gid, gid + 1, ...) whose FP32 bit patterns
// are in b[], packed together as one run of NG * G values.  Writes the packed
// chunk planes to w[plane][...] and the shared exponents to E_out; nonfinite
// is set if any input was Inf/NaN.  Two 16-value groups fill the 32 inputs of
// the FP6 converter exactly, and their codes are the two groups' codes side by
// side, as stored.
//
// Alignment is done in floating point, exactly: with the shared exponent E,
// one LSB is 2^(E-127-(m-1)), so a = |x| / LSB = ldexp(|x|, 127 + (m-1) - E)
// is a power-of-two scaling of an FP32 value into [0, 2^m) and has no
// rounding.  Truncating conversions to integer then implement the three
// rounding rules exactly:
//   truncate:   q = floor(a)
//   nearest:    q = (floor(2a) + 1) >> 1           (half an LSB added, ties up)
//   stochastic: q = (floor(256a) + U) >> 8         (U = the noise byte)
// Subnormal inputs are read as zero: explicitly, or (FTZ true, only for
// files built with FP32 denormals flushed) by the ldexp's own input flush.
//
// Plane formats P0 / P1 (launch.h): kPlaneFP4 (chunks of at most 2 bits: the
// code is the sign bit above the chunk itself, 4 bits per value, G/8 words);
// kPlaneFP6 (3G/16 words) and kPlaneLo2 (G/8 words: the FP6 codes of
// +-chunk/8, squeezed by lo2_pack), whose codes come from the gfx950 FP6
// converter.  That converter interleaves its two 16-value inputs: output
// value 2i is a[i] / scale and 2i+1 is b[i] / scale.  Two chunk planes split
// q at 2 bits when plane 1 is a Lo2 plane (q >> 2, q & 3: m = 5, 6) and at 4
// otherwise (q >> 4, q & 15: m = 7, 8).
//
// ADAPT (m = 4 only; section V-D and Eq. 2): plane 0 gets the 4-bit magnitude
// q as one code, plane 1 (if NCH = 2) the 2-bit mantissa left when the low
// chunk is discarded, q >> 2; s_lo and s_hi return the group's sums of q & 3
// and q >> 2 (the magnitudes BFP(X,4) - BFP(X,2) and BFP(X,2) in units of
// 2^(E-130) and 2^(E-128)).
template <int G, int NG, int MODE, int NCH, bool ADAPT, int P0, int P1, bool FTZ>
__device__ __forceinline__ void quantize_groups(const uint32_t (&b)[NG * G], uint32_t m, uint64_t gid, uint32_t key0,
                                                uint32_t key1, uint32_t (&w)[NCH][NG * G * 6 / 32],
                                                uint32_t (&E_out)[NG], bool& nonfinite, uint32_t (&s_lo)[NG],
                                                uint32_t (&s_hi)[NG]) {
  static_assert(NG == 1 || NG * G == 16 || NG * G == 32, "several groups per call: one or two 16-value units");
  constexpr int PK[2] = {P0, P1};
  constexpr int LEN = NG * G;  // values converted together (one packing unit)
#pragma unroll
  for (int gi = 0; gi < NG; ++gi) {
    s_lo[gi] = 0u;
    s_hi[gi] = 0u;
  }
  nonfinite = false;
  // (a) shared exponent of each group: the largest biased exponent field.
  uint32_t E[NG];
#pragma unroll
  for (int gi = 0; gi < NG; ++gi) {
    E[gi] = group_exponent<G>(b + gi * G);
    E_out[gi] = E[gi];
    nonfinite |= (E[gi] == 255u);
  }

  uint32_t noise[LEN / 4];
  if (MODE == kStochastic) {
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) group_noise<G>(gid + (uint64_t)gi, key0, key1, noise + gi * G / 4);
  }

  const uint32_t qmax = (1u << m) - 1u;
  // (b) the exponent that aligns a value to its group's LSB (times 2 for
  // nearest, 256 for stochastic rounding).
  int align[NG];
#pragma unroll
  for (int gi = 0; gi < NG; ++gi) align[gi] = magnitude_align<MODE>(m, E[gi]);
  typedef float v16f __attribute__((ext_vector_type(16)));
  constexpr int NH = LEN / 32 + (LEN % 32 != 0);
  v16f ev[NCH][NH], od[NCH][NH];
#pragma unroll
  for (int p = 0; p < NCH; ++p) {
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      ev[p][h] = v16f{};
      od[p][h] = v16f{};
    }
#pragma unroll
    for (int i = 0; i < LEN * 6 / 32; ++i) w[p][i] = 0u;
  }
#pragma unroll
  for (int t = 0; t < LEN; ++t) {
    const uint32_t q = value_magnitude<MODE, FTZ>(b[t], align[t / G], MODE == kStochastic ? noise[t >> 2] : 0u, t,
                                                  qmax);
    if (ADAPT) {
      s_lo[t / G] += q & 3u;
      s_hi[t / G] += q >> 2;
    }
    // the chunk of each plane
    uint32_t c[2];
    if (ADAPT) {
      c[0] = q;
      c[1] = q >> 2;
    } else if (NCH == 1) {
      c[0] = q;
      c[1] = 0u;
    } else if (P1 == kPlaneLo2) {
      c[0] = q >> 2;
      c[1] = q & 3u;
    } else {
      c[0] = q >> 4;
      c[1] = q & 15u;
    }
    const float nh = __uint_as_float((b[t] & 0x80000000u) | 0x3F000000u);  // +-0.5
    const uint32_t sgn = (b[t] >> 28) & 8u;                                  // the FP4 sign bit
    const int h = t / 32, k = (t % 32) / 2;
#pragma unroll
    for (int p = 0; p < NCH; ++p) {
      if (PK[p] == kPlaneFP4) {
        w[p][t >> 3] |= (c[p] ? (sgn | c[p]) : 0u) << (4 * (t & 7));
      } else {
        // +-c/2, or +-c/8 for a Lo2 plane (exact either way; zero as +0)
        const float f = signed_half(c[p], PK[p] == kPlaneLo2 ? 0.25f * nh : nh);
        if (t % 2 == 0) ev[p][h][k] = f; else od[p][h][k] = f;
      }
    }
  }
  typedef uint32_t v6u __attribute__((ext_vector_type(6)));
#pragma unroll
  for (int p = 0; p < NCH; ++p) {
    if (PK[p] == kPlaneFP4) continue;
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const v6u cv = cvt_fp6_x32(ev[p][h], od[p][h]);
#pragma unroll
      for (int i = 0; i < 6 && 6 * h + i < LEN * 6 / 32; ++i) w[p][6 * h + i] = cv[i];
    }
    if (PK[p] == kPlaneLo2) {
      // squeeze each 16 values' three code dwords into two (in order: the
      // dwords written never come after those still to be read)
#pragma unroll
      for (int u = 0; u < LEN / 16; ++u) {
        const uint2 d = lo2_pack(w[p][3 * u], w[p][3 * u + 1], w[p][3 * u + 2]);
        w[p][2 * u] = d.x;
        w[p][2 * u + 1] = d.y;
      }
    }
  }
}


// One group (the common case).
template <int G, int MODE, int NCH, bool ADAPT, int P0, int P1, bool FTZ = false>
__device__ __forceinline__ void quantize_group(const uint32_t (&b)[G], uint32_t m, uint64_t gid, uint32_t key0,
                                               uint32_t key1, uint32_t (&w)[NCH][G * 6 / 32], uint32_t& E_out,
                                               bool& nonfinite, uint32_t& s_lo, uint32_t& s_hi) {
  uint32_t E[1], lo[1], hi[1];
  quantize_groups<G, 1, MODE, NCH, ADAPT, P0, P1, FTZ>(b, m, gid, key0, key1, w, E, nonfinite, lo, hi);
  E_out = E[0];
  s_lo = lo[0];
  s_hi = hi[0];
}

// Stores plane p's codes of group gid (from quantize_group) at
// mant_p + gid * bytes-per-group: 8 (FOUR: an FP4 or Lo2 plane) or 12 bytes
// per 16 values.
template <class T, bool STREAM>
__device__ __forceinline__ void put(T* p, T v) {
  if constexpr (STREAM) stream_store(p, v);
  else *p = v;
}
// STREAM: nt stores (for a wave that writes whole contiguous lines).
template <int G, bool FOUR, bool STREAM = false>
__device__ __forceinline__ void store_plane(uint8_t* __restrict__ mant, int64_t gid, const uint32_t* w) {
  typedef uint32_t u2 __attribute__((ext_vector_type(2)));
  typedef uint32_t u3 __attribute__((ext_vector_type(3)));
  if (FOUR) {
    u2* dst = reinterpret_cast<u2*>(mant + gid * (G / 2));
#pragma unroll
    for (int i = 0; i < G / 16; ++i) put<u2, STREAM>(dst + i, u2{w[2 * i], w[2 * i + 1]});
  } else {
    uint8_t* dst = mant + gid * (G * 3 / 4);
#pragma unroll
    for (int i = 0; i < G / 16; ++i)
      put<u3, STREAM>(reinterpret_cast<u3*>(dst + 12 * i), u3{w[3 * i], w[3 * i + 1], w[3 * i + 2]});
  }
}

}  // namespace fastbfp
