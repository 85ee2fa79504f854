// quantize.hip -- FP32 -> BFP conversion on gfx950 (section III-A steps
// (a)-(d); the converter of section V-C), plus the inverse (dequantize).
//
// One lane owns one group of G values end to end: it loads the group, finds
// the shared exponent with an in-register max (the comparator tree), aligns
// each significand with one clamped shift (the barrel shifter), adds the
// rounding term (half an LSB, nothing, or an 8-bit Philox noise byte), keeps
// the carry, saturates, and writes the magnitudes as packed FP6 E2M3 chunk
// codes (3G/4 bytes per chunk plane) plus one exponent byte.  Owning a whole
// group per lane makes one Philox call serve 16 values, which keeps stochastic
// rounding within the HBM-bound budget.
#include "bfp_device.h"
#include "launch.h"

namespace fastbfp {

// Quantize one group whose FP32 bit patterns are in b[].  Writes the packed
// chunk planes to w[plane][...] and the shared exponent to E_out; nonfinite is
// set if any input was Inf/NaN.
template <int G, int MODE, int NCH>
__device__ __forceinline__ void quantize_group(const uint32_t (&b)[G], uint32_t m, uint64_t gid, uint32_t key0,
                                               uint32_t key1, uint32_t (&w)[NCH][G * 6 / 32], uint32_t& E_out,
                                               bool& nonfinite) {
  // (a) shared exponent: the largest biased exponent field in the group.
  uint32_t E = 0;
#pragma unroll
  for (int t = 0; t < G; ++t) E = max(E, (b[t] >> 23) & 0xFFu);
  E_out = E;
  nonfinite = (E == 255u);

  uint32_t noise[G / 4];
  if (MODE == kStochastic) {
#pragma unroll
    for (int blk = 0; blk < G / 16; ++blk) {
      const uint4 r = philox4x32_10(make_uint4((uint32_t)gid, (uint32_t)(gid >> 32), (uint32_t)blk, 0u), key0, key1);
      noise[4 * blk + 0] = r.x;
      noise[4 * blk + 1] = r.y;
      noise[4 * blk + 2] = r.z;
      noise[4 * blk + 3] = r.w;
    }
  }

#pragma unroll
  for (int p = 0; p < NCH; ++p)
#pragma unroll
    for (int i = 0; i < G * 6 / 32; ++i) w[p][i] = 0u;

  const uint32_t qmax = (1u << m) - 1u;
  // The value's 24-bit significand S is worth S * 2^(ef-150); one LSB of the
  // group is 2^(E-127-(m-1)); so the magnitude in LSBs is S >> sh with
  // sh = E - ef + 24 - m (>= 16 because m <= 8).
  const uint32_t base = E + 24u - m;
#pragma unroll
  for (int t = 0; t < G; ++t) {
    const uint32_t ef = (b[t] >> 23) & 0xFFu;
    const uint32_t S = ef ? ((b[t] & 0x7FFFFFu) | 0x800000u) : 0u;  // subnormals flush to zero
    const uint32_t sh = base - ef;
    uint32_t q;
    if (MODE == kNearest) {
      // (c)+(d): add half an LSB, truncate.
      q = ((S >> min(sh - 1u, 31u)) + 1u) >> 1;
    } else if (MODE == kTruncate) {
      q = S >> min(sh, 31u);
    } else {
      // (b) keep 8 bits below the LSB, (c) add the noise byte, (d) truncate.
      const uint32_t u = (noise[t >> 2] >> (8 * (t & 3))) & 0xFFu;
      q = ((S >> min(sh - 8u, 31u)) + u) >> 8;
    }
    q = min(q, qmax);  // a group maximum that rounds up to 2^m saturates
    const uint32_t sbit = (b[t] >> 26) & 0x20u;
    uint32_t code[NCH];
    if (NCH == 1) {
      code[0] = e2m3_half_code(q) | (q ? sbit : 0u);
    } else {
      const uint32_t hi = q >> 4, lo = q & 15u;
      code[0] = e2m3_half_code(hi) | (hi ? sbit : 0u);
      code[NCH - 1] = e2m3_half_code(lo) | (lo ? sbit : 0u);
    }
    const int bit = 6 * t, wi = bit / 32, bs = bit % 32;
#pragma unroll
    for (int p = 0; p < NCH; ++p) {
      w[p][wi] |= code[p] << bs;
      if (bs > 26) w[p][wi + 1] |= code[p] >> (32 - bs);
    }
  }
}

template <int G, int NCH>
__device__ __forceinline__ void store_group(uint8_t* __restrict__ mant, int64_t plane_bytes, int64_t gid,
                                            const uint32_t (&w)[NCH][G * 6 / 32]) {
#pragma unroll
  for (int p = 0; p < NCH; ++p) {
    uint3* dst = reinterpret_cast<uint3*>(mant + p * plane_bytes + gid * (G * 3 / 4));
#pragma unroll
    for (int i = 0; i < G / 16; ++i) dst[i] = make_uint3(w[p][3 * i], w[p][3 * i + 1], w[p][3 * i + 2]);
  }
}

// Groups along the contiguous last axis: group gid covers x[gid*G, gid*G+G).
template <int G, int MODE, int NCH>
__global__ __launch_bounds__(256) void k_quantize_rows(const float* __restrict__ x, int64_t ngroups, uint32_t m,
                                                       uint32_t key0, uint32_t key1, uint8_t* __restrict__ mant,
                                                       uint8_t* __restrict__ exps, uint32_t* status) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= ngroups) return;
  uint32_t b[G];
  const u32x4* src = reinterpret_cast<const u32x4*>(x) + gid * (G / 4);
#pragma unroll
  for (int i = 0; i < G / 4; ++i) {
    const u32x4 v = __builtin_nontemporal_load(src + i);  // read once: bypass cache retention
    b[4 * i + 0] = v[0];
    b[4 * i + 1] = v[1];
    b[4 * i + 2] = v[2];
    b[4 * i + 3] = v[3];
  }
  uint32_t w[NCH][G * 6 / 32];
  uint32_t E;
  bool nonfinite;
  quantize_group<G, MODE, NCH>(b, m, (uint64_t)gid, key0, key1, w, E, nonfinite);
  exps[gid] = (uint8_t)E;
  store_group<G, NCH>(mant, ngroups * (G * 3 / 4), gid, w);
  if (status && nonfinite) atomicOr(status, 1u);
}

// Groups down the columns of x[R][C] (transpose-on-quantize).  Output row c is
// column c of x; its group j covers x[j*G .. j*G+G-1][c] and has
// gid = c * (R/G) + j.  A block is 64 columns x 4 group slots; each thread
// walks NGT consecutive groups of its column, so its output bytes are
// contiguous and a wave's loads are 256 contiguous bytes.
template <int G, int MODE, int NCH, int NGT>
__global__ __launch_bounds__(256) void k_quantize_cols(const float* __restrict__ x, int64_t R, int64_t C,
                                                       int64_t nbx, uint32_t m, uint32_t key0, uint32_t key1,
                                                       uint8_t* __restrict__ mant, uint8_t* __restrict__ exps,
                                                       uint32_t* status) {
  const int64_t bx = blockIdx.x % nbx, by = blockIdx.x / nbx;
  const int64_t c = bx * 64 + (threadIdx.x & 63);
  if (c >= C) return;
  const int64_t gpr = R / G;
  const int64_t ngroups = C * gpr;
  const int64_t j0 = (by * 4 + (threadIdx.x >> 6)) * NGT;
  bool any_bad = false;
  for (int i = 0; i < NGT; ++i) {
    const int64_t j = j0 + i;
    if (j >= gpr) break;
    uint32_t b[G];
    const float* src = x + (j * G) * C + c;
#pragma unroll
    for (int t = 0; t < G; ++t) b[t] = __float_as_uint(__builtin_nontemporal_load(src + t * C));
    uint32_t w[NCH][G * 6 / 32];
    uint32_t E;
    bool nonfinite;
    const int64_t gid = c * gpr + j;
    quantize_group<G, MODE, NCH>(b, m, (uint64_t)gid, key0, key1, w, E, nonfinite);
    exps[gid] = (uint8_t)E;
    store_group<G, NCH>(mant, ngroups * (G * 3 / 4), gid, w);
    any_bad |= nonfinite;
  }
  if (status && any_bad) atomicOr(status, 1u);
}

// BFP -> FP32: y = +-q * 2^(E-127-(m-1)).  One lane per group.
template <int G, int NCH>
__global__ __launch_bounds__(256) void k_dequantize(const uint8_t* __restrict__ mant, const uint8_t* __restrict__ exps,
                                                    int64_t ngroups, int m, float* __restrict__ y) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= ngroups) return;
  uint32_t w[NCH][G * 6 / 32];
#pragma unroll
  for (int p = 0; p < NCH; ++p) {
    const uint3* src = reinterpret_cast<const uint3*>(mant + p * ngroups * (G * 3 / 4) + gid * (G * 3 / 4));
#pragma unroll
    for (int i = 0; i < G / 16; ++i) {
      const uint3 v = src[i];
      w[p][3 * i] = v.x;
      w[p][3 * i + 1] = v.y;
      w[p][3 * i + 2] = v.z;
    }
  }
  const int e = (int)exps[gid] - 127 - (m - 1);
  float4* dst = reinterpret_cast<float4*>(y + gid * G);
#pragma unroll
  for (int i = 0; i < G / 4; ++i) {
    float v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int t = 4 * i + k;
      int q = e2m3_half_decode(fp6_field(w[0], t));
      if (NCH == 2) {
        const int lo = e2m3_half_decode(fp6_field(w[NCH - 1], t));
        q = q * 16 + lo;  // both chunks carry the value's sign
      }
      v[k] = ldexpf((float)q, e);
    }
    dst[i] = make_float4(v[0], v[1], v[2], v[3]);
  }
}

template <int G, int MODE, int NCH>
static hipError_t launch_rows_t(const float* x, int64_t ngroups, int m, uint64_t seed, uint8_t* mant, uint8_t* exps,
                                uint32_t* status, hipStream_t s) {
  const int64_t blocks = (ngroups + 255) / 256;
  hipLaunchKernelGGL((k_quantize_rows<G, MODE, NCH>), dim3((unsigned)blocks), dim3(256), 0, s, x, ngroups,
                     (uint32_t)m, (uint32_t)seed, (uint32_t)(seed >> 32), mant, exps, status);
  return hipGetLastError();
}

template <int G, int MODE, int NCH>
static hipError_t launch_cols_t(const float* x, int64_t R, int64_t C, int m, uint64_t seed, uint8_t* mant,
                                uint8_t* exps, uint32_t* status, hipStream_t s) {
  constexpr int NGT = 8;
  const int64_t gpr = R / G;
  const int64_t nbx = (C + 63) / 64, nby = (gpr + 4 * NGT - 1) / (4 * NGT);
  hipLaunchKernelGGL((k_quantize_cols<G, MODE, NCH, NGT>), dim3((unsigned)(nbx * nby)), dim3(256), 0, s, x, R, C, nbx,
                     (uint32_t)m, (uint32_t)seed, (uint32_t)(seed >> 32), mant, exps, status);
  return hipGetLastError();
}

#define FASTBFP_DISPATCH_QUANT(FN, ...)                                  \
  do {                                                                   \
    const bool two = m > 4;                                              \
    if (g == 16) {                                                       \
      if (mode == kNearest) return two ? FN<16, kNearest, 2>(__VA_ARGS__) : FN<16, kNearest, 1>(__VA_ARGS__); \
      if (mode == kStochastic) return two ? FN<16, kStochastic, 2>(__VA_ARGS__) : FN<16, kStochastic, 1>(__VA_ARGS__); \
      return two ? FN<16, kTruncate, 2>(__VA_ARGS__) : FN<16, kTruncate, 1>(__VA_ARGS__); \
    } else {                                                             \
      if (mode == kNearest) return two ? FN<32, kNearest, 2>(__VA_ARGS__) : FN<32, kNearest, 1>(__VA_ARGS__); \
      if (mode == kStochastic) return two ? FN<32, kStochastic, 2>(__VA_ARGS__) : FN<32, kStochastic, 1>(__VA_ARGS__); \
      return two ? FN<32, kTruncate, 2>(__VA_ARGS__) : FN<32, kTruncate, 1>(__VA_ARGS__); \
    }                                                                    \
  } while (0)

hipError_t launch_quantize_rows(const float* x, int64_t rows, int64_t len, int g, int m, int mode, uint64_t seed,
                                uint8_t* mant, uint8_t* exps, uint32_t* status, hipStream_t s) {
  const int64_t ngroups = rows * (len / g);
  if (ngroups == 0) return hipSuccess;
  FASTBFP_DISPATCH_QUANT(launch_rows_t, x, ngroups, m, seed, mant, exps, status, s);
}

hipError_t launch_quantize_cols(const float* x, int64_t R, int64_t C, int g, int m, int mode, uint64_t seed,
                                uint8_t* mant, uint8_t* exps, uint32_t* status, hipStream_t s) {
  if (R == 0 || C == 0) return hipSuccess;
  FASTBFP_DISPATCH_QUANT(launch_cols_t, x, R, C, m, seed, mant, exps, status, s);
}

hipError_t launch_dequantize(const uint8_t* mant, const uint8_t* exps, int64_t rows, int64_t len, int g, int m,
                             float* y, hipStream_t s) {
  const int64_t ngroups = rows * (len / g);
  if (ngroups == 0) return hipSuccess;
  const unsigned blocks = (unsigned)((ngroups + 255) / 256);
  const bool two = m > 4;
  if (g == 16) {
    if (two) hipLaunchKernelGGL((k_dequantize<16, 2>), dim3(blocks), dim3(256), 0, s, mant, exps, ngroups, m, y);
    else hipLaunchKernelGGL((k_dequantize<16, 1>), dim3(blocks), dim3(256), 0, s, mant, exps, ngroups, m, y);
  } else {
    if (two) hipLaunchKernelGGL((k_dequantize<32, 2>), dim3(blocks), dim3(256), 0, s, mant, exps, ngroups, m, y);
    else hipLaunchKernelGGL((k_dequantize<32, 1>), dim3(blocks), dim3(256), 0, s, mant, exps, ngroups, m, y);
  }
  return hipGetLastError();
}

}  // namespace fastbfp
