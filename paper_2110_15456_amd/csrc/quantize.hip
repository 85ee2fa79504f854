// quantize.hip -- FP32 -> BFP conversion on gfx950 (section III-A steps
// (a)-(d); the converter of section V-C), plus the inverse (dequantize).
//
// One lane owns one group of G values end to end: it loads the group, finds
// the shared exponent with an in-register max (the comparator tree), aligns
// each significand with one clamped shift (the barrel shifter), adds the
// rounding term (half an LSB, nothing, or an 8-bit Philox noise byte), keeps
// the carry, saturates, and writes the magnitudes as packed chunk codes
// (FP4 E2M1 for chunks of at most 2 bits, G/2 bytes per plane; FP6 E2M3
// otherwise, 3G/4 bytes) plus one exponent byte.  Owning a whole
// group per lane makes one Philox call serve 16 values, which keeps stochastic
// rounding within the HBM-bound budget.
#include <mutex>

#include "bfp_quant.h"

namespace fastbfp {

// Plane p of the group goes to mant_p (plane 1 of a two-chunk tensor, or the
// separate 2-bit tensor of the adaptive path).
template <int G, int NCH, int P0, int P1, bool STREAM = false>
__device__ __forceinline__ void store_group(uint8_t* __restrict__ mant0, uint8_t* __restrict__ mant1, int64_t gid,
                                            const uint32_t (&w)[NCH][G * 6 / 32]) {
  store_plane<G, P0 != kPlaneFP6, STREAM>(mant0, gid, w[0]);
  if (NCH == 2) store_plane<G, P1 != kPlaneFP6, STREAM>(mant1, gid, w[NCH - 1]);
}

// Writes the block's Eq. 2 partial sums to part[2 * blockIdx.x + {0, 1}]:
// a fixed-order reduction over the lanes of each wave, then over the four
// waves.  Every thread of the block must call it.
__device__ __forceinline__ void block_improvement(double num, double den, double* part) {
  __shared__ double red[2][4];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    num += __shfl_xor(num, off);
    den += __shfl_xor(den, off);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[0][wave] = num;
    red[1][wave] = den;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    part[2 * blockIdx.x + 1] = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
  }
}

// out[0..1] = the sums of the nparts partial pairs at part, in a fixed order
// (one block of 1024 threads: thread t adds pairs t, t + 1024, ... in order,
// reading them in batches of eight independent pairs, then a fixed tree over
// the threads): the result does not depend on scheduling.
__global__ __launch_bounds__(1024) void k_improvement_finalize(double* out, const double* part, int64_t nparts) {
  __shared__ double red[2][1024];
  double num = 0.0, den = 0.0;
  int64_t i = threadIdx.x;
  for (; i + 7 * 1024 < nparts; i += 8 * 1024) {
    double a[8], b[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      a[j] = part[2 * (i + 1024 * j)];
      b[j] = part[2 * (i + 1024 * j) + 1];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      num += a[j];
      den += b[j];
    }
  }
  for (; i < nparts; i += 1024) {
    num += part[2 * i];
    den += part[2 * i + 1];
  }
  red[0][threadIdx.x] = num;
  red[1][threadIdx.x] = den;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      red[0][threadIdx.x] += red[0][threadIdx.x + w];
      red[1][threadIdx.x] += red[1][threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    out[0] = red[0][0];
    out[1] = red[1][0];
  }
}

// Groups along the contiguous last axis: group gid covers x[gid*G, gid*G+G).
// A lane owns GPL consecutive groups (two of 16 -- one 32-value packing unit
// of the FP6 converter, also on the adaptive path -- or one of 32), a
// wave 64 * GPL groups.  Their FP32 values are brought into the wave's LDS
// region by direct global->LDS 16-byte loads, each of which reads 1 KB
// contiguous (one lane per 16-byte chunk), and every lane then reads its own
// groups back.  The chunk c of lane l's run lands in 16-byte slot
// CPL*l + (c ^ swz(l)): the XOR spreads the 16 lanes served together across
// all 64 banks on the read-back.  (Reading 64 contiguous bytes per lane
// straight from global memory instead leaves each load instruction touching
// 64 scattered 16-byte pieces, which costs about a third of HBM bandwidth.)
template <int G, int MODE, int NCH, bool ADAPT, int P0, int P1>
__global__ __launch_bounds__(256) void k_quantize_rows(const float* __restrict__ x, int64_t ngroups, uint32_t m,
                                                       uint32_t key0, uint32_t key1, uint8_t* __restrict__ mant0,
                                                       uint8_t* __restrict__ mant1, uint8_t* __restrict__ exps,
                                                       uint32_t* status, double* part) {
  constexpr int GPL = G <= 16 ? 32 / G : 1;  // groups per lane: 32 values for g <= 16
  constexpr int CPG = G / 4;                         // 16-byte chunks per group
  constexpr int CPL = GPL * CPG;                     // 16-byte chunks per lane
  constexpr int LANES_PER_SWZ = 16 / CPL;
  __shared__ __attribute__((aligned(16))) uint32_t stage[4][64 * 4 * CPL];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t g0 = ((int64_t)blockIdx.x * 4 + wave) * 64 * GPL;  // first group of this wave
  if (!ADAPT && g0 >= ngroups) return;  // (the adaptive path keeps every wave for its block sums)
  const int nvalid = (int)max((int64_t)0, min((int64_t)(64 * GPL), ngroups - g0));
  typedef __attribute__((address_space(3))) void lds_void;
  // (a wave with no valid group, kept by the adaptive path, reads x's first groups)
  const uint8_t* base = reinterpret_cast<const uint8_t*>(x) + (nvalid > 0 ? g0 * (G * 4) : 0);
  const int qmax_chunk = max(nvalid, 1) * CPG - 1;  // the wave's last valid chunk
#pragma unroll
  for (int k = 0; k < CPL; ++k) {
    const int slot = 64 * k + lane;
    const int l = slot / CPL;
    const int c = (slot % CPL) ^ ((l / LANES_PER_SWZ) % CPL);
    // chunks of groups past the end reread the wave's last valid chunk (unused)
    const int off = min(l * CPL + c, qmax_chunk) * 16;
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(base + off),
                                     (lds_void*)(&stage[wave][64 * 4 * k]), 16, 0, kStreamPolicy);
  }
  __builtin_amdgcn_s_waitcnt(0);  // the wave reads back what its own loads wrote
  const int nmine = min(GPL, max(0, nvalid - lane * GPL));  // this lane's valid groups
  if (!ADAPT && nmine == 0) return;  // (the adaptive path keeps every lane for its wave sums)
  uint32_t b[GPL * G];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int slot = CPL * lane + (c ^ ((lane / LANES_PER_SWZ) % CPL));
    const u32x4 v = *reinterpret_cast<const u32x4*>(&stage[wave][4 * slot]);
    b[4 * c + 0] = v[0];
    b[4 * c + 1] = v[1];
    b[4 * c + 2] = v[2];
    b[4 * c + 3] = v[3];
  }
  const int64_t gid = g0 + lane * GPL;
  uint32_t w[NCH][GPL * G * 6 / 32];
  uint32_t E[GPL], s_lo[GPL], s_hi[GPL];
  bool nonfinite;
  quantize_groups<G, GPL, MODE, NCH, ADAPT, P0, P1, true>(b, m, (uint64_t)gid, key0, key1, w, E, nonfinite, s_lo,
                                                          s_hi);
  if (GPL > 1 && nmine == GPL) {
    // every group: one packing unit of 32 values (its bytes are the groups'
    // bytes side by side) and GPL exponent bytes
    if constexpr (GPL == 2) {
      stream_store(reinterpret_cast<uint16_t*>(exps + gid), (uint16_t)(E[0] | (E[GPL - 1] << 8)));
    } else if constexpr (GPL >= 4) {
      uint32_t e4[GPL / 4];
#pragma unroll
      for (int k = 0; k < GPL / 4; ++k)
        e4[k] = E[4 * k] | (E[4 * k + 1] << 8) | (E[4 * k + 2] << 16) | (E[4 * k + 3] << 24);
#pragma unroll
      for (int k = 0; k < GPL / 4; ++k) stream_store(reinterpret_cast<uint32_t*>(exps + gid) + k, e4[k]);
    }
    store_group<GPL * G, NCH, P0, P1, true>(mant0, mant1, gid / GPL, w);
    if (status && nonfinite) atomicOr(status, 1u);
  } else if (nmine > 0) {
    // GPL = 1, or the last 16 values of the wave (every row holds whole
    // 16-value units): their own bytes
    constexpr int U = G < 16 ? 16 : G;  // values stored
#pragma unroll
    for (int k = 0; k < (G < 16 ? 16 / G : 1); ++k) exps[gid + k] = (uint8_t)E[k];
    store_plane<U, P0 != kPlaneFP6, true>(mant0, gid * G / U, w[0]);
    if (NCH == 2) store_plane<U, P1 != kPlaneFP6, true>(mant1, gid * G / U, w[NCH - 1]);
    if (status && nonfinite) atomicOr(status, 1u);
  }
  if (ADAPT) {
    double num = 0.0, den = 0.0;
#pragma unroll
    for (int gi = 0; gi < GPL; ++gi)
      if (gi < nmine) {
        num += ldexp((double)s_lo[gi], (int)E[gi] - 130);
        den += ldexp((double)s_hi[gi], (int)E[gi] - 128);
      }
    block_improvement(num, den, part);
  }
}

// Groups down the columns of x[R][C] (transpose-on-quantize).  Output row c is
// column c of x; its group j covers x[j*G .. j*G+G-1][c] and has
// gid = c * (R/G) + j.  A block takes 64 columns (one per lane: every load
// instruction reads 256 contiguous bytes of a row of x) and JB = 4 * NGT
// consecutive group rows (NGT per wave).  The packed codes and exponents of
// the 64 x JB groups are gathered in LDS and then written row by row, so that
// every store instruction writes contiguous bytes of one output row.
template <int G, int MODE, int NCH, int NGT, bool ADAPT, int P0, int P1>
__global__ __launch_bounds__(256) void k_quantize_cols(const float* __restrict__ x, int64_t R, int64_t C,
                                                       int64_t nbx, int64_t nbxy, uint32_t m, uint32_t key0,
                                                       uint32_t key1,
                                                       uint8_t* __restrict__ mant0, uint8_t* __restrict__ mant1,
                                                       uint8_t* __restrict__ exps, uint32_t* status, double* part) {
  // A step converts U = max(G, 16) consecutive values of a column: NGU = U / G
  // groups (a 16-value unit of groups of 4 or 8, or one group).
  constexpr int U = G < 16 ? 16 : G, NGU = U / G;
  constexpr int JB = 4 * NGT;             // unit rows per block
  constexpr int WPG = U * 6 / 32;         // code dwords per unit of an FP6 plane (an FP4 or Lo2 plane: U / 8)
  constexpr int WP[2] = {P0 != kPlaneFP6 ? U / 8 : WPG, P1 != kPlaneFP6 ? U / 8 : WPG};
  constexpr int ROWW = JB * WPG;          // LDS row stride, code dwords per output row
  __shared__ uint32_t sc[NCH][64][ROWW];
  __shared__ uint8_t se[64][JB * NGU];
  // A batch of matrices x[nbatch][R][C] (one launch for every slice of a
  // tensor grouped along an axis that is neither first nor last): slice b's
  // output rows are b * C .. b * C + C - 1.
  const int64_t batch = blockIdx.x / nbxy, bid = blockIdx.x % nbxy;
  const int64_t bx = bid % nbx, by = bid / nbx;
  x += batch * R * C;
  const int64_t row_base = batch * C;
  const int lane = threadIdx.x & 63, slot = threadIdx.x >> 6;
  const int64_t c0 = bx * 64, c = c0 + lane;
  const int64_t gpr = R / G, upr = R / U;  // groups and units per output row
  const int64_t jb = by * JB;
  const int jn = (int)min((int64_t)JB, upr - jb);  // unit rows this block covers
  bool any_bad = false;
  double num = 0.0, den = 0.0;
  if (c < C) {
    for (int i = 0; i < NGT; ++i) {
      const int jl = slot * NGT + i;
      if (jl >= jn) break;
      const int64_t j = jb + jl;
      uint32_t b[U];
      const float* src = x + (j * U) * C + c;
#pragma unroll
      for (int t = 0; t < U; ++t) b[t] = __float_as_uint(stream_load(src + t * C));
      uint32_t w[NCH][WPG];
      uint32_t E[NGU], s_lo[NGU], s_hi[NGU];
      bool nonfinite;
      quantize_groups<G, NGU, MODE, NCH, ADAPT, P0, P1, true>(b, m, (uint64_t)((row_base + c) * gpr + j * NGU), key0,
                                                             key1, w, E,
                                                             nonfinite, s_lo, s_hi);
      if (ADAPT) {
        num += ldexp((double)s_lo[0], (int)E[0] - 130);
        den += ldexp((double)s_hi[0], (int)E[0] - 128);
      }
#pragma unroll
      for (int p = 0; p < NCH; ++p)
#pragma unroll
        for (int k = 0; k < WP[p]; ++k) sc[p][lane][jl * WP[p] + k] = w[p][k];
#pragma unroll
      for (int k = 0; k < NGU; ++k) se[lane][jl * NGU + k] = (uint8_t)E[k];
      any_bad |= nonfinite;
    }
  }
  if (ADAPT) block_improvement(num, den, part);
  __syncthreads();
  // Write-out: output row c0 + r gets jn units starting at unit jb.
  const int ncols = (int)min((int64_t)64, C - c0);
#pragma unroll
  for (int p = 0; p < NCH; ++p) {
    const int rw = JB * WP[p];  // code dwords of a full output row of this block in plane p
    for (int d = threadIdx.x; d < ncols * rw; d += 256) {
      const int r = d / rw, k = d % rw;
      if (k < jn * WP[p]) {
        const int64_t o = ((row_base + c0 + r) * upr + jb) * WP[p] + k;
        reinterpret_cast<uint32_t*>(p ? mant1 : mant0)[o] = sc[p][r][k];
      }
    }
  }
  for (int d = threadIdx.x; d < ncols * JB * NGU; d += 256) {
    const int r = d / (JB * NGU), k = d % (JB * NGU);
    if (k < jn * NGU) exps[(row_base + c0 + r) * gpr + jb * NGU + k] = se[r][k];
  }
  if (status && any_bad) atomicOr(status, 1u);
}

// BFP -> FP32: y = +-q * 2^(E-127-(m-1)).  One lane per U = max(G, 16)
// values (a 16-value unit of groups of 4 or 8, or one group).  P0 / P1: the
// plane formats (launch.h); with two planes q = c0 * 2^s + c1, s = 2 when
// plane 1 is a Lo2 plane and 4 otherwise (both chunks carry the sign).
template <int G, int NCH, int P0, int P1>
__global__ __launch_bounds__(256) void k_dequantize(const uint8_t* __restrict__ mant, const uint8_t* __restrict__ exps,
                                                    int64_t nunits, int m, float* __restrict__ y) {
  constexpr int U = G < 16 ? 16 : G, NGU = U / G;
  const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (u >= nunits) return;
  constexpr int PK[2] = {P0, P1};
  constexpr int B0 = P0 != kPlaneFP6 ? U / 2 : U * 3 / 4;  // bytes per unit in plane 0
  uint32_t w[NCH][U * 6 / 32];
#pragma unroll
  for (int p = 0; p < NCH; ++p) {
    const int gb = PK[p] != kPlaneFP6 ? U / 2 : U * 3 / 4;
    const uint32_t* src = reinterpret_cast<const uint32_t*>(mant + p * nunits * B0 + u * gb);
#pragma unroll
    for (int i = 0; i < U * 6 / 32; ++i) w[p][i] = i < gb / 4 ? src[i] : 0u;
    if (PK[p] == kPlaneLo2) {
      // back to three FP6 code dwords per 16 values (last half first: in place)
#pragma unroll
      for (int h = U / 16 - 1; h >= 0; --h) {
        uint32_t t0, t1, t2;
        lo2_unpack(w[p][2 * h], w[p][2 * h + 1], t0, t1, t2);
        w[p][3 * h] = t0;
        w[p][3 * h + 1] = t1;
        w[p][3 * h + 2] = t2;
      }
    }
  }
  int e[NGU];
#pragma unroll
  for (int k = 0; k < NGU; ++k) e[k] = (int)exps[u * NGU + k] - 127 - (m - 1);
  auto chunk = [&](int p, int t) {
    if (PK[p] == kPlaneFP4) {
      const uint32_t nib = (w[p][t >> 3] >> (4 * (t & 7))) & 0xFu;
      return (nib & 8u) ? -(int)(nib & 7u) : (int)(nib & 7u);
    }
    if (PK[p] == kPlaneLo2) return e2m3_eighth_decode(fp6_field(w[p], t));
    return e2m3_half_decode(fp6_field(w[p], t));
  };
  float4* dst = reinterpret_cast<float4*>(y + u * U);
#pragma unroll
  for (int i = 0; i < U / 4; ++i) {
    float v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int t = 4 * i + k;
      int q = chunk(0, t);
      if (NCH == 2) q = q * (P1 == kPlaneLo2 ? 4 : 16) + chunk(NCH - 1, t);
      v[k] = ldexpf((float)q, e[t / G]);
    }
    dst[i] = make_float4(v[0], v[1], v[2], v[3]);
  }
}

template <int G, int MODE, int NCH, int P0, bool ADAPT = false, int P1 = kPlaneFP6>
static hipError_t launch_rows_t(const float* x, int64_t ngroups, int m, uint64_t seed, uint8_t* mant0, uint8_t* mant1,
                                uint8_t* exps, uint32_t* status, double* part, hipStream_t s) {
  constexpr int GPL = G <= 16 ? 32 / G : 1;  // groups per lane (as in the kernel)
  const int64_t blocks = (ngroups + 256 * GPL - 1) / (256 * GPL);
  hipLaunchKernelGGL((k_quantize_rows<G, MODE, NCH, ADAPT, P0, P1>), dim3((unsigned)blocks), dim3(256), 0, s, x, ngroups,
                     (uint32_t)m, (uint32_t)seed, (uint32_t)(seed >> 32), mant0, mant1, exps, status, part);
  return hipGetLastError();
}

template <int G, int MODE, int NCH, int P0, bool ADAPT = false, int P1 = kPlaneFP6>
static hipError_t launch_cols_t(const float* x, int64_t R, int64_t C, int m, uint64_t seed, uint8_t* mant0,
                                uint8_t* mant1, uint8_t* exps, uint32_t* status, double* part, hipStream_t s,
                                int64_t nbatch = 1) {
  constexpr int NGT = G == 64 ? 2 : 8;  // (the LDS gather holds 4 * NGT units of 64 columns)
  const int64_t upr = R / (G < 16 ? 16 : G);  // units per output row (as in the kernel)
  const int64_t nbx = (C + 63) / 64, nby = (upr + 4 * NGT - 1) / (4 * NGT);
  const int64_t nbxy = nbx * nby;
  hipLaunchKernelGGL((k_quantize_cols<G, MODE, NCH, NGT, ADAPT, P0, P1>), dim3((unsigned)(nbxy * nbatch)), dim3(256), 0,
                     s, x, R, C, nbx, nbxy, (uint32_t)m, (uint32_t)seed, (uint32_t)(seed >> 32), mant0, mant1, exps,
                     status, part);
  return hipGetLastError();
}

// Specialisation for (g, rounding mode, m): planes and plane formats.
#define FASTBFP_QUANT_M(FN, G, MODE, ...)                                         \
  do {                                                                            \
    if (m <= 2) return FN<G, MODE, 1, kPlaneFP4>(__VA_ARGS__);                    \
    if (m <= 4) return FN<G, MODE, 1, kPlaneFP6>(__VA_ARGS__);                    \
    if (m <= 6) return FN<G, MODE, 2, kPlaneFP6, false, kPlaneLo2>(__VA_ARGS__);  \
    return FN<G, MODE, 2, kPlaneFP6>(__VA_ARGS__);                                \
  } while (0)
#define FASTBFP_QUANT_G(FN, G, ...)                                               \
  do {                                                                            \
    if (mode == kNearest) FASTBFP_QUANT_M(FN, G, kNearest, __VA_ARGS__);          \
    if (mode == kStochastic) FASTBFP_QUANT_M(FN, G, kStochastic, __VA_ARGS__);    \
    FASTBFP_QUANT_M(FN, G, kTruncate, __VA_ARGS__);                               \
  } while (0)
#define FASTBFP_DISPATCH_QUANT(FN, ...)                                           \
  do {                                                                            \
    if (g == 4) FASTBFP_QUANT_G(FN, 4, __VA_ARGS__);                              \
    if (g == 8) FASTBFP_QUANT_G(FN, 8, __VA_ARGS__);                              \
    if (g == 16) FASTBFP_QUANT_G(FN, 16, __VA_ARGS__);                            \
    if (g == 32) FASTBFP_QUANT_G(FN, 32, __VA_ARGS__);                            \
    FASTBFP_QUANT_G(FN, 64, __VA_ARGS__);                                         \
  } while (0)

hipError_t launch_quantize_rows(const float* x, int64_t rows, int64_t len, int g, int m, int mode, uint64_t seed,
                                uint8_t* mant, uint8_t* exps, uint32_t* status, hipStream_t s) {
  const int64_t ngroups = rows * (len / g);
  if (ngroups == 0) return hipSuccess;
  uint8_t* mant1 = mant + ngroups * plane_group_bytes(g, m, 0);  // plane 1 when m > 4
  FASTBFP_DISPATCH_QUANT(launch_rows_t, x, ngroups, m, seed, mant, mant1, exps, status, nullptr, s);
}

hipError_t launch_quantize_cols(const float* x, int64_t R, int64_t C, int g, int m, int mode, uint64_t seed,
                                uint8_t* mant, uint8_t* exps, uint32_t* status, hipStream_t s, int64_t nbatch) {
  if (R == 0 || C == 0 || nbatch == 0) return hipSuccess;
  uint8_t* mant1 = mant + nbatch * C * (R / g) * plane_group_bytes(g, m, 0);  // plane 1 when m > 4
  FASTBFP_DISPATCH_QUANT(launch_cols_t, x, R, C, m, seed, mant, mant1, exps, status, nullptr, s, nbatch);
}

int64_t quantize_rows_blocks(int64_t rows, int64_t len, int g) {
  const int64_t per_block = 256 * (g <= 16 ? 32 / g : 1);  // groups per k_quantize_rows workgroup
  const int64_t ngroups = (len / g) > 0 && rows > INT64_MAX / (len / g) ? INT64_MAX : rows * (len / g);
  return (ngroups + per_block - 1) / per_block;
}

int64_t quantize_cols_blocks(int64_t R, int64_t C, int g, int64_t nbatch) {
  const int64_t U = g < 16 ? 16 : g, NGT = g == 64 ? 2 : 8;
  return ((C + 63) / 64) * ((R / U + 4 * NGT - 1) / (4 * NGT)) * nbatch;
}

// The adaptive specialisations: plane 0 the m = 4 codes (FP6), plane 1 (if
// two) the 2-bit tensor (FP4).
#define FASTBFP_ADAPT_M(FN, G, MODE, ...)                                         \
  do {                                                                            \
    if (two) return FN<G, MODE, 2, kPlaneFP6, true, kPlaneFP4>(__VA_ARGS__);      \
    return FN<G, MODE, 1, kPlaneFP6, true, kPlaneFP4>(__VA_ARGS__);               \
  } while (0)
#define FASTBFP_DISPATCH_ADAPT(FN, ...)                                           \
  do {                                                                            \
    if (g == 16) {                                                                \
      if (mode == kNearest) FASTBFP_ADAPT_M(FN, 16, kNearest, __VA_ARGS__);       \
      if (mode == kStochastic) FASTBFP_ADAPT_M(FN, 16, kStochastic, __VA_ARGS__); \
      FASTBFP_ADAPT_M(FN, 16, kTruncate, __VA_ARGS__);                            \
    } else {                                                                      \
      if (mode == kNearest) FASTBFP_ADAPT_M(FN, 32, kNearest, __VA_ARGS__);       \
      if (mode == kStochastic) FASTBFP_ADAPT_M(FN, 32, kStochastic, __VA_ARGS__); \
      FASTBFP_ADAPT_M(FN, 32, kTruncate, __VA_ARGS__);                            \
    }                                                                             \
  } while (0)

int64_t adaptive_parts(int64_t R, int64_t C, int group_axis, int g) {
  if (R == 0 || C == 0) return 0;
  if (group_axis == 1) {  // one partial pair per k_quantize_rows block (two groups per lane when g = 16)
    const int64_t per_block = g == 16 ? 512 : 256;
    return (R * (C / g) + per_block - 1) / per_block;
  }
  const int64_t gpr = R / g;
  return ((C + 63) / 64) * ((gpr + 31) / 32);  // one per k_quantize_cols block (NGT = 8)
}

static hipError_t launch_adaptive_kernel(const float* x, int64_t R, int64_t C, int group_axis, int g, int mode,
                                         uint64_t seed, uint8_t* mant4, uint8_t* mant2, uint8_t* exps, double* part,
                                         uint32_t* status, hipStream_t s) {
  const int m = 4;
  const bool two = mant2 != nullptr;  // second output plane: the 2-bit mantissas
  if (group_axis == 1) {
    const int64_t ngroups = R * (C / g);
    FASTBFP_DISPATCH_ADAPT(launch_rows_t, x, ngroups, m, seed, mant4, mant2, exps, status, part, s);
  }
  FASTBFP_DISPATCH_ADAPT(launch_cols_t, x, R, C, m, seed, mant4, mant2, exps, status, part, s);
}

// part: the per-workgroup partial pairs (2 * adaptive_parts doubles); out:
// the two sums.
static hipError_t launch_adaptive_parts(const float* x, int64_t R, int64_t C, int group_axis, int g, int mode,
                                        uint64_t seed, uint8_t* mant4, uint8_t* mant2, uint8_t* exps, double* out,
                                        double* part, uint32_t* status, hipStream_t s) {
  const int64_t nparts = adaptive_parts(R, C, group_axis, g);
  if (nparts > 0) {
    const hipError_t e = launch_adaptive_kernel(x, R, C, group_axis, g, mode, seed, mant4, mant2, exps, part, status, s);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_improvement_finalize, dim3(1), dim3(1024), 0, s, out, part, nparts);
  return hipGetLastError();
}

hipError_t launch_quantize_adaptive(const float* x, int64_t R, int64_t C, int group_axis, int g, int mode,
                                    uint64_t seed, uint8_t* mant4, uint8_t* mant2, uint8_t* exps, double* sums,
                                    uint32_t* status, hipStream_t s) {
  return launch_adaptive_parts(x, R, C, group_axis, g, mode, seed, mant4, mant2, exps, sums, sums + 2, status, s);
}

// The allocation-free variant: the partial pairs go to a file-scope device
// array (one copy per GPU, kept until the process ends) instead of a caller
// workspace.  Its address is looked up once per device, with that device
// current; host code uses only that address, never the array's name.
static __device__ __align__(256) double scratch[kAdaptiveScratchDoubles];

static hipError_t scratch_address(double** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static double* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = static_cast<double*>(p);
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_quantize_adaptive_static(const float* x, int64_t R, int64_t C, int group_axis, int g, int mode,
                                           uint64_t seed, uint8_t* mant4, uint8_t* mant2, uint8_t* exps,
                                           double* sums, uint32_t* status, hipStream_t s) {
  double* part = nullptr;
  const hipError_t e = scratch_address(&part);
  if (e != hipSuccess) return e;
  return launch_adaptive_parts(x, R, C, group_axis, g, mode, seed, mant4, mant2, exps, sums, part, status, s);
}

// Both groupings of a matrix from one read (and, with UPD, the weight update
// in front of them).  x[R][C] is converted with groups of 16 along its rows
// (output "r": rows = R, len = C, gid = r * C/16 + j) and along its columns
// (output "c": rows = C, len = R, gid = c * R/16 + i), each byte for byte what
// the single-axis kernels write with that output's seed.  UPD: the matrix is
// x' = x + alpha * dx, computed as the two FP32 roundings of the product and
// the sum (no fused multiply-add), written to x_out and converted.
//
// A block owns a 64 x 64 tile, staged in LDS once (16 KB, so that several
// blocks per CU overlap one another's loads and conversions): row r's 16-byte
// granule g sits at granule g ^ s(r), s(r) = (r & 15) ^ 4 ((r >> 4) & 3), so
// that 16 lanes reading one granule of 16 consecutive rows (a row group
// each), and 64 lanes reading one float of 16 columns x 4 group rows (a
// column group each), both hit distinct banks.  Each thread then converts one
// row group and one column group; the lanes of a wave store 16 output rows x
// 4 consecutive groups in either grouping, i.e. contiguous 4-group runs.  Tile
// rows past R read zero (the buffer resource ends at the last row); columns
// past C read whatever follows in memory, and only whole groups past C are
// affected, which are never stored.
template <int MODE, int NCH, int P0, int P1, bool UPD>
__global__ __launch_bounds__(256) void k_quantize_dual(const float* x, const float* dx, float alpha, float* x_out,
                                                       int64_t R, int64_t C, int tiles_c, uint32_t m, uint32_t kr0,
                                                       uint32_t kr1, uint32_t kc0, uint32_t kc1,
                                                       uint8_t* __restrict__ mr0, uint8_t* __restrict__ mr1,
                                                       uint8_t* __restrict__ er, uint8_t* __restrict__ mc0,
                                                       uint8_t* __restrict__ mc1, uint8_t* __restrict__ ec,
                                                       uint32_t* status) {
  constexpr int T = 64;
  __shared__ __attribute__((aligned(16))) float tile[T * T];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // Tile order: each XCD (workgroups are dealt to the 8 XCDs in turn) takes a
  // contiguous run of tiles, walked in bands of 8 tile rows, down each band's
  // column first: an output row of either grouping then receives 8
  // neighbouring tiles' groups (384 bytes) at about the same time.
  int lid = blockIdx.x;
  if (gridDim.x % 8 == 0) lid = (blockIdx.x % 8) * (gridDim.x / 8) + blockIdx.x / 8;
  const int tiles_r = (int)((R + T - 1) / T), band = lid / (8 * tiles_c), in = lid % (8 * tiles_c);
  const int band_rows = min(8, tiles_r - 8 * band);
  const int64_t r0 = (int64_t)(8 * band + in % band_rows) * T, c0 = (int64_t)(in / band_rows) * T;
  const int rows = (int)min((int64_t)T, R - r0);
  typedef __attribute__((address_space(3))) void lds_void;
  // Tile rows [r0, r0 + rows) of x (and dx); offsets are within 64 rows of C floats.
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(x + r0 * C), (short)0, (int)(rows * C * 4), 0x00020000);
  // Granule slot q = 64 * (4 * wave + n) + lane: row q / 16, slot q % 16,
  // which holds the row's granule (q % 16) ^ s(row).
  auto swz = [](int row) { return (row & 15) ^ (((row >> 4) & 3) << 2); };
#pragma unroll
  for (int n = 0; n < 4; ++n) {
    const int q = 64 * (4 * wave + n) + lane, row = q >> 4, g = (q & 15) ^ swz(row);
    const uint32_t off = (uint32_t)(row * C + c0 + 4 * g) * 4u;
    if constexpr (UPD) {
      const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(dx + r0 * C), (short)0, (int)(rows * C * 4), 0x00020000);
      const v4i a = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, kStreamPolicy));
      const v4i d = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rd, off, 0, kStreamPolicy));
      float4 v;
      {
        // Two roundings, never a fused multiply-add.
#pragma clang fp contract(off)
        v.x = __int_as_float(a[0]) + alpha * __int_as_float(d[0]);
        v.y = __int_as_float(a[1]) + alpha * __int_as_float(d[1]);
        v.z = __int_as_float(a[2]) + alpha * __int_as_float(d[2]);
        v.w = __int_as_float(a[3]) + alpha * __int_as_float(d[3]);
      }
      *reinterpret_cast<float4*>(&tile[4 * q]) = v;
      if (row < rows && c0 + 4 * g < C) {
        typedef float f4 __attribute__((ext_vector_type(4)));
        stream_store(reinterpret_cast<f4*>(x_out + (r0 + row) * C + c0 + 4 * g), f4{v.x, v.y, v.z, v.w});
      }
    } else {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)&tile[4 * 64 * (4 * wave + n)], 16, off, 0, 0,
                                               kStreamPolicy);
    }
  }
  if constexpr (!UPD) __builtin_amdgcn_s_waitcnt(0);  // this wave's direct loads have landed
  __syncthreads();

  bool bad = false;
  uint32_t b[16], w[NCH][3], E, s_lo, s_hi;
  bool nonfinite;
  {
    // Row group: wave w covers rows 16 w .. 16 w + 15, lane block lb group lb.
    const int row = 16 * wave + (lane & 15), cg = lane >> 4;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(&tile[row * T + 4 * ((4 * cg + u) ^ swz(row))]);
      b[4 * u] = v[0];
      b[4 * u + 1] = v[1];
      b[4 * u + 2] = v[2];
      b[4 * u + 3] = v[3];
    }
    if (r0 + row < R && c0 + 16 * cg < C) {
      const int64_t gid = (r0 + row) * (C / 16) + c0 / 16 + cg;
      quantize_group<16, MODE, NCH, false, P0, P1, true>(b, m, (uint64_t)gid, kr0, kr1, w, E, nonfinite, s_lo,
                                                            s_hi);
      er[gid] = (uint8_t)E;
      store_group<16, NCH, P0, P1>(mr0, mr1, gid, w);
      bad |= nonfinite;
    }
  }
  {
    // Column group: wave w covers columns 16 w .. 16 w + 15, lane block lb
    // group row lb.
    const int rg = lane >> 4, col = 16 * wave + (lane & 15);
#pragma unroll
    for (int u = 0; u < 16; ++u)
      b[u] = __float_as_uint(tile[(16 * rg + u) * T + 4 * ((col >> 2) ^ swz(16 * rg + u)) + (col & 3)]);
    if (c0 + col < C && r0 + 16 * rg < R) {
      const int64_t gid = (c0 + col) * (R / 16) + r0 / 16 + rg;
      quantize_group<16, MODE, NCH, false, P0, P1, true>(b, m, (uint64_t)gid, kc0, kc1, w, E, nonfinite, s_lo,
                                                            s_hi);
      ec[gid] = (uint8_t)E;
      store_group<16, NCH, P0, P1>(mc0, mc1, gid, w);
      bad |= nonfinite;
    }
  }
  if (status && bad) atomicOr(status, 1u);
}

template <int MODE, int NCH, int P0, int P1, bool UPD>
static hipError_t launch_dual_t(const float* x, const float* dx, float alpha, float* x_out, int64_t R, int64_t C, int m,
                                uint64_t seed_r, uint64_t seed_c, uint8_t* mr, uint8_t* er, uint8_t* mc, uint8_t* ec,
                                uint32_t* status, hipStream_t s) {
  const int64_t tiles_r = (R + 63) / 64, tiles_c = (C + 63) / 64;
  const int64_t ng = R * (C / 16);  // groups per output (either grouping)
  const int64_t b0 = plane_group_bytes(16, m, 0);
  hipLaunchKernelGGL((k_quantize_dual<MODE, NCH, P0, P1, UPD>), dim3((unsigned)(tiles_r * tiles_c)), dim3(256), 0, s, x,
                     dx, alpha, x_out, R, C, (int)tiles_c, (uint32_t)m, (uint32_t)seed_r, (uint32_t)(seed_r >> 32),
                     (uint32_t)seed_c, (uint32_t)(seed_c >> 32), mr, mr + ng * b0, er, mc, mc + ng * b0, ec, status);
  return hipGetLastError();
}

template <bool UPD>
static hipError_t launch_dual_any(const float* x, const float* dx, float alpha, float* x_out, int64_t R, int64_t C,
                                  int m, int mode, uint64_t seed_r, uint64_t seed_c, uint8_t* mr, uint8_t* er,
                                  uint8_t* mc, uint8_t* ec, uint32_t* status, hipStream_t s) {
  if (R == 0 || C == 0) return hipSuccess;
#define FASTBFP_DUAL(MODE)                                                                                        \
  do {                                                                                                            \
    if (m <= 2) return launch_dual_t<MODE, 1, kPlaneFP4, kPlaneFP6, UPD>(x, dx, alpha, x_out, R, C, m, seed_r,    \
                                                                         seed_c, mr, er, mc, ec, status, s);      \
    if (m <= 4) return launch_dual_t<MODE, 1, kPlaneFP6, kPlaneFP6, UPD>(x, dx, alpha, x_out, R, C, m, seed_r,    \
                                                                         seed_c, mr, er, mc, ec, status, s);      \
    if (m <= 6) return launch_dual_t<MODE, 2, kPlaneFP6, kPlaneLo2, UPD>(x, dx, alpha, x_out, R, C, m, seed_r,    \
                                                                         seed_c, mr, er, mc, ec, status, s);      \
    return launch_dual_t<MODE, 2, kPlaneFP6, kPlaneFP6, UPD>(x, dx, alpha, x_out, R, C, m, seed_r, seed_c, mr, er, \
                                                             mc, ec, status, s);                                  \
  } while (0)
  if (mode == kNearest) FASTBFP_DUAL(kNearest);
  if (mode == kStochastic) FASTBFP_DUAL(kStochastic);
  FASTBFP_DUAL(kTruncate);
#undef FASTBFP_DUAL
}

hipError_t launch_quantize_dual(const float* x, int64_t R, int64_t C, int m, int mode, uint64_t seed_r,
                                uint64_t seed_c, uint8_t* mr, uint8_t* er, uint8_t* mc, uint8_t* ec,
                                uint32_t* status, hipStream_t s) {
  return launch_dual_any<false>(x, nullptr, 0.0f, nullptr, R, C, m, mode, seed_r, seed_c, mr, er, mc, ec, status, s);
}

hipError_t launch_weight_update(const float* w, const float* dw, float alpha, float* w_out, int64_t R, int64_t C,
                                int m, int mode, uint64_t seed_r, uint64_t seed_c, uint8_t* mr, uint8_t* er,
                                uint8_t* mc, uint8_t* ec, uint32_t* status, hipStream_t s) {
  return launch_dual_any<true>(w, dw, alpha, w_out, R, C, m, mode, seed_r, seed_c, mr, er, mc, ec, status, s);
}

template <int G, int NCH, int P0, int P1 = kPlaneFP6>
static hipError_t launch_deq_t(const uint8_t* mant, const uint8_t* exps, int64_t ngroups, int m, float* y,
                               hipStream_t s) {
  const int64_t nunits = G < 16 ? ngroups * G / 16 : ngroups;
  const unsigned blocks = (unsigned)((nunits + 255) / 256);
  hipLaunchKernelGGL((k_dequantize<G, NCH, P0, P1>), dim3(blocks), dim3(256), 0, s, mant, exps, nunits, m, y);
  return hipGetLastError();
}

template <int G>
static hipError_t launch_deq_g(const uint8_t* mant, const uint8_t* exps, int64_t ngroups, int m, float* y,
                               hipStream_t s) {
  if (m <= 2) return launch_deq_t<G, 1, kPlaneFP4>(mant, exps, ngroups, m, y, s);
  if (m <= 4) return launch_deq_t<G, 1, kPlaneFP6>(mant, exps, ngroups, m, y, s);
  if (m <= 6) return launch_deq_t<G, 2, kPlaneFP6, kPlaneLo2>(mant, exps, ngroups, m, y, s);
  return launch_deq_t<G, 2, kPlaneFP6, kPlaneFP6>(mant, exps, ngroups, m, y, s);
}

hipError_t launch_dequantize(const uint8_t* mant, const uint8_t* exps, int64_t rows, int64_t len, int g, int m,
                             float* y, hipStream_t s) {
  const int64_t ngroups = rows * (len / g);
  if (ngroups == 0) return hipSuccess;
  switch (g) {
    case 4: return launch_deq_g<4>(mant, exps, ngroups, m, y, s);
    case 8: return launch_deq_g<8>(mant, exps, ngroups, m, y, s);
    case 16: return launch_deq_g<16>(mant, exps, ngroups, m, y, s);
    case 32: return launch_deq_g<32>(mant, exps, ngroups, m, y, s);
    default: return launch_deq_g<64>(mant, exps, ngroups, m, y, s);
  }
}

}  // namespace fastbfp
