// packed.hip -- the paper's packed BFP storage (section V-D): every 2-bit
// chunk of a mantissa stored with its value's sign in 3 bits, chunk planes
// most significant first, and a 3-bit exponent per group of 16 above one
// base for the tensor.  Conversion (FP32 -> packed) and the inverse; the GEMM
// on packed operands runs on the general kernel (gemm_general.hip).
//
// Layout (include/fastbfp.h): NP = ceil(m / 2) planes; plane c holds chunk c
// of every value (q >> 2 (NP - 1 - c) & 3) as a 3-bit field -- the sign at bit 2
// (only for a nonzero chunk), the chunk at bits 0-1 -- value t of group gid at
// bits 3t .. 3t + 2 of the group's 6 bytes, group gid at byte offset
// (c * ngroups + gid) * 6.  The exponent array starts with a 32-bit word
// holding the tensor's largest exponent field E_max; base B = max(E_max - 7,
// 0); then group gid's offset e = E - B in bits 3 gid .. 3 gid + 2 of the
// stream that follows (64 groups per 24 bytes).  Group gid is converted with
// the shared exponent E = max(its largest exponent field, B).
#include "bfp_quant.h"

namespace fastbfp {

namespace {

__global__ void k_packed_header_clear(uint32_t* hdr) { *hdr = 0u; }

// hdr = max(hdr, the largest exponent field of x[0 .. 4 n4)): kExpMaxGranules
// 16-byte granules per block, in rounds of four independent loads per thread.
// The word only grows, so a block whose maximum is not above the value it
// reads skips its atomic.
constexpr int kExpMaxGranules = 4096;
__global__ __launch_bounds__(256) void k_exponent_max(const u32x4* __restrict__ x, int64_t n4, uint32_t* hdr) {
  const int64_t i0 = (int64_t)blockIdx.x * kExpMaxGranules + threadIdx.x;
  uint32_t e = 0;
#pragma unroll
  for (int r = 0; r < kExpMaxGranules / 1024; ++r) {
    u32x4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t i = i0 + 1024 * r + 256 * j;
      v[j] = i < n4 ? stream_load(x + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      e = max(max(e, (v[j].x >> 23) & 0xFFu), (v[j].y >> 23) & 0xFFu);
      e = max(max(e, (v[j].z >> 23) & 0xFFu), (v[j].w >> 23) & 0xFFu);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) e = max(e, (uint32_t)__shfl_xor((int)e, off));
  __shared__ uint32_t red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = e;
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t bmax = max(max(red[0], red[1]), max(red[2], red[3]));
    if (bmax > __atomic_load_n(hdr, __ATOMIC_RELAXED)) atomicMax(hdr, bmax);
  }
}

// One lane per group of 16 values along the rows, a wave per 64 groups.  The
// wave's 4 KB of input come into its LDS region by four direct global->LDS
// loads of 1 KB contiguous each; chunk c (16 bytes) of lane l's group lands in
// slot 4 l + (c ^ ((l / 4) % 4)), so that the 16 lanes served together on the
// read-back hit all 64 banks.  NP = ceil(m / 2) chunk planes.
template <int MODE, int NP>
__global__ __launch_bounds__(256) void k_quantize_packed(const float* __restrict__ x, int64_t ngroups, uint32_t m,
                                                         uint32_t key0, uint32_t key1, uint8_t* __restrict__ mant,
                                                         uint32_t* __restrict__ expw, uint32_t* status) {
  __shared__ __attribute__((aligned(16))) uint32_t stage[4][64 * 16];
  __shared__ uint32_t e3s[256];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t g0 = ((int64_t)blockIdx.x * 4 + wave) * 64;  // the wave's first group
  const int64_t gid = g0 + lane;
  const int nvalid = (int)max((int64_t)0, min((int64_t)64, ngroups - g0));
  const uint32_t base = packed_base(expw[0]);
  uint32_t e3 = 0;
  if (nvalid > 0) {
    typedef __attribute__((address_space(3))) void lds_void;
    const uint8_t* src = reinterpret_cast<const uint8_t*>(x) + g0 * 64;
    const int last = nvalid * 4 - 1;  // chunks of groups past the end reread the last valid one (unused)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int slot = 64 * k + lane, l = slot / 4, c = (slot % 4) ^ ((l / 4) % 4);
      __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(src + min(4 * l + c, last) * 16),
                                       (lds_void*)&stage[wave][64 * 4 * k], 16, 0, kStreamPolicy);
    }
    __builtin_amdgcn_s_waitcnt(0);  // the wave reads back what its own loads wrote
  }
  if (lane < nvalid) {
    uint32_t b[16];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(&stage[wave][4 * (4 * lane + (c ^ ((lane / 4) % 4)))]);
      b[4 * c] = v.x;
      b[4 * c + 1] = v.y;
      b[4 * c + 2] = v.z;
      b[4 * c + 3] = v.w;
    }
    // (a) the group's exponent, raised to the tensor base
    const uint32_t Eg = group_exponent<16>(b);
    const uint32_t E = max(Eg, base);
    if (status && Eg == 255u) atomicOr(status, 1u);
    uint32_t noise[4] = {0u, 0u, 0u, 0u};
    if (MODE == kStochastic) group_noise<16>((uint64_t)gid, key0, key1, noise);
    // (b)-(d) the magnitudes, split into 2-bit chunks with the sign
    const int align = magnitude_align<MODE>(m, E);
    const uint32_t qmax = (1u << m) - 1u;
    uint64_t plane[NP];
#pragma unroll
    for (int c = 0; c < NP; ++c) plane[c] = 0;
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const uint32_t q = value_magnitude<MODE, true>(b[t], align, noise[t >> 2], t, qmax);
      const uint32_t sgn = (b[t] >> 29) & 4u;  // the sign at bit 2 of a field
#pragma unroll
      for (int c = 0; c < NP; ++c) {
        const uint32_t ch = (q >> (2 * (NP - 1 - c))) & 3u;
        plane[c] |= (uint64_t)(ch ? (sgn | ch) : 0u) << (3 * t);
      }
    }
#pragma unroll
    for (int c = 0; c < NP; ++c) {
      uint16_t* dst = reinterpret_cast<uint16_t*>(mant + (c * ngroups + gid) * 6);
      dst[0] = (uint16_t)plane[c];
      dst[1] = (uint16_t)(plane[c] >> 16);
      dst[2] = (uint16_t)(plane[c] >> 32);
    }
    e3 = E - base;
  }
  // The wave's 64 exponent offsets, 192 bits: lane d < 6 assembles dword d
  // from the fields of lanes 32d/3 .. (32d + 31)/3.
  e3s[threadIdx.x] = e3;
  __syncthreads();
  if (lane < 6 && nvalid > 0) {
    uint32_t w = 0;
    for (int l = (32 * lane) / 3; l <= (32 * lane + 31) / 3; ++l) {
      const int sh = 3 * l - 32 * lane;  // -2 .. 31
      const uint32_t f = e3s[wave * 64 + l];
      w |= sh >= 0 ? f << sh : f >> -sh;
    }
    expw[1 + (g0 / 64) * 6 + lane] = w;
  }
}

// One lane per group: y = +-q * 2^(E - 127 - (m - 1)).
template <int NP>
__global__ __launch_bounds__(256) void k_dequantize_packed(const uint8_t* __restrict__ mant,
                                                           const uint32_t* __restrict__ expw, int64_t ngroups, int m,
                                                           float* __restrict__ y) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= ngroups) return;
  const uint32_t base = packed_base(expw[0]);
  const int e = (int)(base + packed_exponent_offset(expw, gid)) - 127 - (m - 1);
  uint64_t plane[NP];
#pragma unroll
  for (int c = 0; c < NP; ++c) {
    const uint16_t* src = reinterpret_cast<const uint16_t*>(mant + (c * ngroups + gid) * 6);
    plane[c] = (uint64_t)src[0] | ((uint64_t)src[1] << 16) | ((uint64_t)src[2] << 32);
  }
  float4* dst = reinterpret_cast<float4*>(y + gid * 16);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int t = 4 * i + k;
      int q = 0;
      bool neg = false;
#pragma unroll
      for (int c = 0; c < NP; ++c) {
        const uint32_t f = (uint32_t)(plane[c] >> (3 * t)) & 7u;
        q = 4 * q + (int)(f & 3u);
        neg |= (f & 4u) != 0;
      }
      v[k] = ldexpf((float)(neg ? -q : q), e);
    }
    dst[i] = make_float4(v[0], v[1], v[2], v[3]);
  }
}

template <int MODE>
hipError_t quantize_packed_mode(const float* x, int64_t ngroups, int m, uint64_t seed, uint8_t* mant, uint32_t* expw,
                                uint32_t* status, hipStream_t s) {
  const dim3 grid((unsigned)((ngroups + 255) / 256));
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  switch ((m + 1) / 2) {
    case 1: hipLaunchKernelGGL((k_quantize_packed<MODE, 1>), grid, dim3(256), 0, s, x, ngroups, (uint32_t)m, k0, k1,
                               mant, expw, status); break;
    case 2: hipLaunchKernelGGL((k_quantize_packed<MODE, 2>), grid, dim3(256), 0, s, x, ngroups, (uint32_t)m, k0, k1,
                               mant, expw, status); break;
    case 3: hipLaunchKernelGGL((k_quantize_packed<MODE, 3>), grid, dim3(256), 0, s, x, ngroups, (uint32_t)m, k0, k1,
                               mant, expw, status); break;
    default: hipLaunchKernelGGL((k_quantize_packed<MODE, 4>), grid, dim3(256), 0, s, x, ngroups, (uint32_t)m, k0, k1,
                                mant, expw, status); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize_packed(const float* x, int64_t rows, int64_t len, int m, int mode, uint64_t seed,
                                  uint8_t* mant, uint8_t* exps, uint32_t* status, hipStream_t s) {
  const int64_t n = rows * len, ngroups = n / 16;
  uint32_t* expw = reinterpret_cast<uint32_t*>(exps);
  // E_max of the tensor first (the base every group's exponent is stored above)
  hipLaunchKernelGGL(k_packed_header_clear, dim3(1), dim3(1), 0, s, expw);
  const int64_t n4 = n / 4;
  hipLaunchKernelGGL(k_exponent_max, dim3((unsigned)((n4 + kExpMaxGranules - 1) / kExpMaxGranules)), dim3(256), 0, s,
                     reinterpret_cast<const u32x4*>(x), n4, expw);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (mode == kStochastic) return quantize_packed_mode<kStochastic>(x, ngroups, m, seed, mant, expw, status, s);
  if (mode == kNearest) return quantize_packed_mode<kNearest>(x, ngroups, m, seed, mant, expw, status, s);
  return quantize_packed_mode<kTruncate>(x, ngroups, m, seed, mant, expw, status, s);
}

hipError_t launch_dequantize_packed(const uint8_t* mant, const uint8_t* exps, int64_t rows, int64_t len, int m,
                                    float* y, hipStream_t s) {
  const int64_t ngroups = rows * len / 16;
  const dim3 grid((unsigned)((ngroups + 255) / 256));
  const uint32_t* expw = reinterpret_cast<const uint32_t*>(exps);
  switch ((m + 1) / 2) {
    case 1: hipLaunchKernelGGL(k_dequantize_packed<1>, grid, dim3(256), 0, s, mant, expw, ngroups, m, y); break;
    case 2: hipLaunchKernelGGL(k_dequantize_packed<2>, grid, dim3(256), 0, s, mant, expw, ngroups, m, y); break;
    case 3: hipLaunchKernelGGL(k_dequantize_packed<3>, grid, dim3(256), 0, s, mant, expw, ngroups, m, y); break;
    default: hipLaunchKernelGGL(k_dequantize_packed<4>, grid, dim3(256), 0, s, mant, expw, ngroups, m, y); break;
  }
  return hipGetLastError();
}

}  // namespace fastbfp
