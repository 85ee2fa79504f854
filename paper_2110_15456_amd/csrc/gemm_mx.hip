// gemm_mx.hip -- the variable-precision BFP GEMM on gfx950's block-scaled MFMA
// (section III-B dot product; fMAC of section V-B).
//
// C[M][N] = A[M][K] * B[N][K]^T, both operands BFP with groups of 16 along K,
// stored as FP6 E2M3 chunk planes (value +-chunk/2) and one exponent byte per
// group.
//
// What the fMAC does per group pair -- g integer products, an adder tree, one
// exponent addition, conversion to FP and an FP32 accumulation -- is what one
// v_mfma_scale_f32_16x16x128_f8f6f4 does per 32-value block: the FP6 products
// of 4-bit chunks are exact, the block sum is scaled by 2^(sa-127) * 2^(sb-127)
// with the shared exponents as the E8M0 block scales, and the result is added
// to an FP32 accumulator.  The hardware block is 32 values and a BFP group is
// 16, so a block carries one group of the A row next to 16 zeros: the "even"
// instruction of a pair takes A = [group 2t | 0] and the "odd" one
// A = [0 | group 2t+1], each with that group's exponent as the block scale,
// while B's block holds both groups [2t | 2t+1] in the same registers and is
// scaled by the matching B exponent (selected with op_sel from a packed pair).
// FP6 has no NaN or Inf encodings, so the B values facing A's zeros are harmless.
//
// Variable precision (section V-B): an m-bit magnitude is one 4-bit chunk when
// m <= 4 and two when m > 4; each chunk-plane pair (ca, cb) is one pass of
// MFMAs over the group with the chunk's scale raised by 4 per chunk of
// significance (the paper lowers the exponent of the lower chunk instead; both
// give the same weights).  Passes per group pair = chunks(m_a) * chunks(m_b).
// The one remaining constant factor, 2^(4 - m_a - m_b) (the E2M3 halving of
// both operands and the (m-1) in the LSB), is applied exactly in the epilogue.
//
// Tiling: a 256-thread workgroup computes a 128x128 tile of C with four waves
// of 64x64 (4x4 MFMA tiles of 16x16, 64 FP32 accumulators per lane).  K is
// walked in slabs of 8 groups (128 values); each slab's codes and exponents
// are staged global -> registers -> LDS, and the next slab's global loads are
// in flight while the current slab's MFMAs run.
#include "bfp_device.h"
#include "launch.h"

namespace fastbfp {

namespace mx {
constexpr int BM = 128, BN = 128;
constexpr int KG = 8;            // groups per K slab
constexpr int ROWB = KG * 12;    // code bytes per row per plane per slab
constexpr int PITCH = 112;       // LDS row pitch: conflict-free 8-byte reads
constexpr int NT = 256;          // threads per workgroup
}  // namespace mx

// Staging registers for one operand tile of one slab.
template <int NP, int VEC>
struct TileRegs {
  static constexpr int CHUNKS = mx::BM * mx::ROWB / VEC;  // VEC-byte pieces per plane
  static constexpr int PER_T = CHUNKS / mx::NT;
  uint32_t v[NP][PER_T][VEC / 4];
  uint32_t e;  // 4 exponent bytes
};

// Load one slab of a 128-row operand tile: codes of planes [0, NP) and the
// exponents, zero-filled past row_end / past the last group.
template <int NP, int VEC>
__device__ __forceinline__ void load_tile(TileRegs<NP, VEC>& r, const uint8_t* __restrict__ mant,
                                          const uint8_t* __restrict__ exps, int64_t plane_stride, int row0,
                                          int row_end, int ng, int slab, int tid) {
  constexpr int PIECES_PER_ROW = mx::ROWB / VEC;
  const int gvalid = min(mx::KG, ng - slab * mx::KG);
  const int bvalid = gvalid * 12;
  const int64_t row_bytes = (int64_t)ng * 12;
#pragma unroll
  for (int u = 0; u < TileRegs<NP, VEC>::PER_T; ++u) {
    const int id = tid + u * mx::NT;
    const int row = id / PIECES_PER_ROW, part = id % PIECES_PER_ROW;
    const bool ok = (row0 + row < row_end) && (part * VEC < bvalid);
    const int64_t off = (int64_t)(row0 + row) * row_bytes + slab * mx::ROWB + part * VEC;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      if (VEC == 16) {
        uint4 x = make_uint4(0, 0, 0, 0);
        if (ok) x = *reinterpret_cast<const uint4*>(mant + p * plane_stride + off);
        r.v[p][u][0] = x.x;
        r.v[p][u][1] = x.y;
        r.v[p][u][2] = x.z;
        r.v[p][u][3] = x.w;
      } else {
        r.v[p][u][0] = ok ? *reinterpret_cast<const uint32_t*>(mant + p * plane_stride + off) : 0u;
      }
    }
  }
  // Exponents: 128 rows x 8 groups = 1024 bytes, 4 per thread.
  {
    const int row = tid >> 1, j0 = (tid & 1) * 4;
    uint32_t e = 0;
    if (row0 + row < row_end) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int gidx = slab * mx::KG + j0 + j;
        if (j0 + j < gvalid) e |= (uint32_t)exps[(int64_t)(row0 + row) * ng + gidx] << (8 * j);
      }
    }
    r.e = e;
  }
}

template <int NP, int VEC>
__device__ __forceinline__ void store_tile(const TileRegs<NP, VEC>& r, uint8_t* sm, uint8_t* se, int tid) {
  constexpr int PIECES_PER_ROW = mx::ROWB / VEC;
#pragma unroll
  for (int u = 0; u < TileRegs<NP, VEC>::PER_T; ++u) {
    const int id = tid + u * mx::NT;
    const int row = id / PIECES_PER_ROW, part = id % PIECES_PER_ROW;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      uint8_t* dst = sm + p * (mx::BM * mx::PITCH) + row * mx::PITCH + part * VEC;
      if (VEC == 16)
        *reinterpret_cast<uint4*>(dst) = make_uint4(r.v[p][u][0], r.v[p][u][1], r.v[p][u][2], r.v[p][u][3]);
      else
        *reinterpret_cast<uint32_t*>(dst) = r.v[p][u][0];
    }
  }
  *reinterpret_cast<uint32_t*>(se + (tid >> 1) * mx::KG + (tid & 1) * 4) = r.e;
}

// 24 code bytes (groups 2b and 2b+1 of one row) as six dwords.
__device__ __forceinline__ void read_frag(const uint8_t* p, uint32_t (&d)[6]) {
  const uint2 x0 = *reinterpret_cast<const uint2*>(p);
  const uint2 x1 = *reinterpret_cast<const uint2*>(p + 8);
  const uint2 x2 = *reinterpret_cast<const uint2*>(p + 16);
  d[0] = x0.x; d[1] = x0.y; d[2] = x1.x; d[3] = x1.y; d[4] = x2.x; d[5] = x2.y;
}

template <int NA, int NB, int VEC>
__global__ __launch_bounds__(256) void k_gemm_mx(const uint8_t* __restrict__ a_mant, const uint8_t* __restrict__ a_exp,
                                                 int64_t a_plane_stride, const uint8_t* __restrict__ b_mant,
                                                 const uint8_t* __restrict__ b_exp, int64_t b_plane_stride, int M,
                                                 int N, int ng, float scale, float* __restrict__ C, int64_t ldc,
                                                 int tiles_n) {
  __shared__ __attribute__((aligned(16))) uint8_t sA[NA * mx::BM * mx::PITCH];
  __shared__ __attribute__((aligned(16))) uint8_t sB[NB * mx::BN * mx::PITCH];
  __shared__ __attribute__((aligned(16))) uint8_t sEA[mx::BM * mx::KG];
  __shared__ __attribute__((aligned(16))) uint8_t sEB[mx::BN * mx::KG];

  const int tid = threadIdx.x;
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int row0 = tm * mx::BM, col0 = tn * mx::BN;
  const int wave = tid >> 6, lane = tid & 63;
  const int wr = wave >> 1, wc = wave & 1;
  const int lr = lane & 15, lb = lane >> 4;

  v4f acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  const int nslabs = (ng + mx::KG - 1) / mx::KG;
  TileRegs<NA, VEC> ra;
  TileRegs<NB, VEC> rb;
  load_tile<NA, VEC>(ra, a_mant, a_exp, a_plane_stride, row0, M, ng, 0, tid);
  load_tile<NB, VEC>(rb, b_mant, b_exp, b_plane_stride, col0, N, ng, 0, tid);

  for (int s = 0; s < nslabs; ++s) {
    store_tile<NA, VEC>(ra, sA, sEA, tid);
    store_tile<NB, VEC>(rb, sB, sEB, tid);
    __syncthreads();
    if (s + 1 < nslabs) {
      load_tile<NA, VEC>(ra, a_mant, a_exp, a_plane_stride, row0, M, ng, s + 1, tid);
      load_tile<NB, VEC>(rb, b_mant, b_exp, b_plane_stride, col0, N, ng, s + 1, tid);
    }
#pragma unroll
    for (int ca = 0; ca < NA; ++ca) {
      // A fragments of this wave's four 16-row tiles, with their exponent pairs.
      uint32_t af[4][6];
      int ea[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rl = wr * 64 + i * 16 + lr;
        read_frag(sA + ca * (mx::BM * mx::PITCH) + rl * mx::PITCH + lb * 24, af[i]);
        // +4 per chunk of significance, applied to both packed exponent bytes
        // (no carry: E <= 250).
        ea[i] = (int)*reinterpret_cast<const uint16_t*>(sEA + rl * mx::KG + 2 * lb) + 0x0404 * (NA - 1 - ca);
      }
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int cl = wc * 64 + j * 16 + lr;
          uint32_t bf[6];
          read_frag(sB + cb * (mx::BN * mx::PITCH) + cl * mx::PITCH + lb * 24, bf);
          const int eb = (int)*reinterpret_cast<const uint16_t*>(sEB + cl * mx::KG + 2 * lb) + 0x0404 * (NB - 1 - cb);
          const v8i bv = {(int)bf[0], (int)bf[1], (int)bf[2], (int)bf[3], (int)bf[4], (int)bf[5], 0, 0};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const v8i a_even = {(int)af[i][0], (int)af[i][1], (int)af[i][2], 0, 0, 0, 0, 0};
            const v8i a_odd = {0, 0, 0, (int)af[i][3], (int)af[i][4], (int)af[i][5], 0, 0};
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a_even, bv, acc[i][j], 2, 2, 0, ea[i], 0, eb);
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a_odd, bv, acc[i][j], 2, 2, 1, ea[i], 1, eb);
          }
        }
      }
    }
    __syncthreads();
  }

  // Epilogue: lane holds rows 4*lb + r, column lr of each 16x16 tile.
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = col0 + wc * 64 + j * 16 + lr;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = row0 + wr * 64 + i * 16 + lb * 4 + r;
        if (row < M && col < N) C[(int64_t)row * ldc + col] = acc[i][j][r] * scale;
      }
    }
}

template <int NA, int NB>
static hipError_t launch_mx_t(const uint8_t* a_mant, const uint8_t* a_exp, int64_t a_ps, const uint8_t* b_mant,
                              const uint8_t* b_exp, int64_t b_ps, int M, int N, int ng, float scale, float* C,
                              int64_t ldc, hipStream_t s) {
  const int tiles_m = (M + mx::BM - 1) / mx::BM, tiles_n = (N + mx::BN - 1) / mx::BN;
  const dim3 grid((unsigned)(tiles_m * tiles_n));
  const bool al16 = (reinterpret_cast<uintptr_t>(a_mant) % 16 == 0) && (reinterpret_cast<uintptr_t>(b_mant) % 16 == 0);
  if (ng % 4 == 0 && al16)  // every row starts 16-byte aligned: 16-byte global loads
    hipLaunchKernelGGL((k_gemm_mx<NA, NB, 16>), grid, dim3(mx::NT), 0, s, a_mant, a_exp, a_ps, b_mant, b_exp, b_ps,
                       M, N, ng, scale, C, ldc, tiles_n);
  else
    hipLaunchKernelGGL((k_gemm_mx<NA, NB, 4>), grid, dim3(mx::NT), 0, s, a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M,
                       N, ng, scale, C, ldc, tiles_n);
  return hipGetLastError();
}

hipError_t launch_gemm_mx(const uint8_t* a_mant, const uint8_t* a_exp, int a_planes, int na, const uint8_t* b_mant,
                          const uint8_t* b_exp, int b_planes, int nb, int64_t M, int64_t N, int64_t K, int g,
                          int scale_log2, float* C, int64_t ldc, hipStream_t s) {
  (void)a_planes;
  (void)b_planes;
  (void)g;
  if (M == 0 || N == 0) return hipSuccess;
  const int ng = (int)(K / 16);
  const int64_t a_ps = M * ng * 12, b_ps = N * ng * 12;
  const float scale = ldexpf(1.0f, scale_log2);
  if (na == 1 && nb == 1) return launch_mx_t<1, 1>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, s);
  if (na == 1 && nb == 2) return launch_mx_t<1, 2>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, s);
  if (na == 2 && nb == 1) return launch_mx_t<2, 1>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, s);
  return launch_mx_t<2, 2>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, s);
}

}  // namespace fastbfp
