// gemm_mx.h -- the variable-precision BFP GEMM on gfx950's block-scaled MFMA
// (section III-B dot product; fMAC of section V-B): the kernel template and
// its launcher, instantiated per operand format in gemm_mx_{11,12,21,22}.hip.
//
// C[M][N] = A[M][K] * B[N][K]^T, both operands BFP with groups of 16 (or 32)
// along K, stored as chunk planes (layout of include/fastbfp.h: FP4 or FP6
// codes of +-q/2 for m <= 4; for m = 5, 6 an FP6 plane of q >> 2 and a Lo2
// plane of q & 3; for m = 7, 8 FP6 planes of q >> 4 and q & 15) and one
// exponent byte per group.
//
// What the fMAC does per group pair -- g integer products, an adder tree, one
// exponent addition, conversion to FP and an FP32 accumulation -- is what one
// v_mfma_scale_f32_16x16x128_f8f6f4 does per 32-value block: the FP6/FP4
// products of chunks are exact, the block sum is scaled by 2^(sa-127) *
// 2^(sb-127) with the shared exponents as the E8M0 block scales, and the
// result is added to an FP32 accumulator.  The hardware block is 32 values
// and a BFP group 16: with one chunk plane per operand a lane's block carries
// one active group per operand, arranged so that it meets the other
// operand's active group and everything else meets zeros (FP6 and FP4 have
// no NaN or Inf encodings).  One instruction thus covers 4 groups of K, one
// per lane block; the operand formats of A and B are chosen per instruction.
//
// Variable precision (section V-B): chunk planes are passes over the group
// with the chunk's weight on the scale byte.  An operand split at 2 bits
// (m = 5, 6) fills a whole block with one group: +-(q >> 2)/2 in one half and
// +-(q & 3)/8 in the other, i.e. q/8, against the other operand's group
// repeated in both halves -- one MFMA per chunk plane of the other operand
// and no zero half.  The one remaining constant factor, 2^(4 - m_a - m_b)
// (the halving of both operands' codes and the (m-1) in the LSB), is applied
// exactly in the epilogue.
//
// Staging: a K slab is 8 groups.  In an FP6 plane each group occupies a
// 16-byte LDS slot filled by a direct buffer->LDS 12-byte load, which leaves
// the slot's last dword untouched (zeroed once); in an FP4 or Lo2 plane each
// slot holds a group pair (2p, 2p + 1), filled by one 16-byte load.  Lane
// block lb of K-step ks works on group 2 lb + ks, so such a lane reads one
// slot for both K-steps.  Slot order within a row is XOR-swizzled by the row
// so that the 16-byte fragment reads of 16 rows hit all 64 banks, while each
// load instruction still reads whole runs of consecutive rows.  With full
// slabs of groups of 16, the exponents of two slabs come in one 16-byte load
// per row into a buffer of their own.  Slabs are double buffered in two LDS
// objects: the loads of slab s+1 are issued right after the barrier that
// publishes slab s and have all of slab s's MFMAs to land.  Every load
// instruction costs the MFMA waves that issue it time, so the kernel issues
// no load it does not need (an L2 prefetch of slab s+2 cost more than it
// saved) and spreads a slab's loads between blocks of MFMAs.  A 256-thread
// workgroup (2x2 MFMA waves) computes a 256x256 tile (128 along an operand
// with two chunk planes, except 256 along A when both are split at 2 bits);
// tiles are ordered so that neighbours share panels in L2 on the same XCD.
#pragma once
#include "bfp_quant.h"

namespace fastbfp {

namespace mx {
#ifndef FASTBFP_MX_BM
#define FASTBFP_MX_BM 256
#endif
#ifndef FASTBFP_MX_BN
#define FASTBFP_MX_BN 256
#endif
#ifndef FASTBFP_MX_PIPE11
#define FASTBFP_MX_PIPE11 1
#endif
#ifndef FASTBFP_MX_SPREAD
#define FASTBFP_MX_SPREAD 8  // parts a slab's loads are spread over (explicit pipeline)
#endif
#ifndef FASTBFP_MX_X3
#define FASTBFP_MX_X3 1  // one MFMA for both cross products of two-chunk operands
#endif
#ifndef FASTBFP_MX_PIPE2
#define FASTBFP_MX_PIPE2 1
#endif
#ifndef FASTBFP_MX_GM
#define FASTBFP_MX_GM (CF::BM > CF::BN ? 4 : 8)
#endif
#ifndef FASTBFP_MX11_BM
#define FASTBFP_MX11_BM FASTBFP_MX_BM
#endif
#ifndef FASTBFP_MX11_BN
#define FASTBFP_MX11_BN FASTBFP_MX_BN
#endif
constexpr int KG = 8;            // groups per K slab (two MFMA K-steps)
// NA / NB: chunk planes of A / B read.  FA / FB: with one plane read, 1 if it
// holds FP4 codes (else FP6); with two, 1 if the operand is split at 2 bits
// (m = 5, 6: plane 0 FP6 codes of q >> 2, plane 1 a Lo2 plane of q & 3), 0 if
// at 4 (m = 7, 8: two FP6 planes).  FP4 and Lo2 planes take 8 bytes per
// group of 16 and are staged alike (16-byte LDS slots of group pairs).
// G: the operands' group size, 16 or 32.  A slab is 8 groups of 16 (KG) or
// 4 of 32: the mantissa planes of a g = 32 tensor are laid out exactly like
// those of a g = 16 tensor with twice the groups (each group is its two
// 16-value halves), so the staging works in 16-value halves either way; EK
// exponent bytes per row and slab.
// WGM x WGN: the MFMA wave grid (2 x 2: 256 accumulator registers per wave
// for a 256x256 tile).  A 2 x 4 grid (128 each, two waves per SIMD) compiles
// too; for the one-chunk kernels it was no faster (-4% to +2%).
template <int BM_, int BN_, int NA_, int NB_, int FA_, int FB_, int G_ = 16, int WGN_ = 2>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, NA = NA_, NB = NB_, FA = FA_, FB = FB_, G = G_;
  static constexpr int WGM = 2, WGN = WGN_, NW = WGM * WGN, NT = 64 * NW;  // MFMA wave grid, threads
  static constexpr int EK = KG * 16 / G;      // exponents per row and slab
  static constexpr int KSTEPS = G == 16 ? 2 : 1;  // MFMA K-steps per slab
  static_assert(G == 16 || G == 32, "group size 16 or 32");
  static constexpr int WM = BM / WGM, WN = BN / WGN;  // wave tile
  static constexpr int TM = WM / 16, TN = WN / 16;    // 16x16 MFMA tiles per wave
  // LDS bytes per row of a slab: 8 slots of one group (FP6) or 4 slots of a
  // group pair (FP4, Lo2), 16 bytes each.
  static constexpr int RA0 = (NA == 1 && FA) ? 64 : 128, RB0 = (NB == 1 && FB) ? 64 : 128;
  static constexpr int RA1 = FA ? 64 : 128, RB1 = FB ? 64 : 128;  // plane 1 (two planes read)
  static constexpr int OFF_A1 = BM * RA0;                        // A's plane 1
  static constexpr int OFF_B = OFF_A1 + (NA == 2 ? BM * RA1 : 0);
  static constexpr int OFF_B1 = OFF_B + BN * RB0;                // B's plane 1
  static constexpr int OFF_EA = OFF_B1 + (NB == 2 ? BN * RB1 : 0);
  static constexpr int OFF_EB = OFF_EA + BM * EK;
  static constexpr int SPARE = OFF_EB + BN * EK;  // EK bytes written by threads without an exponent row
  static constexpr int STAGE = SPARE + 16;
  static constexpr int EXP_ROWS_PER_T = (BM + BN + NT - 1) / NT;
  // Explicitly software-pipelined fragment reads (one chunk per operand);
  // otherwise the compiler schedules them.
  static constexpr bool PIPE = FASTBFP_MX_PIPE11 && NA == 1 && NB == 1 && G == 16;
  static_assert(TM * 16 * WGM == BM && TN * 16 * WGN == BN, "wave tiles cover the tile");
  static_assert((BM + BN) % 64 == 0 && BM % 64 == 0 && BN % 64 == 0,
                "loads split evenly over the waves; whole waves skip exponent rows past BM + BN");
  static_assert((BN / 16) % NW == 0 && (BM / 16) % NW == 0, "plane loads split evenly over the waves");
  static_assert(2 * STAGE <= 160 * 1024, "two stages fit in LDS");
};
// LDS offset of plane p of A / B within a stage, and its format: a_fp4 /
// b_fp4 (FP4 codes, read by the MFMA as FP4), a_lo2 / b_lo2 (a Lo2 plane,
// unpacked to FP6 codes), a_four / b_four (either: 8 bytes per group, staged
// in group-pair slots).
template <class CF> __device__ constexpr int a_plane(int p) { return p ? CF::OFF_A1 : 0; }
template <class CF> __device__ constexpr int b_plane(int p) { return p ? CF::OFF_B1 : CF::OFF_B; }
template <class CF> __device__ constexpr int a_fp4(int p) { return p == 0 && CF::NA == 1 && CF::FA; }
template <class CF> __device__ constexpr int b_fp4(int p) { return p == 0 && CF::NB == 1 && CF::FB; }
template <class CF> __device__ constexpr int a_lo2(int p) { return p == 1 && CF::NA == 2 && CF::FA; }
template <class CF> __device__ constexpr int b_lo2(int p) { return p == 1 && CF::NB == 2 && CF::FB; }
template <class CF> __device__ constexpr int a_four(int p) { return a_fp4<CF>(p) || a_lo2<CF>(p); }
template <class CF> __device__ constexpr int b_four(int p) { return b_fp4<CF>(p) || b_lo2<CF>(p); }
template <class CF> __device__ constexpr int a_kind(int p) {
  return a_fp4<CF>(p) ? kPlaneFP4 : a_lo2<CF>(p) ? kPlaneLo2 : kPlaneFP6;
}
template <class CF> __device__ constexpr int b_kind(int p) {
  return b_fp4<CF>(p) ? kPlaneFP4 : b_lo2<CF>(p) ? kPlaneLo2 : kPlaneFP6;
}
// Scale-byte offset of chunk plane p of an operand, relative to one FP6 or
// FP4 plane of codes of +-q/2 (the unit the epilogue's 2^(4 - m_a - m_b)
// assumes): split at 4 bits, the upper plane +-(q >> 4)/2 weighs 2^4 and the
// lower one 2^0; split at 2 bits, the upper plane +-(q >> 2)/2 weighs 2^2 and
// the lower one, unpacked to +-(q & 3)/8, 2^2 as well.
template <int NP, int SPLIT2> __device__ constexpr int plane_weight(int p) {
  return NP == 1 ? 0 : SPLIT2 ? 2 : (p == 0 ? 4 : 0);
}
}  // namespace mx

// Calls f(ic<0>{}), ..., f(ic<N-1>{}): a loop whose index is a constant
// expression (the MFMA's operand formats must be).
template <int I> struct ic { static constexpr int value = I; };
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(ic<I>{});
    static_for<N, I + 1>(f);
  }
}

// Workgroup id -> (tile_m, tile_n).  Dispatch places consecutive workgroup ids
// on consecutive XCDs; the remap gives each XCD a contiguous run of logical
// tiles, and logical tiles are walked in column-major groups of GROUP_M tile
// rows so that concurrently running workgroups share A and B panels in L2:
// the 32 workgroups an XCD runs at once cover GROUP_M x (32 / GROUP_M) tiles.
template <int GROUP_M>
__device__ __forceinline__ void tile_of(int bid, int nblocks, int tiles_m, int tiles_n, int& tm, int& tn) {
  constexpr int NXCD = 8;
  int lid = bid;
  if (nblocks % NXCD == 0) lid = (bid % NXCD) * (nblocks / NXCD) + bid / NXCD;
  const int per_group = GROUP_M * tiles_n;
  const int grp = lid / per_group;
  const int first_m = grp * GROUP_M;
  const int rows_in_group = min(tiles_m - first_m, GROUP_M);
  const int in = lid % per_group;
  tm = first_m + in % rows_in_group;
  tn = in / rows_in_group;
}

// Exponents of one slab for one row (EK bytes of ng_e per row), zero past
// the last group and for rows past the end.  dw: every row starts 4-byte
// aligned and holds a multiple of 4 exponents (K a multiple of 4 groups), so
// a slab's valid bytes are whole dwords: one dword load per 4 exponents
// instead of one byte load each (the ragged-K ResNet shape, K = 576).
template <int EK>
__device__ __forceinline__ uint2 load_exps(const uint8_t* __restrict__ exps, int row, int row_end, int ng, int slab,
                                           bool dw) {
  const bool rok = row < row_end;
  const int64_t base = (int64_t)(rok ? row : 0) * ng + slab * EK;
  const int gvalid = min(EK, ng - slab * EK);
  uint32_t w[2] = {0u, 0u};
  if (dw) {
#pragma unroll
    for (int k = 0; k < (EK + 3) / 4; ++k)
      if (rok && 4 * k < gvalid) w[k] = *reinterpret_cast<const uint32_t*>(exps + base + 4 * k);
    return make_uint2(w[0], w[1]);
  }
#pragma unroll
  for (int j = 0; j < EK; ++j) {
    const uint32_t b = exps[base + min(j, gvalid - 1)];
    w[j >> 2] |= ((rok && j < gvalid) ? b : 0u) << (8 * (j & 3));
  }
  return make_uint2(w[0], w[1]);
}

typedef __attribute__((address_space(3))) void lds_void;

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Buffer resource over [p, p + bytes): loads at offsets past the end read
// zero instead of faulting.  (Third dword: the gfx9 raw-buffer format.)
__device__ __forceinline__ rsrc_t make_rsrc(const uint8_t* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p), (short)0, (int)bytes, 0x00020000);
}

// Direct buffer->LDS loads of one slab of one FP6 operand plane: ROWS rows x
// 8 groups, i.e. ROWS * 8 / 64 load instructions of 64 slots, spread over the
// four waves.  The resource starts at the tile's first row and ends at its
// last valid one, so rows past the end read zero.  Instruction blk covers
// rows 8 blk .. 8 blk + 7; a wave's instructions all have the parity of its
// index, so the lane's part of the offset (row within the 8, swizzled group)
// is one register, lane_off.  RAGGED: groups past K get an offset past the
// resource and read zero.
// (Every loader issues its per-wave instructions u in [u0, u1) only, so that
// a slab's loads can be spread over the MFMAs of the previous slab.)
template <int NW, int ROWS>
constexpr int plane_loads(bool fp4) { return (fp4 ? ROWS / 16 : ROWS * mx::KG / 64) / NW; }  // per wave
template <int NW, int ROWS, bool RAGGED>
__device__ __forceinline__ void load_plane(uint8_t* lds_plane, rsrc_t rsrc, uint32_t lane_off, uint32_t row_bytes,
                                           int slab, bool g_ok, int wave, int u0, int u1) {
  constexpr int INSTR = ROWS * mx::KG / 64;
#pragma unroll
  for (int u = 0; u < INSTR / NW; ++u) {
    if (u < u0 || u >= u1) continue;
    const int blk = wave + NW * u;
    uint32_t off = lane_off + (uint32_t)blk * 8u * row_bytes + (uint32_t)slab * (mx::KG * 12);
    if (RAGGED && !g_ok) off = 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)(lds_plane + blk * 64 * 16), 12, off, 0, 0, 0);
  }
}

// The same for an FP4 plane: a slab row is 4 group pairs of 16 bytes, one
// 16-byte load each, so an instruction covers rows 16 blk .. 16 blk + 15 and
// every wave's lane offset is the same register.  RAGGED: pairs starting past
// K read zero; the second group of a pair that straddles K reads whatever
// follows, which meets a zero exponent (a product scale of 2^-254 or less
// leaves an FP32 accumulator unchanged).
template <int NW, int ROWS, bool RAGGED>
__device__ __forceinline__ void load_plane4(uint8_t* lds_plane, rsrc_t rsrc, uint32_t lane_off, uint32_t row_bytes,
                                            int slab, bool p_ok, int wave, int u0, int u1) {
  constexpr int INSTR = ROWS / 16;
#pragma unroll
  for (int u = 0; u < INSTR / NW; ++u) {
    if (u < u0 || u >= u1) continue;
    const int blk = wave + NW * u;
    uint32_t off = lane_off + (uint32_t)blk * 16u * row_bytes + (uint32_t)slab * (mx::KG * 8);
    if (RAGGED && !p_ok) off = 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)(lds_plane + blk * 64 * 16), 16, off, 0, 0, 0);
  }
}

// Direct buffer->LDS loads of one full slab of exponents (EK bytes per row,
// as DPR = EK / 4 dwords) for ROWS rows: row r lands at lds_exps + EK r.
// lane_off is (lane / DPR) * ng + (lane % DPR) * 4.  Instructions past the
// last (when they do not split evenly over the four waves) go through the
// zero-length resource rnull into the sink.
template <int NW, int ROWS, int EK>
constexpr int exps_loads() { return (ROWS * (EK / 4) / 64 + NW - 1) / NW; }  // per wave
template <int NW, int ROWS, int EK>
__device__ __forceinline__ void load_exps_lds(uint8_t* lds_exps, rsrc_t rsrc, rsrc_t rnull, uint8_t* sink,
                                              uint32_t lane_off, int ng, int slab, int wave, int u0, int u1) {
  constexpr int DPR = EK / 4, INSTR = ROWS * DPR / 64;
#pragma unroll
  for (int u = 0; u < (INSTR + NW - 1) / NW; ++u) {
    if (u < u0 || u >= u1) continue;
    const int blk = wave + NW * u;
    const bool ok = INSTR % NW == 0 || blk < INSTR;
    const uint32_t off = lane_off + (uint32_t)blk * (64u / DPR) * (uint32_t)ng + (uint32_t)slab * EK;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ok ? rsrc : rnull, (lds_void*)(ok ? lds_exps + blk * 256 : sink), 4, off,
                                             0, 0, 0);
  }
}

// Direct loads of the exponents of one slab pair (EK = 8 bytes for each of
// two slabs: 16 contiguous bytes per row) for ROWS rows, one row per lane:
// row r lands at lds_x + 16 r.  lane_off is lane * ng.  When the instructions
// do not split evenly over the four waves, the extra waves repeat the last one
// (the same bytes to the same place).
template <int NW, int ROWS>
constexpr int pair_loads() { return (ROWS / 64 + NW - 1) / NW; }  // per wave
template <int NW, int ROWS>
__device__ __forceinline__ void load_exps_pair(uint8_t* lds_x, rsrc_t rsrc, uint32_t lane_off, int ng, int pair,
                                               int wave, int u0, int u1) {
  constexpr int INSTR = ROWS / 64;
#pragma unroll
  for (int u = 0; u < (INSTR + NW - 1) / NW; ++u) {
    if (u < u0 || u >= u1) continue;
    const int blk = min(wave + NW * u, INSTR - 1);
    const uint32_t off = lane_off + (uint32_t)blk * 64u * (uint32_t)ng + (uint32_t)pair * 16u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)(lds_x + blk * 1024), 16, off, 0, 0, 0);
  }
}

// MFMA operands of one K-step from the 16-byte slots read for A (x) and B (y).
// A lane's block is values 0..15 (half 0) and 16..31 (half 1).  An FP6 slot
// has its group in half 0 (dwords 0-2; dword 3 is the slot's zero dword and
// A's upper registers are zero); an FP4 slot has the pair (2 lb, 2 lb + 1) in
// dwords 0-1 and 2-3, the active group 2 lb + ks in half ks.  The two active
// groups must meet, and every other product must meet a zero:
//   FP6 x FP6: A has zeros in half 1, B as read;
//   FP4 x FP4: A as read, B keeps its active half and zeroes the other;
//   FP6 x FP4: B's active group moves to half 0 (A's half 1 is zero);
//   FP4 x FP6: A's active group moves to half 0, B's half 1 is zeroed.
template <int FA, int FB>
__device__ __forceinline__ v8i op_a(const u32x4& x, int ks) {
  const v4i& v = reinterpret_cast<const v4i&>(x);
  if constexpr (!FA) return v8i{v[0], v[1], v[2], v[3], 0, 0, 0, 0};
  else if constexpr (FB) return __builtin_shufflevector(v, v, 0, 1, 2, 3, -1, -1, -1, -1);
  else return ks ? __builtin_shufflevector(v, v, 2, 3, -1, -1, -1, -1, -1, -1)
                 : __builtin_shufflevector(v, v, 0, 1, 2, 3, -1, -1, -1, -1);
}
template <int FA, int FB>
__device__ __forceinline__ v8i op_b(const u32x4& y, int ks) {
  const v4i& v = reinterpret_cast<const v4i&>(y);
  if constexpr (!FB && !FA) return __builtin_shufflevector(v, v, 0, 1, 2, 3, -1, -1, -1, -1);
  else if constexpr (!FB) return v8i{v[0], v[1], v[2], v[3], 0, 0, 0, 0};
  else if constexpr (!FA)
    return ks ? __builtin_shufflevector(v, v, 2, 3, -1, -1, -1, -1, -1, -1)
              : __builtin_shufflevector(v, v, 0, 1, 2, 3, -1, -1, -1, -1);
  else return ks ? v8i{0, 0, v[2], v[3], 0, 0, 0, 0} : v8i{v[0], v[1], 0, 0, 0, 0, 0, 0};
}
// The MFMA operand format code of a plane: FP6 E2M3 = 2, FP4 E2M1 = 4 (as a
// template constant: the intrinsic needs a literal).
template <int FP4> struct mfma_fmt { static constexpr int value = FP4 ? 4 : 2; };

#ifndef FASTBFP_MX_TIED
#define FASTBFP_MX_TIED 1
#endif
typedef int v6i __attribute__((ext_vector_type(6)));
// acc += the block-scaled product of one K-step (A format FA, B format FB,
// block scales sa / sb).  The intrinsic's instruction form does not tie the
// result to the accumulator input, so with 256 accumulator registers live the
// register allocator moves accumulators between registers every slab (several
// hundred accumulator moves per 128 MFMAs).  The tied form below keeps every
// accumulator in one register quad for the whole loop.  Written as inline
// assembly the instruction is invisible to the compiler's hazard tracking, so
// it carries its own wait states: two for a VALU write of an operand just
// before it; the accumulators are only ever written by these instructions
// inside the loop (back-to-back accumulation into the same registers needs no
// wait), and mma_drain() covers the reads after it.  The statement is not
// volatile: a volatile one would also keep the scheduler from moving fragment
// reads across it.
// SA / SB: which byte of sa / sb is the block scale (the instruction's
// op_sel bits for its second / first source): 0 for the low byte, 1 for the
// next, so that one 16-bit exponent read serves both K-steps of a slab.
#define FASTBFP_MFMA_ASM(SEL, CB, BG) \
  "s_nop 1\n\tv_mfma_scale_f32_16x16x128_f8f6f4 %0, %1, %2, %0, %3, %4 " SEL " cbsz:" #CB " blgp:" #BG
#define FASTBFP_MFMA_SEL(CB, BG, BOP, AOP)                                                                      \
  {                                                                                                            \
    if constexpr (SA == 0 && SB == 0)                                                                          \
      asm(FASTBFP_MFMA_ASM("op_sel_hi:[0,0,0]", CB, BG) : "+a"(acc) : "v"(BOP), "v"(AOP), "v"(sb), "v"(sa));    \
    else if constexpr (SA == 0)                                                                                \
      asm(FASTBFP_MFMA_ASM("op_sel:[1,0,0] op_sel_hi:[0,0,0]", CB, BG)                                         \
          : "+a"(acc) : "v"(BOP), "v"(AOP), "v"(sb), "v"(sa));                                                 \
    else if constexpr (SB == 0)                                                                                \
      asm(FASTBFP_MFMA_ASM("op_sel:[0,1,0] op_sel_hi:[0,0,0]", CB, BG)                                         \
          : "+a"(acc) : "v"(BOP), "v"(AOP), "v"(sb), "v"(sa));                                                 \
    else                                                                                                       \
      asm(FASTBFP_MFMA_ASM("op_sel:[1,1,0] op_sel_hi:[0,0,0]", CB, BG)                                         \
          : "+a"(acc) : "v"(BOP), "v"(AOP), "v"(sb), "v"(sa));                                                 \
  }
template <int FA, int FB, int SA = 0, int SB = 0>
__device__ __forceinline__ void mma(v4f& acc, const v8i& a, const v8i& b, int sa, int sb) {
  static_assert(SA == 0 || SA == 1, "scale byte 0 or 1");
  static_assert(SB == 0 || SB == 1, "scale byte 0 or 1");
  // B's fragment is the instruction's first operand and A's the second, so
  // the result is the tile of C transposed: a lane's four accumulators are
  // four consecutive columns of one row of C (see the epilogue).
#if FASTBFP_MX_TIED
  const v4i a4 = __builtin_shufflevector(a, a, 0, 1, 2, 3);
  const v4i b4 = __builtin_shufflevector(b, b, 0, 1, 2, 3);
  const v6i a6 = __builtin_shufflevector(a, a, 0, 1, 2, 3, 4, 5);
  const v6i b6 = __builtin_shufflevector(b, b, 0, 1, 2, 3, 4, 5);
  if constexpr (FA && FB)
    FASTBFP_MFMA_SEL(4, 4, b4, a4)
  else if constexpr (FA)
    FASTBFP_MFMA_SEL(2, 4, b6, a4)
  else if constexpr (FB)
    FASTBFP_MFMA_SEL(4, 2, b4, a6)
  else
    FASTBFP_MFMA_SEL(2, 2, b6, a6)
#else
  acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b, a, acc, mfma_fmt<FB>::value, mfma_fmt<FA>::value, SB, sb,
                                                         SA, sa);
#endif
}
#undef FASTBFP_MFMA_SEL
#undef FASTBFP_MFMA_ASM
// Wait states between the last MFMA and any other read of its accumulators
// (a 16x16x128 block-scaled MFMA needs at most 19).  Every accumulator then
// passes through an empty statement that comes after them (volatile
// statements keep their order), so that every later read -- including copies
// the register allocator places at block boundaries, which no scheduling
// barrier orders -- depends on it.
template <int TM, int TN>
__device__ __forceinline__ void mma_drain(v4f (&acc)[TM][TN]) {
#if FASTBFP_MX_TIED
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) asm volatile("" : "+a"(acc[i][j]));
#endif
}

// Where the epilogue puts C: FP32 rows (QNCH = 0), or BFP with groups of 16
// along each row of C (the next GEMM's K) at c_m bits in QNCH chunk planes --
// the converter of section V-C applied to the FP32 results in the epilogue.
struct OutBFP {
  uint8_t* mant0;
  uint8_t* mant1;
  uint8_t* exps;
  uint32_t* status;
  int m, mode;
  int four;  // one plane: it holds FP4 codes (m <= 2); two planes: plane 1 is a Lo2 plane (m = 5, 6)
  uint32_t key0, key1;
};

template <class CF, bool EXP_FULL, int QNCH>
__global__ __launch_bounds__(CF::NT) void k_gemm_mx(const uint8_t* __restrict__ a_mant, const uint8_t* __restrict__ a_exp,
                                                 int64_t a_plane_stride, const uint8_t* __restrict__ b_mant,
                                                 const uint8_t* __restrict__ b_exp, int64_t b_plane_stride, int M,
                                                 int N, int ng, float scale, float* __restrict__ C, int64_t ldc,
                                                 int tiles_m, int tiles_n, OutBFP qo) {
  constexpr int TM = CF::TM, TN = CF::TN, NA = CF::NA, NB = CF::NB, FA = CF::FA, FB = CF::FB;
  // Groups of 16 with full slabs (XP): the exponents of slab pair p (slabs 2p
  // and 2p + 1: 16 contiguous bytes per row) come in one 16-byte load per row,
  // with slab 2p's mantissas, into their own buffer xe[p % 2] -- a quarter of
  // the load instructions of per-slab dword loads.  The stages then hold only mantissas (and the converted output's
  // strips).  Otherwise each stage holds its slab's exponents.
  constexpr bool XP = EXP_FULL && CF::G == 16;
  constexpr bool X3 = FASTBFP_MX_X3 && NA == 2 && NB == 2 && CF::G == 16 && !CF::PIPE && !FA && !FB;
  // an operand split at 2 bits fills whole MFMA blocks (groups of 16)
  constexpr bool COMB = CF::G == 16 && ((NA == 2 && FA) || (NB == 2 && FB));
  // explicit pipeline of the two-chunk loop (operands split at 4 bits)
  constexpr bool PIPE2 = FASTBFP_MX_PIPE2 && (NA == 2 || NB == 2) && CF::G == 16 && !X3 && !COMB;
  constexpr int NTHR = CF::NT;
  constexpr int STRIP_BYTES = QNCH ? CF::NW * 16 * (CF::WN + 4) * 4 : 0;
  constexpr int SB = XP ? (CF::OFF_EA > STRIP_BYTES ? CF::OFF_EA : STRIP_BYTES) : CF::STAGE;
  constexpr int XEB = XP ? (CF::BM + CF::BN) * 16 : 16;
  // Two stages (and two exponent buffers) as separate LDS objects: the
  // compiler then knows that the direct loads into one do not alias the
  // fragment reads of the other, and does not wait for the next slab's loads
  // before computing on this one.
  __shared__ __attribute__((aligned(16))) uint8_t stage0[SB];
  __shared__ __attribute__((aligned(16))) uint8_t stage1[SB];
  __shared__ __attribute__((aligned(16))) uint8_t xe0[XEB];
  __shared__ __attribute__((aligned(16))) uint8_t xe1[XEB];
  __shared__ __attribute__((aligned(16))) uint8_t sink[CF::NW * 256];  // destination of padding loads, never read
  const int tid = threadIdx.x;
  int tm, tn;
  tile_of<FASTBFP_MX_GM>(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int row0 = tm * CF::BM, col0 = tn * CF::BN;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;  // wave index in an SGPR
  const int wr = wave / CF::WGN, wc = wave % CF::WGN;
  const int lr = lane & 15, lb = lane >> 4;

  // Zero both stages once: the slot dwords that the 12-byte loads never write
  // are the zero padding of the FP6 operands.
  for (int i = tid; i < SB / 16; i += NTHR) {
    reinterpret_cast<u32x4*>(stage0)[i] = u32x4{0u, 0u, 0u, 0u};
    reinterpret_cast<u32x4*>(stage1)[i] = u32x4{0u, 0u, 0u, 0u};
  }
  __syncthreads();

  v4f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  const int nslabs = (ng + mx::KG - 1) / mx::KG;
  auto exp_row = [&](int k, const uint8_t*& src, int& grow, int& gend, int& lds) {
    const int r = tid + k * CF::NT;
    const bool is_a = r < CF::BM;
    const int rr = is_a ? r : r - CF::BM;
    src = is_a ? a_exp : b_exp;
    grow = (is_a ? row0 : col0) + rr;
    gend = is_a ? M : N;
    lds = (is_a ? CF::OFF_EA : CF::OFF_EB) + rr * CF::EK;
  };
  // Per-tile resources and the lane parts of the load offsets.  Row bytes in
  // HBM: 12 per group in an FP6 plane, 8 in an FP4 plane.
  const uint32_t rb6 = (uint32_t)ng * 12u, rb4 = (uint32_t)ng * 8u;
  auto rbytes = [&](int fp4) { return fp4 ? rb4 : rb6; };
  const int a_rows = min(CF::BM, M - row0), b_rows = min(CF::BN, N - col0);
  rsrc_t ra[NA], rb[NB];
#pragma unroll
  for (int p = 0; p < NA; ++p) {
    const uint32_t r = rbytes(mx::a_four<CF>(p));
    ra[p] = make_rsrc(a_mant + p * a_plane_stride + (int64_t)row0 * r, (uint32_t)a_rows * r);
  }
#pragma unroll
  for (int p = 0; p < NB; ++p) {
    const uint32_t r = rbytes(mx::b_four<CF>(p));
    rb[p] = make_rsrc(b_mant + p * b_plane_stride + (int64_t)col0 * r, (uint32_t)b_rows * r);
  }
  // FP6: lane -> (row lane / 8 of the instruction's 8, slot lane % 8), loading
  // the group that the row's swizzle puts in that slot.
  // FP4: lane -> (row lane / 4 of the instruction's 16, slot lane % 4), the
  // slot of row r holding pair slot ^ ((r >> 2) & 3).
  const int p_lane = (lane & 3) ^ ((lane >> 4) & 3);
  const uint32_t m4_lane_off = (uint32_t)(lane >> 2) * rb4 + (uint32_t)p_lane * 16u;
  // Exponents: ng_e per row (one per group of G).
  const int ng_e = ng * 16 / CF::G;
  const bool exp_dw = (ng_e & 3) == 0 && (reinterpret_cast<uintptr_t>(a_exp) & 3) == 0 &&
                      (reinterpret_cast<uintptr_t>(b_exp) & 3) == 0;
  const rsrc_t rea = make_rsrc(a_exp + (int64_t)row0 * ng_e, (uint32_t)(a_rows * ng_e));
  const rsrc_t reb = make_rsrc(b_exp + (int64_t)col0 * ng_e, (uint32_t)(b_rows * ng_e));
  constexpr int DPR = CF::EK / 4;
  const uint32_t e_lane_off = (uint32_t)(lane / DPR) * (uint32_t)ng_e + (uint32_t)(lane % DPR) * 4u;
  const uint32_t x_lane_off = (uint32_t)lane * (uint32_t)ng_e;

  // Exponents: with full slabs, direct loads like the mantissas.  Otherwise
  // through registers (zeros are needed past K): this thread handles rows
  // tid + k*NT of the BM + BN exponent rows, A's first, loaded with the slab's
  // mantissas and written to LDS after the MFMAs.
  //
  // Branch-free: with live false (no next slab) the direct loads go through
  // zero-length resources and the register loads reread slab `slab`, so that
  // a whole step is one basic block and the MFMAs cannot be moved past the
  // next step's barrier.
  const rsrc_t rnull = make_rsrc(a_exp, 0u);
  // A slab's per-wave load instructions in a fixed order (A's planes, B's
  // planes, then the exponents of A and B); part `part` of `nparts` issues the
  // instructions [part * NLOAD / nparts, (part + 1) * NLOAD / nparts) of that
  // order (the register exponent loads of the ragged path go with part 0).
  // XP: the exponent loads are those of a slab pair, issued only where xe
  // (their destination) is given.
  constexpr int LA0 = plane_loads<CF::NW, CF::BM>(mx::a_four<CF>(0));
  constexpr int LA1 = NA == 2 ? plane_loads<CF::NW, CF::BM>(mx::a_four<CF>(1)) : 0;
  constexpr int LB0 = plane_loads<CF::NW, CF::BN>(mx::b_four<CF>(0));
  constexpr int LB1 = NB == 2 ? plane_loads<CF::NW, CF::BN>(mx::b_four<CF>(1)) : 0;
  constexpr int LEA = XP ? pair_loads<CF::NW, CF::BM>() : EXP_FULL ? exps_loads<CF::NW, CF::BM, CF::EK>() : 0;
  constexpr int LEB = XP ? pair_loads<CF::NW, CF::BN>() : EXP_FULL ? exps_loads<CF::NW, CF::BN, CF::EK>() : 0;
  constexpr int OFS[6] = {0, LA0, LA0 + LA1, LA0 + LA1 + LB0, LA0 + LA1 + LB0 + LB1, LA0 + LA1 + LB0 + LB1 + LEA};
  constexpr int NLOAD = OFS[5] + LEB;
  auto issue = [&](uint8_t* stage, int slab, bool live, uint2 (&e)[CF::EXP_ROWS_PER_T], uint8_t* xe, int part = 0,
                   int nparts = 1) {
    const int vw = wave;
    const int g_lane = (lane & 7) ^ ((4 * (vw & 1) + (lane >> 4)) & 7);
    const uint32_t m_lane_off = (uint32_t)(lane >> 3) * rb6 + (uint32_t)g_lane * 12u;
    const int lo = part * NLOAD / nparts, hi = (part + 1) * NLOAD / nparts;
    // the range of loader q's own instructions that falls in [lo, hi)
    auto u0 = [&](int q) { return lo > OFS[q] ? lo - OFS[q] : 0; };
    auto u1 = [&](int q) { return hi - OFS[q]; };
    if (!EXP_FULL && part == 0) {
#pragma unroll
      for (int k = 0; k < CF::EXP_ROWS_PER_T; ++k) {
        e[k] = make_uint2(0u, 0u);
        if (tid + k * CF::NT >= CF::BM + CF::BN) break;
        const uint8_t* src;
        int grow, gend, lds;
        exp_row(k, src, grow, gend, lds);
        e[k] = load_exps<CF::EK>(src, grow, gend, ng_e, slab, exp_dw);
      }
    }
    const bool g_ok = slab * mx::KG + g_lane < ng;
    const bool p_ok = slab * mx::KG + 2 * p_lane < ng;
#pragma unroll
    for (int p = 0; p < NA; ++p) {
      if (mx::a_four<CF>(p))
        load_plane4<CF::NW, CF::BM, !EXP_FULL>(stage + mx::a_plane<CF>(p), live ? ra[p] : rnull, m4_lane_off, rb4, slab, p_ok,
                                       vw, u0(p), u1(p));
      else
        load_plane<CF::NW, CF::BM, !EXP_FULL>(stage + mx::a_plane<CF>(p), live ? ra[p] : rnull, m_lane_off, rb6, slab, g_ok,
                                      vw, u0(p), u1(p));
    }
#pragma unroll
    for (int p = 0; p < NB; ++p) {
      if (mx::b_four<CF>(p))
        load_plane4<CF::NW, CF::BN, !EXP_FULL>(stage + mx::b_plane<CF>(p), live ? rb[p] : rnull, m4_lane_off, rb4, slab, p_ok,
                                       vw, u0(2 + p), u1(2 + p));
      else
        load_plane<CF::NW, CF::BN, !EXP_FULL>(stage + mx::b_plane<CF>(p), live ? rb[p] : rnull, m_lane_off, rb6, slab, g_ok,
                                      vw, u0(2 + p), u1(2 + p));
    }
    if constexpr (XP) {
      if (xe) {
        load_exps_pair<CF::NW, CF::BM>(xe, live ? rea : rnull, x_lane_off, ng_e, slab / 2, vw, u0(4), u1(4));
        load_exps_pair<CF::NW, CF::BN>(xe + CF::BM * 16, live ? reb : rnull, x_lane_off, ng_e, slab / 2, vw, u0(5), u1(5));
      }
    } else if constexpr (EXP_FULL) {
      load_exps_lds<CF::NW, CF::BM, CF::EK>(stage + CF::OFF_EA, live ? rea : rnull, rnull, sink + vw * 256, e_lane_off,
                                    ng_e, slab, vw, u0(4), u1(4));
      load_exps_lds<CF::NW, CF::BN, CF::EK>(stage + CF::OFF_EB, live ? reb : rnull, rnull, sink + vw * 256, e_lane_off,
                                    ng_e, slab, vw, u0(5), u1(5));
    }
  };
  // Branch-free, so that it stays behind the MFMAs in one basic block: rows
  // past BM + BN write to a spare 8 bytes after the exponents.
  auto put_exps = [&](uint8_t* stage, const uint2 (&e)[CF::EXP_ROWS_PER_T]) {
    if constexpr (!EXP_FULL) {
#pragma unroll
      for (int k = 0; k < CF::EXP_ROWS_PER_T; ++k) {
        const uint8_t* src;
        int grow, gend, lds;
        exp_row(k, src, grow, gend, lds);
        if (tid + k * CF::NT >= CF::BM + CF::BN) lds = CF::SPARE;
        if constexpr (CF::EK == 8) *reinterpret_cast<uint2*>(stage + lds) = e[k];
        else *reinterpret_cast<uint32_t*>(stage + lds) = e[k].x;
      }
    }
  };

  uint2 e_regs[CF::EXP_ROWS_PER_T];
  if (nslabs > 0) {
    issue(stage0, 0, true, e_regs, XP ? xe0 : nullptr);
    put_exps(stage0, e_regs);
  }

  // One slab: publish slab s (its direct loads and exponent writes, from
  // every wave), start the loads of slab s + 1 into the other stage (which
  // held slab s - 1, finished by every wave), compute slab s, then write the
  // next slab's exponents.
  // XP: xcur is the exponent buffer of slab s's pair, xnext (or null) the one
  // that receives the next pair with slab s + 1, half = s & 1.  Otherwise the
  // exponents are in cur.
  auto step = [&](const uint8_t* cur, uint8_t* nxt, int s, const uint8_t* xcur, uint8_t* xnext, int half) {
    // Every wave's direct loads into cur must have landed before any wave
    // passes the barrier (the compiler only orders them against this wave's
    // own LDS reads): wait for them explicitly (s_waitcnt 0: vmcnt, expcnt
    // and lgkmcnt zero).  The empty asm statements keep the compiler from
    // moving memory accesses across the barrier.
    __builtin_amdgcn_s_waitcnt(0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    const bool more = s + 1 < nslabs;
    const int nslab = more ? s + 1 : s;
    // With an FP6 operand the loads go out in NPART parts between the blocks
    // of MFMAs, so that the wave keeps issuing MFMAs while the load path works
    // through them (FP6 x FP6: 10-14% faster, two
    // chunk planes 1-12%).  FP4 x FP4 slabs have half the load instructions,
    // and there issuing them all at once, here, is faster (their latency, not
    // their issue, is what shows).
    // (The same holds for groups of 32, whose slabs are one K-step: there
    // spreading was 1-4% slower.)
    constexpr int NPART = ((NA == 1 && NB == 1 && FA && FB) || CF::G == 32)
                              ? 1
                              : (NLOAD < FASTBFP_MX_SPREAD ? NLOAD : FASTBFP_MX_SPREAD);
    // The parts go after MFMA blocks spread over the first half of the slab's
    // nblk blocks (part k after block k * (nblk / 2) / NPART), each fenced so
    // that the compiler keeps it there.
    auto issue_after = [&](int b, int nblk) {
#pragma unroll
      for (int k = 0; k < NPART; ++k)
        if (NPART > 1 && k * (nblk / 2) / NPART == b) {
          issue(nxt, nslab, more, e_regs, xnext, k, NPART);
          __builtin_amdgcn_sched_barrier(0);
        }
    };
    if constexpr (NPART == 1) issue(nxt, nslab, more, e_regs, xnext);
    __builtin_amdgcn_sched_barrier(0);
    // Fragment addresses.  Row rl = wr*WM + 16*i + lr has the FP6 swizzle
    // ((rl >> 1) & 7) = ((lr >> 1) & 7) and the FP4 swizzle ((rl >> 2) & 3) =
    // ((lr >> 2) & 3) (WM and 16*i are multiples of 16), so for a K-step the
    // slot column is a lane constant and fragment i / j sits at an immediate
    // offset of 16 rows.  A lane's block scale is the exponent byte of its row
    // and group: one byte read.
    const int swz6 = (lr >> 1) & 7, swz4 = (lr >> 2) & 3;
    // (Every address is one offset from the stage base, which keeps the
    // accesses attributable to the stage object.)
    const int a_r = wr * CF::WM + lr, b_r = wc * CF::WN + lr;
    // the exponent of lane block lb's group in K-step ks: group 2 lb + ks
    // (G = 16) or lb (G = 32, one K-step)
    // (XP: rows of 16 bytes in the pair buffer, this slab's 8 at half * 8.)
    constexpr int ER = XP ? 16 : CF::EK;  // exponent bytes per row
    const int ea_lane = (XP ? 0 : CF::OFF_EA) + a_r * ER + (XP ? 8 * half : 0) + (CF::G == 16 ? 2 * lb : lb);
    const int eb_lane =
        (XP ? 16 * CF::BM : CF::OFF_EB) + b_r * ER + (XP ? 8 * half : 0) + (CF::G == 16 ? 2 * lb : lb);
    // Byte offset of the 16-byte slot of row tile t, K-step ks, in a plane of
    // format fp4 starting at plane_off, for a lane of row r.
    auto slot_addr = [&](int plane_off, int fp4, int r, int t, int ks) {
      return fp4 ? plane_off + (r + 16 * t) * 64 + ((lb ^ swz4) * 16)
                 : plane_off + (r + 16 * t) * 128 + (((2 * lb + ks) ^ swz6) * 16);
    };
    auto rd = [&](int off) { return *reinterpret_cast<const u32x4*>(cur + off); };
    // G = 32: the operand is the whole group, with no padding -- the FP4 slot
    // as read, the 12 bytes of each of the two FP6 half-group slots, or a Lo2
    // slot's two halves unpacked to FP6 codes.  kind: kPlaneFP6 / FP4 / Lo2.
    auto op32 = [&](int kind, int plane_off, int r, int t) -> v8i {
      const u32x4 x = rd(slot_addr(plane_off, kind != kPlaneFP6, r, t, 0));
      if (kind == kPlaneFP4) return v8i{(int)x[0], (int)x[1], (int)x[2], (int)x[3], 0, 0, 0, 0};
      if (kind == kPlaneLo2) {
        uint32_t t0, t1, t2, u0, u1, u2;
        lo2_unpack(x[0], x[1], t0, t1, t2);
        lo2_unpack(x[2], x[3], u0, u1, u2);
        return v8i{(int)t0, (int)t1, (int)t2, (int)u0, (int)u1, (int)u2, 0, 0};
      }
      const u32x4 y = rd(slot_addr(plane_off, 0, r, t, 1));
      return v8i{(int)x[0], (int)x[1], (int)x[2], (int)y[0], (int)y[1], (int)y[2], 0, 0};
    };
    if constexpr (CF::PIPE) {
      // Software pipeline.  A block is the TN MFMAs of one A fragment (row
      // tile i) against the B fragments of K-step ks; a phase is one K-step,
      // TM blocks.  Each block reads the next block's A fragment and a share
      // of the next phase's B fragments, and a scheduling barrier closes it,
      // so that about two blocks' fragments are live at a time.
      constexpr int BPP = TM;           // blocks per phase
      constexpr int NPH = CF::KSTEPS;   // phases per slab
      v8i bf[2][TN], af[2];
      // A lane's exponents of both K-steps (groups 2 lb and 2 lb + 1) are
      // adjacent bytes: one 16-bit read per fragment in the first phase, and
      // each MFMA takes its K-step's byte of it as the block scale.
      int be[TN], ae[TM];
      auto rd16 = [&](int off) { return (int)*reinterpret_cast<const uint16_t*>(xcur + off); };
      auto read_b = [&](int ks, int j) {
        bf[ks & 1][j] = op_b<FA, FB>(rd(slot_addr(CF::OFF_B, FB, b_r, j, ks)), ks);
        if (ks == 0) be[j] = rd16(eb_lane + j * 16 * ER);
      };
      auto read_a = [&](int blk) {
        const int ks = blk / BPP, i = blk % BPP;
        af[blk & 1] = op_a<FA, FB>(rd(slot_addr(0, FA, a_r, i, ks)), ks);
        if (ks == 0) ae[i] = rd16(ea_lane + i * 16 * ER);
      };
#pragma unroll
      for (int j = 0; j < TN; ++j) read_b(0, j);
      read_a(0);
      // An FP4 slot serves both K-steps; the empty asm statements (here and
      // at the phase boundary) keep the compiler from merging the two phases'
      // reads of it, which would hold every raw fragment for the whole slab.
      if constexpr ((FA || FB) && NPH == 2) asm volatile("" ::: "memory");
#pragma unroll
      for (int blk = 0; blk < NPH * BPP; ++blk) {
        const int ph = blk / BPP, bi = blk % BPP, i = blk % TM;
        if constexpr ((FA || FB) && NPH == 2)
          if (blk == BPP) asm volatile("" ::: "memory");
        if (blk + 1 < NPH * BPP) read_a(blk + 1);
        if (ph + 1 < NPH) {
#pragma unroll
          for (int j = bi * TN / BPP; j < (bi + 1) * TN / BPP; ++j) read_b(ph + 1, j);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          if (ph == 0)
            mma<FA, FB, 0, 0>(acc[i][j], af[blk & 1], bf[0][j], ae[i], be[j]);
          else
            mma<FA, FB, 1, 1>(acc[i][j], af[blk & 1], bf[1][j], ae[i], be[j]);
        }
        issue_after(blk, NPH * BPP);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else if constexpr (CF::G == 32) {
      // Compiler-scheduled, one K-step: per B chunk the B fragments, then each
      // A fragment against them.
      static_for<NB>([&](auto cbc) {
        constexpr int cb = decltype(cbc)::value, fb = mx::b_fp4<CF>(cb);
        v8i bv[TN];
        int eb[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          bv[j] = op32(mx::b_kind<CF>(cb), mx::b_plane<CF>(cb), b_r, j);
          eb[j] = (int)xcur[eb_lane + j * 16 * ER] + mx::plane_weight<NB, FB>(cb);  // the chunk's weight
        }
        static_for<NA>([&](auto cac) {
          constexpr int ca = decltype(cac)::value, fa = mx::a_fp4<CF>(ca);
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const v8i av = op32(mx::a_kind<CF>(ca), mx::a_plane<CF>(ca), a_r, i);
            const int ea = (int)xcur[ea_lane + i * 16 * ER] + mx::plane_weight<NA, FA>(ca);
#pragma unroll
            for (int j = 0; j < TN; ++j)
              mma<fa, fb>(acc[i][j], av, bv[j], ea, eb[j]);
            issue_after((cb * NA + ca) * TM + i, NB * NA * TM);
          }
        });
      });
    } else if constexpr (COMB) {
      // An operand split at 2 bits (q = 4 (q >> 2) + (q & 3)) fills a whole
      // 32-value MFMA block with one group of 16: the codes of +-(q >> 2)/2
      // (its FP6 plane) in half 0 and those of +-(q & 3)/8 (its Lo2 plane,
      // unpacked) in half 1, i.e. q/8 per value.  The other operand's group
      // is repeated in both halves, one block per chunk plane of it.  So a
      // fragment pair takes one MFMA per chunk plane of the repeated operand
      // and no block holds zeros: (6,6) 2 MFMAs per group of 16 where
      // separate chunk passes over half-empty blocks take 4, (6, m <= 4) 1
      // where they take 2.  The combined operand C is A when A is split at 2
      // bits, else B; D is the other.  The scale bytes carry the chunk
      // weights: 2 for the combined block (q/8 against the unit q/2) plus the
      // repeated plane's.
      //
      // Software pipeline: a block is one C fragment (K-step ks, fragment c)
      // against every D fragment and plane (TD * ND MFMAs).  Each block first
      // reads the next block's C slots (a Lo2 slot holds both K-steps' groups
      // and is read once), and the blocks of K-step 0 read a share of K-step
      // 1's D slots; D's repeated operands are built from the raw slots at
      // the start of each K-step; a scheduling barrier closes each block.
      constexpr bool CA = NA == 2 && FA;
      constexpr int TC = CA ? TM : TN, TD = CA ? TN : TM, ND = CA ? NB : NA;
      constexpr int C0 = CA ? mx::a_plane<CF>(0) : mx::b_plane<CF>(0);  // FP6 plane of q >> 2
      constexpr int C1 = CA ? mx::a_plane<CF>(1) : mx::b_plane<CF>(1);  // Lo2 plane of q & 3
      constexpr int DP0 = CA ? mx::b_plane<CF>(0) : mx::a_plane<CF>(0);
      constexpr int DP1 = CA ? mx::b_plane<CF>(1) : mx::a_plane<CF>(1);
      constexpr int DK0 = CA ? mx::b_kind<CF>(0) : mx::a_kind<CF>(0);
      constexpr int DK1 = CA ? mx::b_kind<CF>(1) : mx::a_kind<CF>(1);
      constexpr int FD = CA ? FB : FA;
      const int c_r = CA ? a_r : b_r, d_r = CA ? b_r : a_r;
      const int c_e = CA ? ea_lane : eb_lane, d_e = CA ? eb_lane : ea_lane;
      u32x4 dr[2][ND][TD];  // D's raw slots per K-step (an FP4 / Lo2 slot only in [0])
      int de[TD];
      v8i dd[ND][TD];       // D's repeated operands of the current K-step
      u32x4 ch[2], cl[TC];  // C's FP6 slots (per block) and Lo2 slots (per fragment)
      // Exponents: both K-steps' bytes of a fragment in one 16-bit read (in
      // K-step 0); each MFMA takes its K-step's byte (the weights added to
      // both bytes stay below 256 for exponents up to 250).
      int ce[TC];
      auto rd16 = [&](int off) { return (int)*reinterpret_cast<const uint16_t*>(xcur + off); };
      auto read_d = [&](int ks, int t) {
        static_for<ND>([&](auto pc) {
          constexpr int p = decltype(pc)::value, k = p == 0 ? DK0 : DK1, off = p == 0 ? DP0 : DP1;
          if (k == kPlaneFP6 || ks == 0) dr[k == kPlaneFP6 ? ks : 0][p][t] = rd(slot_addr(off, k != kPlaneFP6, d_r, t, ks));
        });
        if (ks == 0) de[t] = rd16(d_e + t * 16 * ER);
      };
      auto read_c = [&](int blk) {
        const int ks = blk / TC, c = blk % TC;
        ch[blk & 1] = rd(slot_addr(C0, 0, c_r, c, ks));
        if (ks == 0) {
          cl[c] = rd(slot_addr(C1, 1, c_r, c, 0));
          ce[c] = rd16(c_e + c * 16 * ER);
        }
      };
      // the group repeated in both halves, from a raw slot of a plane of kind k
      auto make_dup = [&](int k, const u32x4& x, int ks) -> v8i {
        if (k == kPlaneFP6) return v8i{(int)x[0], (int)x[1], (int)x[2], (int)x[0], (int)x[1], (int)x[2], 0, 0};
        if (k == kPlaneFP4)
          return v8i{(int)x[2 * ks], (int)x[2 * ks + 1], (int)x[2 * ks], (int)x[2 * ks + 1], 0, 0, 0, 0};
        uint32_t t0, t1, t2;
        lo2_unpack(x[2 * ks], x[2 * ks + 1], t0, t1, t2);
        return v8i{(int)t0, (int)t1, (int)t2, (int)t0, (int)t1, (int)t2, 0, 0};
      };
#pragma unroll
      for (int t = 0; t < TD; ++t) read_d(0, t);
      read_c(0);
      static_for<2 * TC>([&](auto bc) {
        constexpr int blk = decltype(bc)::value, ks = blk / TC, c = blk % TC;
        if constexpr (c == 0) {
#pragma unroll
          for (int t = 0; t < TD; ++t)
            static_for<ND>([&](auto pc) {
              constexpr int p = decltype(pc)::value, k = p == 0 ? DK0 : DK1;
              dd[p][t] = make_dup(k, dr[k == kPlaneFP6 ? ks : 0][p][t], ks);
            });
        }
        if constexpr (blk + 1 < 2 * TC) read_c(blk + 1);
        if constexpr (ks == 0) {
#pragma unroll
          for (int t = c * TD / TC; t < (c + 1) * TD / TC; ++t) read_d(1, t);
        }
        uint32_t t0, t1, t2;
        lo2_unpack(cl[c][2 * ks], cl[c][2 * ks + 1], t0, t1, t2);
        const u32x4& h = ch[blk & 1];
        const v8i cv = v8i{(int)h[0], (int)h[1], (int)h[2], (int)t0, (int)t1, (int)t2, 0, 0};
        const int e_c = ce[c];
        // plane-major: consecutive MFMAs accumulate into different tiles
        static_for<ND>([&](auto pc) {
          constexpr int p = decltype(pc)::value;
          constexpr int W = 2 + mx::plane_weight<ND, FD>(p);
          constexpr int dfp4 = (p == 0 ? DK0 : DK1) == kPlaneFP4;
          constexpr int W1 = 0x0101 * ((W + 1) / 2), W0 = 0x0101 * (W / 2);  // added to both bytes
#pragma unroll
          for (int t = 0; t < TD; ++t) {
            if constexpr (CA)
              mma<0, dfp4, ks, ks>(acc[c][t], cv, dd[p][t], e_c + W1, de[t] + W0);
            else
              mma<dfp4, 0, ks, ks>(acc[t][c], dd[p][t], cv, de[t] + W1, e_c + W0);
          }
        });
        issue_after(blk, 2 * TC);
        __builtin_amdgcn_sched_barrier(0);
      });
    } else if constexpr (PIPE2) {
      // Software pipeline of the two-chunk kernels (an operand in two chunk
      // planes, groups of 16).  A block is one A fragment (row tile i, chunk
      // plane ca) against the B fragments of every chunk plane: NB TN MFMAs;
      // a K-step is the blocks (i, 0 .. NA-1) for each i.  Each block first
      // reads the next block's A fragment (and with a row's first plane its
      // exponent byte, which serves every plane), and the blocks of K-step 0
      // also read a share of K-step 1's B fragments, so that every LDS read
      // has a block of MFMAs to land in; the next slab's load parts go
      // between blocks, and a scheduling
      // barrier closes each block.  A B plane of FP4 slots holds the group
      // pairs of both K-steps and is read once.
      constexpr int BPK = NA * TM;   // blocks per K-step
      constexpr int NBLK = 2 * BPK;  // blocks per slab
      u32x4 yb[2][NB][TN], xa[2];
      int ebr[2][TN], ear[2];
      auto read_b = [&](int ks, int j) {
        static_for<NB>([&](auto cbc) {
          constexpr int cb = decltype(cbc)::value, fb = mx::b_fp4<CF>(cb);
          if (!fb || ks == 0) yb[ks][cb][j] = rd(slot_addr(mx::b_plane<CF>(cb), fb, b_r, j, fb ? 0 : ks));
        });
        ebr[ks][j] = (int)xcur[eb_lane + j * 16 * ER + ks];
      };
      auto read_a = [&](int blk) {
        const int ks = blk / BPK, i = (blk % BPK) / NA, ca = blk % NA;
        xa[blk & 1] = rd(slot_addr(mx::a_plane<CF>(ca), mx::a_fp4<CF>(ca), a_r, i, ks));
        if (ca == 0) ear[(blk / NA) & 1] = (int)xcur[ea_lane + i * 16 * ER + ks];
      };
#pragma unroll
      for (int j = 0; j < TN; ++j) read_b(0, j);
      read_a(0);
      static_for<NBLK>([&](auto bc) {
        constexpr int blk = decltype(bc)::value;
        constexpr int ks = blk / BPK, i = (blk % BPK) / NA, ca = blk % NA;
        constexpr int fa = mx::a_fp4<CF>(ca);
        if constexpr (blk + 1 < NBLK) read_a(blk + 1);
        if constexpr (ks == 0) {
#pragma unroll
          for (int j = blk * TN / BPK; j < (blk + 1) * TN / BPK; ++j) read_b(1, j);
        }
        const int ea = ear[(blk / NA) & 1] + 4 * (NA - 1 - ca);  // +4 per chunk of significance
        static_for<NB>([&](auto cbc) {
          constexpr int cb = decltype(cbc)::value, fb = mx::b_fp4<CF>(cb);
          const v8i av = op_a<fa, fb>(xa[blk & 1], ks);
#pragma unroll
          for (int j = 0; j < TN; ++j)
            mma<fa, fb>(acc[i][j], av, op_b<fa, fb>(yb[fb ? 0 : ks][cb][j], ks), ea,
                        ebr[ks][j] + 4 * (NB - 1 - cb));
        });
        issue_after(blk, NBLK);
        __builtin_amdgcn_sched_barrier(0);
      });
    } else if constexpr (X3) {
      // Both operands in two chunk planes: the cross products (A's upper
      // chunk with B's lower, A's lower with B's upper) carry the same weight,
      // one chunk of significance, and with groups of 16 each fills only half
      // of a 32-value block, so the two share one MFMA: A's block holds its
      // upper group then its lower one, B's block its lower then its upper,
      // both as FP6, and the scales are those of the cross weight.  Three
      // MFMAs per fragment pair and K-step instead of four.
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        u32x4 y0[TN], y1[TN];
        int eb[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          y0[j] = rd(slot_addr(mx::b_plane<CF>(0), FB, b_r, j, ks));
          y1[j] = rd(slot_addr(mx::b_plane<CF>(1), 0, b_r, j, ks));
          eb[j] = (int)xcur[eb_lane + j * 16 * ER + ks];
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const u32x4 x0 = rd(slot_addr(mx::a_plane<CF>(0), FA, a_r, i, ks));
          const u32x4 x1 = rd(slot_addr(mx::a_plane<CF>(1), 0, a_r, i, ks));
          const int ea = (int)xcur[ea_lane + i * 16 * ER + ks];
          const v8i a0 = op_a<FA, FB>(x0, ks), a1 = op_a<0, 0>(x1, ks);
#pragma unroll
          for (int j = 0; j < TN; ++j) mma<FA, FB>(acc[i][j], a0, op_b<FA, FB>(y0[j], ks), ea + 4, eb[j] + 4);
#pragma unroll
          for (int j = 0; j < TN; ++j) mma<0, 0>(acc[i][j], a1, op_b<0, 0>(y1[j], ks), ea, eb[j]);
          const v8i ax = v8i{(int)x0[0], (int)x0[1], (int)x0[2], (int)x1[0], (int)x1[1], (int)x1[2], 0, 0};
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const v8i bx = v8i{(int)y1[j][0], (int)y1[j][1], (int)y1[j][2], (int)y0[j][0], (int)y0[j][1],
                               (int)y0[j][2], 0, 0};
            mma<0, 0>(acc[i][j], ax, bx, ea + 4, eb[j]);
          }
          issue_after(ks * TM + i, 2 * TM);
        }
      }
    } else {
      // Compiler-scheduled: per K-step, the B fragments of every chunk plane,
      // then each A fragment (read once, its exponent byte once) against
      // them.  A block is one A fragment's MFMAs; the load parts go between
      // blocks.
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        u32x4 y[NB][TN];
        int eb[NB][TN];
        static_for<NB>([&](auto cbc) {
          constexpr int cb = decltype(cbc)::value, fb = mx::b_fp4<CF>(cb);
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            y[cb][j] = rd(slot_addr(mx::b_plane<CF>(cb), fb, b_r, j, ks));
            // +4 per chunk of significance
            eb[cb][j] = (int)xcur[eb_lane + j * 16 * ER + ks] + 4 * (NB - 1 - cb);
          }
        });
        static_for<NA>([&](auto cac) {
          constexpr int ca = decltype(cac)::value, fa = mx::a_fp4<CF>(ca);
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const u32x4 x = rd(slot_addr(mx::a_plane<CF>(ca), fa, a_r, i, ks));
            const int ea = (int)xcur[ea_lane + i * 16 * ER + ks] + 4 * (NA - 1 - ca);
            static_for<NB>([&](auto cbc) {
              constexpr int cb = decltype(cbc)::value, fb = mx::b_fp4<CF>(cb);
              const v8i av = op_a<fa, fb>(x, ks);
#pragma unroll
              for (int j = 0; j < TN; ++j) mma<fa, fb>(acc[i][j], av, op_b<fa, fb>(y[cb][j], ks), ea, eb[cb][j]);
            });
            issue_after((ks * NA + ca) * TM + i, 2 * NA * TM);
          }
        });
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    put_exps(nxt, e_regs);  // stale but harmless after the last slab
  };
  int s = 0;
  if constexpr (XP) {
    // Unrolled by four: slab s in stage s % 2, its exponents in xe[(s / 2) % 2].
    for (; s + 4 <= nslabs; s += 4) {
      step(stage0, stage1, s, xe0, nullptr, 0);
      step(stage1, stage0, s + 1, xe0, xe1, 1);
      step(stage0, stage1, s + 2, xe1, nullptr, 0);
      step(stage1, stage0, s + 3, xe1, xe0, 1);
    }
    if (s < nslabs) step(stage0, stage1, s, xe0, nullptr, 0);
    if (s + 1 < nslabs) step(stage1, stage0, s + 1, xe0, xe1, 1);
    if (s + 2 < nslabs) step(stage0, stage1, s + 2, xe1, nullptr, 0);
  } else {
    for (; s + 2 <= nslabs; s += 2) {
      step(stage0, stage1, s, stage0, nullptr, 0);
      step(stage1, stage0, s + 1, stage1, nullptr, 1);
    }
    if (s < nslabs) step(stage0, stage1, s, stage0, nullptr, 0);
  }
  mma_drain(acc);

  // Epilogue: lane holds row lr, columns 4*lb .. 4*lb + 3 of each 16x16
  // tile (B was the MFMAs' first operand): one 16-byte store per tile where
  // C's rows are 16-byte aligned and the four columns exist.
  if constexpr (QNCH == 0) {
    const bool vec = (ldc & 3) == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int row = row0 + wr * CF::WM + i * 16 + lr;
      if (row >= M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = col0 + wc * CF::WN + j * 16 + 4 * lb;
        float* p = C + (int64_t)row * ldc + col;
        if (vec && col + 3 < N) {
          *reinterpret_cast<float4*>(p) =
              make_float4(acc[i][j][0] * scale, acc[i][j][1] * scale, acc[i][j][2] * scale, acc[i][j][3] * scale);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (col + r < N) p[r] = acc[i][j][r] * scale;
        }
      }
    }
  } else {
    // Converted output.  A row group of C (16 consecutive columns) is spread
    // over the four lane blocks, so each wave stages one 16-row
    // strip of its tile at a time in LDS (the stage memory, free now), and
    // then every lane converts whole groups with the quantizer's converter:
    // the same FP32 values and the same noise addressing (gid = the group's
    // index in the output exponent array) as converting C separately.
    constexpr int SROW = CF::WN + 4;  // strip row stride in floats (padding spreads the banks)
    static_assert(CF::NW * 16 * SROW * 4 <= SB, "a strip per wave fits in one stage");
    // Every wave is done with the stages, and no direct load (the last
    // steps' no-op loads included) can still write them.
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    float* strip = reinterpret_cast<float*>(stage0) + wave * (16 * SROW);
    const int ngN = N / 16;
    bool bad = false;
    // Convert and store one group: FOUR as OutBFP::four.
    auto convert = [&](auto f0c, const uint32_t (&b)[16], int64_t gid) {
      constexpr bool FOUR = decltype(f0c)::value;
      constexpr int P0 = (QNCH == 1 && FOUR) ? kPlaneFP4 : kPlaneFP6;
      constexpr int P1 = (QNCH == 2 && FOUR) ? kPlaneLo2 : kPlaneFP6;
      uint32_t w[QNCH][16 * 6 / 32];
      uint32_t E, s_lo, s_hi;
      bool nonfinite;
      const uint32_t m = (uint32_t)qo.m;
      if (qo.mode == kStochastic)
        quantize_group<16, kStochastic, QNCH, false, P0, P1>(b, m, (uint64_t)gid, qo.key0, qo.key1, w, E, nonfinite,
                                                                s_lo, s_hi);
      else if (qo.mode == kNearest)
        quantize_group<16, kNearest, QNCH, false, P0, P1>(b, m, (uint64_t)gid, qo.key0, qo.key1, w, E, nonfinite,
                                                             s_lo, s_hi);
      else
        quantize_group<16, kTruncate, QNCH, false, P0, P1>(b, m, (uint64_t)gid, qo.key0, qo.key1, w, E, nonfinite,
                                                              s_lo, s_hi);
      qo.exps[gid] = (uint8_t)E;
      store_plane<16, P0 != kPlaneFP6>(qo.mant0, gid, w[0]);
      if (QNCH == 2) store_plane<16, P1 != kPlaneFP6>(qo.mant1, gid, w[QNCH - 1]);
      bad |= nonfinite;
    };
    // The strips, with the output format fixed outside the loop (one copy of
    // the loop per format keeps the register pressure of one converter).
    auto strips = [&](auto f0c) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int j = 0; j < TN; ++j)
        *reinterpret_cast<float4*>(&strip[lr * SROW + j * 16 + 4 * lb]) =
            make_float4(acc[i][j][0] * scale, acc[i][j][1] * scale, acc[i][j][2] * scale, acc[i][j][3] * scale);
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's strip writes are done
      __builtin_amdgcn_wave_barrier();
      for (int gi = lane; gi < 16 * TN; gi += 64) {
        const int rr = gi / TN, jj = gi % TN;
        const int row = row0 + wr * CF::WM + i * 16 + rr;
        const int gcol = (col0 + wc * CF::WN) / 16 + jj;
        uint32_t b[16];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float4 v = *reinterpret_cast<const float4*>(&strip[rr * SROW + jj * 16 + 4 * k]);
          b[4 * k] = __float_as_uint(v.x);
          b[4 * k + 1] = __float_as_uint(v.y);
          b[4 * k + 2] = __float_as_uint(v.z);
          b[4 * k + 3] = __float_as_uint(v.w);
        }
        if (row < M && gcol < ngN) convert(f0c, b, (int64_t)row * ngN + gcol);
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // the strip's reads are done before the next strip overwrites it
      __builtin_amdgcn_wave_barrier();
    }
    };
    if (qo.four) strips(ic<1>{});
    else strips(ic<0>{});
    if (qo.status && bad) atomicOr(qo.status, 1u);
  }
}

template <class CF, bool EXP_FULL>
static hipError_t launch_mx_v(const uint8_t* a_mant, const uint8_t* a_exp, int64_t a_ps, const uint8_t* b_mant,
                              const uint8_t* b_exp, int64_t b_ps, int M, int N, int ng, float scale, float* C,
                              int64_t ldc, const OutBFP* qo, hipStream_t s) {
  const int tiles_m = (M + CF::BM - 1) / CF::BM, tiles_n = (N + CF::BN - 1) / CF::BN;
  const dim3 grid((unsigned)(tiles_m * tiles_n)), block(CF::NT);
  if (!qo)
    hipLaunchKernelGGL((k_gemm_mx<CF, EXP_FULL, 0>), grid, dim3(CF::NT), 0, s, a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N,
                       ng, scale, C, ldc, tiles_m, tiles_n, OutBFP{});
  else if (qo->m > 4)
    hipLaunchKernelGGL((k_gemm_mx<CF, EXP_FULL, 2>), grid, block, 0, s, a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N,
                       ng, scale, C, ldc, tiles_m, tiles_n, *qo);
  else
    hipLaunchKernelGGL((k_gemm_mx<CF, EXP_FULL, 1>), grid, block, 0, s, a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N,
                       ng, scale, C, ldc, tiles_m, tiles_n, *qo);
  return hipGetLastError();
}

// One operand-format combination: NA / NB planes read, FA / FB plane 0 of A /
// B in FP4, G the group size.  a_ps / b_ps: byte offset of plane 1 (the stored
// plane 0's size); ng: 16-value halves (K / 16) per row.
template <int NA, int NB, int FA, int FB, int G>
hipError_t launch_mx_t(const uint8_t* a_mant, const uint8_t* a_exp, int64_t a_ps, const uint8_t* b_mant,
                       const uint8_t* b_exp, int64_t b_ps, int M, int N, int ng, float scale, float* C, int64_t ldc,
                       const OutBFP* qo, hipStream_t s) {
  // The tile shrinks along an operand with two chunk planes so that two LDS
  // stages fit in 160 KB; with FP4 upper planes on both sides (192 bytes per
  // slab row instead of 256) A keeps 256 rows.
  constexpr bool WIDE22 = NA == 2 && NB == 2 && FA && FB;
  using CF = mx::Cfg<(NA == 1 && NB == 1) ? FASTBFP_MX11_BM : (NA == 1 || WIDE22) ? FASTBFP_MX_BM : FASTBFP_MX_BM / 2,
                     (NA == 1 && NB == 1) ? FASTBFP_MX11_BN : NB == 1 ? FASTBFP_MX_BN : FASTBFP_MX_BN / 2, NA, NB, FA,
                     FB, G>;
  auto al = [](const void* p, uintptr_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; };
  // direct exponent loads need full slabs and 4-byte aligned exponent rows
  const bool ef = ng % mx::KG == 0 && al(a_exp, 4) && al(b_exp, 4);  // (K a multiple of 128 either way)
  if (ef) return launch_mx_v<CF, true>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, qo, s);
  return launch_mx_v<CF, false>(a_mant, a_exp, a_ps, b_mant, b_exp, b_ps, M, N, ng, scale, C, ldc, qo, s);
}

// One chunk plane per operand, groups of 16, on a BM x BN tile smaller than
// the default 256 x 256: for GEMMs with few columns (a 64-wide tile wastes no
// MFMAs on padding when N = 64) or too few 256 x 256 tiles to give every CU
// work (the ResNet im2col shapes: 98 to 196 tiles on 256 CUs).  C in FP32, or
// converted to BFP in the epilogue (qo).
template <int BM, int BN, int FA, int FB>
hipError_t launch_mx_11_tile(const uint8_t* a_mant, const uint8_t* a_exp, const uint8_t* b_mant,
                             const uint8_t* b_exp, int M, int N, int ng, float scale, float* C, int64_t ldc,
                             const OutBFP* qo, hipStream_t s) {
  using CF = mx::Cfg<BM, BN, 1, 1, FA, FB, 16>;
  auto al = [](const void* p, uintptr_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; };
  const bool ef = ng % mx::KG == 0 && al(a_exp, 4) && al(b_exp, 4);
  if (ef) return launch_mx_v<CF, true>(a_mant, a_exp, 0, b_mant, b_exp, 0, M, N, ng, scale, C, ldc, qo, s);
  return launch_mx_v<CF, false>(a_mant, a_exp, 0, b_mant, b_exp, 0, M, N, ng, scale, C, ldc, qo, s);
}

#define FASTBFP_MX11_TILE_DECLARE(BM, BN, FA, FB)                                                              \
  extern template hipError_t launch_mx_11_tile<BM, BN, FA, FB>(const uint8_t*, const uint8_t*, const uint8_t*, \
                                                               const uint8_t*, int, int, int, float, float*,   \
                                                               int64_t, const OutBFP*, hipStream_t);
#define FASTBFP_MX11_TILE_INSTANTIATE(BM, BN, FA, FB)                                                         \
  template hipError_t launch_mx_11_tile<BM, BN, FA, FB>(const uint8_t*, const uint8_t*, const uint8_t*,       \
                                                        const uint8_t*, int, int, int, float, float*, int64_t, \
                                                        const OutBFP*, hipStream_t);

#define FASTBFP_MX_DECLARE(NA, NB, FA, FB, G)                                                          \
  extern template hipError_t launch_mx_t<NA, NB, FA, FB, G>(const uint8_t*, const uint8_t*, int64_t,       \
                                                            const uint8_t*, const uint8_t*, int64_t, int, int, \
                                                            int, float, float*, int64_t, const OutBFP*,         \
                                                            hipStream_t);
#define FASTBFP_MX_INSTANTIATE(NA, NB, FA, FB, G)                                                           \
  template hipError_t launch_mx_t<NA, NB, FA, FB, G>(const uint8_t*, const uint8_t*, int64_t, const uint8_t*, \
                                                     const uint8_t*, int64_t, int, int, int, float, float*,     \
                                                     int64_t, const OutBFP*, hipStream_t);

}  // namespace fastbfp
