"""GPU parity of bfp_gemm (block-scaled MFMA) and bfp_gemm_group_partials
(int8 MFMA) with the oracle.  Group partials must be bit-exact; every FP32
output must satisfy |C_gpu - C_oracle| <= 1e-6 * sum_G |T_G| (the oracle sums
in double).  Operands are quantized on both sides from the same FP32 inputs,
and their quantized bytes are checked bit-exact first."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2110_15456_amd as fb
from paper_2110_15456_amd import synth
from gpu_util import announce, check_quantize, chunk_drops, THREADS

pytestmark = pytest.mark.gpu
TOL = 1e-6


def operands(xa, xb, m_a_st, m_b_st, a_axis=-1, b_axis=-1, mode_a="nearest", mode_b="nearest", seed=0,
             rows=None, g=16):
    """GPU BFP tensors plus the oracle's own quantization of the same inputs."""
    A, qa, ea = check_quantize(xa, a_axis, g, m_a_st, mode_a, seed=seed, rows=None)
    B, qb, eb = check_quantize(xb, b_axis, g, m_b_st, mode_b, seed=seed + 1)
    return A, B, (qa, ea), (qb, eb)


def check_gemm(A, B, oa, ob, m_a=None, m_b=None, rows=None, partials=False, tile=None):
    m_a = A.m if m_a is None else m_a
    m_b = B.m if m_b is None else m_b
    C = fb.gemm(A, B, m_a, m_b, tile=tile)
    torch.cuda.synchronize()
    Cg = C.cpu().numpy().astype(np.float64)
    idx = np.arange(A.rows) if rows is None else np.asarray(rows)
    Co, S = oracle.gemm(oa[0], oa[1], A.m, ob[0], ob[1], B.m, g=A.g, m_a=m_a, m_b=m_b, rows=idx, threads=THREADS)
    err = np.abs(Cg[idx] - Co)
    ratio = err / np.maximum(S, 1e-300)
    worst = np.unravel_index(np.argmax(ratio), ratio.shape)
    assert np.all(err <= TOL * S), "max err/sum|T| = %.3g at %s (gpu %r oracle %r)" % (
        ratio[worst], worst, Cg[idx][worst], Co[worst])
    if partials:
        P = fb.gemm_group_partials(A, B, m_a, m_b).cpu().numpy()
        Po = oracle.group_partials(oa[0], A.m, ob[0], B.m, g=A.g, m_a=m_a, m_b=m_b, rows=idx)
        assert np.array_equal(P[:, idx, :].astype(np.int64), Po)
    return float(ratio.max())


@pytest.mark.parametrize("K", [16, 32])
def test_tiny_all_precisions(K):
    """M = N = 4, K = 16 and 32: every stored (m_a, m_b) in 1..8, and the
    low-chunk drop where an operand has two chunks; C and the int32 partials."""
    x = synth.draw("normal", (8, K), 300 + K)
    for am in range(1, 9):
        for bm in range(1, 9):
            announce("gemm tiny K=%d stored (%d,%d)" % (K, am, bm))
            A, B, oa, ob = operands(x[:4], x[4:], am, bm)
            for m_a in chunk_drops(am):
                for m_b in chunk_drops(bm):
                    check_gemm(A, B, oa, ob, m_a, m_b, partials=True)


def test_config1_256():
    """A 256x256 and B 256x256 from N(0,1) (seed 0, one stream); A at m=2
    along K, B [K, N] quantized along axis 0 (its K) at m=4; round to nearest."""
    a, b = synth.gemm_pair_normal(256, 256, 256, seed=0)
    announce("gemm config 256^3 (2,4)")
    A, B, oa, ob = operands(a, b, 2, 4, a_axis=-1, b_axis=0)
    check_gemm(A, B, oa, ob, partials=True)


SHAPES = [(300, 200, 592), (257, 129, 576), (129, 257, 144), (1, 1, 16), (5, 300, 4096), (64, 64, 2048)]
# Every kernel variant: the operand formats of A x B, where m = 1, 2 is one FP4
# plane, 3, 4 one FP6 plane, 5, 6 an FP6 + Lo2 pair (split at 2 bits: whole
# MFMA blocks) and 7, 8 two FP6 planes (split at 4 bits).
PAIRS = [(2, 2), (2, 4), (4, 2), (4, 4),          # one plane each
         (1, 5), (2, 8), (4, 6), (3, 7),          # one x two
         (5, 2), (6, 3), (8, 1), (7, 4),          # two x one
         (6, 6), (6, 8), (8, 6), (8, 8)]          # two x two


@pytest.mark.parametrize("shape", SHAPES)
def test_ragged_shapes(shape):
    M, N, K = shape
    xa = synth.draw("half_normal", (M, K), M + K)
    xb = synth.draw("weights", (N, K), N + 2 * K)
    for pa, pb in PAIRS:
        announce("gemm %dx%dx%d (%d,%d)" % (M, N, K, pa, pb))
        A, B, oa, ob = operands(xa, xb, pa, pb)
        check_gemm(A, B, oa, ob, partials=(M * N * K <= 64 * 64 * 2048))


@pytest.mark.parametrize("tile", [0, 1, 2, 3, 4])
def test_one_chunk_tiles(tile):
    """Every workgroup tile of the one-chunk, g = 16 GEMM (256x256, 256x128,
    256x64, 128x64, 128x128), forced through bfp_gemm_tiled, on shapes that span several
    tiles with ragged tails, partial and full slabs, and every one-plane operand
    format pair (FP4 / FP6 codes, and the FP6 upper plane of m = 5, 6 read
    alone)."""
    # K = 576, 192, 64: ragged K whose exponent rows are whole dwords (the
    # dword exponent loads, last slab half full); 592, 144, 16: byte loads
    for M, N, K in [(300, 200, 592), (520, 72, 1024), (129, 257, 144), (1, 1, 16), (5, 300, 4096),
                    (384, 64, 128 * 5), (260, 136, 576), (130, 70, 192), (70, 130, 64)]:
        xa = synth.draw("half_normal", (M, K), 900 + M + K)
        xb = synth.draw("weights", (N, K), 901 + N + K)
        for am, bm, m_a, m_b in [(2, 2, 2, 2), (2, 4, 2, 4), (4, 2, 4, 2), (3, 4, 3, 4), (6, 1, 4, 1),
                                 (4, 5, 4, 3)]:
            announce("gemm tile %d %dx%dx%d stored (%d,%d) at (%d,%d)" % (tile, M, N, K, am, bm, m_a, m_b))
            A, B, oa, ob = operands(xa, xb, am, bm)
            check_gemm(A, B, oa, ob, m_a, m_b, tile=tile)


def test_tiled_auto_matches_default_tile():
    """bfp_gemm (tile chosen from the shape) and bfp_gemm_tiled with every
    tile: the same products, per-group scales and per-output order of the
    MFMA accumulations, so the FP32 results are identical."""
    M, N, K = 700, 64, 576
    xa = synth.draw("half_normal", (M, K), 951)
    xb = synth.draw("weights", (N, K), 952)
    A, B, oa, ob = operands(xa, xb, 2, 4)
    announce("gemm auto tile %dx%dx%d" % (M, N, K))
    check_gemm(A, B, oa, ob, partials=True)
    ref = fb.gemm(A, B, tile=0).cpu().numpy()
    for t in (1, 2, 3, 4):
        c = fb.gemm(A, B, tile=t).cpu().numpy()
        assert np.array_equal(c, ref), "tile %d differs from the default tile" % t


@pytest.mark.parametrize("nslabs", range(1, 10))
def test_full_slab_counts(nslabs):
    """K = 128 * nslabs (full slabs: exponents by direct loads, two slabs' per
    16-byte load, and the slab loop unrolled by four): every slab count mod 4
    (the loop's tail) for each kernel family, with ragged M and N."""
    M, N, K = 260, 136, 128 * nslabs
    xa = synth.draw("normal", (M, K), 700 + nslabs)
    xb = synth.draw("weights", (N, K), 800 + nslabs)
    for pa, pb in [(2, 2), (4, 4), (2, 4), (4, 2), (6, 6), (4, 6), (6, 3), (8, 8)]:
        announce("gemm full slabs %dx%dx%d (%d,%d)" % (M, N, K, pa, pb))
        A, B, oa, ob = operands(xa, xb, pa, pb)
        check_gemm(A, B, oa, ob)


@pytest.mark.parametrize("g", [16, 32])
def test_degenerate_shapes(g):
    """K = 0: every kernel family (one chunk, two chunks, the cross-product
    and the load-issuing-wave variants) runs zero slabs and writes C = 0;
    M = 0 or N = 0: an empty C, nothing launched."""
    for pa, pb in [(2, 2), (4, 4), (2, 4), (4, 6), (6, 6), (8, 8)]:
        announce("gemm K=0 g=%d (%d,%d)" % (g, pa, pb))
        A = fb.quantize(torch.zeros((300, 0), device="cuda"), g=g, m=pa)
        B = fb.quantize(torch.zeros((200, 0), device="cuda"), g=g, m=pb)
        C = fb.gemm(A, B)
        torch.cuda.synchronize()
        assert tuple(C.shape) == (300, 200) and not torch.any(C != 0).item()
        announce("gemm M=0 / N=0 g=%d (%d,%d)" % (g, pa, pb))
        xa = torch.ones((0, 256), device="cuda")
        xb = torch.ones((64, 256), device="cuda")
        A0, B1 = fb.quantize(xa, g=g, m=pa), fb.quantize(xb, g=g, m=pb)
        assert tuple(fb.gemm(A0, B1).shape) == (0, 64)
        assert tuple(fb.gemm(B1, fb.quantize(xa, g=g, m=pb)).shape) == (64, 0)
        torch.cuda.synchronize()


def test_strided_output():
    """bfp_gemm through the C-ABI into a wider row-major buffer (ldc > N): at a
    16-byte-aligned base with ldc a multiple of 4 (the 16-byte store path) and
    at a 4-byte-aligned base with an odd ldc (the 4-byte path).  The values are
    the oracle's, and the columns between the rows and the words around the
    output stay untouched."""
    import ctypes
    M, N, K = 130, 72, 384
    xa = synth.draw("normal", (M, K), 901)
    xb = synth.draw("weights", (N, K), 902)
    lib = fb._lib.load()
    P = ctypes.c_void_p
    for pa, pb in [(2, 2), (4, 4), (2, 4), (4, 6), (6, 6), (8, 8)]:
        A, B, oa, ob = operands(xa, xb, pa, pb)
        Co, S = oracle.gemm(oa[0], oa[1], A.m, ob[0], ob[1], B.m, g=16, rows=np.arange(M), threads=THREADS)
        for off, ldc in [(4, 80), (1, 81)]:
            announce("gemm strided out (%d,%d) offset %d ldc %d" % (pa, pb, off, ldc))
            big = torch.full((off + M * ldc + 8,), -7.0, dtype=torch.float32, device="cuda")
            rc = lib.bfp_gemm(P(A.mant.data_ptr()), P(A.exp.data_ptr()), A.m, P(B.mant.data_ptr()),
                              P(B.exp.data_ptr()), B.m, M, N, K, 16, A.m, B.m, P(big.data_ptr() + 4 * off), ldc,
                              P(torch.cuda.current_stream().cuda_stream))
            assert rc == 0
            torch.cuda.synchronize()
            h = big.cpu().numpy()
            Cw = h[off:off + M * ldc].reshape(M, ldc).astype(np.float64)
            assert np.all(np.abs(Cw[:, :N] - Co) <= TOL * S)
            assert np.all(Cw[:, N:] == -7.0) and np.all(h[:off] == -7.0) and np.all(h[off + M * ldc:] == -7.0)


def test_precision_lowering():
    xa = synth.draw("half_normal", (130, 320), 5)
    xb = synth.draw("grads", (70, 320), 6)
    announce("gemm stored (8,6) used at (4,4) and mixed")
    A, B, oa, ob = operands(xa, xb, 8, 6, mode_b="stochastic", seed=3)
    for m_a, m_b in [(4, 4), (8, 4), (4, 6), (8, 6)]:
        check_gemm(A, B, oa, ob, m_a, m_b, partials=True)


def test_gradient_operands_wide_exponents():
    """Laplace gradients with outliers on both sides, stochastic rounding."""
    xa = synth.draw("grads", (256, 1024), 51)
    xb = synth.draw("grads", (192, 1024), 52)
    for pair in [(2, 2), (4, 4), (6, 8)]:
        announce("gemm grads x grads %s" % (pair,))
        A, B, oa, ob = operands(xa, xb, *pair, mode_a="stochastic", mode_b="stochastic", seed=17)
        check_gemm(A, B, oa, ob)


def sampled_rows(M, n, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, M - 1], rng.choice(M, n, replace=False)]))


def big_case(M, N, K, pa, pb, dist_a, dist_b, seed, b_axis=-1, nrows=24):
    xa = synth.draw(dist_a, (M, K), seed)
    xb = synth.draw(dist_b, (N, K) if b_axis == -1 else (K, N), seed + 1)
    rows = sampled_rows(M, nrows, seed)
    announce("gemm %dx%dx%d (%d,%d) %s x %s sampled rows" % (M, N, K, pa, pb, dist_a, dist_b))
    A = fb.quantize(torch.from_numpy(xa).cuda(), g=16, m=pa)
    B = fb.quantize(torch.from_numpy(xb).cuda(), group_axis=b_axis, g=16, m=pb)
    # oracle operands: A only on the sampled rows, B in full
    qa = np.zeros((M, K), np.int16)
    ea = np.zeros((M, K // 16), np.uint8)
    for r in rows:
        q1, e1, _ = oracle.quantize(xa, g=16, m=pa, rows=(int(r), int(r) + 1))
        qa[r], ea[r] = q1[0], e1[0]
    qb, eb, _ = oracle.quantize(xb, axis=b_axis, g=16, m=pb, threads=THREADS)
    return check_gemm(A, B, (qa, ea), (qb, eb), rows=rows)


@pytest.mark.parametrize("shape", [(8192, 12288, 4096), (8192, 4096, 4096), (8192, 16384, 4096),
                                   (8192, 4096, 16384)])
def test_transformer_shapes_sampled(shape):
    M, N, K = shape
    for pa, pb in [(2, 4), (8, 8)]:
        big_case(M, N, K, pa, pb, "normal", "weights", seed=41)


@pytest.mark.parametrize("shape", [(802816, 64, 576), (200704, 128, 1152), (50176, 256, 2304),
                                   (12544, 512, 4608)])
def test_resnet_im2col_shapes_sampled(shape):
    M, N, K = shape
    big_case(M, N, K, 2, 4, "half_normal", "weights", seed=61)


def test_ffn_backward_shapes_sampled():
    """dX = dY . W^T (K = 16384) and dW = X^T . dY (operands regrouped along
    the token axis by transpose-on-quantize)."""
    big_case(8192, 4096, 16384, 4, 4, "grads", "weights", seed=53)
    # dW[4096, 16384] = X^T [4096, 8192] . dY [8192, 16384]: quantize X and dY
    # along axis 0 (tokens); the oracle does the same from the untransposed arrays
    x = synth.draw("half_normal", (8192, 4096), 51)
    dy = synth.draw("grads", (8192, 16384), 54)
    rows = sampled_rows(4096, 16, 9)
    announce("gemm dW 4096x16384x8192 regrouped operands")
    A = fb.quantize(torch.from_numpy(x).cuda(), group_axis=0, g=16, m=6)
    B = fb.quantize(torch.from_numpy(dy).cuda(), group_axis=0, g=16, m=6, rounding="stochastic", seed=7)
    qa, ea, _ = oracle.quantize(x, axis=0, g=16, m=6, threads=THREADS)
    qb, eb, _ = oracle.quantize(dy, axis=0, g=16, m=6, mode="stochastic", seed=7, threads=THREADS)
    check_gemm(A, B, (qa, ea), (qb, eb), rows=rows)


# Groups of 32: one whole group per MFMA block (no padding), every kernel
# variant, full and ragged K slabs, at sizes spanning several tiles.
G32_SHAPES = [(300, 200, 608), (257, 129, 512), (1, 1, 32), (64, 300, 4096)]


@pytest.mark.parametrize("K", [32, 64, 96])
def test_g32_tiny_all_precisions(K):
    x = synth.draw("normal", (8, K), 700 + K)
    for am in range(1, 9):
        for bm in range(1, 9):
            announce("gemm g=32 tiny K=%d stored (%d,%d)" % (K, am, bm))
            A, B, oa, ob = operands(x[:4], x[4:], am, bm, g=32)
            for m_a in chunk_drops(am):
                for m_b in chunk_drops(bm):
                    check_gemm(A, B, oa, ob, m_a, m_b, partials=True)


@pytest.mark.parametrize("shape", G32_SHAPES)
def test_g32_ragged_shapes(shape):
    M, N, K = shape
    xa = synth.draw("half_normal", (M, K), 710 + M + K)
    xb = synth.draw("grads", (N, K), 720 + N + K)
    for pa, pb in PAIRS:
        announce("gemm g=32 %dx%dx%d (%d,%d)" % (M, N, K, pa, pb))
        A, B, oa, ob = operands(xa, xb, pa, pb, g=32, mode_b="stochastic", seed=4)
        check_gemm(A, B, oa, ob, partials=(M * N * K <= 64 * 64 * 2048))


def test_g32_ffn_shape_sampled():
    """The FFN up-projection (8192 x 16384 x 4096) with groups of 32 at (4,4) and
    (6,6): sampled rows against the oracle."""
    M, N, K = 8192, 16384, 4096
    xa = synth.draw("half_normal", (M, K), 730)
    xb = synth.draw("weights", (N, K), 731)
    rows = np.random.default_rng(5).choice(M, 48, replace=False)
    for pair in [(4, 4), (6, 6)]:
        announce("gemm g=32 ffn_up %s" % (pair,))
        A = fb.quantize(torch.from_numpy(xa).cuda(), g=32, m=pair[0])
        B = fb.quantize(torch.from_numpy(xb).cuda(), g=32, m=pair[1])
        qa, ea, _ = oracle.quantize(xa, g=32, m=pair[0], threads=THREADS, rows=None)
        qb, eb, _ = oracle.quantize(xb, g=32, m=pair[1], threads=THREADS)
        check_gemm(A, B, (qa, ea), (qb, eb), rows=rows)
