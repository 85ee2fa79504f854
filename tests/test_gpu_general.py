"""GPU parity of the general cases against the oracle: group sizes 4, 8 and 64
(quantize, dequantize, GEMM, group partials) and a GEMM taken at any
precision below the stored one (magnitudes truncated to their top m_use bits,
section V-D), which bfp_gemm runs on its general kernel.  Quantized bytes are
bit-exact, int32 group partials bit-exact, and every FP32 output within
1e-6 * sum_G |T_G| of the oracle; with K = g (one group) the output equals the
oracle's exact value."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2110_15456_amd as fb
from paper_2110_15456_amd import synth
from gpu_util import announce, check_quantize, gpu_quantize, THREADS

pytestmark = pytest.mark.gpu
MODES = ("nearest", "stochastic", "truncate")


@pytest.mark.parametrize("g", [4, 8, 64])
@pytest.mark.parametrize("m", range(1, 9))
def test_quantize_group_sizes(g, m):
    """Rows (37 x 768: several workgroups, a partial last one) and columns
    (transpose-on-quantize, 320 x 200) in every rounding mode."""
    x = synth.draw("grads", (37, 768), 40 + m)
    xc = synth.draw("normal", (320, 200), 50 + m)
    for mode in MODES:
        announce("quantize rows 37x768 g=%d m=%d %s" % (g, m, mode))
        check_quantize(x, -1, g, m, mode, seed=3 + m)
        announce("quantize cols 320x200 g=%d m=%d %s" % (g, m, mode))
        t, _, _ = check_quantize(xc, 0, g, m, mode, seed=5 + m)
        t2, _ = gpu_quantize(np.ascontiguousarray(xc.T), -1, g, m, mode, seed=5 + m)
        assert torch.equal(t.mant, t2.mant) and torch.equal(t.exp, t2.exp)


@pytest.mark.parametrize("g", [4, 8, 64])
def test_dequantize_group_sizes(g):
    x = synth.draw("grads", (33, 512), 7)
    for m in (2, 4, 6, 8):
        announce("dequantize g=%d m=%d" % (g, m))
        t, _ = gpu_quantize(x, -1, g, m, "stochastic", seed=9)
        y = fb.dequantize(t).cpu().numpy().astype(np.float64)
        q_o, E_o, _ = oracle.quantize(x, g=g, m=m, mode="stochastic", seed=9)
        assert np.array_equal(y, oracle.dequantize(q_o, E_o, g, m))


def check(A, B, qa, ea, qb, eb, g, m_a, m_b, exact=False, partials=False):
    C = fb.gemm(A, B, m_a, m_b, workspace=False)  # bfp_gemm: the general kernel for these cases
    torch.cuda.synchronize()
    Cg = C.cpu().numpy().astype(np.float64)
    Co, S = oracle.gemm(qa, ea, A.m, qb, eb, B.m, g=g, m_a=m_a, m_b=m_b, threads=THREADS)
    err = np.abs(Cg - Co)
    assert np.all(err <= 1e-6 * S), "max err/sum|T| = %.3g" % float((err / np.maximum(S, 1e-300)).max())
    if exact:
        assert np.array_equal(Cg, Co)
    if partials:
        P = fb.gemm_group_partials(A, B, m_a, m_b).cpu().numpy().astype(np.int64)
        Po = oracle.group_partials(qa, A.m, qb, B.m, g=g, m_a=m_a, m_b=m_b)
        assert np.array_equal(P, Po)


# stored widths and the precisions each is taken at: every lower width of
# one operand with the other at its stored width
STORED = [(2, 4), (4, 4), (4, 6), (6, 6), (6, 8), (8, 8), (3, 7), (5, 1)]


@pytest.mark.parametrize("g", [4, 8, 16, 32, 64])
def test_gemm_every_lower_precision(g):
    """Tiny stacked cases (40 seeds of M = N = 4, so 160 x 160 outputs), K =
    max(g, 16) (one group and exact for g >= 16; rows hold whole 16-value
    units) and K = 128, every precision 1..stored of A and of B, with int32
    group partials."""
    for K in sorted({max(g, 16), 128}):
        xs = [synth.draw("normal", (8, K), 7000 + K + s) for s in range(40)]
        xa = np.ascontiguousarray(np.concatenate([x[:4] for x in xs]))
        xb = np.ascontiguousarray(np.concatenate([x[4:] for x in xs]))
        for am, bm in STORED:
            A, qa, ea = check_quantize(xa, -1, g, am, "stochastic", seed=11)
            B, qb, eb = check_quantize(xb, -1, g, bm, "nearest")
            pairs = {(ma, bm) for ma in range(1, am + 1)} | {(am, mb) for mb in range(1, bm + 1)}
            for m_a, m_b in sorted(pairs):
                announce("gemm g=%d K=%d stored (%d,%d) at (%d,%d)" % (g, K, am, bm, m_a, m_b))
                check(A, B, qa, ea, qb, eb, g, m_a, m_b, exact=(K == g), partials=(K <= 64))


@pytest.mark.parametrize("g", [4, 8, 64])
def test_gemm_group_sizes_ragged(g):
    """Several 32 x 32 tiles with ragged edges, at every operand format, with
    group partials on the smaller shape."""
    for M, N, K in [(70, 45, 192), (129, 257, 576)]:
        xa = synth.draw("half_normal", (M, K), 80 + M + g)
        xb = synth.draw("weights", (N, K), 81 + N + g)
        for am, bm in [(2, 2), (4, 4), (2, 6), (6, 6), (8, 8), (6, 3)]:
            announce("gemm g=%d %dx%dx%d (%d,%d)" % (g, M, N, K, am, bm))
            A, qa, ea = check_quantize(xa, -1, g, am, "nearest")
            B, qb, eb = check_quantize(xb, -1, g, bm, "stochastic", seed=4)
            check(A, B, qa, ea, qb, eb, g, am, bm, partials=(M < 100))


def test_lowered_gemm_matches_chunk_drop_fast_path():
    """Where both kernels apply -- a two-plane operand with its low chunk
    plane dropped -- bfp_gemm takes the block-scaled kernel; the same product
    one bit lower goes to the general kernel.  Both against the oracle on a
    full-slab shape (transformer-like, 1024 x 512 x 1024)."""
    M, N, K = 1024, 512, 1024
    xa = synth.draw("normal", (M, K), 91)
    xb = synth.draw("weights", (N, K), 92)
    A, qa, ea = check_quantize(xa, -1, 16, 6, "nearest")
    B, qb, eb = check_quantize(xb, -1, 16, 8, "nearest")
    for m_a, m_b in [(4, 4), (3, 4), (4, 3), (6, 7), (5, 8), (1, 1)]:
        announce("gemm 1024x512x1024 stored (6,8) at (%d,%d)" % (m_a, m_b))
        check(A, B, qa, ea, qb, eb, 16, m_a, m_b)
