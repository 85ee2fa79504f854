"""GPU parity of bfp_gemm on the tiny cases, held to exact equality where the
arithmetic allows it.

With K = g (one group) each output is one group's T_G = P_G * 2^(ea + eb -
254 - (m_a-1) - (m_b-1)): the chunk products are exact, and every partial sum
of a group's chunk passes is an integer below 2^24 in units of the product's
LSB, so the FP32 result must equal the oracle's exact value bit for bit
(section III-B: the group dot product is exact; only the cross-group sum is
floating point).  With K = 2g and one chunk plane per operand the result is
one FP32 addition of two exact terms, so it must equal the oracle's exact
sum rounded once to FP32.  Every other output is held to
|C_gpu - C_oracle| <= 1e-6 * sum_G |T_G|.

Inputs: the tiny cases of M = N = 4 for 100 seeds, stacked into 400-row
operands (rows are independent, so every 4 x 4 block of C is one seed's
case), for every stored (m_a, m_b) in 1..8, every lower precision that drops
a low chunk plane, and all three rounding modes."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2110_15456_amd as fb
from paper_2110_15456_amd import synth
from gpu_util import announce, check_quantize, chunk_drops, THREADS

pytestmark = pytest.mark.gpu
SEEDS = range(100)


def stacked(K: int):
    xs = [synth.draw("normal", (8, K), 5000 + 7 * K + s) for s in SEEDS]
    return (np.ascontiguousarray(np.concatenate([x[:4] for x in xs])),
            np.ascontiguousarray(np.concatenate([x[4:] for x in xs])))


@pytest.mark.parametrize("mode", ["nearest", "stochastic", "truncate"])
@pytest.mark.parametrize("g,K", [(16, 16), (16, 32), (32, 32), (32, 64)])
def test_tiny_cases_exact(g, K, mode):
    xa, xb = stacked(K)
    A, B = {}, {}
    for m in range(1, 9):
        announce("quantize stacked tiny g=%d K=%d m=%d %s" % (g, K, m, mode))
        A[m] = check_quantize(xa, -1, g, m, mode, seed=31)
        B[m] = check_quantize(xb, -1, g, m, mode, seed=32)
    for am in range(1, 9):
        for bm in range(1, 9):
            (Ta, qa, ea), (Tb, qb, eb) = A[am], B[bm]
            for m_a in chunk_drops(am):
                for m_b in chunk_drops(bm):
                    announce("gemm stacked tiny g=%d K=%d %s stored (%d,%d) at (%d,%d)"
                             % (g, K, mode, am, bm, m_a, m_b))
                    C = fb.gemm(Ta, Tb, m_a, m_b)
                    torch.cuda.synchronize()
                    Cg = C.cpu().numpy()
                    Co, S = oracle.gemm(qa, ea, am, qb, eb, bm, g=g, m_a=m_a, m_b=m_b, threads=THREADS)
                    assert np.all(np.abs(Cg.astype(np.float64) - Co) <= 1e-6 * S)
                    if K == g:
                        bad = np.argwhere(Cg.astype(np.float64) != Co)
                        assert bad.size == 0, "K = g not exact at %s: gpu %r oracle %r" % (
                            bad[0].tolist(), float(Cg[tuple(bad[0])]), float(Co[tuple(bad[0])]))
                    elif m_a <= 4 and m_b <= 4:
                        bad = np.argwhere(Cg != Co.astype(np.float32))
                        assert bad.size == 0, "K = 2g not one rounding at %s: gpu %r oracle %r" % (
                            bad[0].tolist(), float(Cg[tuple(bad[0])]), float(Co[tuple(bad[0])]))


def _at_exponent(x: np.ndarray, g: int, E: int) -> np.ndarray:
    """x with every group of g along the rows scaled so that its largest
    magnitude lies in [2^(E-127), 2^(E-126)): every shared exponent is E."""
    x = x.astype(np.float64).reshape(x.shape[0], -1, g)
    top = np.abs(x).max(axis=2, keepdims=True)
    y = x / top * 1.5 * 2.0 ** (E - 127)
    return np.ascontiguousarray(y.reshape(x.shape[0], -1).astype(np.float32))


@pytest.mark.parametrize("g", [16, 32])
@pytest.mark.parametrize("big", ["A", "B"])
def test_exponent_range_edge_exact(g, big):
    """The stated domain's top edge: one operand's group exponents all at 250
    (the largest the header allows; a chunk weight of up to +4 then still fits
    the 8-bit block scale), the other's near 100, K = g, every operand-format
    variant (m = 2, 4, 6, 8 on either side) and its chunk drops: C must equal
    the oracle exactly."""
    xa = synth.draw("normal", (64, g), 9100 + g)
    xb = synth.draw("normal", (48, g), 9200 + g)
    hi, lo = 250, 100
    xa = _at_exponent(xa, g, hi if big == "A" else lo)
    xb = _at_exponent(xb, g, lo if big == "A" else hi)
    A, B = {}, {}
    for m in (2, 4, 6, 8):
        announce("quantize exponent edge g=%d big=%s m=%d" % (g, big, m))
        A[m] = check_quantize(xa, -1, g, m, "nearest")
        B[m] = check_quantize(xb, -1, g, m, "nearest")
        assert A[m][2].max() == (hi if big == "A" else lo) and B[m][2].max() == (lo if big == "A" else hi)
    for am in (2, 4, 6, 8):
        for bm in (2, 4, 6, 8):
            (Ta, qa, ea), (Tb, qb, eb) = A[am], B[bm]
            for m_a in chunk_drops(am):
                for m_b in chunk_drops(bm):
                    announce("gemm exponent edge g=%d big=%s stored (%d,%d) at (%d,%d)" % (g, big, am, bm, m_a, m_b))
                    Cg = fb.gemm(Ta, Tb, m_a, m_b).cpu().numpy()
                    Co, _ = oracle.gemm(qa, ea, am, qb, eb, bm, g=g, m_a=m_a, m_b=m_b, threads=THREADS)
                    assert np.isfinite(Co).all()
                    bad = np.argwhere(Cg.astype(np.float64) != Co)
                    assert bad.size == 0, "exponent edge not exact at %s: gpu %r oracle %r" % (
                        bad[0].tolist(), float(Cg[tuple(bad[0])]), float(Co[tuple(bad[0])]))
