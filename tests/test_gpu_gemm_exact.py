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
