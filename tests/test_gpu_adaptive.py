"""GPU parity of the adaptive converter (bfp_quantize_adaptive; Algorithm 1,
Eqs. 1-2, section V-D) with the oracle: the 4-bit tensor and the 2-bit tensor
left by discarding the low chunk are bit-exact, the two sums of Eq. 2 agree
to double rounding, the 2-bit tensor feeds bfp_gemm, and Algorithm 1 makes the
oracle's choices on a small layered schedule."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import bfp_codec
import paper_2110_15456_amd as fb
from paper_2110_15456_amd import synth
from gpu_util import announce, THREADS

pytestmark = pytest.mark.gpu
MODES = ("nearest", "stochastic", "truncate")
REL = 1e-12  # the sums are exact per group and rounded only when summed in double


def run_adaptive(x, axis, g, mode, seed=0, with_m2=True):
    xt = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    t4, t2, sums = fb.quantize_adaptive(xt, group_axis=axis, g=g, rounding=mode, seed=seed, with_m2=with_m2,
                                        status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    return t4, t2, sums.cpu().numpy()


def check_adaptive(x, axis, g, mode, seed=0, with_m2=True):
    t4, t2, sums = run_adaptive(x, axis, g, mode, seed, with_m2)
    q4, e4, bad = oracle.quantize(x, axis=axis, g=g, m=4, mode=mode, seed=seed, threads=THREADS)
    assert bad == 0
    assert np.array_equal(t4.exp.cpu().numpy(), e4), "shared exponents differ"
    assert np.array_equal(t4.mant.cpu().numpy(), bfp_codec.encode(q4, 4).reshape(-1)), "4-bit mantissas differ"
    if with_m2:
        assert t2.exp is t4.exp and t2.m == 2
        q2 = oracle.drop_low_chunk(q4)
        assert np.array_equal(t2.mant.cpu().numpy(), bfp_codec.encode(q2, 2).reshape(-1)), "2-bit mantissas differ"
    num, den = oracle.improvement_sums(q4, e4, g=g)
    assert abs(sums[0] - num) <= REL * abs(num) and abs(sums[1] - den) <= REL * abs(den), (sums, num, den)
    return t4, t2, sums, (q4, e4)


@pytest.mark.parametrize("g", [16, 32])
@pytest.mark.parametrize("dist", ["normal", "grads", "half_normal", "weights"])
def test_rows_ragged(g, dist):
    x = synth.draw(dist, (37, 768), 3100 + g)
    for mode in MODES:
        announce("adaptive rows 37x768 g=%d %s %s" % (g, dist, mode))
        check_adaptive(x, -1, g, mode, seed=11)


@pytest.mark.parametrize("shape", [(16 * 37, 100), (512, 64), (32 * 9, 130)])
@pytest.mark.parametrize("g", [16, 32])
def test_cols_transposed(shape, g):
    R, C = shape
    if R % g:
        pytest.skip("group size must divide R")
    x = synth.draw("grads", shape, 3200 + R + C)
    for mode in MODES:
        announce("adaptive cols %dx%d g=%d %s" % (R, C, g, mode))
        t4, t2, sums, _ = check_adaptive(x, 0, g, mode, seed=5)
        # the same bytes and sums as the transposed copy quantized along rows
        u4, u2, usums = run_adaptive(np.ascontiguousarray(x.T), -1, g, mode, seed=5)
        assert torch.equal(t4.mant, u4.mant) and torch.equal(t4.exp, u4.exp) and torch.equal(t2.mant, u2.mant)
        assert np.allclose(sums, usums, rtol=REL, atol=0)


def test_without_second_tensor_and_edges():
    announce("adaptive edges")
    x = synth.draw("normal", (8, 256), 3300)
    check_adaptive(x, -1, 16, "nearest", with_m2=False)
    # all zero: both sums 0, Algorithm 1 keeps 2 bits for any positive threshold
    z = np.zeros((4, 64), np.float32)
    _, _, sums, _ = check_adaptive(z, -1, 16, "nearest")
    assert sums[0] == 0.0 and sums[1] == 0.0
    assert fb.adaptive_mantissa(sums, 0.1) == 2
    # one group with 1.75: r = 1/6 exactly
    one = np.zeros((1, 16), np.float32)
    one[0, 3] = -1.75
    _, _, sums, _ = check_adaptive(one, -1, 16, "nearest")
    assert sums[0] == 0.25 and sums[1] == 1.5
    # empty tensor: sums are zeroed, nothing else is written
    e = torch.zeros((0, 64), dtype=torch.float32, device="cuda")
    _, _, s = fb.quantize_adaptive(e)
    assert s.cpu().tolist() == [0.0, 0.0]


def test_quantize_sweep_size_sums():
    """The 64M-element quantize workload (8192 x 8192, half-normal): full
    comparison of the sums and sampled rows of both tensors."""
    announce("adaptive 8192x8192 half_normal nearest")
    x = synth.draw("half_normal", (8192, 8192), 21)
    t4, t2, sums = run_adaptive(x, -1, 16, "nearest")
    q4, e4, _ = oracle.quantize(x, g=16, m=4, threads=THREADS)
    num, den = oracle.improvement_sums(q4, e4, g=16)
    assert abs(sums[0] - num) <= REL * num and abs(sums[1] - den) <= REL * den
    rows = np.random.default_rng(0).choice(8192, 64, replace=False)
    m4 = t4.mant.cpu().numpy().reshape(8192, -1)  # 6-bit codes: 6144 bytes per row
    m2 = t2.mant.cpu().numpy().reshape(8192, -1)  # 4-bit codes: 4096 bytes per row
    for r in rows:
        assert np.array_equal(m4[r], bfp_codec.encode(q4[r:r + 1], 4).reshape(-1))
        assert np.array_equal(m2[r], bfp_codec.encode(oracle.drop_low_chunk(q4[r:r + 1]), 2).reshape(-1))


def test_two_bit_tensor_feeds_the_gemm():
    """bfp_gemm on the discarded-chunk tensor equals the oracle GEMM of
    sign * (|q4| >> 2) at m = 2 (the paper's 2-bit choice, section V-D)."""
    announce("adaptive m=2 tensor into gemm")
    a = synth.draw("half_normal", (96, 512), 3400)
    b = synth.draw("weights", (80, 512), 3401)
    ta4, ta2, _ = run_adaptive(a, -1, 16, "nearest")
    tb4, tb2, _ = run_adaptive(b, -1, 16, "nearest")
    qa4, ea, _ = oracle.quantize(a, g=16, m=4)
    qb4, eb, _ = oracle.quantize(b, g=16, m=4)
    qa2, qb2 = oracle.drop_low_chunk(qa4), oracle.drop_low_chunk(qb4)
    for (A, qa, ma), (B, qb, mb) in (((ta2, qa2, 2), (tb2, qb2, 2)), ((ta2, qa2, 2), (tb4, qb4, 4)),
                                     ((ta4, qa4, 4), (tb2, qb2, 2))):
        C = fb.gemm(A, B).cpu().numpy().astype(np.float64)
        Co, S = oracle.gemm(qa, ea, ma, qb, eb, mb, g=16)
        assert np.all(np.abs(C - Co) <= 1e-6 * S), (ma, mb)


def test_algorithm1_schedule():
    """Algorithm 1 over a small schedule of layers and iterations (alpha 0.6,
    beta 0.3): every choice equals the oracle's."""
    I, L = 4, 3
    tensors = {"A": ("half_normal", (64, 256)), "W": ("weights", (64, 256)), "G": ("grads", (64, 256))}
    for i in range(I):
        for l in range(L):
            eps = fb.adaptive_threshold(0.6, 0.3, i, I, l, L)
            assert eps == oracle.threshold(0.6, 0.3, i, I, l, L)
            for k, (name, (dist, shape)) in enumerate(tensors.items()):
                announce("algorithm 1 i=%d l=%d %s" % (i, l, name))
                x = synth.draw(dist, shape, 3500 + 100 * i + 10 * l + k)
                _, _, sums = run_adaptive(x, -1, 16, "stochastic" if name == "G" else "nearest", seed=i)
                q4, e4, _ = oracle.quantize(x, g=16, m=4, mode="stochastic" if name == "G" else "nearest", seed=i)
                num, den = oracle.improvement_sums(q4, e4)
                if abs(num / den - eps) > 1e-9:  # a choice decided by the last bits would be ambiguous
                    assert fb.adaptive_mantissa(sums, eps) == oracle.select_mantissa(num, den, eps)


def test_sums_are_deterministic():
    """The partials are added in a fixed order: repeated runs agree bitwise."""
    announce("adaptive determinism")
    x = synth.draw("grads", (1024, 2048), 3600)
    _, _, s1 = run_adaptive(x, -1, 16, "stochastic", seed=3)
    _, _, s2 = run_adaptive(x, -1, 16, "stochastic", seed=3)
    assert s1.tobytes() == s2.tobytes()
    xc = synth.draw("grads", (2048, 1024), 3601)
    _, _, c1 = run_adaptive(xc, 0, 16, "nearest")
    _, _, c2 = run_adaptive(xc, 0, 16, "nearest")
    assert c1.tobytes() == c2.tobytes()
