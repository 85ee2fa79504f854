"""GPU parity of bfp_gemm_bfp, the GEMM whose epilogue converts C to BFP
(groups of 16 along each row of C; the converter of section V-C at the array
output, section V-A).

Two checks: (1) the fused output is bit-exact with converting the FP32 C of
bfp_gemm separately (same values, same noise addressing); (2) against the
oracle: its double-precision GEMM, rounded to FP32, then its quantizer.  The
GPU's FP32 accumulation may differ from the oracle's C by up to 1e-6 * sum|T|
(the GEMM tolerance), so an element's (E, q) is required to match exactly
wherever the oracle gives the same (E, q) for C - tol, C and C + tol, and to
be one of those three results elsewhere."""
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


def operands(shape_a, shape_b, m_a, m_b, seed):
    a = synth.draw("half_normal", shape_a, seed)
    b = synth.draw("weights", shape_b, seed + 1)
    A = fb.quantize(torch.from_numpy(a).cuda(), g=16, m=m_a)
    B = fb.quantize(torch.from_numpy(b).cuda(), g=16, m=m_b)
    return a, b, A, B


def decode(t):
    q = bfp_codec.decode(t.mant.cpu().numpy(), t.rows, t.len, t.m)
    return q, t.exp.cpu().numpy()


@pytest.mark.parametrize("mm", [(4, 4), (2, 4), (6, 6), (4, 8), (8, 4)])
@pytest.mark.parametrize("shape", [(300, 208, 512), (256, 256, 4096), (130, 48, 576), (17, 16, 16)])
def test_fused_equals_separate_conversion(mm, shape):
    m_a, m_b = mm
    M, N, K = shape
    _, _, A, B = operands((M, K), (N, K), m_a, m_b, 4000 + M + N + K)
    C = fb.gemm(A, B)
    for c_m in (1, 2, 4, 6, 8):
        for mode in MODES:
            announce("gemm_bfp %dx%dx%d (%d,%d) -> m=%d %s" % (M, N, K, m_a, m_b, c_m, mode))
            st = torch.zeros(1, dtype=torch.int32, device="cuda")
            T = fb.gemm_bfp(A, B, c_m, rounding=mode, seed=99, status=st)
            R = fb.quantize(C, g=16, m=c_m, rounding=mode, seed=99)
            torch.cuda.synchronize()
            assert int(st.item()) == 0
            assert torch.equal(T.exp, R.exp), "exponents differ"
            assert torch.equal(T.mant, R.mant), "mantissas differ"


@pytest.mark.parametrize("mm", [(4, 4), (6, 6), (2, 8)])
@pytest.mark.parametrize("mode", MODES)
def test_fused_against_oracle(mm, mode):
    m_a, m_b = mm
    M, N, K = 96, 160, 1024
    a, b, A, B = operands((M, K), (N, K), m_a, m_b, 4100 + m_a * 10 + m_b)
    qa, ea, _ = oracle.quantize(a, g=16, m=m_a)
    qb, eb, _ = oracle.quantize(b, g=16, m=m_b)
    Co, S = oracle.gemm(qa, ea, m_a, qb, eb, m_b, g=16, threads=THREADS)
    tol = 1e-6 * S
    for c_m in (2, 4, 8):
        announce("gemm_bfp vs oracle (%d,%d) -> m=%d %s" % (m_a, m_b, c_m, mode))
        T = fb.gemm_bfp(A, B, c_m, rounding=mode, seed=7)
        q, E = decode(T)
        var = []
        for d in (-1.0, 0.0, 1.0):
            x = (Co + d * tol).astype(np.float32)
            qo, eo, _ = oracle.quantize(x, g=16, m=c_m, mode=mode, seed=7)
            var.append((qo, np.repeat(eo, 16, axis=1)))
        Ee = np.repeat(E, 16, axis=1)
        stable = ((var[0][0] == var[1][0]) & (var[1][0] == var[2][0]) &
                  (var[0][1] == var[1][1]) & (var[1][1] == var[2][1]))
        assert stable.mean() > 0.95
        assert np.array_equal(q[stable], var[1][0][stable]) and np.array_equal(Ee[stable], var[1][1][stable])
        ok = np.zeros_like(stable)
        for qo, eo in var:
            ok |= (q == qo) & (Ee == eo)
        assert ok.all(), "unstable elements outside the perturbed results: %d" % (~ok).sum()


def test_fused_edges():
    # all-zero product: every group has E = 0 and q = 0
    announce("gemm_bfp zero operand")
    z = torch.zeros((64, 256), dtype=torch.float32, device="cuda")
    A = fb.quantize(z, g=16, m=4)
    _, _, _, B = operands((64, 256), (48, 256), 4, 4, 4200)
    T = fb.gemm_bfp(A, B, 4)
    assert int(T.exp.max()) == 0 and int(T.mant.max()) == 0
    # N not a multiple of 16 is a shape error
    _, _, A2, B2 = operands((32, 64), (40, 64), 4, 4, 4201)
    with pytest.raises(fb.BFPError):
        fb.gemm_bfp(A2, B2, 4)


@pytest.mark.parametrize("mode", ["nearest", "stochastic"])
@pytest.mark.parametrize("m", [2, 4, 6])
def test_fused_full_size(m, mode):
    """The FFN up-projection shape (8192 x 16384 x 4096) at (m, m) -> m, the
    bench's fused-epilogue cases: every exponent and mantissa byte equal to
    the separate GEMM and conversion."""
    announce("gemm_bfp ffn_up (%d,%d)->m%d %s" % (m, m, m, mode))
    M, N, K = 8192, 16384, 4096
    x = torch.from_numpy(synth.draw("normal", (M, K), 41)).cuda()
    w = torch.from_numpy(synth.draw("weights", (N, K), 42)).cuda()
    A, B = fb.quantize(x, g=16, m=m), fb.quantize(w, g=16, m=m)
    del x, w
    T = fb.gemm_bfp(A, B, m, rounding=mode, seed=5)
    C = fb.gemm(A, B)
    R = fb.quantize(C, g=16, m=m, rounding=mode, seed=5)
    torch.cuda.synchronize()
    assert torch.equal(T.exp, R.exp)
    assert torch.equal(T.mant, R.mant)


@pytest.mark.parametrize("name,shape", [("conv2_x", (802816, 64, 576)), ("conv3_x", (200704, 128, 1152)),
                                        ("conv4_x", (50176, 256, 2304)), ("conv5_x", (12544, 512, 4608))])
def test_fused_resnet_full_size(name, shape):
    """The ResNet-18 im2col shapes at full size, in the bench's launch
    configuration (the small tiles bfp_gemm picks for them): every exponent and
    mantissa byte of the fused output equal to the separate GEMM and
    conversion, for the one-chunk pairs the bench times and both rounding
    modes."""
    M, N, K = shape
    g = torch.Generator(device="cuda").manual_seed(4400 + N)
    x = torch.randn((M, K), generator=g, device="cuda").abs_()
    w = torch.randn((N, K), generator=g, device="cuda").mul_(0.02)
    for m_a, m_b in ((2, 2), (2, 4), (4, 4)):
        A, B = fb.quantize(x, g=16, m=m_a), fb.quantize(w, g=16, m=m_b)
        C = fb.gemm(A, B)
        for mode in ("nearest", "stochastic"):
            announce("gemm_bfp %s (%d,%d)->m%d %s" % (name, m_a, m_b, m_a, mode))
            T = fb.gemm_bfp(A, B, m_a, rounding=mode, seed=9)
            R = fb.quantize(C, g=16, m=m_a, rounding=mode, seed=9)
            torch.cuda.synchronize()
            assert torch.equal(T.exp, R.exp) and torch.equal(T.mant, R.mant)
        del A, B, C


def test_fused_with_g32_operands():
    """Operands grouped by 32 (the output is still grouped by 16 along N)."""
    M, N, K = 200, 208, 640
    a = synth.draw("half_normal", (M, K), 4300)
    b = synth.draw("weights", (N, K), 4301)
    for m_a, m_b in ((4, 4), (2, 6), (8, 3)):
        A = fb.quantize(torch.from_numpy(a).cuda(), g=32, m=m_a)
        B = fb.quantize(torch.from_numpy(b).cuda(), g=32, m=m_b)
        C = fb.gemm(A, B)
        for c_m in (2, 4, 6):
            announce("gemm_bfp g=32 operands (%d,%d) -> m=%d" % (m_a, m_b, c_m))
            T = fb.gemm_bfp(A, B, c_m, rounding="stochastic", seed=8)
            R = fb.quantize(C, g=16, m=c_m, rounding="stochastic", seed=8)
            torch.cuda.synchronize()
            assert torch.equal(T.exp, R.exp) and torch.equal(T.mant, R.mant)
