"""GPU parity of the two-grouping conversion (bfp_quantize_dual) and the weight
update with re-conversion (bfp_weight_update): bit-exact with the oracle's
conversions along each axis and its FP32 update, and with the single-axis
kernels of the library."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import bfp_codec
import paper_2110_15456_amd as fb
from paper_2110_15456_amd import synth
from gpu_util import announce, check_tensor, THREADS

pytestmark = pytest.mark.gpu
MODES = ("nearest", "stochastic", "truncate")


def check_against_oracle(x, tr, tc, m, mode, seed_r, seed_c, rows=None):
    """Bytes of both outputs against the oracle's two conversions (optionally
    only the output rows listed in ``rows`` = (row indices of tr, of tc))."""
    (qr, er), (qc, ec), bad = oracle.quantize_dual(x, m=m, mode=mode, seed_rows=seed_r, seed_cols=seed_c,
                                                   threads=THREADS)
    assert bad == 0
    for t, q, e in ((tr, qr, er), (tc, qc, ec)):
        assert np.array_equal(t.exp.cpu().numpy(), e), "exponents differ"
        assert np.array_equal(t.mant.cpu().numpy(), bfp_codec.encode(q, m)), "mantissas differ"


@pytest.mark.parametrize("shape", [(128, 128), (272, 400), (16, 16), (48, 1040), (1040, 48)])
@pytest.mark.parametrize("m", [2, 4, 6, 8, 3])
def test_dual_matches_oracle(shape, m):
    x = synth.draw("grads", shape, 5000 + shape[0] + m)
    xt = torch.from_numpy(x).cuda()
    for mode in MODES:
        announce("dual %s m=%d %s" % (shape, m, mode))
        st = torch.zeros(1, dtype=torch.int32, device="cuda")
        tr, tc = fb.quantize_dual(xt, m=m, rounding=mode, seed_rows=11, seed_cols=12, status=st)
        torch.cuda.synchronize()
        assert int(st.item()) == 0
        check_against_oracle(x, tr, tc, m, mode, 11, 12)


def test_dual_equals_single_axis_kernels():
    """The FFN activation shape (8192 x 4096, stochastic): both outputs equal
    the single-axis kernels' outputs byte for byte."""
    announce("dual 8192x4096 vs single-axis")
    x = torch.from_numpy(synth.draw("half_normal", (8192, 4096), 5100)).cuda()
    for m in (2, 4, 6):
        tr, tc = fb.quantize_dual(x, m=m, rounding="stochastic", seed_rows=3, seed_cols=4)
        ur = fb.quantize(x, g=16, m=m, rounding="stochastic", seed=3)
        uc = fb.quantize(x, group_axis=0, g=16, m=m, rounding="stochastic", seed=4)
        torch.cuda.synchronize()
        assert torch.equal(tr.mant, ur.mant) and torch.equal(tr.exp, ur.exp)
        assert torch.equal(tc.mant, uc.mant) and torch.equal(tc.exp, uc.exp)


@pytest.mark.parametrize("shape", [(256, 384), (272, 400), (16, 48)])
def test_weight_update_matches_oracle(shape):
    w = synth.draw("weights", shape, 5200 + shape[1])
    dw = synth.draw("grads", shape, 5300 + shape[1]) * np.float32(0.01)
    for alpha, m, mode in ((-0.1, 4, "nearest"), (1.0, 2, "stochastic"), (-1e-3, 6, "truncate")):
        announce("weight update %s alpha=%g m=%d %s" % (shape, alpha, m, mode))
        wt, dwt = torch.from_numpy(w).cuda(), torch.from_numpy(dw).cuda()
        w_out, tr, tc = fb.weight_update(wt, dwt, alpha, m=m, rounding=mode, seed_rows=21, seed_cols=22)
        torch.cuda.synchronize()
        w_o = oracle.weight_update(w, dw, alpha)
        assert np.array_equal(w_out.cpu().numpy().view(np.uint32), w_o.view(np.uint32)), "updated weights differ"
        check_against_oracle(w_o, tr, tc, m, mode, 21, 22)


def test_weight_update_in_place_and_fma_case():
    """In place (w_out = w), and the value a fused multiply-add would change:
    w = -(1 + 2^-22), alpha = dw = 1 + 2^-23 gives exactly 0."""
    announce("weight update in place")
    a = np.float32(1.0 + 2.0 ** -23)
    w = np.full((16, 16), -(1.0 + 2.0 ** -22), np.float32)
    w[0, 0] = 3.0
    dw = np.full((16, 16), a, np.float32)
    wt = torch.from_numpy(w).cuda()
    w_out, tr, tc = fb.weight_update(wt, torch.from_numpy(dw).cuda(), float(a), m=4, w_out=wt)
    torch.cuda.synchronize()
    got = wt.cpu().numpy()
    assert w_out.data_ptr() == wt.data_ptr()
    want = oracle.weight_update(w, dw, float(a))
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    assert got[1, 1] == 0.0 and got[0, 0] == want[0, 0]
    check_against_oracle(want, tr, tc, 4, "nearest", 0, 0)


def test_weight_update_subnormals_flush_to_signed_zero():
    """Subnormal inputs, products and sums become zeros of the same sign, as
    in the oracle's definition."""
    announce("weight update subnormals")
    tiny = np.float32(np.finfo(np.float32).tiny)
    w = np.zeros((16, 16), np.float32)
    dw = np.ones((16, 16), np.float32)
    w[0, :4] = [-0.0, -0.0, 0.25 * tiny, -0.0]
    dw[0, :4] = [-0.5 * tiny, -1e-30, 1.0, 0.5 * tiny]
    w[1, :] = 0.75 * tiny
    dw[1, :] = -0.75 * tiny
    w_out, _, _ = fb.weight_update(torch.from_numpy(w).cuda(), torch.from_numpy(dw).cuda(), 1e-9, m=4)
    torch.cuda.synchronize()
    want = oracle.weight_update(w, dw, 1e-9)
    assert np.array_equal(w_out.cpu().numpy().view(np.uint32), want.view(np.uint32))


def test_dual_edges():
    announce("dual edges")
    e = torch.zeros((0, 64), dtype=torch.float32, device="cuda")
    tr, tc = fb.quantize_dual(e)
    assert tr.rows == 0 and tc.rows == 64
    with pytest.raises(fb.BFPError):
        fb.quantize_dual(torch.zeros((24, 64), dtype=torch.float32, device="cuda"))  # R not a multiple of 16
    with pytest.raises(fb.BFPError):
        fb.quantize_dual(torch.zeros((32, 64), dtype=torch.float32, device="cuda"), g=32)


def test_dual_special_values():
    """Zeros of both signs, subnormals, powers of two, ties and extremes."""
    x = synth.special_values(64 * 256, seed=9).reshape(64, 256)
    xt = torch.from_numpy(x).cuda()
    for m in (2, 4, 8):
        for mode in MODES:
            announce("dual special values m=%d %s" % (m, mode))
            tr, tc = fb.quantize_dual(xt, m=m, rounding=mode, seed_rows=1, seed_cols=2)
            torch.cuda.synchronize()
            check_against_oracle(x, tr, tc, m, mode, 1, 2)


@pytest.mark.parametrize("m", [2, 4, 6])
def test_step_dy_full_size(m):
    """dY of the FFN training step (8192 x 16384, the gradient distribution)
    in both groupings with stochastic rounding, at the step's size and launch
    configuration: byte for byte what the single-axis kernels write (those are
    pinned to the oracle at full size by the quantize tests), and the first and
    last 16 output rows of each grouping against the oracle directly."""
    announce("dual full-size dY 8192x16384 m=%d stochastic" % m)
    x = synth.draw("grads", (8192, 16384), 5400 + m)
    xt = torch.from_numpy(x).cuda()
    sr, sc = 1000 + 2 * m, 1001 + 2 * m
    tr, tc = fb.quantize_dual(xt, g=16, m=m, rounding="stochastic", seed_rows=sr, seed_cols=sc)
    ur = fb.quantize(xt, g=16, m=m, rounding="stochastic", seed=sr)
    uc = fb.quantize(xt, group_axis=0, g=16, m=m, rounding="stochastic", seed=sc)
    torch.cuda.synchronize()
    assert torch.equal(tr.exp, ur.exp) and torch.equal(tr.mant, ur.mant), "row grouping differs from k_quantize_rows"
    assert torch.equal(tc.exp, uc.exp) and torch.equal(tc.mant, uc.mant), "column grouping differs from k_quantize_cols"
    for rows in ((0, 16), (8192 - 16, 8192)):
        check_tensor(tr, x, -1, 16, m, "stochastic", sr, rows)
    for rows in ((0, 16), (16384 - 16, 16384)):
        check_tensor(tc, x, 0, 16, m, "stochastic", sc, rows)


@pytest.mark.parametrize("m", [2, 4, 6])
def test_step_weight_update_full_size(m):
    """The step's weight update at full size (W 4096 x 16384, alpha = -1e-3),
    in place as the step runs it: W' bit for bit the oracle's two FP32
    roundings, and both groupings of W' byte for byte what the single-axis
    kernels write for W'."""
    announce("weight update full-size 4096x16384 m=%d" % m)
    w = synth.draw("weights", (4096, 16384), 5500 + m)
    dw = synth.draw("grads", (4096, 16384), 5600 + m)
    wt, dwt = torch.from_numpy(w).cuda(), torch.from_numpy(dw).cuda()
    w_out, tr, tc = fb.weight_update(wt, dwt, -1e-3, g=16, m=m, w_out=wt)
    ur = fb.quantize(w_out, g=16, m=m)
    uc = fb.quantize(w_out, group_axis=0, g=16, m=m)
    torch.cuda.synchronize()
    want = oracle.weight_update(w, dw, -1e-3)
    assert np.array_equal(w_out.cpu().numpy().view(np.uint32), want.view(np.uint32)), "updated weights differ"
    assert torch.equal(tr.exp, ur.exp) and torch.equal(tr.mant, ur.mant), "row grouping of W' differs"
    assert torch.equal(tc.exp, uc.exp) and torch.equal(tc.mant, uc.mant), "column grouping of W' differs"
    check_tensor(tr, want, -1, 16, m, "nearest", 0, (0, 16))
    check_tensor(tc, want, 0, 16, m, "nearest", 0, (16384 - 16, 16384))
