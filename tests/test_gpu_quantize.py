"""GPU parity of bfp_quantize / bfp_dequantize with the oracle: exponents and
packed mantissas bit-exact, on small ragged shapes, edge values, both group
axes, every m and rounding mode, and the full 64M-element quantize sweep."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import bfp_codec
import paper_2110_15456_amd as fb
from paper_2110_15456_amd import synth
from gpu_util import announce, check_quantize, gpu_quantize, THREADS

pytestmark = pytest.mark.gpu
MODES = ("nearest", "stochastic", "truncate")


@pytest.mark.parametrize("g", [16, 32])
@pytest.mark.parametrize("m", range(1, 9))
@pytest.mark.parametrize("dist", ["normal", "grads"])
def test_rows_small_ragged(g, m, dist):
    # 37 x 768: 1776 groups at g=16 (7 workgroups, the last one partial)
    x = synth.draw(dist, (37, 768), 1000 + m)
    for mode in MODES:
        announce("quantize rows 37x768 g=%d m=%d %s %s" % (g, m, dist, mode))
        check_quantize(x, -1, g, m, mode, seed=77 + m)


@pytest.mark.parametrize("shape", [(16 * 37, 100), (512, 64), (32 * 9, 130), (16, 1)])
@pytest.mark.parametrize("g", [16, 32])
def test_cols_transposed(shape, g):
    R, C = shape
    if R % g:
        pytest.skip("group size must divide R")
    x = synth.draw("grads", shape, 2000 + R + C)
    for m in (1, 2, 4, 6, 8):
        for mode in MODES:
            announce("quantize cols %dx%d g=%d m=%d %s" % (R, C, g, m, mode))
            t, q_o, _ = check_quantize(x, 0, g, m, mode, seed=5)
            # the same bytes as quantizing the transposed copy along rows
            t2, _ = gpu_quantize(np.ascontiguousarray(x.T), -1, g, m, mode, seed=5)
            assert torch.equal(t.mant, t2.mant) and torch.equal(t.exp, t2.exp)


def test_special_values():
    x = synth.special_values(64 * 256, seed=3).reshape(64, 256)
    for m in range(1, 9):
        for mode in MODES:
            announce("quantize special values m=%d %s" % (m, mode))
            check_quantize(x, -1, 16, m, mode, seed=11)
            check_quantize(np.ascontiguousarray(x.T), 0, 16, m, mode, seed=11)


def test_nonfinite_sets_status():
    x = synth.draw("normal", (8, 64), 1)
    x[3, 17] = np.inf
    announce("quantize with an Inf input")
    _, st = gpu_quantize(x, -1, 16, 4, "nearest")
    assert st == 1
    x[3, 17] = np.nan
    _, st = gpu_quantize(np.ascontiguousarray(x.T), 0, 16, 4, "nearest")
    assert st == 1


def test_empty_inputs():
    announce("quantize empty tensors")
    t, st = gpu_quantize(np.zeros((0, 64), np.float32), -1, 16, 4, "nearest")
    assert t.rows == 0 and st == 0
    y = fb.dequantize(t)
    assert y.shape == (0, 64)


@pytest.mark.parametrize("m", [1, 2, 4, 5, 8])
def test_dequantize_matches_oracle(m):
    x = synth.draw("grads", (33, 512), 7)
    announce("dequantize m=%d" % m)
    t, _ = gpu_quantize(x, -1, 16, m, "stochastic", seed=9)
    y = fb.dequantize(t).cpu().numpy().astype(np.float64)
    q_o, E_o, _ = oracle.quantize(x, g=16, m=m, mode="stochastic", seed=9)
    assert np.array_equal(y, oracle.dequantize(q_o, E_o, 16, m))


@pytest.mark.parametrize("dist,seed", [("half_normal", 21), ("weights", 22), ("grads", 23)])
def test_full_size_sweep(dist, seed):
    """The 64M-element quantize sweep (8192 x 8192, g=16 along the last axis):
    m in {2,4,6,8}, nearest and stochastic (Philox seed 1234); full parity for
    one mode per m, the other on a 1024-row slice."""
    x = synth.draw(dist, (8192, 8192), seed)
    for m in (2, 4, 6, 8):
        for mode in ("nearest", "stochastic"):
            full = (mode == "nearest") == (m % 4 == 0)
            rows = None if full else (8192 - 1024, 8192)
            announce("quantize 8192x8192 %s m=%d %s rows=%s" % (dist, m, mode, rows))
            check_quantize(x, -1, 16, m, mode, seed=1234, rows=rows)


def test_stochastic_unbiased_over_1000_seeds():
    """First 4096 values of the gradient tensor, Philox seeds 1234..2233.  For
    each value the exact expectation of the magnitude is the average over all
    256 noise bytes (taken from the oracle); the GPU's average over 1000 seeds
    must match it within sampling error (per-value and pooled z scores)."""
    x = synth.draw("grads", (8192, 8192), 23)[:1, :4096].copy()
    m = 2
    announce("SR unbiasedness, 1000 seeds, 4096 values")
    xt = torch.from_numpy(x).cuda()
    out = fb.BFPTensor.empty(1, 4096, 16, m, "cuda")
    acc = torch.zeros(4096, dtype=torch.float64)
    accsq = torch.zeros(4096, dtype=torch.float64)
    for s in range(1234, 2234):
        fb.quantize(xt, g=16, m=m, rounding="stochastic", seed=s, out=out)
        qv = torch.from_numpy(bfp_codec.decode(out.mant.cpu().numpy(), 1, 4096, m).astype(np.float64))[0]
        acc += qv.abs()
        accsq += qv.abs() ** 2
    mean = (acc / 1000).numpy()
    # exact expectation per value from the oracle, enumerating the noise byte
    expect = np.zeros(4096)
    for G in range(256):
        grp = x[0, 16 * G:16 * G + 16]
        tot = np.zeros(16)
        for u in range(256):
            qg, _, _ = oracle.quantize_group(grp, m, "stochastic", np.full(16, u))
            tot += np.abs(qg)
        expect[16 * G:16 * G + 16] = tot / 256
    p = expect - np.floor(expect)
    var = p * (1 - p)
    live = var > 0
    z = (mean[live] - expect[live]) / np.sqrt(var[live] / 1000)
    assert np.all(mean[~live] == expect[~live])
    assert np.max(np.abs(z)) < 5.5
    pooled = (mean[live] - expect[live]).sum() / np.sqrt((var[live] / 1000).sum())
    assert abs(pooled) < 4.0


def test_stochastic_rounding_frequencies_64M():
    """Theorem 1 on the GPU's output of the 64M-element gradient tensor (SR,
    Philox seed 1234, m = 4): a value whose magnitude is a LSBs, with
    r = floor(256 * frac(a)), rounds up with probability exactly r / 256 (the
    8-bit noise byte is uniform).  The round-up counts in each of the 255 bins
    r = 1..255 are tested together (chi-square, 255 degrees of freedom);
    values with r = 0 never round up.  Computed from the GPU's dequantized
    output and the FP32 input only."""
    from scipy import stats
    m = 4
    x = synth.draw("grads", (8192, 8192), 23)
    announce("SR round-up frequencies, 8192x8192 grads m=%d" % m)
    t = fb.quantize(torch.from_numpy(x).cuda(), g=16, m=m, rounding="stochastic", seed=1234)
    y = np.abs(fb.dequantize(t).cpu().numpy().astype(np.float64)).ravel()
    E = np.repeat(t.exp.cpu().numpy().astype(np.int64).ravel(), 16)
    del t
    lsb_exp = E - 127 - (m - 1)
    a = np.ldexp(np.abs(x.astype(np.float64)).ravel(), -lsb_exp)
    del x
    fl = np.floor(a)
    up = np.ldexp(y, -lsb_exp) - fl
    r = np.floor(256.0 * (a - fl)).astype(np.int64)
    live = (E > 0) & (fl < 2 ** m - 1)  # not saturated
    assert np.all((up[live] == 0) | (up[live] == 1))
    assert np.all(up[live & (r == 0)] == 0)
    n_r = np.bincount(r[live], minlength=256)[1:]
    ups = np.bincount(r[live], weights=up[live], minlength=256)[1:]
    p = np.arange(1, 256) / 256.0
    keep = n_r > 0
    x2 = float((((ups - n_r * p) ** 2) / (n_r * p * (1 - p)))[keep].sum())
    assert stats.chi2.sf(x2, int(keep.sum())) > 1e-7, "chi2 = %.1f over %d bins" % (x2, int(keep.sum()))
    # and no bias overall
    z = float((ups - n_r * p).sum() / np.sqrt((n_r * p * (1 - p)).sum()))
    assert abs(z) < 5.0


def test_stochastic_noise_independent_on_gpu():
    """Every value sits exactly half an LSB above a grid point (r = 128), so it
    rounds up exactly when its noise byte is at least 128: the round-up bits
    are the noise bytes' top bits.  They must be balanced, and independent
    between positions of a group (the same Philox word, neighbouring words,
    the two 16-value blocks of a group of 32), between neighbouring groups
    and between seeds (2 x 2 chi-square)."""
    from scipy import stats
    rng = np.random.default_rng(4)
    R, C = 4096, 512
    m = 4
    # magnitudes k + 1/2 for k in 0..14 with one value of each group at 14.5,
    # which fixes the shared exponent at 130 (LSB = 1)
    k = rng.integers(0, 15, (R, C)).astype(np.float64)
    k[:, ::32] = 14
    x = ((k + 0.5) * rng.choice([-1.0, 1.0], (R, C))).astype(np.float32)
    bits = {}
    for seed in (1234, 1235):
        announce("SR noise top bits on the GPU, seed %d" % seed)
        t = fb.quantize(torch.from_numpy(x).cuda(), g=32, m=m, rounding="stochastic", seed=seed)
        assert np.all(t.exp.cpu().numpy() == 130)
        y = np.abs(fb.dequantize(t).cpu().numpy().astype(np.float64))
        bits[seed] = (y - np.floor(np.abs(x.astype(np.float64)))).astype(np.int64).reshape(-1, 32)
    u = bits[1234]
    assert set(np.unique(u)) <= {0, 1}
    n = u.size
    assert abs(int(u.sum()) - n / 2) < 6 * np.sqrt(n / 4)

    def indep(a, b):
        tab = np.bincount(2 * a + b, minlength=4).reshape(2, 2)
        return stats.chi2_contingency(tab, correction=False)[1]

    for p, q in [(0, 1), (0, 4), (2, 6), (3, 4), (0, 16), (5, 21), (15, 16)]:
        assert indep(u[:, p], u[:, q]) > 1e-7, (p, q)
    assert indep(u[:-1, 7].ravel(), u[1:, 7].ravel()) > 1e-7
    assert indep(u.ravel(), bits[1235].ravel()) > 1e-7


@pytest.mark.parametrize("shape,axis", [((3, 64, 5), 1), ((2, 3, 48, 7), 2), ((2, 96, 3, 2), 1), ((32, 2, 5), 0),
                                        ((4, 6, 32), 2), ((128,), 0), ((7, 64), 1), ((64, 7), 0)])
def test_quantize_nd_any_axis(shape, axis):
    """bfp_quantize_nd: an N-D tensor grouped along any axis is the 2-D
    row-grouped conversion of the tensor with that axis moved last (the other
    axes in order as rows), noise included; through the binding and through
    the C ABI directly."""
    import ctypes
    x = synth.draw("grads", shape, 60 + len(shape) + axis)
    L = shape[axis]
    if L % 16:
        pytest.skip("grouped axis not a multiple of 16")
    moved = np.ascontiguousarray(np.moveaxis(x, axis, -1).reshape(-1, L))
    for g in (16, 8) if L % 16 == 0 else (16,):
        for m, mode in [(4, "stochastic"), (6, "nearest"), (2, "truncate")]:
            announce("quantize nd %s axis %d g=%d m=%d %s" % (shape, axis, g, m, mode))
            t = fb.quantize(torch.from_numpy(x).cuda(), group_axis=axis, g=g, m=m, rounding=mode, seed=21)
            torch.cuda.synchronize()
            q_o, E_o, _ = oracle.quantize(moved, g=g, m=m, mode=mode, seed=21)
            assert (t.rows, t.len) == moved.shape
            assert np.array_equal(t.exp.cpu().numpy(), E_o)
            assert np.array_equal(t.mant.cpu().numpy(), bfp_codec.encode(q_o, m))
            # the N-D entry point directly, also where the binding uses the 2-D one
            lib = fb._lib.load()
            u = fb.BFPTensor.empty(t.rows, t.len, g, m, "cuda")
            xt = torch.from_numpy(x).cuda()
            arr = (ctypes.c_int64 * len(shape))(*shape)
            rc = lib.bfp_quantize_nd(ctypes.c_void_p(xt.data_ptr()), len(shape), arr, axis, g, m,
                                     fb.ROUNDING[mode], ctypes.c_uint64(21), ctypes.c_void_p(u.mant.data_ptr()),
                                     ctypes.c_void_p(u.exp.data_ptr()), None,
                                     ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            assert rc == 0
            torch.cuda.synchronize()
            assert torch.equal(u.mant, t.mant) and torch.equal(u.exp, t.exp)
