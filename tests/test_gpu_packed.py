"""GPU parity of the packed storage (section V-D: 2-bit chunks with their sign
in 3 bits, a 3-bit exponent above a per-tensor base) against the oracle.

Quantized bytes -- the E_max word, the exponent stream and every chunk field
-- are compared bit for bit with the oracle's (q, E) encoded by the test codec;
dequantized values exactly; the GEMM on packed operands within
1e-6 * sum_G |T_G| of the oracle's exact sum, and equal to it with K = 16 (one
group: the FP32 result is the exact value)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import bfp_codec
import oracle
import paper_2110_15456_amd as fb
from paper_2110_15456_amd import synth
from gpu_util import announce, THREADS

pytestmark = pytest.mark.gpu
MODES = ("nearest", "stochastic", "truncate")


def max_exponent_field(x: np.ndarray) -> int:
    return int(((np.ascontiguousarray(x, np.float32).view(np.uint32) >> 23) & 255).max()) if x.size else 0


def check_packed(x: np.ndarray, m: int, mode: str, seed: int = 0):
    """Quantize x on the GPU into packed storage; compare every byte with the
    oracle's.  Returns (tensor, q, E)."""
    xt = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    t = fb.quantize_packed(xt, m=m, rounding=mode, seed=seed, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    q_o, E_o, base, bad = oracle.quantize_packed(x, g=16, m=m, mode=mode, seed=seed, threads=THREADS)
    assert bad == 0
    emax = max_exponent_field(x)
    assert base == max(emax - 7, 0)
    mant, exp = t.mant.cpu().numpy(), t.exp.cpu().numpy()
    want_mant, want_exp = bfp_codec.encode_packed(q_o, E_o, emax, m)
    assert np.array_equal(exp, want_exp), "exponent stream differs"
    if not np.array_equal(mant, want_mant):
        q_g, _, _ = bfp_codec.decode_packed(mant, exp, t.rows, t.len, m)
        bad_idx = np.argwhere(q_g != q_o)
        raise AssertionError("packed mantissas differ at %d positions, first %s" % (len(bad_idx), bad_idx[:3].tolist()))
    return t, q_o, E_o


def wide_range(shape, seed):
    """Gradient-like values whose group maxima span far more than 7 binades,
    so that many groups sit below the tensor base and are raised to it."""
    x = synth.draw("grads", shape, seed).astype(np.float32)
    scale = np.float32(2.0) ** np.random.default_rng(seed).integers(-20, 1, size=(shape[0], 1)).astype(np.float32)
    return np.ascontiguousarray(x * scale)


@pytest.mark.parametrize("m", range(1, 9))
def test_quantize_packed(m):
    """37 x 768 (1776 groups: a partial workgroup and a partial 64-group
    exponent block), one value distribution within the exponent window and
    one far outside it, every rounding mode."""
    for name, x in [("normal", synth.draw("normal", (37, 768), 10 + m)), ("wide", wide_range((37, 768), 20 + m))]:
        for mode in MODES:
            announce("quantize_packed %s 37x768 m=%d %s" % (name, m, mode))
            check_packed(x, m, mode, seed=7 + m)


def test_packed_matches_chunk_plane_quantize_within_the_window():
    """Where every group's exponent is within 7 of the tensor's largest, the
    packed conversion is bfp_quantize's: the same magnitudes and exponents."""
    x = synth.draw("normal", (64, 1024), 5)
    emax = max_exponent_field(x)
    for m in (2, 4, 6, 8):
        for mode in MODES:
            announce("packed vs chunk-plane 64x1024 m=%d %s" % (m, mode))
            t, q_o, E_o = check_packed(x, m, mode, seed=3)
            assert E_o.min() >= emax - 7  # the input stays inside the window
            tp = fb.quantize(torch.from_numpy(x).cuda(), g=16, m=m, rounding=mode, seed=3)
            torch.cuda.synchronize()
            assert np.array_equal(tp.exp.cpu().numpy().astype(np.int64), E_o)
            assert np.array_equal(bfp_codec.decode(tp.mant.cpu().numpy(), 64, 1024, m), q_o)


def test_packed_edge_cases():
    """All zeros (E_max 0, base 0), one row of one group, a tensor whose
    largest exponent field is below 7 (base 0 clamps), and Inf input
    (status bit 0)."""
    for shape in [(3, 32), (1, 16)]:
        announce("quantize_packed zeros %s" % (shape,))
        t, q, E = check_packed(np.zeros(shape, np.float32), 4, "stochastic", seed=1)
        assert not q.any() and not E.any()
    tiny = (synth.draw("normal", (4, 64), 2) * np.float32(2.0 ** -124)).astype(np.float32)
    assert max_exponent_field(tiny) < 7
    for mode in MODES:
        announce("quantize_packed base clamped at 0, %s" % mode)
        check_packed(tiny, 6, mode, seed=2)
    x = synth.draw("normal", (2, 64), 3)
    x[1, 5] = np.inf
    announce("quantize_packed Inf input")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    fb.quantize_packed(torch.from_numpy(x).cuda(), m=4, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) & 1


@pytest.mark.parametrize("m", [1, 2, 4, 5, 6, 8])
def test_dequantize_packed(m):
    x = wide_range((33, 512), 30 + m)
    announce("dequantize_packed 33x512 m=%d" % m)
    t, q_o, E_o = check_packed(x, m, "stochastic", seed=9)
    y = fb.dequantize_packed(t).cpu().numpy().astype(np.float64)
    want = oracle.dequantize(q_o, E_o, 16, m)
    # FP32 flushes results below the normal range to zero
    want = np.where(np.abs(want) < 2.0 ** -126, 0.0, want)
    assert np.array_equal(y, want)


def check_gemm(A, B, qa, ea, qb, eb, m_a, m_b, exact=False):
    """bfp_gemm_packed (general kernel) and bfp_gemm_ws (unpacked into a
    workspace, block-scaled kernel), each against the oracle."""
    Co, S = oracle.gemm(qa, ea, A.m, qb, eb, B.m, g=16, m_a=m_a, m_b=m_b, threads=THREADS)
    for ws in (False, True):
        C = fb.gemm_packed(A, B, m_a, m_b, workspace=ws)
        torch.cuda.synchronize()
        Cg = C.cpu().numpy().astype(np.float64)
        err = np.abs(Cg - Co)
        assert np.all(err <= 1e-6 * S), "workspace=%s: max err/sum|T| = %.3g" % (
            ws, float((err / np.maximum(S, 1e-300)).max()))
        if exact:
            assert np.array_equal(Cg, Co), "workspace=%s: not exact" % ws


STORED = [(2, 2), (2, 4), (4, 2), (4, 4), (6, 6), (8, 8), (3, 5), (8, 1)]


@pytest.mark.parametrize("K", [16, 32, 128])
def test_gemm_packed_tiny_stacked(K):
    """100 seeds of M = N = 4 stacked (400 x 400 outputs) at every stored pair
    above and every lower precision of each operand; exact at K = 16."""
    xs = [synth.draw("normal", (8, K), 9000 + K + s) for s in range(100)]
    xa = np.ascontiguousarray(np.concatenate([x[:4] for x in xs]))
    xb = np.ascontiguousarray(np.concatenate([x[4:] for x in xs]))
    for am, bm in STORED:
        announce("gemm_packed stacked tiny K=%d stored (%d,%d)" % (K, am, bm))
        A, qa, ea = check_packed(xa, am, "stochastic", seed=11)
        B, qb, eb = check_packed(xb, bm, "nearest")
        pairs = {(ma, bm) for ma in range(1, am + 1)} | {(am, mb) for mb in range(1, bm + 1)}
        for m_a, m_b in sorted(pairs):
            check_gemm(A, B, qa, ea, qb, eb, m_a, m_b, exact=(K == 16))


def test_gemm_packed_ragged_and_wide_range():
    """Several 32 x 32 tiles with ragged edges; operands whose groups are
    raised to their tensor base."""
    for M, N, K in [(70, 45, 192), (257, 129, 1024)]:
        xa = wide_range((M, K), 40 + M)
        xb = synth.draw("weights", (N, K), 41 + N)
        for am, bm in [(2, 2), (4, 4), (2, 4), (4, 2), (6, 8)]:
            announce("gemm_packed %dx%dx%d (%d,%d)" % (M, N, K, am, bm))
            A, qa, ea = check_packed(xa, am, "stochastic", seed=5)
            B, qb, eb = check_packed(xb, bm, "nearest")
            check_gemm(A, B, qa, ea, qb, eb, am, bm)


def test_packed_full_size_sampled():
    """The bench's packed conversion (8192 x 8192 half-normal, seed 1234): the
    whole exponent stream (E_max word and every group's 3-bit offset), and the
    mantissa bytes of 32 sampled rows, against the oracle."""
    R = C = 8192
    x = synth.draw("half_normal", (R, C), 21)
    xt = torch.from_numpy(x).cuda()
    ng = R * C // 16
    emax = max_exponent_field(x)
    for m, mode in [(2, "stochastic"), (4, "nearest")]:
        announce("quantize_packed full size 8192x8192 m=%d %s" % (m, mode))
        t = fb.quantize_packed(xt, m=m, rounding=mode, seed=1234)
        torch.cuda.synchronize()
        q, E, base, bad = oracle.quantize_packed(x, g=16, m=m, mode=mode, seed=1234, threads=THREADS)
        assert bad == 0 and base == max(emax - 7, 0)
        exp = t.exp.cpu().numpy()
        stream = exp[4:]
        assert int(np.frombuffer(exp[:4].tobytes(), np.uint32)[0]) == emax
        gid = np.arange(ng)
        e3 = np.zeros(ng, np.int64)
        for b in range(3):
            pos = 3 * gid + b
            e3 |= ((stream[pos // 8].astype(np.int64) >> (pos % 8)) & 1) << b
        assert np.array_equal(base + e3, E.reshape(-1).astype(np.int64)), "exponent stream differs"
        mant = t.mant.cpu().numpy()
        npl = (m + 1) // 2
        for r0 in np.random.default_rng(m).choice(R // 8, 4, replace=False) * 8:
            g0, g1 = int(r0) * (C // 16), (int(r0) + 8) * (C // 16)
            sl = np.concatenate([mant[(c * ng + g0) * 6:(c * ng + g1) * 6] for c in range(npl)])
            want, _ = bfp_codec.encode_packed(q[r0:r0 + 8], E[r0:r0 + 8], emax, m)
            assert np.array_equal(sl, want), "mantissas of rows %d..%d differ" % (r0, r0 + 7)
