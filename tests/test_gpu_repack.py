"""GPU parity of bfp_repack against the oracle: the repacked bytes must be the
oracle's magnitudes truncated to m_use bits (sign * (|q| >> (m - m_use)),
the discard of low-order bits of section V-D), laid out as the header says --
groups of 4 and 8 as zero-padded 16-value units, groups of 64 as two groups of
32 sharing the exponent, packed storage unpacked -- and encoded by the test
codec, exponents alike."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import bfp_codec
import oracle
import paper_2110_15456_amd as fb
from paper_2110_15456_amd import synth
from gpu_util import announce, check_quantize, THREADS

pytestmark = pytest.mark.gpu


def expected(q, E, g, m, m_use):
    """The repacked (q, E) the oracle's stored (q, E) stand for."""
    q = np.asarray(q, np.int64)
    mag = np.abs(q) >> (m - m_use)
    qu = np.where(q < 0, -mag, mag)
    rows, length = q.shape
    if g < 16:
        out = np.zeros((rows, length // g, 16), np.int64)
        out[:, :, :g] = qu.reshape(rows, length // g, g)
        return out.reshape(rows, -1), np.asarray(E)
    if g == 64:
        return qu, np.repeat(np.asarray(E), 2, axis=1)
    return qu, np.asarray(E)


def check_repacked(r, q_want, E_want, m_use):
    assert r.m == m_use and r.len == q_want.shape[1]
    assert np.array_equal(r.exp.cpu().numpy().astype(np.int64), E_want.astype(np.int64)), "exponents differ"
    got = r.mant.cpu().numpy()
    want = bfp_codec.encode(q_want, m_use)
    if not np.array_equal(got, want):
        gq = bfp_codec.decode(got, r.rows, r.len, m_use)
        bad = np.argwhere(gq != q_want)
        raise AssertionError("repacked magnitudes differ at %d positions, first %s" % (len(bad), bad[:3].tolist()))


@pytest.mark.parametrize("g", [4, 8, 16, 32, 64])
def test_repack_chunk_planes(g):
    """37 x 512 (several workgroups, a partial last one), every stored width
    and every lower precision of it."""
    x = synth.draw("grads", (37, 512), 60 + g)
    for m in range(1, 9):
        t, q, E = check_quantize(x, -1, g, m, "stochastic", seed=m)
        for m_use in range(1, m + 1):
            announce("repack g=%d stored %d used %d" % (g, m, m_use))
            r = fb.repack(t, m_use)
            torch.cuda.synchronize()
            assert r.g == (16 if g <= 16 else 32)
            q_want, E_want = expected(q, E, g, m, m_use)
            check_repacked(r, q_want, E_want, m_use)


def test_repack_packed_storage():
    x = synth.draw("normal", (21, 256), 71)
    for m in (2, 4, 5, 8):
        xt = torch.from_numpy(x).cuda()
        t = fb.quantize_packed(xt, m=m, rounding="nearest")
        q, E, base, bad = oracle.quantize_packed(x, g=16, m=m, mode="nearest", threads=THREADS)
        assert bad == 0
        for m_use in sorted({1, m // 2 or 1, m}):
            announce("repack packed stored %d used %d" % (m, m_use))
            r = fb.repack(t, m_use)
            torch.cuda.synchronize()
            q_want, E_want = expected(q, E, 16, m, m_use)
            check_repacked(r, q_want, E_want, m_use)


def check_both_paths(A, B, qa, ea, qb, eb, g, m_a, m_b, exact=False):
    """The workspace path (repack + block-scaled kernel) and the general
    kernel, each against the oracle."""
    gemm = fb.gemm_packed if isinstance(A, fb.PackedBFPTensor) else fb.gemm
    Co, S = oracle.gemm(qa, ea, A.m, qb, eb, B.m, g=g, m_a=m_a, m_b=m_b, threads=THREADS)
    for ws in (True, False):
        C = gemm(A, B, m_a, m_b, workspace=ws)
        torch.cuda.synchronize()
        Cg = C.cpu().numpy().astype(np.float64)
        err = np.abs(Cg - Co)
        assert np.all(err <= 1e-6 * S), "workspace=%s: max err/sum|T| = %.3g" % (
            ws, float((err / np.maximum(S, 1e-300)).max()))
        if exact:
            assert np.array_equal(Cg, Co), "workspace=%s: not exact" % ws


@pytest.mark.parametrize("g", [4, 8, 64])
def test_gemm_ws_group_sizes(g):
    """Several tiles of the block-scaled kernel with ragged edges, groups of
    4, 8 and 64 at every operand format pair shown."""
    for M, N, K in [(70, 45, 192), (300, 257, 1024)]:
        xa = synth.draw("half_normal", (M, K), 90 + M + g)
        xb = synth.draw("weights", (N, K), 91 + N + g)
        for am, bm in [(2, 2), (4, 4), (2, 6), (6, 6), (8, 8), (6, 3), (5, 7)]:
            announce("gemm_ws g=%d %dx%dx%d (%d,%d)" % (g, M, N, K, am, bm))
            A, qa, ea = check_quantize(xa, -1, g, am, "nearest")
            B, qb, eb = check_quantize(xb, -1, g, bm, "stochastic", seed=4)
            check_both_paths(A, B, qa, ea, qb, eb, g, am, bm)


@pytest.mark.parametrize("g", [16, 32])
def test_gemm_ws_lowered_precisions(g):
    """Every precision between chunk boundaries on a full-slab shape with a
    ragged edge (the paper's stored 4 used at 2 among them)."""
    M, N, K = 260, 130, 512
    xa = synth.draw("normal", (M, K), 93)
    xb = synth.draw("weights", (N, K), 94)
    for am, bm in [(4, 4), (6, 6), (8, 8), (3, 7)]:
        A, qa, ea = check_quantize(xa, -1, g, am, "stochastic", seed=2)
        B, qb, eb = check_quantize(xb, -1, g, bm, "nearest")
        pairs = {(ma, bm) for ma in range(1, am + 1)} | {(am, mb) for mb in range(1, bm + 1)} | {(2, 2)}
        for m_a, m_b in sorted(p for p in pairs if p[0] <= am and p[1] <= bm):
            announce("gemm_ws g=%d stored (%d,%d) at (%d,%d)" % (g, am, bm, m_a, m_b))
            check_both_paths(A, B, qa, ea, qb, eb, g, m_a, m_b)


@pytest.mark.parametrize("g", [4, 8, 16, 32, 64])
def test_gemm_ws_one_group_exact(g):
    """K = max(g, 16) on stacked tiny cases (40 seeds of M = N = 4): with g >= 16
    one group, so the FP32 result is the oracle's exact value."""
    K = max(g, 16)
    xs = [synth.draw("normal", (8, K), 7100 + K + s) for s in range(40)]
    xa = np.ascontiguousarray(np.concatenate([x[:4] for x in xs]))
    xb = np.ascontiguousarray(np.concatenate([x[4:] for x in xs]))
    for am, bm in [(4, 4), (6, 8), (8, 2)]:
        A, qa, ea = check_quantize(xa, -1, g, am, "stochastic", seed=5)
        B, qb, eb = check_quantize(xb, -1, g, bm, "nearest")
        for m_a, m_b in [(am, bm), (am - 1, bm), (1, 1)]:
            announce("gemm_ws tiny g=%d K=%d stored (%d,%d) at (%d,%d)" % (g, K, am, bm, m_a, m_b))
            check_both_paths(A, B, qa, ea, qb, eb, g, m_a, m_b, exact=(K == g))


def test_gemm_ws_packed():
    """Packed operands through the workspace (unpacked, block-scaled kernel)
    and on the general kernel."""
    for M, N, K in [(70, 45, 192), (257, 129, 1024)]:
        xa = synth.draw("grads", (M, K), 95 + M)
        xb = synth.draw("weights", (N, K), 96 + N)
        for am, bm in [(2, 2), (4, 4), (2, 4), (6, 8)]:
            announce("gemm_ws packed %dx%dx%d (%d,%d)" % (M, N, K, am, bm))
            A = fb.quantize_packed(torch.from_numpy(xa).cuda(), m=am, rounding="stochastic", seed=6)
            B = fb.quantize_packed(torch.from_numpy(xb).cuda(), m=bm, rounding="nearest")
            qa, ea, _, _ = oracle.quantize_packed(xa, g=16, m=am, mode="stochastic", seed=6, threads=THREADS)
            qb, eb, _, _ = oracle.quantize_packed(xb, g=16, m=bm, mode="nearest", threads=THREADS)
            check_both_paths(A, B, qa, ea, qb, eb, 16, am, bm)
            check_both_paths(A, B, qa, ea, qb, eb, 16, max(1, am - 1), bm)


def test_gemm_ws_caller_workspace_reused():
    """One caller workspace for two calls in a row, the second smaller."""
    ws = torch.empty(1 << 22, dtype=torch.uint8, device="cuda")
    for M, N, K in [(128, 96, 256), (40, 24, 64)]:
        xa = synth.draw("normal", (M, K), 97)
        xb = synth.draw("normal", (N, K), 98)
        A, qa, ea = check_quantize(xa, -1, 8, 4, "nearest")
        B, qb, eb = check_quantize(xb, -1, 8, 4, "nearest")
        announce("gemm_ws caller workspace %dx%dx%d" % (M, N, K))
        assert fb.gemm_ws_size(A, B) <= ws.numel()
        C = fb.gemm(A, B, workspace=ws)
        torch.cuda.synchronize()
        Co, S = oracle.gemm(qa, ea, 4, qb, eb, 4, g=8, threads=THREADS)
        assert np.all(np.abs(C.cpu().numpy().astype(np.float64) - Co) <= 1e-6 * S)


def test_gemm_ws_full_size_sampled():
    """The format sweep's out-projection GEMM (8192 x 4096 x 4096, the bench's
    inputs) on both routes: 48 sampled rows of C (all 4096 columns) against the
    oracle, for packed operands, groups of 8 and 64, and precisions below the
    stored width."""
    M, N, K = 8192, 4096, 4096
    xa = synth.bf16_round(synth.draw("normal", (M, K), 41))
    xb = synth.bf16_round(synth.draw("weights", (N, K), 42))
    ta, tb = torch.from_numpy(xa).cuda(), torch.from_numpy(xb).cuda()
    rows = np.sort(np.random.default_rng(7).choice(M, 48, replace=False))
    cases = [("packed", 16, 2, 2, 2, 2), ("packed", 16, 4, 4, 3, 4), ("chunk", 8, 4, 4, 4, 4),
             ("chunk", 64, 4, 4, 4, 4), ("chunk", 16, 4, 4, 2, 2), ("chunk", 16, 6, 6, 3, 3)]
    for kind, g, am, bm, m_a, m_b in cases:
        announce("gemm_ws full size 8192x4096x4096 %s g=%d stored (%d,%d) at (%d,%d)" % (kind, g, am, bm, m_a, m_b))
        if kind == "packed":
            A, B = fb.quantize_packed(ta, m=am), fb.quantize_packed(tb, m=bm)
            qa, ea, _, _ = oracle.quantize_packed(xa, g=16, m=am, threads=THREADS)
            qb, eb, _, _ = oracle.quantize_packed(xb, g=16, m=bm, threads=THREADS)
        else:
            A, B = fb.quantize(ta, g=g, m=am), fb.quantize(tb, g=g, m=bm)
            qa, ea, _ = oracle.quantize(xa, g=g, m=am, threads=THREADS)
            qb, eb, _ = oracle.quantize(xb, g=g, m=bm, threads=THREADS)
        if kind == "chunk":  # (the packed exponent stream is checked in full in test_gpu_packed.py)
            assert np.array_equal(A.exp.cpu().numpy()[rows], ea[rows])
        Co, S = oracle.gemm(qa, ea, am, qb, eb, bm, g=g, m_a=m_a, m_b=m_b, rows=rows, threads=THREADS)
        gemm = fb.gemm_packed if kind == "packed" else fb.gemm
        for ws in (True, False):
            C = gemm(A, B, m_a, m_b, workspace=ws)
            torch.cuda.synchronize()
            Cg = C[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
            err = np.abs(Cg - Co)
            assert np.all(err <= 1e-6 * S), "workspace=%s: max err/sum|T| = %.3g" % (
                ws, float((err / np.maximum(S, 1e-300)).max()))
        del A, B, C
