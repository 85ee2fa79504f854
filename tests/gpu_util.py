"""Helpers for the GPU parity tests: run a case through the C ABI (via the
binding) and the oracle on the same seeded inputs."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import bfp_codec
import paper_2110_15456_amd as fb

THREADS = 16


def chunk_drops(m: int):
    """The precisions bfp_gemm takes an m-bit operand at by reading fewer
    chunk planes: m itself, and for two planes the upper plane alone (q >> 2
    for m = 5, 6; q >> 4 for m = 7, 8)."""
    return [m] if m <= 4 else [m, m - (2 if m <= 6 else 4)]


def announce(msg: str) -> None:
    """Name the case on stdout before its GPU work starts."""
    sys.stdout.write("\n[case] %s\n" % msg)
    sys.stdout.flush()


def gpu_quantize(x: np.ndarray, axis: int, g: int, m: int, mode: str, seed: int = 0):
    xt = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    t = fb.quantize(xt, group_axis=axis, g=g, m=m, rounding=mode, seed=seed, status=st)
    torch.cuda.synchronize()
    return t, int(st.item())


def check_quantize(x: np.ndarray, axis: int, g: int, m: int, mode: str, seed: int = 0, rows=None):
    """Bit-exact comparison of exponents and packed mantissa bytes with the
    oracle (the oracle's magnitudes encoded by the test codec).  ``rows``: an
    output-row range (start, stop) to compare; default all."""
    t, st = gpu_quantize(x, axis, g, m, mode, seed)
    assert st == 0
    q_o, E_o = check_tensor(t, x, axis, g, m, mode, seed, rows)
    return t, q_o, E_o


def check_tensor(t, x: np.ndarray, axis: int, g: int, m: int, mode: str, seed: int = 0, rows=None):
    """A BFP tensor the library wrote (by any entry point) against the oracle's
    conversion of x along ``axis``: exponents and mantissa bytes of the output
    rows in ``rows`` (start, stop), default all.  Returns the oracle's (q, E)."""
    q_o, E_o, bad = oracle.quantize(x, axis=axis, g=g, m=m, mode=mode, seed=seed, threads=THREADS, rows=rows)
    assert bad == 0
    E = t.exp.cpu().numpy()
    mant = t.mant.cpu().numpy()
    r0, r1 = (0, t.rows) if rows is None else rows
    assert np.array_equal(E[r0:r1], E_o), "shared exponents differ"
    # the compared rows of every plane (each plane is rows x len codes)
    got, off = [], 0
    for p in range(bfp_codec.n_planes(m)):
        per_row = bfp_codec.plane_bytes(1, t.len, m, p)
        got.append(mant[off + r0 * per_row: off + r1 * per_row])
        off += bfp_codec.plane_bytes(t.rows, t.len, m, p)
    assert off == mant.size
    got = np.concatenate(got)
    want = bfp_codec.encode(q_o, m)
    if not np.array_equal(got, want):
        got_q = bfp_codec.decode(got, r1 - r0, t.len, m)
        bad_idx = np.argwhere(got_q != q_o)
        raise AssertionError("mantissas differ at %d positions, first %s: gpu %s oracle %s"
                             % (len(bad_idx), bad_idx[:3].tolist(), got_q[tuple(bad_idx[0])] if len(bad_idx) else None,
                                q_o[tuple(bad_idx[0])] if len(bad_idx) else None))
    return q_o, E_o
