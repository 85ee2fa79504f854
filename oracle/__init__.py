"""Plain CPU oracle for the FAST BFP hot path (test infrastructure only).

The arithmetic lives in ``oracle.c`` (plain C, exact integer / double
arithmetic, following the paper's conversion steps of section III-A and the
group dot product of section III-B).  This module only builds it with gcc,
loads it with ctypes and splits rows over host threads; ctypes releases the
GIL during each call, so the threads run the C loops in parallel.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
import subprocess
import threading
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

NEAREST, STOCHASTIC, TRUNCATE = 0, 1, 2
_MODES = {"nearest": NEAREST, "stochastic": STOCHASTIC, "truncate": TRUNCATE}

_lock = threading.Lock()
_lib = None


def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile oracle.c (or another C source, e.g. a planted-mistake copy in a
    test) into a shared library (gcc, no GPU code)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared",
                               src, "-o", tmp, "-lm"])
        os.replace(tmp, out)
    return out


def _bind(lib):
    """Declare the ctypes signatures of the oracle's C functions on ``lib``."""
    P = ctypes.c_void_p
    i64, i32, u64 = ctypes.c_int64, ctypes.c_int, ctypes.c_uint64
    lib.oracle_philox4x32_10.argtypes = [P, P, P]
    lib.oracle_noise_byte.argtypes = [u64, u64, ctypes.c_uint32]
    lib.oracle_noise_byte.restype = ctypes.c_uint32
    lib.oracle_noise_bytes.argtypes = [u64, u64, i64, i32, P]
    lib.oracle_quantize_group.argtypes = [P, i64, i32, i32, i32, P, P, i64, P]
    lib.oracle_quantize_group.restype = i32
    lib.oracle_quantize.argtypes = [P, i64, i64, i32, i32, i32, i32, u64, i64, i64, P, P]
    lib.oracle_quantize.restype = i64
    lib.oracle_quantize_group_floor.argtypes = [P, i64, i32, i32, i32, P, P, i64, P, i32]
    lib.oracle_quantize_group_floor.restype = i32
    lib.oracle_quantize_floor.argtypes = [P, i64, i64, i32, i32, i32, i32, u64, i32, i64, i64, P, P]
    lib.oracle_quantize_floor.restype = i64
    lib.oracle_exponent_base.argtypes = [P, i64, i32]
    lib.oracle_exponent_base.restype = i32
    lib.oracle_dequantize.argtypes = [P, P, i64, i32, i32, i64, i64, P]
    lib.oracle_gemm.argtypes = [P, P, i32, P, P, i32, i64, i64, i64, i32, i32, i32, P, i64, P, P]
    lib.oracle_group_partials.argtypes = [P, i32, P, i32, i64, i64, i32, i32, i32, P, i64, P]
    lib.oracle_relative_improvement.argtypes = [P, P, P, P, i64, i32, i64, i64, P, P]
    lib.oracle_drop_low_chunk.argtypes = [P, i64, P]
    lib.oracle_threshold.argtypes = [ctypes.c_double, ctypes.c_double, i64, i64, i64, i64]
    lib.oracle_threshold.restype = ctypes.c_double
    lib.oracle_select_mantissa.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_double]
    lib.oracle_select_mantissa.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
            _lib = _bind(ctypes.CDLL(_LIB))
    return _lib


@contextlib.contextmanager
def use_library(path: str):
    """Run the oracle's Python functions on another build of its C source (the
    mutation test plants mistakes in copies of oracle.c this way); the
    default library is restored on exit."""
    global _lib
    prev = _load()
    with _lock:
        _lib = _bind(ctypes.CDLL(path))
    try:
        yield
    finally:
        with _lock:
            _lib = prev


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def _split(n: int, threads: int):
    threads = max(1, min(threads, n)) if n > 0 else 1
    step = (n + threads - 1) // threads if n > 0 else 0
    return [(s, min(n, s + step)) for s in range(0, n, step)] if n > 0 else []


def _run(chunks, fn, threads):
    if len(chunks) <= 1 or threads <= 1:
        return [fn(a, b) for a, b in chunks]
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(lambda ab: fn(*ab), chunks))


def philox4x32_10(counter, key) -> np.ndarray:
    """One Philox4x32-10 block: 4 uint32 counter words, 2 uint32 key words."""
    lib = _load()
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, np.uint32)
    lib.oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def noise_byte(seed: int, gid: int, p: int) -> int:
    """Stochastic-rounding noise byte of position p in group gid."""
    return int(_load().oracle_noise_byte(seed, gid, p))


def noise_bytes(seed: int, gid0: int, ngroups: int, g: int = 16) -> np.ndarray:
    """Noise bytes of groups gid0 .. gid0 + ngroups - 1: uint8 [ngroups, g]."""
    out = np.zeros((ngroups, g), np.uint8)
    _load().oracle_noise_bytes(seed, gid0, ngroups, g, _ptr(out))
    return out


def quantize_group(x, m: int, mode="nearest", noise=None):
    """Quantize one group (1-D float32 array).  Returns (q int16 array, E int, bad)."""
    lib = _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    g = x.shape[0]
    nz = np.zeros(g, np.uint8) if noise is None else np.ascontiguousarray(noise, dtype=np.uint8)
    q = np.zeros(g, np.int16)
    E = np.zeros(1, np.uint8)
    bad = lib.oracle_quantize_group(_ptr(x), 1, g, m, _MODES.get(mode, mode), _ptr(nz), _ptr(q), 1, _ptr(E))
    return q, int(E[0]), bool(bad)


def quantize_group_floor(x, m: int, mode="nearest", noise=None, emin: int = 0):
    """quantize_group with the shared exponent raised to at least emin."""
    lib = _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    g = x.shape[0]
    nz = np.zeros(g, np.uint8) if noise is None else np.ascontiguousarray(noise, dtype=np.uint8)
    q = np.zeros(g, np.int16)
    E = np.zeros(1, np.uint8)
    bad = lib.oracle_quantize_group_floor(_ptr(x), 1, g, m, _MODES.get(mode, mode), _ptr(nz), _ptr(q), 1, _ptr(E), emin)
    return q, int(E[0]), bool(bad)


def exponent_base(x, ebits: int = 3) -> int:
    """The packed layout's tensor exponent base: max exponent field - (2^ebits - 1), at least 0."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return int(_load().oracle_exponent_base(_ptr(x), x.size, ebits))


def quantize_packed(x, g: int = 16, m: int = 2, mode="nearest", seed: int = 0, ebits: int = 3, threads: int = 1):
    """The packed layout's conversion (groups along rows): the tensor base, then
    every group at max(its exponent, base).  Returns (q, E, base, bad)."""
    lib = _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim != 2:
        raise ValueError("oracle.quantize_packed takes a 2-D array")
    R, C = x.shape
    base = exponent_base(x, ebits)
    q = np.zeros((R, C), np.int16)
    E = np.zeros((R, C // g), np.uint8)
    md = _MODES.get(mode, mode)

    def work(a, b):
        return lib.oracle_quantize_floor(_ptr(x), R, C, 1, g, m, md, seed, base, a, b, _ptr(q[a:]), _ptr(E[a:]))

    bad = sum(_run(_split(R, threads), work, threads))
    return q, E, base, bad


def quantize(x, axis: int = -1, g: int = 16, m: int = 4, mode="nearest", seed: int = 0, threads: int = 1,
             rows=None):
    """Quantize a 2-D float32 matrix along ``axis`` (-1/1: rows, 0: columns).

    Returns ``(q, E, bad)``: q int16 [out_rows, out_len] holds sign * magnitude,
    E uint8 [out_rows, out_len // g] the shared exponents, with the group axis
    last (for axis 0 the output is laid out transposed).  ``rows`` optionally
    restricts the computation to a contiguous output-row range (start, stop);
    the returned arrays then hold only those rows.
    """
    lib = _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim != 2:
        raise ValueError("oracle.quantize takes a 2-D array")
    R, C = x.shape
    ax = 1 if axis in (-1, 1) else 0
    out_rows, out_len = (R, C) if ax == 1 else (C, R)
    if out_len % g:
        raise ValueError("group size must divide the grouped axis")
    r0, r1 = (0, out_rows) if rows is None else rows
    q = np.zeros((r1 - r0, out_len), np.int16)
    E = np.zeros((r1 - r0, out_len // g), np.uint8)
    md = _MODES.get(mode, mode)

    def work(a, b):
        # a, b are absolute output rows; the C code offsets its writes by r0
        # only through the base pointers given here.
        qa = q[a - r0:]
        ea = E[a - r0:]
        return lib.oracle_quantize(_ptr(x), R, C, ax, g, m, md, seed, a, b, _ptr(qa), _ptr(ea))

    bad = sum(_run([(a + r0, b + r0) for a, b in _split(r1 - r0, threads)], work, threads))
    return q, E, bad


def dequantize(q, E, g: int, m: int) -> np.ndarray:
    lib = _load()
    q = np.ascontiguousarray(q, dtype=np.int16)
    E = np.ascontiguousarray(E, dtype=np.uint8)
    rows, n = q.shape
    y = np.zeros((rows, n), np.float64)
    lib.oracle_dequantize(_ptr(q), _ptr(E), n, g, m, 0, rows, _ptr(y))
    return y


def gemm(qa, ea, a_m, qb, eb, b_m, g: int = 16, m_a=None, m_b=None, rows=None, threads: int = 1):
    """BFP C = A * B^T in double.  Returns (C, sumabs) for the selected A rows.

    qa [M, K], ea [M, K/g]; qb [N, K], eb [N, K/g]; ``rows``: optional 1-D
    array of A row indices (default: all rows).
    """
    lib = _load()
    qa = np.ascontiguousarray(qa, dtype=np.int16)
    qb = np.ascontiguousarray(qb, dtype=np.int16)
    ea = np.ascontiguousarray(ea, dtype=np.uint8)
    eb = np.ascontiguousarray(eb, dtype=np.uint8)
    M, K = qa.shape
    N = qb.shape[0]
    m_a = a_m if m_a is None else m_a
    m_b = b_m if m_b is None else m_b
    idx = np.arange(M, dtype=np.int64) if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    n = idx.shape[0]
    C = np.zeros((n, N), np.float64)
    S = np.zeros((n, N), np.float64)

    def work(a, b):
        sub = np.ascontiguousarray(idx[a:b])
        lib.oracle_gemm(_ptr(qa), _ptr(ea), a_m, _ptr(qb), _ptr(eb), b_m, M, N, K, g, m_a, m_b,
                        _ptr(sub), b - a, _ptr(C[a:b]), _ptr(S[a:b]))

    _run(_split(n, threads), work, threads)
    return C, S


def group_partials(qa, a_m, qb, b_m, g: int = 16, m_a=None, m_b=None, rows=None) -> np.ndarray:
    """Integer group partials P [K/g, len(rows), N] (int64)."""
    lib = _load()
    qa = np.ascontiguousarray(qa, dtype=np.int16)
    qb = np.ascontiguousarray(qb, dtype=np.int16)
    M, K = qa.shape
    N = qb.shape[0]
    m_a = a_m if m_a is None else m_a
    m_b = b_m if m_b is None else m_b
    idx = np.arange(M, dtype=np.int64) if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    P = np.zeros((K // g, idx.shape[0], N), np.int64)
    lib.oracle_group_partials(_ptr(qa), a_m, _ptr(qb), b_m, N, K, g, m_a, m_b, _ptr(idx), idx.shape[0], _ptr(P))
    return P


def relative_improvement(q4, e4, q2, e2, g: int = 16) -> float:
    """r(X) of Eq. 2 from the m=4 and m=2 quantizations of the same tensor."""
    lib = _load()
    arrs = [np.ascontiguousarray(a, dtype=t) for a, t in
            ((q4, np.int16), (e4, np.uint8), (q2, np.int16), (e2, np.uint8))]
    rows, n = arrs[0].shape
    num = np.zeros(1, np.float64)
    den = np.zeros(1, np.float64)
    lib.oracle_relative_improvement(*[_ptr(a) for a in arrs], n, g, 0, rows, _ptr(num), _ptr(den))
    return float(num[0] / den[0]) if den[0] != 0 else 0.0


def drop_low_chunk(q4) -> np.ndarray:
    """BFP(X,2) mantissas from the stored 4-bit ones: sign * (|q4| >> 2) (section V-D)."""
    lib = _load()
    q4 = np.ascontiguousarray(q4, dtype=np.int16)
    q2 = np.empty_like(q4)
    lib.oracle_drop_low_chunk(_ptr(q4), q4.size, _ptr(q2))
    return q2


def improvement_sums(q4, e4, g: int = 16):
    """Numerator and denominator of Eq. 2 with BFP(X,2) the chunk-dropped BFP(X,4)."""
    lib = _load()
    q4 = np.ascontiguousarray(q4, dtype=np.int16)
    e4 = np.ascontiguousarray(e4, dtype=np.uint8)
    q2 = drop_low_chunk(q4)
    rows, n = q4.shape
    num = np.zeros(1, np.float64)
    den = np.zeros(1, np.float64)
    lib.oracle_relative_improvement(_ptr(q4), _ptr(e4), _ptr(q2), _ptr(e4), n, g, 0, rows, _ptr(num), _ptr(den))
    return float(num[0]), float(den[0])


def threshold(alpha: float, beta: float, i: int, I: int, l: int, L: int) -> float:
    """Eq. 1."""
    return float(_load().oracle_threshold(alpha, beta, i, I, l, L))


def select_mantissa(num: float, den: float, eps: float) -> int:
    """Algorithm 1's per-tensor choice (2 or 4 bits)."""
    return int(_load().oracle_select_mantissa(num, den, eps))



def quantize_dual(x, g: int = 16, m: int = 4, mode="nearest", seed_rows: int = 0, seed_cols: int = 0,
                  threads: int = 1):
    """Both groupings of one matrix, by definition two conversions (section
    III-A): along its rows with seed_rows and down its columns with seed_cols.
    Returns ((q_r, E_r), (q_c, E_c), nonfinite groups)."""
    qr, er, br = quantize(x, axis=-1, g=g, m=m, mode=mode, seed=seed_rows, threads=threads)
    qc, ec, bc = quantize(x, axis=0, g=g, m=m, mode=mode, seed=seed_cols, threads=threads)
    return (qr, er), (qc, ec), br + bc


def _flush(x: np.ndarray) -> np.ndarray:
    """Subnormal FP32 values to zero of the same sign."""
    x = np.asarray(x, dtype=np.float32)
    return np.where(np.abs(x) < np.finfo(np.float32).tiny, np.copysign(np.float32(0.0), x), x).astype(np.float32)


def weight_update(w, dw, alpha: float) -> np.ndarray:
    """The updated weights of the training workflow's last step (the weight
    gradient added to the weights, section V-A): w + alpha * dw in FP32, the
    product and the sum each rounded to nearest-even (numpy's float32
    arithmetic; no fused multiply-add).  Subnormal inputs, product and sum
    are read as / flushed to zero of the same sign, as the converter reads
    subnormal inputs."""
    w = _flush(w)
    dw = _flush(dw)
    prod = _flush(np.float32(_flush(np.float32(alpha))) * dw)
    return _flush(w + prod)
