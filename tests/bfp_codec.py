"""Test-side codec for the BFP chunk-plane layout of include/fastbfp.h.

Written from the OCP MX definitions of FP6 E2M3 (1 sign bit, 2 exponent bits
with bias 1, 3 mantissa bits) and FP4 E2M1 (1 sign bit, 2 exponent bits with
bias 1, 1 mantissa bit); exponent field 0 is subnormal in both.  Independent
of the HIP kernels: it turns the library's packed mantissa bytes into signed
integer magnitudes +-q, and the oracle's +-q into the bytes the library must
write.  A plane whose chunk has at most 2 bits (plane 0 of m = 1, 2, 5, 6)
holds FP4 codes, every other plane FP6 codes; both encode +-chunk/2.
"""
from __future__ import annotations

import numpy as np


def e2m3_value(code: int) -> float:
    """Real value of a 6-bit FP6 E2M3 code."""
    s, e, f = (code >> 5) & 1, (code >> 3) & 3, code & 7
    v = f / 8.0 if e == 0 else 2.0 ** (e - 1) * (1.0 + f / 8.0)
    return -v if s else v


# Each code's chunk value (2 x its real value) where that is an integer 0..15.
_CODE_TO_CHUNK = np.full(64, 10 ** 6, dtype=np.int64)
_CHUNK_TO_CODE = {}
for _c in range(64):
    _v = 2.0 * e2m3_value(_c)
    if _v == int(_v) and abs(_v) <= 15:
        _CODE_TO_CHUNK[_c] = int(_v)
        if _c & 0x20 == 0 or _v != 0:
            _CHUNK_TO_CODE.setdefault(int(_v), _c)
_CHUNK_TO_CODE[0] = 0  # zero magnitudes are stored without a sign
assert sorted(_CHUNK_TO_CODE) == list(range(-15, 16))


def e2m1_value(code: int) -> float:
    """Real value of a 4-bit FP4 E2M1 code."""
    s, e, f = (code >> 3) & 1, (code >> 1) & 3, code & 1
    v = f / 2.0 if e == 0 else 2.0 ** (e - 1) * (1.0 + f / 2.0)
    return -v if s else v


# FP4: each code's chunk value (2 x its real value) where that is an integer 0..3.
_CODE4_TO_CHUNK = np.full(16, 10 ** 6, dtype=np.int64)
_CHUNK_TO_CODE4 = {}
for _c in range(16):
    _v = 2.0 * e2m1_value(_c)
    if _v == int(_v) and abs(_v) <= 3:
        _CODE4_TO_CHUNK[_c] = int(_v)
        if _c & 0x8 == 0 or _v != 0:
            _CHUNK_TO_CODE4.setdefault(int(_v), _c)
_CHUNK_TO_CODE4[0] = 0
assert sorted(_CHUNK_TO_CODE4) == list(range(-3, 4))


def n_planes(m: int) -> int:
    return 1 if m <= 4 else 2


def plane_fp4(m: int, p: int) -> bool:
    """True if plane p of an m-bit tensor holds FP4 codes (its chunk has at most 2 bits)."""
    chunk_bits = m if m <= 4 else (m - 4 if p == 0 else 4)
    return chunk_bits <= 2


def plane_bytes(rows: int, length: int, m: int, p: int) -> int:
    return rows * length * (4 if plane_fp4(m, p) else 6) // 8


def _split_planes(mant: np.ndarray, rows: int, length: int, m: int):
    b = np.ascontiguousarray(mant, dtype=np.uint8).reshape(-1)
    out, off = [], 0
    for p in range(n_planes(m)):
        nb = plane_bytes(rows, length, m, p)
        out.append(b[off:off + nb])
        off += nb
    assert off == b.size, "mantissa buffer size does not match the layout"
    return out


def unpack_codes(mant: np.ndarray, rows: int, length: int, m: int) -> list:
    """Per plane: the codes [rows, length] from the packed little-endian bytes
    (6-bit FP6 codes or 4-bit FP4 codes)."""
    planes = []
    for p, b in enumerate(_split_planes(mant, rows, length, m)):
        if plane_fp4(m, p):
            codes = np.stack([b & 15, b >> 4], axis=-1).astype(np.uint32)
        else:
            t = b.reshape(rows * length // 4, 3).astype(np.uint32)
            v = t[:, 0] | (t[:, 1] << 8) | (t[:, 2] << 16)
            codes = np.stack([(v >> (6 * k)) & 63 for k in range(4)], axis=-1)
        planes.append(codes.reshape(rows, length))
    return planes


def decode(mant: np.ndarray, rows: int, length: int, m: int) -> np.ndarray:
    """Signed magnitudes +-q [rows, length] (int32) from mantissa bytes."""
    codes = unpack_codes(mant, rows, length, m)
    chunks = [(_CODE4_TO_CHUNK if plane_fp4(m, p) else _CODE_TO_CHUNK)[c] for p, c in enumerate(codes)]
    if any(np.any(c == 10 ** 6) for c in chunks):
        raise AssertionError("a code does not stand for an integer chunk")
    if n_planes(m) == 1:
        return chunks[0].astype(np.int32)
    hi, lo = chunks[0], chunks[1]
    if np.any((hi != 0) & (lo != 0) & (np.sign(hi) != np.sign(lo))):
        raise AssertionError("the two chunks of a value carry different signs")
    return (hi * 16 + lo).astype(np.int32)


def encode(q: np.ndarray, m: int) -> np.ndarray:
    """The packed bytes (flat uint8) the library must write for +-q [rows, length]."""
    q = np.asarray(q, dtype=np.int64)
    rows, length = q.shape
    if n_planes(m) == 1:
        planes = [q]
    else:
        mag, sgn = np.abs(q), np.sign(q)
        planes = [sgn * (mag >> 4), sgn * (mag & 15)]
    lut = np.zeros(31, dtype=np.uint32)
    for c, code in _CHUNK_TO_CODE.items():
        lut[c + 15] = code
    lut4 = np.full(31, 1 << 20, dtype=np.uint32)  # out-of-range chunks make an invalid byte below
    for c, code in _CHUNK_TO_CODE4.items():
        lut4[c + 15] = code
    out = []
    for p, pl in enumerate(planes):
        if plane_fp4(m, p):
            codes = lut4[pl + 15].reshape(rows * length // 2, 2)
            if np.any(codes > 15):
                raise ValueError("a chunk does not fit an FP4 plane")
            out.append((codes[:, 0] | (codes[:, 1] << 4)).astype(np.uint8))
        else:
            codes = lut[pl + 15].reshape(rows * length // 4, 4)
            v = codes[:, 0] | (codes[:, 1] << 6) | (codes[:, 2] << 12) | (codes[:, 3] << 18)
            out.append(np.stack([v & 255, (v >> 8) & 255, (v >> 16) & 255], axis=-1).astype(np.uint8).reshape(-1))
    return np.concatenate(out)
