"""Test-side codec for the BFP chunk-plane layout of include/fastbfp.h.

Written from the OCP MX definition of FP6 E2M3 (1 sign bit, 2 exponent bits
with bias 1, 3 mantissa bits; exponent field 0 is subnormal), independently of
the HIP kernels: it turns the library's packed mantissa bytes into signed
integer magnitudes +-q, and the oracle's +-q into the bytes the library must
write.
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


def n_planes(m: int) -> int:
    return 1 if m <= 4 else 2


def unpack_codes(mant: np.ndarray, rows: int, length: int, m: int) -> np.ndarray:
    """6-bit codes [planes, rows, length] from the packed little-endian bytes."""
    p = n_planes(m)
    b = np.ascontiguousarray(mant, dtype=np.uint8).reshape(p, rows * length // 4, 3).astype(np.uint32)
    v = b[..., 0] | (b[..., 1] << 8) | (b[..., 2] << 16)
    codes = np.stack([(v >> (6 * k)) & 63 for k in range(4)], axis=-1)
    return codes.reshape(p, rows, length)


def decode(mant: np.ndarray, rows: int, length: int, m: int) -> np.ndarray:
    """Signed magnitudes +-q [rows, length] (int32) from mantissa bytes."""
    codes = unpack_codes(mant, rows, length, m)
    chunks = _CODE_TO_CHUNK[codes]
    if np.any(chunks == 10 ** 6):
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
    out = []
    for pl in planes:
        codes = lut[pl + 15].reshape(rows * length // 4, 4)
        v = codes[:, 0] | (codes[:, 1] << 6) | (codes[:, 2] << 12) | (codes[:, 3] << 18)
        out.append(np.stack([v & 255, (v >> 8) & 255, (v >> 16) & 255], axis=-1).astype(np.uint8).reshape(-1))
    return np.concatenate(out)
