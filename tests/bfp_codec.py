"""Test-side codec for the BFP chunk-plane layout of include/fastbfp.h.

Written from the OCP MX definitions of FP6 E2M3 (1 sign bit, 2 exponent bits
with bias 1, 3 mantissa bits) and FP4 E2M1 (1 sign bit, 2 exponent bits with
bias 1, 1 mantissa bit); exponent field 0 is subnormal in both.  Independent
of the HIP kernels: it turns the library's packed mantissa bytes into signed
integer magnitudes +-q, and the oracle's +-q into the bytes the library must
write.

Planes: m = 1, 2: FP4 codes of +-q/2.  m = 3, 4: FP6 codes of +-q/2.
m = 5, 6: FP6 codes of +-(q >> 2)/2, then a "Lo2" plane of the 2-bit chunk
q & 3: per 16 values, the 96 bits T of their FP6 codes of +-(q & 3)/8 (three
little-endian dwords T0, T1, T2), stored as the two dwords T0 | (T1 >> 1) and
T2 (the FP6 code of a value below 1/2 has only its sign and two lowest bits
set, and T1's such bits moved down by one fill T0's zero bits).
m = 7, 8: FP6 codes of +-(q >> 4)/2 and of +-(q & 15)/2.
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
    """True if plane p of an m-bit tensor holds FP4 codes."""
    return m <= 2 and p == 0


def plane_lo2(m: int, p: int) -> bool:
    """True if plane p of an m-bit tensor is a Lo2 plane (the 2-bit low chunk of m = 5, 6)."""
    return m in (5, 6) and p == 1


def low_bits(m: int) -> int:
    """Bits of the lower chunk of a two-plane magnitude."""
    return 2 if m <= 6 else 4


def plane_bytes(rows: int, length: int, m: int, p: int) -> int:
    return rows * length * (4 if plane_fp4(m, p) or plane_lo2(m, p) else 6) // 8


def _field_bits():
    """Positions, in the 96 bits of 16 FP6 codes, that a code of +-c/8 with
    c <= 3 can set: each field's two lowest bits and its sign bit."""
    return [6 * t + b for t in range(16) for b in (0, 1, 5)]


_LO2_MASK = [sum(1 << (b - 32 * w) for b in _field_bits() if b // 32 == w) for w in range(3)]
assert _LO2_MASK[0] & (_LO2_MASK[1] >> 1) == 0 and _LO2_MASK[0] | (_LO2_MASK[1] >> 1) == 0xFFFFFFFF


def _e2m3_eighth_code(c: np.ndarray) -> np.ndarray:
    """FP6 E2M3 code of +-|c|/8 for |c| <= 3 (subnormal: mantissa field |c|),
    zero as code 0."""
    c = np.asarray(c, dtype=np.int64)
    if np.any(np.abs(c) > 3):
        raise ValueError("a chunk does not fit a Lo2 plane")
    code = np.abs(c) | np.where(c < 0, 32, 0)
    return code.astype(np.uint64)


# the subnormal codes 0..3 stand for 0, 1/8, 2/8, 3/8
assert [8 * e2m3_value(k) for k in range(4)] == [0, 1, 2, 3]


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
    (6-bit FP6 codes, also for a Lo2 plane after undoing its squeeze, or 4-bit
    FP4 codes)."""
    planes = []
    for p, b in enumerate(_split_planes(mant, rows, length, m)):
        if plane_lo2(m, p):
            d = b.reshape(-1, 8).astype(np.uint64)
            d0 = d[:, 0] | (d[:, 1] << 8) | (d[:, 2] << 16) | (d[:, 3] << 24)
            d1 = d[:, 4] | (d[:, 5] << 8) | (d[:, 6] << 16) | (d[:, 7] << 24)
            t0 = d0 & _LO2_MASK[0]
            t1 = (d0 << 1) & _LO2_MASK[1]
            if np.any(d1 & ~np.uint64(_LO2_MASK[2])):
                raise AssertionError("a Lo2 plane has bits set outside its codes")
            codes = np.zeros((d.shape[0], 16), np.uint32)
            for k in range(16):
                bit = 6 * k
                words = (t0, t1, d1)
                v = words[bit // 32] >> np.uint64(bit % 32)
                if bit % 32 > 26:
                    v = v | (words[bit // 32 + 1] << np.uint64(32 - bit % 32))
                codes[:, k] = (v & np.uint64(63)).astype(np.uint32)
        elif plane_fp4(m, p):
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
    chunks = []
    for p, c in enumerate(codes):
        if plane_lo2(m, p):
            v = np.array([8 * e2m3_value(int(k)) for k in range(64)])[c]
            if np.any((v != np.round(v)) | (np.abs(v) > 3)):
                raise AssertionError("a Lo2 code does not stand for a 2-bit chunk")
            chunks.append(v.astype(np.int64))
        else:
            chunks.append((_CODE4_TO_CHUNK if plane_fp4(m, p) else _CODE_TO_CHUNK)[c])
    if any(np.any(c == 10 ** 6) for c in chunks):
        raise AssertionError("a code does not stand for an integer chunk")
    if n_planes(m) == 1:
        return chunks[0].astype(np.int32)
    hi, lo = chunks[0], chunks[1]
    if np.any((hi != 0) & (lo != 0) & (np.sign(hi) != np.sign(lo))):
        raise AssertionError("the two chunks of a value carry different signs")
    return (hi * (1 << low_bits(m)) + lo).astype(np.int32)


def encode(q: np.ndarray, m: int) -> np.ndarray:
    """The packed bytes (flat uint8) the library must write for +-q [rows, length]."""
    q = np.asarray(q, dtype=np.int64)
    rows, length = q.shape
    if n_planes(m) == 1:
        planes = [q]
    else:
        mag, sgn = np.abs(q), np.sign(q)
        w = low_bits(m)
        planes = [sgn * (mag >> w), sgn * (mag & ((1 << w) - 1))]
    lut = np.zeros(31, dtype=np.uint32)
    for c, code in _CHUNK_TO_CODE.items():
        lut[c + 15] = code
    lut4 = np.full(31, 1 << 20, dtype=np.uint32)  # out-of-range chunks make an invalid byte below
    for c, code in _CHUNK_TO_CODE4.items():
        lut4[c + 15] = code
    out = []
    for p, pl in enumerate(planes):
        if plane_lo2(m, p):
            codes = _e2m3_eighth_code(pl).reshape(rows * length // 16, 16)
            t = [np.zeros(codes.shape[0], np.uint64) for _ in range(3)]
            for k in range(16):
                bit = 6 * k
                t[bit // 32] |= (codes[:, k] << np.uint64(bit % 32)) & np.uint64(0xFFFFFFFF)
                if bit % 32 > 26:
                    t[bit // 32 + 1] |= codes[:, k] >> np.uint64(32 - bit % 32)
            d0 = t[0] | (t[1] >> np.uint64(1))
            d1 = t[2]
            words = np.stack([d0, d1], axis=-1).astype(np.uint32)
            out.append(words.view(np.uint8).reshape(-1))
        elif plane_fp4(m, p):
            codes = lut4[pl + 15].reshape(rows * length // 2, 2)
            if np.any(codes > 15):
                raise ValueError("a chunk does not fit an FP4 plane")
            out.append((codes[:, 0] | (codes[:, 1] << 4)).astype(np.uint8))
        else:
            codes = lut[pl + 15].reshape(rows * length // 4, 4)
            v = codes[:, 0] | (codes[:, 1] << 6) | (codes[:, 2] << 12) | (codes[:, 3] << 18)
            out.append(np.stack([v & 255, (v >> 8) & 255, (v >> 16) & 255], axis=-1).astype(np.uint8).reshape(-1))
    return np.concatenate(out)


# ---------------------------------------------------------------------------
# Packed storage (section V-D): 2-bit chunks with the value's sign in 3-bit
# fields, ceil(m/2) planes, 16 fields per group in 6 bytes; a uint32 E_max
# word, then 3-bit exponent offsets above B = max(E_max - 7, 0).


def packed_planes(m: int) -> int:
    return (m + 1) // 2


def encode_packed(q: np.ndarray, E: np.ndarray, emax: int, m: int):
    """(mant, exp) bytes for +-q [rows, length] with group exponents E
    [rows, length/16] and the tensor's largest exponent field emax."""
    q = np.asarray(q, dtype=np.int64)
    rows, length = q.shape
    ng = rows * length // 16
    base = max(emax - 7, 0)
    e3 = np.asarray(E, dtype=np.int64).reshape(-1) - base
    if np.any((e3 < 0) | (e3 > 7)):
        raise ValueError("a group exponent is outside base .. base + 7")
    mag, neg = np.abs(q).reshape(ng, 16), (q < 0).reshape(ng, 16)
    npl = packed_planes(m)
    mant = np.zeros((npl, ng, 6), np.uint8)
    for c in range(npl):
        ch = (mag >> (2 * (npl - 1 - c))) & 3
        field = np.where(ch != 0, ch | (neg.astype(np.int64) << 2), 0)
        bits = np.zeros(ng, np.uint64)
        for t in range(16):
            bits |= field[:, t].astype(np.uint64) << np.uint64(3 * t)
        for k in range(6):
            mant[c, :, k] = ((bits >> np.uint64(8 * k)) & np.uint64(255)).astype(np.uint8)
    stream = np.zeros(24 * ((ng + 63) // 64), np.uint8)
    gid = np.arange(ng)
    for b in range(3):
        pos = 3 * gid + b
        np.add.at(stream, pos // 8, (((e3 >> b) & 1) << (pos % 8)).astype(np.uint8))  # distinct bits: add is OR
    exp = np.concatenate([np.frombuffer(np.uint32(emax).tobytes(), np.uint8), stream])
    return mant.reshape(-1), exp


def decode_packed(mant: np.ndarray, exp: np.ndarray, rows: int, length: int, m: int):
    """(+-q [rows, length] int32, E [rows, length/16] int64, emax) from packed
    bytes; raises if a nonzero chunk's sign disagrees with another's."""
    ng = rows * length // 16
    npl = packed_planes(m)
    mb = np.ascontiguousarray(mant, dtype=np.uint8).reshape(npl, ng, 6).astype(np.uint64)
    mag = np.zeros((ng, 16), np.int64)
    sgn = np.full((ng, 16), -1, np.int64)  # -1: no nonzero chunk seen yet
    for c in range(npl):
        bits = np.zeros(ng, np.uint64)
        for k in range(6):
            bits |= mb[c, :, k] << np.uint64(8 * k)
        for t in range(16):
            f = ((bits >> np.uint64(3 * t)) & np.uint64(7)).astype(np.int64)
            ch, s = f & 3, f >> 2
            if np.any((ch == 0) & (s == 1)):
                raise AssertionError("a zero chunk is stored with a sign")
            nz = ch != 0
            if np.any(nz & (sgn[:, t] >= 0) & (sgn[:, t] != s)):
                raise AssertionError("the chunks of a value carry different signs")
            sgn[nz, t] = s[nz]
            mag[:, t] = 4 * mag[:, t] + ch
    q = np.where(sgn == 1, -mag, mag).reshape(rows, length).astype(np.int32)
    eb = np.ascontiguousarray(exp, dtype=np.uint8)
    emax = int(np.frombuffer(eb[:4].tobytes(), np.uint32)[0])
    base = max(emax - 7, 0)
    stream = eb[4:]
    E = np.full(ng, base, np.int64)
    gid = np.arange(ng)
    for b in range(3):
        pos = 3 * gid + b
        E += ((stream[pos // 8].astype(np.int64) >> (pos % 8)) & 1) << b
    return q, E.reshape(rows, length // 16), emax
