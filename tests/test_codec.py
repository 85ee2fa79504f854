"""The test-side codec of the chunk-plane layout (CPU only): its FP6 and FP4
value tables against the OCP MX element-format definitions written out as
literal tables, and encode/decode round trips at every width, so that a codec
mistake cannot hide a kernel mistake (or invent one)."""
from __future__ import annotations

import numpy as np
import pytest

import bfp_codec

# OCP MX v1.0, FP4 E2M1: the eight positive values of codes 0..7.
E2M1_POSITIVE = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
# FP6 E2M3: codes 0..7 are subnormal (k/8), then 1.0..1.875, 2..3.75, 4..7.5.
E2M3_POSITIVE = [k / 8 for k in range(8)] + [1 + k / 8 for k in range(8)] + [2 + k / 4 for k in range(8)] + \
                [4 + k / 2 for k in range(8)]


def test_value_tables_match_the_format_definitions():
    assert [bfp_codec.e2m1_value(c) for c in range(8)] == E2M1_POSITIVE
    assert [bfp_codec.e2m1_value(c | 8) for c in range(8)] == [-v for v in E2M1_POSITIVE]
    assert [bfp_codec.e2m3_value(c) for c in range(32)] == E2M3_POSITIVE
    assert [bfp_codec.e2m3_value(c | 32) for c in range(32)] == [-v for v in E2M3_POSITIVE]


def test_fp4_code_is_sign_above_the_chunk():
    # +-c/2 for a 2-bit chunk c is the code (sign << 3) | c
    for c in range(4):
        assert bfp_codec.e2m1_value(c) == c / 2
        assert bfp_codec.e2m1_value(8 | c) == -c / 2


@pytest.mark.parametrize("m", range(1, 9))
def test_round_trip_and_sizes(m):
    rng = np.random.default_rng(m)
    rows, length = 3, 64
    q = rng.integers(-(2 ** m - 1), 2 ** m, size=(rows, length))
    b = bfp_codec.encode(q, m)
    bits = {1: 4, 2: 4, 3: 6, 4: 6, 5: 10, 6: 10, 7: 12, 8: 12}[m]  # m = 5, 6: FP6 + Lo2
    assert b.size == rows * length * bits // 8
    assert np.array_equal(bfp_codec.decode(b, rows, length, m), q)


def test_fp4_plane_packing_order():
    # value t of a group sits at bits 4t..4t+3 (low nibble first)
    q = np.zeros((1, 16), np.int64)
    q[0, 0], q[0, 1], q[0, 15] = 1, -3, 2
    b = bfp_codec.encode(q, 2)
    assert b.size == 8
    assert b[0] == (0x8 | 3) << 4 | 1 and b[7] == 2 << 4 and not b[1:7].any()
    # m = 6: the upper chunk q >> 2 = 13 in FP6 (-6.5: sign 32, exponent 3,
    # mantissa 5 -> code 61), then the 2-bit chunk q & 3 = 1 in the Lo2 plane
    # (-1/8: the subnormal code 32 | 1)
    q6 = np.zeros((1, 16), np.int64)
    q6[0, 0] = -(3 * 16 + 5)
    b6 = bfp_codec.encode(q6, 6)
    assert b6.size == 12 + 8
    assert b6[0] == 61 and not b6[1:12].any()
    assert b6[12] == 33 and not b6[13:].any()
    assert bfp_codec.decode(b6, 1, 16, 6)[0, 0] == -53


def test_lo2_plane_is_the_squeezed_fp6_codes():
    """The Lo2 plane of m = 5, 6 holds the FP6 codes of +-(q & 3)/8: per 16
    values the 96-bit code string T (dwords T0, T1, T2) stored as T0 | T1 >> 1
    and T2.  Checked on every value position against a direct bit string."""
    rng = np.random.default_rng(3)
    for _ in range(20):
        lo = rng.integers(-3, 4, 16)
        q = np.sign(lo) * (4 * rng.integers(0, 8, 16) + np.abs(lo))
        q[lo == 0] = 4 * rng.integers(0, 8, int((lo == 0).sum()))
        b = bfp_codec.encode(q.reshape(1, 16), 5)
        lo_bytes = b[12:20]
        T = 0
        for t in range(16):
            c = int(abs(q[t]) & 3)
            code = c | (32 if (q[t] < 0 and c) else 0)
            assert bfp_codec.e2m3_value(code) * 8 == (c if q[t] >= 0 else -c)
            T |= code << (6 * t)
        t0, t1, t2 = T & 0xFFFFFFFF, (T >> 32) & 0xFFFFFFFF, T >> 64
        d0, d1 = t0 | (t1 >> 1), t2
        assert int.from_bytes(lo_bytes[:4].tobytes(), "little") == d0
        assert int.from_bytes(lo_bytes[4:].tobytes(), "little") == d1
        assert np.array_equal(bfp_codec.decode(b, 1, 16, 5)[0], q)


def test_fp4_rejects_wide_chunks():
    with pytest.raises(ValueError):
        bfp_codec.encode(np.full((1, 16), 4), 2)


def test_packed_fields_worked_by_hand():
    """Section V-D's chunk storage at m = 4: q = 5 (chunks 01, 01), q = -3
    (chunks 00, 11 with the sign), q = 0 and q = -12 (chunks 11, 00 with the
    sign) as the first four values of one group; the other values are zero."""
    q = np.zeros((1, 16), np.int64)
    q[0, :4] = [5, -3, 0, -12]
    mant, exp = bfp_codec.encode_packed(q, np.array([[130]]), emax=133, m=4)
    # plane 0 (upper chunks): fields 1, 0, 0, 4|3 -> bits 1 | 7 << 9
    # plane 1 (lower chunks): fields 1, 4|3, 0, 0 -> bits 1 | 7 << 3
    p0 = 1 | (7 << 9)
    p1 = 1 | (7 << 3)
    assert mant.tolist() == [p0 & 255, p0 >> 8, 0, 0, 0, 0, p1 & 255, p1 >> 8, 0, 0, 0, 0]
    # E_max 133 -> base 126; the group's offset 130 - 126 = 4 in bits 0..2
    assert exp.tolist() == [133, 0, 0, 0, 4] + [0] * 23
    q2, E2, emax = bfp_codec.decode_packed(mant, exp, 1, 16, 4)
    assert np.array_equal(q2, q) and E2.tolist() == [[130]] and emax == 133


@pytest.mark.parametrize("m", range(1, 9))
def test_packed_round_trip_and_sizes(m):
    rng = np.random.default_rng(100 + m)
    rows, length = 5, 16 * 29  # 145 groups: two full blocks of 64 and a partial one
    q = rng.integers(-(2 ** m - 1), 2 ** m, size=(rows, length))
    E = rng.integers(200, 208, size=(rows, length // 16))
    mant, exp = bfp_codec.encode_packed(q, E, emax=207, m=m)
    ng = rows * length // 16
    assert mant.size == ((m + 1) // 2) * 6 * ng and exp.size == 4 + 24 * 3
    q2, E2, emax = bfp_codec.decode_packed(mant, exp, rows, length, m)
    assert np.array_equal(q2, q) and np.array_equal(E2, E) and emax == 207
    # the exponent fields cross byte boundaries: group 1's bits are 3..5, group 2's 6..8
    assert (int(exp[4]) >> 3) & 7 == E.reshape(-1)[1] - 200
    assert ((int(exp[4]) >> 6) | (int(exp[5]) << 2)) & 7 == E.reshape(-1)[2] - 200


def test_packed_rejects_exponents_outside_the_window():
    q = np.zeros((1, 16), np.int64)
    with pytest.raises(ValueError):
        bfp_codec.encode_packed(q, np.array([[100]]), emax=120, m=2)  # 100 < 113
