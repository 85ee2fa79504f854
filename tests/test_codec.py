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
    bits = {1: 4, 2: 4, 3: 6, 4: 6, 5: 10, 6: 10, 7: 12, 8: 12}[m]
    assert b.size == rows * length * bits // 8
    assert np.array_equal(bfp_codec.decode(b, rows, length, m), q)


def test_fp4_plane_packing_order():
    # value t of a group sits at bits 4t..4t+3 (low nibble first)
    q = np.zeros((1, 16), np.int64)
    q[0, 0], q[0, 1], q[0, 15] = 1, -3, 2
    b = bfp_codec.encode(q, 2)
    assert b.size == 8
    assert b[0] == (0x8 | 3) << 4 | 1 and b[7] == 2 << 4 and not b[1:7].any()
    # m = 6: the upper chunk (q >> 4, two bits) in FP4, then the lower chunk in FP6
    q6 = np.zeros((1, 16), np.int64)
    q6[0, 0] = -(3 * 16 + 5)
    b6 = bfp_codec.encode(q6, 6)
    assert b6.size == 8 + 12
    assert b6[0] == 0x8 | 3 and not b6[1:8].any()
    assert bfp_codec.decode(b6, 1, 16, 6)[0, 0] == -53


def test_fp4_rejects_wide_chunks():
    with pytest.raises(ValueError):
        bfp_codec.encode(np.full((1, 16), 4), 2)
