"""The C-ABI library: it loads without a GPU, exports every symbol the header
declares, and rejects bad arguments on the host before any launch.  CPU only:
every call here returns before touching the HIP runtime."""
from __future__ import annotations

import ctypes
import math
import os
import re
import subprocess
import sys

import pytest

from paper_2110_15456_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fastbfp.h")
OK, E_ARG, E_SHAPE, E_UNSUP, E_PREC, E_HIP = range(6)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bfp_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libfastbfp.so is not built; run __graft_entry__.build()")
    return _lib.load()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 8
    for n in names:
        assert hasattr(lib, n), n
    # and the binding's signature table covers exactly the header
    assert sorted(_lib.SIGNATURES) == names


def _header_abi_version():
    import re
    txt = open(os.path.join(ROOT, "include", "fastbfp.h")).read()
    return int(re.search(r"#define FASTBFP_ABI_VERSION (\d+)", txt).group(1))


def test_version_and_status_strings(lib):
    assert lib.bfp_abi_version() == _header_abi_version()
    for s in range(6):
        assert len(lib.bfp_status_str(s)) > 0
    assert lib.bfp_status_str(99) == b"unknown status"


def test_chunks(lib):
    assert [lib.bfp_chunks(m) for m in range(0, 10)] == [0, 1, 1, 1, 1, 2, 2, 2, 2, 0]


def test_quantized_sizes(lib):
    mb, eb = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.bfp_quantized_sizes(8192, 8192, 16, 4, ctypes.byref(mb), ctypes.byref(eb)) == OK
    assert (mb.value, eb.value) == (8192 * 8192 * 3 // 4, 8192 * 512)
    assert lib.bfp_quantized_sizes(3, 64, 32, 8, ctypes.byref(mb), ctypes.byref(eb)) == OK
    assert (mb.value, eb.value) == (2 * 3 * 64 * 3 // 4, 6)
    # chunks of at most 2 bits take 4-bit codes: m = 1, 2 (one plane), 5, 6 (the upper plane)
    for m, bits in ((1, 4), (2, 4), (3, 6), (4, 6), (5, 10), (6, 10), (7, 12), (8, 12)):
        assert lib.bfp_quantized_sizes(5, 96, 16, m, ctypes.byref(mb), ctypes.byref(eb)) == OK
        assert (mb.value, eb.value) == (5 * 96 * bits // 8, 5 * 6), m
    assert lib.bfp_quantized_sizes(3, 40, 16, 4, ctypes.byref(mb), ctypes.byref(eb)) == E_SHAPE
    # g in {4, 8, 16, 32, 64}; rows hold whole 16-value units
    for g, m, nbytes in ((4, 4, 3 * 64 * 6 // 8), (8, 2, 3 * 64 * 4 // 8), (64, 6, 3 * 64 * 10 // 8)):
        assert lib.bfp_quantized_sizes(3, 64, g, m, ctypes.byref(mb), ctypes.byref(eb)) == OK
        assert (mb.value, eb.value) == (nbytes, 3 * 64 // g), g
    assert lib.bfp_quantized_sizes(3, 40, 8, 4, ctypes.byref(mb), ctypes.byref(eb)) == E_SHAPE  # 40 % 16
    assert lib.bfp_quantized_sizes(3, 64, 12, 4, ctypes.byref(mb), ctypes.byref(eb)) == E_UNSUP
    assert lib.bfp_quantized_sizes(3, 128, 128, 4, ctypes.byref(mb), ctypes.byref(eb)) == E_UNSUP
    assert lib.bfp_quantized_sizes(3, 64, 16, 9, ctypes.byref(mb), ctypes.byref(eb)) == E_PREC
    assert lib.bfp_quantized_sizes(3, 64, 16, 0, ctypes.byref(mb), ctypes.byref(eb)) == E_PREC
    assert lib.bfp_quantized_sizes(-1, 64, 16, 4, ctypes.byref(mb), ctypes.byref(eb)) == E_ARG
    assert lib.bfp_quantized_sizes(3, 64, 16, 4, None, ctypes.byref(eb)) == E_ARG


FAKE = ctypes.c_void_p(0x100000)  # never dereferenced: every call below fails validation first


def q(lib, x=FAKE, R=4, C=64, axis=1, g=16, m=4, mode=0, mant=FAKE, exp=FAKE, st=None):
    return lib.bfp_quantize(x, R, C, axis, g, m, mode, 0, mant, exp, st, None)


def test_quantize_validation(lib):
    assert q(lib, x=None) == E_ARG
    assert q(lib, mant=None) == E_ARG
    assert q(lib, axis=2) == E_ARG
    assert q(lib, mode=3) == E_ARG
    assert q(lib, mode=-1) == E_ARG
    assert q(lib, C=40) == E_SHAPE
    assert q(lib, R=40, axis=0) == E_SHAPE
    assert q(lib, g=12) == E_UNSUP and q(lib, g=128, C=128) == E_UNSUP
    assert q(lib, g=8, C=40) == E_SHAPE
    assert q(lib, g=0) == E_ARG
    assert q(lib, m=9) == E_PREC
    assert q(lib, m=0) == E_PREC
    assert q(lib, R=-1) == E_ARG
    assert q(lib, x=ctypes.c_void_p(0x100004)) == E_ARG  # FP32 rows must be 16-byte aligned
    assert q(lib, R=0) == OK  # empty: nothing to launch
    assert q(lib, x=None, C=0, R=0) == OK


def gm(lib, a=FAKE, ae=FAKE, am=4, b=FAKE, be=FAKE, bm=4, M=8, N=8, K=64, g=16, ma=4, mb=4, C=FAKE, ldc=8):
    return lib.bfp_gemm(a, ae, am, b, be, bm, M, N, K, g, ma, mb, C, ldc, None)


def test_gemm_validation(lib):
    assert gm(lib, a=None) == E_ARG
    assert gm(lib, C=None) == E_ARG
    assert gm(lib, ae=None) == E_ARG
    assert gm(lib, K=40) == E_SHAPE
    assert gm(lib, ldc=7) == E_SHAPE
    assert gm(lib, g=128, K=128) == E_UNSUP and gm(lib, g=8, K=24) == E_SHAPE
    assert gm(lib, g=8, M=0) == OK and gm(lib, g=64, M=0) == OK and gm(lib, g=4, M=0) == OK
    assert gm(lib, M=-1) == E_ARG
    assert gm(lib, am=9) == E_PREC
    # any precision from 1 to the stored width (M = 0: accepted, nothing launched)
    assert gm(lib, ma=3, M=0) == OK and gm(lib, am=8, ma=5, M=0) == OK and gm(lib, bm=6, mb=1, M=0) == OK
    assert gm(lib, am=4, ma=5) == E_PREC    # cannot raise precision
    assert gm(lib, ma=0) == E_PREC and gm(lib, bm=6, mb=7) == E_PREC
    assert gm(lib, a=ctypes.c_void_p(0x100001)) == E_ARG
    assert gm(lib, M=0) == OK and gm(lib, N=0, ldc=0) == OK
    # 32-bit tile offsets: K up to 11184784 (256 rows of FP6 codes < 2^31 bytes)
    kmax = ((1 << 31) // (256 * 12) - 1) * 16
    assert gm(lib, K=kmax + 16) == E_UNSUP and gm(lib, K=kmax + 16, g=32, ma=4, mb=4) == E_UNSUP
    assert gm(lib, M=0, K=kmax) == OK
    # workgroup count of the smallest tile beyond 31 bits
    assert gm(lib, M=(1 << 31) - 1, N=(1 << 31) - 1, ldc=(1 << 31) - 1) == E_UNSUP


def gmt(lib, tile, a=FAKE, ae=FAKE, am=4, b=FAKE, be=FAKE, bm=4, M=8, N=8, K=64, g=16, ma=4, mb=4, C=FAKE, ldc=8):
    return lib.bfp_gemm_tiled(a, ae, am, b, be, bm, M, N, K, g, ma, mb, C, ldc, tile, None)


def test_gemm_tiled_validation(lib):
    assert gmt(lib, 5) == E_ARG and gmt(lib, -2) == E_ARG
    assert gmt(lib, 1, am=6, ma=6) == E_UNSUP            # two chunk planes: default tile only
    assert gmt(lib, 2, bm=8, mb=8) == E_UNSUP
    assert gmt(lib, 3, g=32) == E_UNSUP                  # groups of 32: default tile only
    assert gmt(lib, 1, am=6, ma=4, M=0) == OK            # the low chunk dropped: one plane, empty
    assert gmt(lib, 0, am=6, ma=6, M=0) == OK and gmt(lib, -1, g=32, N=0, ldc=0) == OK
    # products the block-scaled kernel does not take run on the general kernel: no tile to force
    assert gmt(lib, 0, am=6, ma=3, M=0) == E_UNSUP and gmt(lib, 3, g=8, M=0) == E_UNSUP
    assert gmt(lib, -1, am=6, ma=3, M=0) == OK and gmt(lib, -1, g=8, M=0) == OK
    assert gmt(lib, 2, K=40) == E_SHAPE and gmt(lib, 3, C=None) == E_ARG and gmt(lib, 1, ldc=7) == E_SHAPE


def test_group_partials_validation(lib):
    f = lib.bfp_gemm_group_partials
    assert f(None, 4, FAKE, 4, 8, 8, 64, 16, 4, 4, FAKE, None) == E_ARG
    assert f(FAKE, 4, FAKE, 4, 8, 8, 64, 16, 4, 4, None, None) == E_ARG
    assert f(FAKE, 4, FAKE, 4, 8, 8, 60, 16, 4, 4, FAKE, None) == E_SHAPE
    assert f(FAKE, 8, FAKE, 4, 8, 8, 64, 16, 9, 4, FAKE, None) == E_PREC
    assert f(FAKE, 8, FAKE, 4, 8, 8, 64, 16, 3, 4, None, None) == E_ARG  # any lowering; P is null
    assert f(FAKE, 4, FAKE, 4, 0, 8, 64, 16, 4, 4, FAKE, None) == OK


def test_quantize_nd_validation(lib):
    f = lib.bfp_quantize_nd

    def qn(shape, axis, g=16, m=4, mode=0, x=FAKE, mant=FAKE, exp=FAKE):
        arr = (ctypes.c_int64 * max(1, len(shape)))(*shape)
        return f(x, len(shape), arr, axis, g, m, mode, 0, mant, exp, None, None)

    assert qn((4, 64, 8), 3) == E_ARG and qn((4, 64, 8), -1) == E_ARG
    assert qn((), 0) == E_ARG
    assert qn((4, -1, 8), 0) == E_ARG
    assert qn((4, 40, 8), 1) == E_SHAPE          # the grouped axis: a multiple of g and of 16
    assert qn((4, 24, 8), 1, g=8) == E_SHAPE
    assert qn((4, 64, 8), 1, g=12) == E_UNSUP and qn((4, 64, 8), 1, m=9) == E_PREC
    assert qn((4, 64, 8), 1, mode=3) == E_ARG
    assert qn((4, 64, 8), 1, x=None) == E_ARG
    assert qn((0, 64, 8), 1) == OK and qn((4, 64, 0), 1) == OK and qn((4, 0, 8), 1) == OK
    assert qn((1 << 32, 1 << 31, 16), 2) == E_UNSUP  # more than 2^62 rows
    assert qn((1 << 40, 1 << 4), 1) == E_UNSUP       # more than 2^31 workgroups


def test_dequantize_validation(lib):
    f = lib.bfp_dequantize
    assert f(None, FAKE, 4, 64, 16, 4, FAKE, None) == E_ARG
    assert f(FAKE, FAKE, 4, 60, 16, 4, FAKE, None) == E_SHAPE
    assert f(FAKE, FAKE, 4, 64, 16, 10, FAKE, None) == E_PREC
    assert f(FAKE, FAKE, 0, 64, 16, 4, None, None) == OK


def test_binding_fails_loudly_without_library(tmp_path):
    """No CPU fallback: a missing library is an ImportError at first use."""
    code = ("import paper_2110_15456_amd._lib as L; L.LIB_PATH = %r\n"
            "try:\n    L.load()\nexcept ImportError as e:\n    print('raised', e)\n" % str(tmp_path / "missing.so"))
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=ROOT)
    assert "raised" in out.stdout, out.stderr


def test_product_path_does_not_touch_the_oracle():
    pkg = os.path.join(ROOT, "paper_2110_15456_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                pat = r"^\s*(import|from)\s+oracle\b|liboracle|\boracle\.\w+\s*\(|oracle\.c\b"
                assert not re.search(pat, text, flags=re.M), os.path.join(dirpath, f)


def test_adaptive_argument_errors(lib):
    """bfp_quantize_adaptive validates on the host before any launch."""
    P = ctypes.c_void_p
    dummy = P(4096)
    sums = P(8192)
    E_ARG, E_SHAPE = 1, 2
    # bad group axis, bad rounding mode, missing sums, misaligned sums
    assert lib.bfp_quantize_adaptive(dummy, 4, 32, 2, 16, 0, 0, dummy, None, dummy, sums, None, None) == E_ARG
    assert lib.bfp_quantize_adaptive(dummy, 4, 32, 1, 16, 7, 0, dummy, None, dummy, sums, None, None) == E_ARG
    assert lib.bfp_quantize_adaptive(dummy, 4, 32, 1, 16, 0, 0, dummy, None, dummy, None, None, None) == E_ARG
    assert lib.bfp_quantize_adaptive(dummy, 4, 32, 1, 16, 0, 0, dummy, None, dummy, P(8196), None, None) == E_ARG
    # g does not divide the grouped axis
    assert lib.bfp_quantize_adaptive(dummy, 4, 40, 1, 16, 0, 0, dummy, None, dummy, sums, None, None) == E_SHAPE
    assert lib.bfp_quantize_adaptive(dummy, 40, 32, 0, 16, 0, 0, dummy, None, dummy, sums, None, None) == E_SHAPE
    # missing outputs, misaligned second tensor
    assert lib.bfp_quantize_adaptive(dummy, 4, 32, 1, 16, 0, 0, None, None, dummy, sums, None, None) == E_ARG
    assert lib.bfp_quantize_adaptive(dummy, 4, 32, 1, 16, 0, 0, dummy, P(4098), dummy, sums, None, None) == E_ARG


def test_adaptive_host_helpers_match_oracle(lib):
    """Eq. 1 and Algorithm 1's choice: the library's host arithmetic against
    the oracle's."""
    import oracle
    for args in ((0.6, 0.3, 0, 100, 0, 12), (0.6, 0.3, 37, 100, 5, 12), (0.6, 0.3, 100, 100, 12, 12),
                 (0.9, 0.1, 3, 7, 2, 5)):
        assert lib.bfp_adaptive_threshold(*args) == oracle.threshold(*args)
    assert math.isnan(lib.bfp_adaptive_threshold(0.6, 0.3, 1, 0, 1, 4))
    for num, den, eps in ((1.0, 4.0, 0.25), (1.0, 4.0, 0.26), (0.0, 0.0, 0.0), (0.0, 0.0, 0.1), (3.0, 2.0, 0.6)):
        assert lib.bfp_adaptive_mantissa(num, den, eps) == oracle.select_mantissa(num, den, eps)



def test_adaptive_sums_len(lib):
    """Workspace doubles for the adaptive converter: 2 results + 2 per workgroup."""
    assert lib.bfp_adaptive_sums_len(4, 32, 2, 16) == -1
    assert lib.bfp_adaptive_sums_len(4, 40, 1, 16) == -1
    assert lib.bfp_adaptive_sums_len(4, 32, 1, 8) == -1
    assert lib.bfp_adaptive_sums_len(0, 64, 1, 16) == 2
    assert lib.bfp_adaptive_sums_len(4, 32, 1, 16) == 4          # 8 groups: one workgroup
    assert lib.bfp_adaptive_sums_len(8192, 8192, 1, 16) == 2 + 2 * (8192 * 512 // 512)  # 512 groups a block
    assert lib.bfp_adaptive_sums_len(8192, 8192, 1, 32) == 2 + 2 * (8192 * 256 // 256)  # 256 groups a block
    assert lib.bfp_adaptive_sums_len(512, 100, 0, 16) == 2 + 2 * (2 * 1)  # 2 column blocks x 1 group-row block


def gb(lib, a=FAKE, ae=FAKE, am=4, b=FAKE, be=FAKE, bm=4, M=8, N=16, K=64, g=16, ma=4, mb=4, cm=4, mode=0,
       cmant=FAKE, cexp=FAKE, st=None):
    return lib.bfp_gemm_bfp(a, ae, am, b, be, bm, M, N, K, g, ma, mb, cm, mode, 0, cmant, cexp, st, None)


def test_gemm_bfp_validation(lib):
    assert gb(lib, a=None) == E_ARG
    assert gb(lib, cmant=None) == E_ARG
    assert gb(lib, cexp=None) == E_ARG
    assert gb(lib, ae=None) == E_ARG
    assert gb(lib, mode=3) == E_ARG
    assert gb(lib, N=24) == E_SHAPE            # C's rows are grouped by 16
    assert gb(lib, K=40) == E_SHAPE
    assert gb(lib, cm=0) == E_PREC and gb(lib, cm=9) == E_PREC
    assert gb(lib, am=8, ma=5) == E_UNSUP and gb(lib, g=8) == E_UNSUP  # the block-scaled kernel only
    assert gb(lib, g=8, K=64) == E_UNSUP
    assert gb(lib, cmant=ctypes.c_void_p(0x100002)) == E_ARG
    assert gb(lib, st=ctypes.c_void_p(0x100001)) == E_ARG
    assert gb(lib, M=0) == OK and gb(lib, N=0) == OK


def test_dual_and_update_validation(lib):
    d = lib.bfp_quantize_dual
    assert d(FAKE, 32, 64, 16, 4, 3, 0, 0, FAKE, FAKE, FAKE, FAKE, None, None) == E_ARG      # bad rounding mode
    assert d(FAKE, 24, 64, 16, 4, 0, 0, 0, FAKE, FAKE, FAKE, FAKE, None, None) == E_SHAPE    # R % 16
    assert d(FAKE, 32, 40, 16, 4, 0, 0, 0, FAKE, FAKE, FAKE, FAKE, None, None) == E_SHAPE    # C % 16
    assert d(FAKE, 32, 64, 32, 4, 0, 0, 0, FAKE, FAKE, FAKE, FAKE, None, None) == E_UNSUP    # g = 32
    assert d(FAKE, 32, 64, 16, 9, 0, 0, 0, FAKE, FAKE, FAKE, FAKE, None, None) == E_PREC
    assert d(None, 32, 64, 16, 4, 0, 0, 0, FAKE, FAKE, FAKE, FAKE, None, None) == E_ARG
    assert d(FAKE, 32, 64, 16, 4, 0, 0, 0, FAKE, None, FAKE, FAKE, None, None) == E_ARG
    assert d(ctypes.c_void_p(0x100004), 32, 64, 16, 4, 0, 0, 0, FAKE, FAKE, FAKE, FAKE, None, None) == E_ARG
    assert d(None, 0, 64, 16, 4, 0, 0, 0, None, None, None, None, None, None) == OK
    u = lib.bfp_weight_update
    args = lambda w=FAKE, dw=ctypes.c_void_p(0x200000), wo=FAKE, R=32: (w, dw, 1.0, wo, R, 64, 16, 4, 0, 0, 0, FAKE,
                                                                         FAKE, FAKE, FAKE, None, None)
    assert u(*args(dw=None)) == E_ARG
    assert u(*args(wo=None)) == E_ARG
    assert u(*args(dw=FAKE)) == E_ARG        # dw overlaps w_out
    assert u(*args(R=24)) == E_SHAPE
    assert u(*args(w=None, R=0)) == OK


def test_packed_sizes_match_the_paper(lib):
    """Section V-D: a group of g values takes e + g * (m/2) * 3 bits (a 2-bit
    chunk and its sign in 3 bits); with e = 3 and g = 16 that is 51/16 bits per
    value at m = 2 and 99/16 at m = 4 (printed rounded as 3.2 and 6.2).  The
    library's sizes add only the 32-bit E_max word when the group count is a
    multiple of 64."""
    from fractions import Fraction
    mb, eb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    for m, bits in [(2, Fraction(51, 16)), (4, Fraction(99, 16)), (6, Fraction(147, 16)), (8, Fraction(195, 16))]:
        for rows, length in [(64, 16), (8, 1024), (1024, 1024)]:
            assert lib.bfp_packed_sizes(rows, length, m, ctypes.byref(mb), ctypes.byref(eb)) == OK
            n = rows * length
            assert Fraction(8 * (mb.value + eb.value - 4), n) == bits, (m, rows, length)
            assert eb.value == 4 + 3 * n // 16 // 8
    assert round(float(Fraction(51, 16)), 1) == 3.2 and round(float(Fraction(99, 16)), 1) == 6.2
    # odd widths take ceil(m/2) planes; a partial block of 64 groups is padded to 24 bytes
    assert lib.bfp_packed_sizes(3, 32, 3, ctypes.byref(mb), ctypes.byref(eb)) == OK
    assert (mb.value, eb.value) == (2 * 6 * 6, 4 + 24)
    assert lib.bfp_packed_sizes(0, 32, 4, ctypes.byref(mb), ctypes.byref(eb)) == OK and mb.value == 0
    assert lib.bfp_packed_sizes(3, 40, 4, ctypes.byref(mb), ctypes.byref(eb)) == E_SHAPE
    assert lib.bfp_packed_sizes(3, 32, 9, ctypes.byref(mb), ctypes.byref(eb)) == E_PREC
    assert lib.bfp_packed_sizes(3, 32, 0, ctypes.byref(mb), ctypes.byref(eb)) == E_PREC
    assert lib.bfp_packed_sizes(-1, 32, 4, ctypes.byref(mb), ctypes.byref(eb)) == E_ARG
    assert lib.bfp_packed_sizes(3, 32, 4, None, ctypes.byref(eb)) == E_ARG
    assert lib.bfp_packed_sizes(1 << 40, 1 << 21, 4, ctypes.byref(mb), ctypes.byref(eb)) == E_UNSUP


def test_packed_validation(lib):
    qp, dq, gp = lib.bfp_quantize_packed, lib.bfp_dequantize_packed, lib.bfp_gemm_packed
    assert qp(None, 4, 64, 4, 0, 0, FAKE, FAKE, None, None) == E_ARG
    assert qp(FAKE, 4, 64, 4, 0, 0, None, FAKE, None, None) == E_ARG
    assert qp(FAKE, 4, 64, 4, 3, 0, FAKE, FAKE, None, None) == E_ARG
    assert qp(FAKE, 4, 40, 4, 0, 0, FAKE, FAKE, None, None) == E_SHAPE
    assert qp(FAKE, 4, 64, 9, 0, 0, FAKE, FAKE, None, None) == E_PREC
    assert qp(ctypes.c_void_p(0x100004), 4, 64, 4, 0, 0, FAKE, FAKE, None, None) == E_ARG
    assert qp(FAKE, 4, 64, 4, 0, 0, FAKE, ctypes.c_void_p(0x100002), None, None) == E_ARG
    assert qp(None, 0, 64, 4, 0, 0, None, None, None, None) == OK
    assert qp(FAKE, 1 << 40, 1 << 16, 4, 0, 0, FAKE, FAKE, None, None) == E_UNSUP  # > 2^31 workgroups
    assert dq(None, FAKE, 4, 64, 4, FAKE, None) == E_ARG
    assert dq(FAKE, FAKE, 4, 40, 4, FAKE, None) == E_SHAPE
    assert dq(FAKE, FAKE, 4, 64, 0, FAKE, None) == E_PREC
    assert dq(FAKE, FAKE, 4, 64, 4, ctypes.c_void_p(0x100004), None) == E_ARG
    assert dq(FAKE, FAKE, 0, 64, 4, None, None) == OK

    def g(a=FAKE, ae=FAKE, am=4, b=FAKE, be=FAKE, bm=4, M=8, N=8, K=64, ma=4, mb=4, C=FAKE, ldc=8):
        return gp(a, ae, am, b, be, bm, M, N, K, ma, mb, C, ldc, None)

    assert g(a=None) == E_ARG and g(C=None) == E_ARG and g(be=None) == E_ARG
    assert g(ae=ctypes.c_void_p(0x100002)) == E_ARG
    assert g(K=40) == E_SHAPE and g(ldc=7) == E_SHAPE
    assert g(ma=5) == E_PREC and g(am=9) == E_PREC and g(mb=0) == E_PREC
    assert g(M=0) == OK and g(am=8, ma=3, N=0, ldc=0) == OK


def test_general_kernel_grid_bound(lib):
    """The general kernel's 32 x 32 tiles bound M and N more tightly than the
    block-scaled kernel's: such shapes are rejected, not launched."""
    n = 1 << 21  # 2^29 tiles of 128 x 64 (accepted there), 2^32 of 32 x 32
    assert ((n + 127) // 128) * ((n + 63) // 64) < 2 ** 31 <= ((n + 31) // 32) ** 2
    assert gm(lib, g=8, M=n, N=n, ldc=n) == E_UNSUP
    assert gm(lib, g=16, M=n, N=n, ldc=n, am=6, ma=3) == E_UNSUP
    assert lib.bfp_gemm_group_partials(FAKE, 4, FAKE, 4, n, n, 64, 16, 4, 4, FAKE, None) == E_UNSUP
    assert lib.bfp_gemm_packed(FAKE, FAKE, 4, FAKE, FAKE, 4, n, n, 64, 4, 4, FAKE, n, None) == E_UNSUP


def test_repack_sizes(lib):
    mb, eb, lo, go = ctypes.c_size_t(0), ctypes.c_size_t(0), ctypes.c_int64(0), ctypes.c_int(0)
    args = (ctypes.byref(mb), ctypes.byref(eb), ctypes.byref(lo), ctypes.byref(go))
    # groups of 4 and 8: one zero-padded 16-value unit per group; 64: groups of 32
    for g, m, want_len, want_g in [(4, 4, 256, 16), (8, 2, 128, 16), (16, 6, 64, 16), (32, 8, 64, 32), (64, 3, 64, 32)]:
        assert lib.bfp_repack_sizes(3, 64, g, m, *args) == OK
        assert (lo.value, go.value) == (want_len, want_g)
        want_mb, want_eb = ctypes.c_size_t(0), ctypes.c_size_t(0)
        assert lib.bfp_quantized_sizes(3, want_len, want_g, m, ctypes.byref(want_mb), ctypes.byref(want_eb)) == OK
        assert (mb.value, eb.value) == (want_mb.value, want_eb.value)
    assert lib.bfp_repack_sizes(3, 40, 8, 4, *args) == E_SHAPE
    assert lib.bfp_repack_sizes(3, 64, 12, 4, *args) == E_UNSUP
    assert lib.bfp_repack_sizes(3, 64, 16, 9, *args) == E_PREC
    assert lib.bfp_repack_sizes(3, 64, 16, 4, None, *args[1:]) == E_ARG


def test_repack_validation(lib):
    f = lib.bfp_repack
    assert f(FAKE, FAKE, 4, 64, 16, 4, 0, 5, FAKE, FAKE, None) == E_PREC      # cannot raise the width
    assert f(FAKE, FAKE, 4, 64, 16, 4, 0, 0, FAKE, FAKE, None) == E_PREC
    assert f(FAKE, FAKE, 4, 64, 16, 4, 2, 2, FAKE, FAKE, None) == E_ARG       # packed is 0 or 1
    assert f(FAKE, FAKE, 4, 64, 8, 4, 1, 2, FAKE, FAKE, None) == E_UNSUP      # packed storage has g = 16
    assert f(None, FAKE, 4, 64, 16, 4, 0, 2, FAKE, FAKE, None) == E_ARG
    assert f(FAKE, FAKE, 4, 64, 16, 4, 0, 2, None, FAKE, None) == E_ARG
    assert f(FAKE, ctypes.c_void_p(0x100002), 4, 64, 16, 4, 1, 2, FAKE, FAKE, None) == E_ARG  # packed exps
    assert f(FAKE, FAKE, 4, 40, 16, 4, 0, 2, FAKE, FAKE, None) == E_SHAPE
    assert f(None, None, 0, 64, 8, 4, 0, 2, None, None, None) == OK


def test_gemm_ws_size_and_validation(lib):
    nb = ctypes.c_size_t(0)

    def size(am=4, bm=4, M=8, N=8, K=64, g=16, ma=4, mb=4, packed=0):
        st = lib.bfp_gemm_ws_size(am, bm, M, N, K, g, ma, mb, packed, ctypes.byref(nb))
        return st, nb.value

    # products the block-scaled kernel reads as stored need no workspace
    assert size() == (OK, 0) and size(g=32) == (OK, 0) and size(am=6, ma=4) == (OK, 0)
    assert size(am=8, bm=6, ma=4, mb=4) == (OK, 0)
    # the others: the operands that need it, repacked
    st, n_a = size(am=4, ma=2)                   # A lowered: its 8 x 64 at m = 2 (FP4: 4 bytes per row-group) + exps
    assert st == OK and n_a == 256 + 256
    st, n_both = size(g=8)                       # both operands, K_out = 128: 768 mantissa + 64 exponent bytes each
    assert st == OK and n_both == 2 * (768 + 256)
    assert size(packed=1)[0] == OK and size(packed=1)[1] > 0
    assert size(packed=1, g=8)[0] == E_UNSUP
    assert size(packed=2)[0] == E_ARG
    assert size(ma=5)[0] == E_PREC and size(K=40)[0] == E_SHAPE
    kmax = ((1 << 31) // (256 * 12) - 1) * 16
    k4 = (kmax // 64 + 1) * 16                   # K_out = 4 K just beyond the kernel's limit
    assert k4 <= kmax < 4 * k4 and size(K=k4, g=4)[0] == E_UNSUP and size(K=k4 - 16, g=4)[0] == OK
    assert lib.bfp_gemm_ws_size(4, 4, 8, 8, 64, 16, 4, 4, 0, None) == E_ARG
    # the repack kernel's workgroup count (one thread per output unit) beyond 31 bits
    big_m = (1 << 31) - 1
    assert size(M=big_m, N=16, K=16 * 4096, g=8, ma=4, mb=4)[0] == E_UNSUP
    assert size(M=16, N=big_m, K=16 * 4096, g=16, ma=4, mb=2, am=4, bm=4)[0] == E_UNSUP

    def ws(workspace=FAKE, nbytes=1 << 20, ldc=8, C=FAKE, **kw):
        a = dict(am=4, bm=4, M=8, N=8, K=64, g=16, ma=4, mb=4, packed=0)
        a.update(kw)
        return lib.bfp_gemm_ws(FAKE, FAKE, a["am"], FAKE, FAKE, a["bm"], a["M"], a["N"], a["K"], a["g"], a["ma"],
                               a["mb"], a["packed"], C, ldc, workspace, nbytes, None)

    assert ws(g=8, workspace=None) == E_ARG                       # a workspace is needed
    assert ws(g=8, nbytes=n_both - 1) == E_ARG                    # too small
    assert ws(g=8, workspace=ctypes.c_void_p(0x100010)) == E_ARG  # not 256-byte aligned
    assert ws(ldc=7) == E_SHAPE and ws(C=None) == E_ARG
    assert ws(M=0, g=8, workspace=None, nbytes=0) == OK           # empty: nothing launched
