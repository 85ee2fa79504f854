"""MI355X (gfx950) BFP hot path of FAST: FP32 -> BFP quantization and the
variable-precision BFP GEMM.

This module is a thin binding over the C ABI of ``include/fastbfp.h``
(``libfastbfp.so``): it checks tensor arguments, allocates outputs with torch
(device memory is torch's), passes raw pointers and torch's current stream,
and turns non-zero statuses into exceptions.  Every step of the computation
runs in the library's HIP kernels; there is no CPU path.

    A = quantize(x, group_axis=-1, g=16, m=4, rounding="nearest")
    W = quantize(w, group_axis=0, g=16, m=2)        # K-contiguous, transposed
    y = gemm(A, W)                                   # FP32 [M, N] = x . w
"""
from __future__ import annotations

import ctypes
import math
from dataclasses import dataclass

import torch

from ._lib import BFPError, check, load

__all__ = ["BFPTensor", "BFPError", "quantize", "quantize_dual", "weight_update", "dequantize", "gemm", "gemm_bfp",
           "gemm_group_partials", "quantize_adaptive", "quantize_adaptive_noalloc", "adaptive_threshold", "adaptive_mantissa", "chunks", "quantized_sizes", "ROUNDING",
           "PackedBFPTensor", "packed_sizes", "quantize_packed", "dequantize_packed", "gemm_packed", "repack",
           "gemm_ws_size"]

ROUNDING = {"nearest": 0, "stochastic": 1, "truncate": 2}


def chunks(m: int) -> int:
    """4-bit chunk planes used for an m-bit magnitude (1 if m <= 4, else 2)."""
    return int(load().bfp_chunks(int(m)))


def quantized_sizes(rows: int, length: int, g: int, m: int):
    """(mantissa bytes, exponent bytes) of a rows x length BFP tensor."""
    mb, eb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    check(load().bfp_quantized_sizes(rows, length, g, m, ctypes.byref(mb), ctypes.byref(eb)), "bfp_quantized_sizes")
    return mb.value, eb.value


@dataclass
class BFPTensor:
    """A rows x len BFP tensor, groups of g along len (see include/fastbfp.h).

    mant: uint8 chunk planes (flat, chunks(m) * rows * len * 3/4 bytes);
    exp: uint8 [rows, len // g] shared exponents.
    """
    mant: torch.Tensor
    exp: torch.Tensor
    rows: int
    len: int
    g: int
    m: int

    @property
    def planes(self) -> int:
        return chunks(self.m)

    @property
    def device(self) -> torch.device:
        return self.mant.device

    @staticmethod
    def empty(rows: int, length: int, g: int, m: int, device) -> "BFPTensor":
        mb, eb = quantized_sizes(rows, length, g, m)
        return BFPTensor(torch.empty(mb, dtype=torch.uint8, device=device),
                         torch.empty((rows, length // g), dtype=torch.uint8, device=device), rows, length, g, m)


def _stream(dev: torch.device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _need_cuda(t: torch.Tensor, name: str, dtype=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a CUDA (HIP) tensor" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must have dtype %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def quantize(x: torch.Tensor, group_axis: int = -1, g: int = 16, m: int = 4, rounding: str = "nearest",
             seed: int = 0, status: torch.Tensor | None = None, out: BFPTensor | None = None) -> BFPTensor:
    """FP32 -> BFP with groups of g along ``group_axis`` (any axis of an N-D
    tensor): a BFPTensor with the group axis innermost, rows = the other
    axes' indices in order.  So the last axis keeps the leading axes as rows,
    and axis 0 of a 2-D [R, C] tensor is written transposed as a [C, R] BFP
    tensor (K-contiguous for the GEMM).  ``status``: optional int32/uint32
    CUDA scalar whose bit 0 is set on Inf/NaN input.  ``out``: optional
    preallocated BFPTensor of the result shape (no allocation happens then).
    """
    _need_cuda(x, "x", torch.float32)
    if rounding not in ROUNDING:
        raise ValueError("rounding must be one of %s" % sorted(ROUNDING))
    if x.dim() < 1:
        raise ValueError("x must have at least one dimension")
    nd = x.dim()
    ax = group_axis % nd
    length = x.shape[ax]
    rows = math.prod(x.shape[:ax]) * math.prod(x.shape[ax + 1:])
    t = out if out is not None else BFPTensor.empty(rows, length, g, m, x.device)
    if (t.rows, t.len, t.g, t.m) != (rows, length, g, m):
        raise ValueError("out has the wrong shape or format")
    st_ptr = None
    if status is not None:
        _need_cuda(status, "status")
        st_ptr = ctypes.c_void_p(status.data_ptr())
    seed_c = ctypes.c_uint64(seed & 0xFFFFFFFFFFFFFFFF)
    ptrs = (ctypes.c_void_p(t.mant.data_ptr()), ctypes.c_void_p(t.exp.data_ptr()), st_ptr, _stream(x.device))
    if ax == nd - 1 or (nd == 2 and ax == 0):  # the 2-D entry point: rows of [R, C], or its columns
        R, C = (rows, length) if ax == nd - 1 else tuple(x.shape)
        check(load().bfp_quantize(ctypes.c_void_p(x.data_ptr()), R, C, 1 if ax == nd - 1 else 0, g, m,
                                  ROUNDING[rounding], seed_c, *ptrs), "bfp_quantize")
    else:
        shape = (ctypes.c_int64 * nd)(*x.shape)
        check(load().bfp_quantize_nd(ctypes.c_void_p(x.data_ptr()), nd, shape, ax, g, m, ROUNDING[rounding], seed_c,
                                     *ptrs), "bfp_quantize_nd")
    return t


def _status_ptr(status):
    if status is None:
        return None
    _need_cuda(status, "status")
    return ctypes.c_void_p(status.data_ptr())


def _dual_outputs(R, C, g, m, device, out_rows, out_cols):
    tr = out_rows if out_rows is not None else BFPTensor.empty(R, C, g, m, device)
    tc = out_cols if out_cols is not None else BFPTensor.empty(C, R, g, m, device)
    if (tr.rows, tr.len, tr.g, tr.m) != (R, C, g, m) or (tc.rows, tc.len, tc.g, tc.m) != (C, R, g, m):
        raise ValueError("out_rows / out_cols have the wrong shape or format")
    return tr, tc


def quantize_dual(x: torch.Tensor, g: int = 16, m: int = 4, rounding: str = "nearest", seed_rows: int = 0,
                  seed_cols: int = 0, status: torch.Tensor | None = None, out_rows: BFPTensor | None = None,
                  out_cols: BFPTensor | None = None):
    """Both groupings of a 2-D [R, C] FP32 tensor from one read: ``(tr, tc)``
    with tr = quantize(x, -1, seed=seed_rows) ([R, C], groups along rows) and
    tc = quantize(x, 0, seed=seed_cols) ([C, R], groups down the columns)."""
    _need_cuda(x, "x", torch.float32)
    if rounding not in ROUNDING:
        raise ValueError("rounding must be one of %s" % sorted(ROUNDING))
    if x.dim() != 2:
        raise ValueError("x must be 2-D")
    R, C = x.shape
    tr, tc = _dual_outputs(R, C, g, m, x.device, out_rows, out_cols)
    check(load().bfp_quantize_dual(ctypes.c_void_p(x.data_ptr()), R, C, g, m, ROUNDING[rounding],
                                   ctypes.c_uint64(seed_rows & 0xFFFFFFFFFFFFFFFF),
                                   ctypes.c_uint64(seed_cols & 0xFFFFFFFFFFFFFFFF), ctypes.c_void_p(tr.mant.data_ptr()),
                                   ctypes.c_void_p(tr.exp.data_ptr()), ctypes.c_void_p(tc.mant.data_ptr()),
                                   ctypes.c_void_p(tc.exp.data_ptr()), _status_ptr(status), _stream(x.device)),
          "bfp_quantize_dual")
    return tr, tc


def weight_update(w: torch.Tensor, dw: torch.Tensor, alpha: float, g: int = 16, m: int = 4,
                  rounding: str = "nearest", seed_rows: int = 0, seed_cols: int = 0, w_out: torch.Tensor | None = None,
                  status: torch.Tensor | None = None, out_rows: BFPTensor | None = None,
                  out_cols: BFPTensor | None = None):
    """w_out = w + alpha * dw (FP32, product and sum each rounded; w_out = w
    updates in place when passed as w) and both groupings of the result, as
    quantize_dual.  Returns ``(w_out, tr, tc)``."""
    _need_cuda(w, "w", torch.float32)
    _need_cuda(dw, "dw", torch.float32)
    if rounding not in ROUNDING:
        raise ValueError("rounding must be one of %s" % sorted(ROUNDING))
    if w.dim() != 2 or dw.shape != w.shape:
        raise ValueError("w must be 2-D and dw of the same shape")
    R, C = w.shape
    if w_out is None:
        w_out = torch.empty_like(w)
    else:
        _need_cuda(w_out, "w_out", torch.float32)
        if w_out.shape != w.shape:
            raise ValueError("w_out has the wrong shape")
    tr, tc = _dual_outputs(R, C, g, m, w.device, out_rows, out_cols)
    check(load().bfp_weight_update(ctypes.c_void_p(w.data_ptr()), ctypes.c_void_p(dw.data_ptr()), ctypes.c_float(alpha),
                                   ctypes.c_void_p(w_out.data_ptr()), R, C, g, m, ROUNDING[rounding],
                                   ctypes.c_uint64(seed_rows & 0xFFFFFFFFFFFFFFFF),
                                   ctypes.c_uint64(seed_cols & 0xFFFFFFFFFFFFFFFF), ctypes.c_void_p(tr.mant.data_ptr()),
                                   ctypes.c_void_p(tr.exp.data_ptr()), ctypes.c_void_p(tc.mant.data_ptr()),
                                   ctypes.c_void_p(tc.exp.data_ptr()), _status_ptr(status), _stream(w.device)),
          "bfp_weight_update")
    return w_out, tr, tc


def quantize_adaptive(x: torch.Tensor, group_axis: int = -1, g: int = 16, rounding: str = "nearest",
                      seed: int = 0, with_m2: bool = True, status: torch.Tensor | None = None):
    """One pass of the adaptive converter (Algorithm 1, Eq. 2): returns
    ``(t4, t2, sums)`` with t4 = BFP(X, 4), t2 = BFP(X, 2) taken from t4 by
    discarding the low 2-bit chunk (same exponent tensor; None unless
    ``with_m2``), and sums a float64 CUDA tensor [sum |BFP4 - BFP2|,
    sum |BFP2|], so that r(X) = sums[0] / sums[1]."""
    _need_cuda(x, "x", torch.float32)
    if rounding not in ROUNDING:
        raise ValueError("rounding must be one of %s" % sorted(ROUNDING))
    nd = x.dim()
    if nd < 1:
        raise ValueError("x must have at least one dimension")
    ax = group_axis % nd
    if ax == nd - 1:
        C = x.shape[-1]
        R = math.prod(x.shape[:-1])  # leading axes flattened into rows (also when C = 0)
        axis_flag, rows, length = 1, R, C
    elif nd == 2 and ax == 0:
        R, C = x.shape
        axis_flag, rows, length = 0, C, R
    else:
        raise ValueError("group_axis must be the last axis, or 0 of a 2-D tensor")
    t4 = BFPTensor.empty(rows, length, g, 4, x.device)
    t2 = None
    if with_m2:  # its own (4-bit code) mantissa plane, sharing t4's exponents
        t2 = BFPTensor(torch.empty(quantized_sizes(rows, length, g, 2)[0], dtype=torch.uint8, device=x.device), t4.exp,
                       rows, length, g, 2)
    lib = load()
    n_sums = lib.bfp_adaptive_sums_len(R, C, axis_flag, g)
    if n_sums < 2:
        raise ValueError("unsupported shape or group size for the adaptive converter")
    work = torch.empty(n_sums, dtype=torch.float64, device=x.device)
    sums = work[:2]
    st_ptr = None
    if status is not None:
        _need_cuda(status, "status")
        st_ptr = ctypes.c_void_p(status.data_ptr())
    check(lib.bfp_quantize_adaptive(ctypes.c_void_p(x.data_ptr()), R, C, axis_flag, g, ROUNDING[rounding],
                                    ctypes.c_uint64(seed & 0xFFFFFFFFFFFFFFFF), ctypes.c_void_p(t4.mant.data_ptr()),
                                    ctypes.c_void_p(t2.mant.data_ptr()) if t2 is not None else None,
                                    ctypes.c_void_p(t4.exp.data_ptr()), ctypes.c_void_p(work.data_ptr()), st_ptr,
                                    _stream(x.device)), "bfp_quantize_adaptive")
    return t4, t2, sums


def quantize_adaptive_noalloc(x: torch.Tensor, t4: BFPTensor, sums: torch.Tensor, group_axis: int = -1,
                              rounding: str = "nearest", seed: int = 0, t2: BFPTensor | None = None,
                              status: torch.Tensor | None = None):
    """quantize_adaptive into caller-provided outputs, with no allocation
    anywhere (bfp_quantize_adaptive_noalloc: the library's device scratch
    array holds the partial sums): t4 = BFP(X, 4), optional t2 (mantissas of
    BFP(X, 2), sharing t4.exp), sums a float64 CUDA tensor of at least 2."""
    _need_cuda(x, "x", torch.float32)
    _need_cuda(sums, "sums", torch.float64)
    if rounding not in ROUNDING:
        raise ValueError("rounding must be one of %s" % sorted(ROUNDING))
    nd = x.dim()
    ax = group_axis % nd
    if ax == nd - 1:
        C = x.shape[-1]
        R = math.prod(x.shape[:-1])
        axis_flag, rows, length = 1, R, C
    elif nd == 2 and ax == 0:
        R, C = x.shape
        axis_flag, rows, length = 0, C, R
    else:
        raise ValueError("group_axis must be the last axis, or 0 of a 2-D tensor")
    if (t4.rows, t4.len, t4.m) != (rows, length, 4) or (t2 is not None and (t2.rows, t2.len, t2.m) != (rows, length, 2)):
        raise ValueError("t4 / t2 have the wrong shape or format")
    if sums.numel() < 2:
        raise ValueError("sums needs 2 doubles")
    check(load().bfp_quantize_adaptive_noalloc(ctypes.c_void_p(x.data_ptr()), R, C, axis_flag, t4.g, ROUNDING[rounding],
                                               ctypes.c_uint64(seed & 0xFFFFFFFFFFFFFFFF),
                                               ctypes.c_void_p(t4.mant.data_ptr()),
                                               ctypes.c_void_p(t2.mant.data_ptr()) if t2 is not None else None,
                                               ctypes.c_void_p(t4.exp.data_ptr()), ctypes.c_void_p(sums.data_ptr()),
                                               _status_ptr(status), _stream(x.device)), "bfp_quantize_adaptive_noalloc")


def adaptive_threshold(alpha: float, beta: float, i: int, I: int, l: int, L: int) -> float:
    """Eq. 1: epsilon(l, i) = alpha - beta i / I - beta l / L."""
    return float(load().bfp_adaptive_threshold(alpha, beta, i, I, l, L))


def adaptive_mantissa(sums, eps: float) -> int:
    """Algorithm 1's choice (2 or 4 bits) from the two sums of quantize_adaptive
    (reading them back synchronises with the stream)."""
    num, den = (float(v) for v in (sums.tolist() if hasattr(sums, "tolist") else sums))
    return int(load().bfp_adaptive_mantissa(num, den, eps))


def dequantize(t: BFPTensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """BFP -> FP32 [rows, len]: +-q * 2^(E - 127 - (m-1))."""
    y = out if out is not None else torch.empty((t.rows, t.len), dtype=torch.float32, device=t.device)
    _need_cuda(y, "out", torch.float32)
    check(load().bfp_dequantize(ctypes.c_void_p(t.mant.data_ptr()), ctypes.c_void_p(t.exp.data_ptr()), t.rows,
                                t.len, t.g, t.m, ctypes.c_void_p(y.data_ptr()), _stream(t.device)), "bfp_dequantize")
    return y


def _gemm_args(A: BFPTensor, B: BFPTensor, m_a, m_b):
    if A.len != B.len or A.g != B.g:
        raise ValueError("A and B must share K and the group size (A: K=%d g=%d, B: K=%d g=%d)"
                         % (A.len, A.g, B.len, B.g))
    return (A.m if m_a is None else int(m_a)), (B.m if m_b is None else int(m_b))


def gemm_ws_size(A, B, m_a: int | None = None, m_b: int | None = None) -> int:
    """Workspace bytes bfp_gemm_ws needs for this product (0 when the
    block-scaled kernel reads both operands as stored)."""
    m_a, m_b = _gemm_args(A, B, m_a, m_b)
    nb = ctypes.c_size_t(0)
    check(load().bfp_gemm_ws_size(A.m, B.m, A.rows, B.rows, A.len, A.g, m_a, m_b,
                                  1 if isinstance(A, PackedBFPTensor) else 0, ctypes.byref(nb)), "bfp_gemm_ws_size")
    return nb.value


def _gemm_out(A, B, out):
    C = out if out is not None else torch.empty((A.rows, B.rows), dtype=torch.float32, device=A.device)
    _need_cuda(C, "out", torch.float32)
    if C.dim() != 2 or C.shape[0] != A.rows or C.shape[1] != B.rows:
        raise ValueError("out must be [%d, %d]" % (A.rows, B.rows))
    return C


def _gemm_with_workspace(A, B, m_a, m_b, C, workspace):
    """bfp_gemm_ws: operands the block-scaled kernel cannot read as stored are
    repacked into a workspace (torch-allocated unless one is given)."""
    packed = 1 if isinstance(A, PackedBFPTensor) else 0
    need = gemm_ws_size(A, B, m_a, m_b)
    if need == 0:
        ws = None
    elif isinstance(workspace, torch.Tensor):
        _need_cuda(workspace, "workspace", torch.uint8)
        ws = workspace
        if ws.numel() < need:
            raise ValueError("workspace needs %d bytes" % need)
    else:
        ws = torch.empty(need, dtype=torch.uint8, device=A.device)
    check(load().bfp_gemm_ws(ctypes.c_void_p(A.mant.data_ptr()), ctypes.c_void_p(A.exp.data_ptr()), A.m,
                             ctypes.c_void_p(B.mant.data_ptr()), ctypes.c_void_p(B.exp.data_ptr()), B.m, A.rows,
                             B.rows, A.len, A.g, m_a, m_b, packed, ctypes.c_void_p(C.data_ptr()), C.stride(0),
                             ctypes.c_void_p(ws.data_ptr()) if ws is not None else None,
                             ws.numel() if ws is not None else 0, _stream(A.device)), "bfp_gemm_ws")
    return C


def gemm(A: BFPTensor, B: BFPTensor, m_a: int | None = None, m_b: int | None = None,
         out: torch.Tensor | None = None, tile: int | None = None, workspace=True) -> torch.Tensor:
    """C = A . B^T in FP32 [A.rows, B.rows] for BFP A [M, K] and B [N, K].

    m_a / m_b: precision of each operand in the product (default: stored m;
    any value from 1 to the stored width).
    tile: None lets the library choose the workgroup tile from the shape;
    0..4 forces one (bfp_gemm_tiled: the default tile, 256x128, 256x64,
    128x64, 128x128 -- the last four for m_a, m_b <= 4 and g = 16 only).
    workspace: True (default) runs every product on the block-scaled kernel,
    repacking an operand it cannot read as stored (groups of 4, 8, 64; a
    precision between chunk boundaries) into a workspace allocated here
    (bfp_gemm_ws), or into a given uint8 CUDA tensor; False calls bfp_gemm,
    which runs such products on its allocation-free general kernel.
    """
    m_a, m_b = _gemm_args(A, B, m_a, m_b)
    C = _gemm_out(A, B, out)
    if tile is None and workspace is not False:
        return _gemm_with_workspace(A, B, m_a, m_b, C, workspace)
    args = (ctypes.c_void_p(A.mant.data_ptr()), ctypes.c_void_p(A.exp.data_ptr()), A.m,
            ctypes.c_void_p(B.mant.data_ptr()), ctypes.c_void_p(B.exp.data_ptr()), B.m, A.rows, B.rows,
            A.len, A.g, m_a, m_b, ctypes.c_void_p(C.data_ptr()), C.stride(0))
    if tile is None:
        check(load().bfp_gemm(*args, _stream(A.device)), "bfp_gemm")
    else:
        check(load().bfp_gemm_tiled(*args, int(tile), _stream(A.device)), "bfp_gemm_tiled")
    return C


def repack(t, m_use: int | None = None) -> BFPTensor:
    """bfp_repack: t (a BFPTensor, or a PackedBFPTensor) re-encoded at m_use
    bits (default: its width) in the chunk-plane layout with groups of 16 (t's
    g <= 16; groups of 4 and 8 zero-padded to 16-value units) or 32."""
    m_use = t.m if m_use is None else int(m_use)
    mb, eb, lo, go = ctypes.c_size_t(0), ctypes.c_size_t(0), ctypes.c_int64(0), ctypes.c_int(0)
    check(load().bfp_repack_sizes(t.rows, t.len, t.g, m_use, ctypes.byref(mb), ctypes.byref(eb), ctypes.byref(lo),
                                  ctypes.byref(go)), "bfp_repack_sizes")
    r = BFPTensor(torch.empty(mb.value, dtype=torch.uint8, device=t.device),
                  torch.empty((t.rows, lo.value // go.value), dtype=torch.uint8, device=t.device), t.rows, lo.value,
                  go.value, m_use)
    check(load().bfp_repack(ctypes.c_void_p(t.mant.data_ptr()), ctypes.c_void_p(t.exp.data_ptr()), t.rows, t.len, t.g,
                            t.m, 1 if isinstance(t, PackedBFPTensor) else 0, m_use, ctypes.c_void_p(r.mant.data_ptr()),
                            ctypes.c_void_p(r.exp.data_ptr()), _stream(t.device)), "bfp_repack")
    return r


def gemm_bfp(A: BFPTensor, B: BFPTensor, c_m: int, m_a: int | None = None, m_b: int | None = None,
             rounding: str = "nearest", seed: int = 0, status: torch.Tensor | None = None,
             out: BFPTensor | None = None) -> BFPTensor:
    """C = A . B^T converted to BFP in the GEMM's epilogue: a [A.rows, B.rows]
    BFP tensor with groups of 16 along each row of C at c_m bits, equal to
    quantize(gemm(A, B), g=16, m=c_m, rounding, seed)."""
    if rounding not in ROUNDING:
        raise ValueError("rounding must be one of %s" % sorted(ROUNDING))
    m_a, m_b = _gemm_args(A, B, m_a, m_b)
    t = out if out is not None else BFPTensor.empty(A.rows, B.rows, 16, c_m, A.device)
    if (t.rows, t.len, t.g, t.m) != (A.rows, B.rows, 16, c_m):
        raise ValueError("out has the wrong shape or format")
    st_ptr = None
    if status is not None:
        _need_cuda(status, "status")
        st_ptr = ctypes.c_void_p(status.data_ptr())
    check(load().bfp_gemm_bfp(ctypes.c_void_p(A.mant.data_ptr()), ctypes.c_void_p(A.exp.data_ptr()), A.m,
                              ctypes.c_void_p(B.mant.data_ptr()), ctypes.c_void_p(B.exp.data_ptr()), B.m, A.rows,
                              B.rows, A.len, A.g, m_a, m_b, c_m, ROUNDING[rounding],
                              ctypes.c_uint64(seed & 0xFFFFFFFFFFFFFFFF), ctypes.c_void_p(t.mant.data_ptr()),
                              ctypes.c_void_p(t.exp.data_ptr()), st_ptr, _stream(A.device)), "bfp_gemm_bfp")
    return t


def gemm_group_partials(A: BFPTensor, B: BFPTensor, m_a: int | None = None, m_b: int | None = None) -> torch.Tensor:
    """Exact int32 group partials P [K/g, M, N] (int8 MFMA)."""
    m_a, m_b = _gemm_args(A, B, m_a, m_b)
    P = torch.empty((A.len // A.g, A.rows, B.rows), dtype=torch.int32, device=A.device)
    check(load().bfp_gemm_group_partials(ctypes.c_void_p(A.mant.data_ptr()), A.m, ctypes.c_void_p(B.mant.data_ptr()),
                                         B.m, A.rows, B.rows, A.len, A.g, m_a, m_b, ctypes.c_void_p(P.data_ptr()),
                                         _stream(A.device)), "bfp_gemm_group_partials")
    return P


def packed_sizes(rows: int, length: int, m: int):
    """(mantissa bytes, exponent bytes) of a rows x length packed BFP tensor."""
    mb, eb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    check(load().bfp_packed_sizes(rows, length, m, ctypes.byref(mb), ctypes.byref(eb)), "bfp_packed_sizes")
    return mb.value, eb.value


@dataclass
class PackedBFPTensor:
    """A rows x len BFP tensor in the packed storage of section V-D (groups of
    16 along len; see include/fastbfp.h): mant holds ceil(m/2) planes of 3-bit
    chunk fields, exp a uint32 E_max word and 3-bit exponent offsets."""
    mant: torch.Tensor
    exp: torch.Tensor
    rows: int
    len: int
    m: int
    g: int = 16

    @property
    def device(self) -> torch.device:
        return self.mant.device

    @staticmethod
    def empty(rows: int, length: int, m: int, device) -> "PackedBFPTensor":
        mb, eb = packed_sizes(rows, length, m)
        # int32 storage keeps the exponent stream 4-byte aligned
        exp = torch.empty((eb + 3) // 4, dtype=torch.int32, device=device).view(torch.uint8)[:eb]
        return PackedBFPTensor(torch.empty(mb, dtype=torch.uint8, device=device), exp, rows, length, m)


def quantize_packed(x: torch.Tensor, m: int = 4, rounding: str = "nearest", seed: int = 0,
                    status: torch.Tensor | None = None) -> PackedBFPTensor:
    """FP32 [..., C] -> packed BFP, groups of 16 along the last axis (leading
    axes flattened into rows), each group's exponent at least the tensor base
    max(E_max - 7, 0)."""
    _need_cuda(x, "x", torch.float32)
    if rounding not in ROUNDING:
        raise ValueError("rounding must be one of %s" % sorted(ROUNDING))
    if x.dim() < 1:
        raise ValueError("x must have at least one dimension")
    C = x.shape[-1]
    R = math.prod(x.shape[:-1])
    t = PackedBFPTensor.empty(R, C, m, x.device)
    check(load().bfp_quantize_packed(ctypes.c_void_p(x.data_ptr()), R, C, m, ROUNDING[rounding],
                                     ctypes.c_uint64(seed & 0xFFFFFFFFFFFFFFFF), ctypes.c_void_p(t.mant.data_ptr()),
                                     ctypes.c_void_p(t.exp.data_ptr()), _status_ptr(status), _stream(x.device)),
          "bfp_quantize_packed")
    return t


def dequantize_packed(t: PackedBFPTensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """Packed BFP -> FP32 [rows, len]."""
    y = out if out is not None else torch.empty((t.rows, t.len), dtype=torch.float32, device=t.device)
    _need_cuda(y, "out", torch.float32)
    check(load().bfp_dequantize_packed(ctypes.c_void_p(t.mant.data_ptr()), ctypes.c_void_p(t.exp.data_ptr()), t.rows,
                                       t.len, t.m, ctypes.c_void_p(y.data_ptr()), _stream(t.device)),
          "bfp_dequantize_packed")
    return y


def gemm_packed(A: PackedBFPTensor, B: PackedBFPTensor, m_a: int | None = None, m_b: int | None = None,
                out: torch.Tensor | None = None, workspace=True) -> torch.Tensor:
    """C = A . B^T in FP32 [A.rows, B.rows] for packed A [M, K] and B [N, K].
    workspace: as for gemm (True: unpacked into a workspace and run on the
    block-scaled kernel; False: bfp_gemm_packed's general kernel)."""
    m_a, m_b = _gemm_args(A, B, m_a, m_b)
    C = _gemm_out(A, B, out)
    if workspace is not False:
        return _gemm_with_workspace(A, B, m_a, m_b, C, workspace)
    check(load().bfp_gemm_packed(ctypes.c_void_p(A.mant.data_ptr()), ctypes.c_void_p(A.exp.data_ptr()), A.m,
                                 ctypes.c_void_p(B.mant.data_ptr()), ctypes.c_void_p(B.exp.data_ptr()), B.m, A.rows,
                                 B.rows, A.len, m_a, m_b, ctypes.c_void_p(C.data_ptr()), C.stride(0),
                                 _stream(A.device)), "bfp_gemm_packed")
    return C
