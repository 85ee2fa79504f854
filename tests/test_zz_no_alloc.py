"""The allocation-free adaptive converter (bfp_quantize_adaptive_noalloc),
called through the C ABI, against bfp_quantize_adaptive (the same outputs
with a caller workspace): codes, exponents and both Eq. 2 sums identical, on
two calls in a row -- the second with a smaller input, so that stale partials
of the first call in the library's scratch array would show -- for both group
axes and both group sizes.  Then the limit: a shape with more partials than
the scratch array holds is rejected before any launch."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest
import torch

import paper_2110_15456_amd as fb
from paper_2110_15456_amd import _lib, synth
from gpu_util import announce

pytestmark = pytest.mark.gpu
P = ctypes.c_void_p


def noalloc_call(lib, x, R, C, axis, g, mode, seed, t4, t2, sums, status=None):
    return lib.bfp_quantize_adaptive_noalloc(P(x.data_ptr()), R, C, axis, g, mode, ctypes.c_uint64(seed),
                                             P(t4.mant.data_ptr()), P(t2.mant.data_ptr()) if t2 is not None else None,
                                             P(t4.exp.data_ptr()), P(sums.data_ptr()),
                                             P(status.data_ptr()) if status is not None else None,
                                             P(torch.cuda.current_stream().cuda_stream))


@pytest.mark.parametrize("axis", [1, 0])
@pytest.mark.parametrize("g", [16, 32])
def test_noalloc_matches_workspace_entry_point(axis, g):
    lib = _lib.load()
    for i, (R, C, dist, mode) in enumerate([(2048, 4096, "grads", 1), (192, 320, "half_normal", 0)]):
        announce("adaptive noalloc call %d: %dx%d axis %d g=%d" % (i, R, C, axis, g))
        x = torch.from_numpy(synth.draw(dist, (R, C), 90 + i)).cuda()
        rows, length = (R, C) if axis == 1 else (C, R)
        ref4, ref2, ref_sums = fb.quantize_adaptive(x, group_axis=-1 if axis == 1 else 0, g=g,
                                                    rounding=("nearest", "stochastic")[mode], seed=55)
        t4 = fb.BFPTensor.empty(rows, length, g, 4, "cuda")
        t2 = fb.BFPTensor(torch.empty_like(ref2.mant), t4.exp, rows, length, g, 2)
        sums = torch.full((2,), -1.0, dtype=torch.float64, device="cuda")
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        assert noalloc_call(lib, x, R, C, axis, g, mode, 55, t4, t2, sums, status) == 0
        torch.cuda.synchronize()
        assert torch.equal(t4.mant, ref4.mant) and torch.equal(t4.exp, ref4.exp)
        assert torch.equal(t2.mant, ref2.mant)
        assert sums.cpu().numpy().tobytes() == ref_sums.cpu().numpy().tobytes()
        assert int(status.item()) == 0


def test_noalloc_limit_and_empty():
    lib = _lib.load()
    cap = lib.bfp_adaptive_noalloc_max_parts()
    assert cap == (1 << 17)
    # 2^26 groups of 16 along rows fill the array exactly; one row more does not fit
    assert lib.bfp_adaptive_parts(1 << 16, 1 << 14, 1, 16) == cap
    fake = P(0x100000)
    sums = torch.zeros(2, dtype=torch.float64, device="cuda")
    rc = lib.bfp_quantize_adaptive_noalloc(fake, (1 << 16) + 1, 1 << 14, 1, 16, 0, ctypes.c_uint64(0), fake, None,
                                           fake, P(sums.data_ptr()), None, None)
    assert rc == 3  # BFP_E_UNSUPPORTED, before any launch
    # an empty tensor: both sums become zero
    announce("adaptive noalloc empty input")
    x = torch.zeros((0, 64), device="cuda")
    t4 = fb.BFPTensor.empty(0, 64, 16, 4, "cuda")
    sums.fill_(5.0)
    assert noalloc_call(lib, x, 0, 64, 1, 16, 0, 0, t4, None, sums) == 0
    torch.cuda.synchronize()
    assert sums.cpu().tolist() == [0.0, 0.0]
