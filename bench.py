#!/usr/bin/env python3
"""Benchmark of the BFP hot path on one MI355X.

A step is one BFP training step of one FFN layer (M = 8192 tokens, 4096 ->
16384, groups of 16): X converted in both groupings from one read (along its
features for the forward GEMM, along the tokens for dW), the forward GEMM
Y = X . W, dY converted in both groupings with stochastic rounding, the
backward GEMMs dX = dY . W^T and dW = X^T . dY, and the weight update
W <- W - lr * dW with W converted in both groupings for the next step (the
forward and dX operands).  The mantissa width follows the schedule
2 -> 4 -> 6 bits over consecutive steps.  Inputs are resident in HBM before
timing (three dY tensors rotate with the schedule).

Printed: one JSON line with the step's effective BFP throughput
(2 M N K summed over the three GEMMs, divided by the step time including the
quantizations), the roofline of the dominant kernel measured with HIP events
inside the timed region, per-kernel figures, a sweep of the GEMM over the
transformer-block shapes and every mantissa pair, the quantize sweep over
64M-element tensors, and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "BFP GEMM effective TOPS per (m_a,m_b) + % int8 MFMA peak; quantize GB/s % HBM"
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
PEAK_FP6_TFLOPS = 10100.0    # dense FP6/FP4 MFMA (the instruction the GEMM issues)
PEAK_INT8_TOPS = 5000.0      # dense int8 MFMA (the metric's reference)
M_TOK, D_IN, D_FF, G = 8192, 4096, 16384, 16
SCHEDULE = (2, 4, 6)


def planes(m):
    return 1 if m <= 4 else 2


def mfma_passes(pa, pb, g=G):
    """MFMAs the block-scaled GEMM issues per group and fragment pair.  With
    groups of 32: one per pair of chunk planes.  With groups of 16: an operand
    split at 2 bits (m = 5, 6) fills a whole block, so it adds no pass (one
    MFMA per chunk plane of the other operand); two operands split at 4 bits
    (m = 7, 8) take 3 (the two cross products share one); otherwise one per
    pair of chunk planes."""
    if g == 32:
        return planes(pa) * planes(pb)
    split2 = lambda m: m in (5, 6)
    if split2(pa):
        return planes(pb)
    if split2(pb):
        return planes(pa)
    if pa >= 7 and pb >= 7:
        return 3
    return planes(pa) * planes(pb)


def mfma_issue_factor(pa, pb, g=G):
    """Issued MFMA work over the algorithmic work 2 M N K: MFMAs per group x 32
    values per block / g values per group."""
    return mfma_passes(pa, pb, g) * 32 // g


def code_bits(m):
    """Mantissa bits per value of the chunk-plane layout: one FP4 plane (4) for
    m = 1, 2; one FP6 plane (6) for m = 3, 4; an FP6 and a Lo2 plane (6 + 4)
    for m = 5, 6; two FP6 planes (12) for m = 7, 8."""
    return {1: 4, 2: 4, 3: 6, 4: 6, 5: 10, 6: 10, 7: 12, 8: 12}[m]


def q_bytes(n_elems, m, g=G):
    """Algorithmic HBM bytes of one quantization: read FP32, write the chunk
    planes and one exponent byte per group."""
    return n_elems * (4 + code_bits(m) / 8.0 + 1.0 / g)


def dual_bytes(n_elems, m, g=G):
    """Algorithmic HBM bytes of a two-grouping conversion: read FP32 once,
    write both BFP tensors."""
    return n_elems * (4 + 2 * (code_bits(m) / 8.0 + 1.0 / g))


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=30)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--no-sweeps", action="store_true", help="skip the GEMM and quantize sweeps")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--quiet", action="store_true")
    p.add_argument("--gemm-only", action="store_true",
                   help="run only the GEMM sweep and print its JSON (no step, no bench line)")
    p.add_argument("--gemm-pairs", choices=("default", "all", "resnet"), default="default",
                   help="GEMM sweep: six pairs on four shapes, all 16 operand-format pairs on ffn_up, or the "
                        "ResNet-18 im2col shapes alone")
    p.add_argument("--formats-only", action="store_true",
                   help="only the packed-storage, group-size and lowered-precision sweep (general kernel)")
    p.add_argument("--quantize-only", action="store_true",
                   help="run only the 64M quantize sweep (per distribution) and print its JSON")
    p.add_argument("--cpu-only", action="store_true",
                   help="run only the CPU oracle baseline (no GPU needed) and print its JSON")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="also run a plain 256 MiB device copy (torch) whose profiler counters calibrate HBM bytes")
    return p.parse_args()


def log(args, *a):
    if not args.quiet:
        print("[bench]", *a, file=sys.stderr, flush=True)


class Step:
    """Buffers and launches of one FFN training step."""

    def __init__(self, torch, fb, synth, dev):
        self.torch, self.fb = torch, fb
        t0 = time.time()
        self.X = torch.from_numpy(synth.draw("half_normal", (M_TOK, D_IN), 51)).to(dev)
        self.W = torch.from_numpy(synth.draw("weights", (D_IN, D_FF), 52)).to(dev)
        self.dY = [torch.from_numpy(synth.draw("grads", (M_TOK, D_FF), 53 + i)).to(dev) for i in range(3)]
        self.gen_s = time.time() - t0
        self.q = {}
        for m in SCHEDULE:
            e = fb.BFPTensor.empty
            self.q[m] = dict(
                xa=e(M_TOK, D_IN, G, m, dev),      # X grouped along features (fwd A)
                wb=e(D_FF, D_IN, G, m, dev),       # W regrouped: rows = output features (fwd B)
                dya=e(M_TOK, D_FF, G, m, dev),     # dY along features (dX A)
                wk=e(D_IN, D_FF, G, m, dev),       # W along its columns (dX B)
                xt=e(D_IN, M_TOK, G, m, dev),      # X regrouped along tokens (dW A)
                dyt=e(D_FF, M_TOK, G, m, dev),     # dY regrouped along tokens (dW B)
            )
        self.Y = torch.empty((M_TOK, D_FF), dtype=torch.float32, device=dev)
        self.dX = torch.empty((M_TOK, D_IN), dtype=torch.float32, device=dev)
        self.dW = torch.empty((D_IN, D_FF), dtype=torch.float32, device=dev)
        # the first step's BFP weights (later steps get them from the update)
        b = self.q[SCHEDULE[0]]
        fb.quantize_dual(self.W, g=G, m=SCHEDULE[0], out_rows=b["wk"], out_cols=b["wb"])

    def run(self, s, ev=None):
        """Enqueue step s.  ev: optional list collecting (name, start, end) events."""
        fb, torch = self.fb, self.torch
        m = SCHEDULE[s % 3]
        b = self.q[m]
        dy = self.dY[s % 3]
        seed = 1000 + 2 * s

        def rec(name, fn):
            if ev is None:
                fn()
                return
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            z.record()
            ev.append((name, m, a, z))

        nb = self.q[SCHEDULE[(s + 1) % 3]]
        rec("quantize_dual", lambda: fb.quantize_dual(self.X, g=G, m=m, out_rows=b["xa"], out_cols=b["xt"]))
        rec("gemm", lambda: fb.gemm(b["xa"], b["wb"], out=self.Y))
        rec("quantize_dual", lambda: fb.quantize_dual(dy, g=G, m=m, rounding="stochastic", seed_rows=seed,
                                                      seed_cols=seed + 1, out_rows=b["dya"], out_cols=b["dyt"]))
        rec("gemm", lambda: fb.gemm(b["dya"], b["wk"], out=self.dX))
        rec("gemm", lambda: fb.gemm(b["xt"], b["dyt"], out=self.dW))
        rec("weight_update", lambda: fb.weight_update(self.W, self.dW, -LR, g=G, m=SCHEDULE[(s + 1) % 3], w_out=self.W,
                                                      out_rows=nb["wk"], out_cols=nb["wb"]))


LR = 1e-3  # SGD step on the raw weight gradient
STEP_OPS = 3 * 2.0 * M_TOK * D_FF * D_IN
GEMM_OPS = 2.0 * M_TOK * D_FF * D_IN  # every one of the three GEMMs has M*N*K = 8192*16384*4096


def gemm_sweep(torch, fb, synth, dev, args):
    """Transformer-block GEMMs at every mantissa pair (effective TOPS)."""
    shapes = {"qkv": (8192, 12288, 4096), "out_proj": (8192, 4096, 4096), "ffn_up": (8192, 16384, 4096),
              "ffn_down": (8192, 4096, 16384)}
    pairs = [(2, 2), (2, 4), (4, 4), (4, 6), (6, 8), (8, 8)]
    if args.gemm_pairs == "all":
        # one pair per kernel variant (the four operand formats on each side:
        # m = 2 FP4, 4 FP6, 6 FP4 + FP6, 8 FP6 + FP6) on the FFN up-projection
        shapes = {"ffn_up": shapes["ffn_up"]}
        pairs = [(pa, pb) for pa in (2, 4, 6, 8) for pb in (2, 4, 6, 8)]
    X = torch.from_numpy(synth.bf16_round(synth.draw("normal", (8192, 16384), 41))).to(dev)
    Wt = torch.from_numpy(synth.bf16_round(synth.draw("weights", (16384, 16384), 42))).to(dev)
    out = {}
    for name, (M, N, K) in shapes.items():
        xa = X[:M, :K].contiguous()
        wb = Wt[:N, :K].contiguous()
        C = torch.empty((M, N), dtype=torch.float32, device=dev)
        for pa, pb in pairs:
            A = fb.quantize(xa, g=G, m=pa)
            B = fb.quantize(wb, g=G, m=pb)
            fb.gemm(A, B, out=C)
            torch.cuda.synchronize()
            reps = 5
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fb.gemm(A, B, out=C)
            z.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(z) / reps
            tops = 2.0 * M * N * K / (ms * 1e-3) / 1e12
            issued = tops * mfma_issue_factor(pa, pb)  # chunk passes and zero-padded half blocks
            out["%s(%d,%d)" % (name, pa, pb)] = {
                "M": M, "N": N, "K": K, "ms": round(ms, 4), "eff_tops": round(tops, 1),
                "frac_int8_peak": round(tops / PEAK_INT8_TOPS, 4),
                "mfma_issued_tflops": round(issued, 1), "frac_fp6_peak_issued": round(issued / PEAK_FP6_TFLOPS, 4)}
            log(args, "gemm %s (%d,%d): %.3f ms, %.0f eff TOPS" % (name, pa, pb, ms, tops))
        del C
    if args.gemm_pairs == "all":
        del X, Wt
        return out
    # groups of 32 (the sensitivity study's other group size): one whole group
    # per MFMA block, no zero padding
    M, N, K = shapes["ffn_up"]
    xa, wb = X[:M, :K].contiguous(), Wt[:N, :K].contiguous()
    C = torch.empty((M, N), dtype=torch.float32, device=dev)
    for pa, pb in [(2, 2), (4, 4), (6, 6), (8, 8)]:
        A, B = fb.quantize(xa, g=32, m=pa), fb.quantize(wb, g=32, m=pb)
        fb.gemm(A, B, out=C)
        torch.cuda.synchronize()
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(5):
            fb.gemm(A, B, out=C)
        z.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(z) / 5
        tops = 2.0 * M * N * K / (ms * 1e-3) / 1e12
        issued = tops * mfma_issue_factor(pa, pb, 32)  # chunk passes, no padding
        out["ffn_up_g32(%d,%d)" % (pa, pb)] = {
            "M": M, "N": N, "K": K, "g": 32, "ms": round(ms, 4), "eff_tops": round(tops, 1),
            "frac_int8_peak": round(tops / PEAK_INT8_TOPS, 4), "mfma_issued_tflops": round(issued, 1),
            "frac_fp6_peak_issued": round(issued / PEAK_FP6_TFLOPS, 4)}
        log(args, "gemm ffn_up g=32 (%d,%d): %.3f ms, %.0f eff TOPS" % (pa, pb, ms, tops))
    del X, Wt, C
    return out


def resnet_sweep(torch, fb, synth, dev, args):
    """ResNet-18 convolutions at batch 256, 224x224 input, as im2col GEMMs
    (C[M,N] = A[M,K] B[N,K]^T, g = 16 along K): half-normal activations, N(0, 0.02)
    weights, round to nearest.  These shapes are HBM-bound: the roofline time is
    max(2MNK / int8 MFMA peak, minimum bytes / HBM peak), with minimum bytes =
    the BFP operands (codes + exponents) read once and the FP32 C written once.
    The same GEMM with C converted to BFP in the epilogue (the next layer's
    activations at the width of A, round to nearest) is timed beside it, with
    its own minimum bytes (the BFP C instead of the FP32 C) and against the
    unfused route (the FP32 GEMM, then a separate quantize of C)."""
    shapes = {"conv2_x": (256 * 56 * 56, 64, 576), "conv3_x": (256 * 28 * 28, 128, 1152),
              "conv4_x": (256 * 14 * 14, 256, 2304), "conv5_x": (256 * 7 * 7, 512, 4608)}
    pairs = [(2, 2), (2, 4), (4, 4)]
    # one activation draw serves every shape: each A is a [M, K] view of its
    # first M*K values (M*K shrinks from conv2_x on)
    n_act = max(M * K for M, _, K in shapes.values())
    act = torch.from_numpy(synth.draw("half_normal", (n_act,), 31)).to(dev)
    out = {}
    for i, (name, (M, N, K)) in enumerate(shapes.items()):
        xa = act[:M * K].view(M, K)
        wb = torch.from_numpy(synth.draw("weights", (N, K), 32 + i)).to(dev)
        C = torch.empty((M, N), dtype=torch.float32, device=dev)
        for pa, pb in pairs:
            A = fb.quantize(xa, g=G, m=pa)
            B = fb.quantize(wb, g=G, m=pb)
            fb.gemm(A, B, out=C)
            torch.cuda.synchronize()
            reps = 10
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fb.gemm(A, B, out=C)
            z.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(z) / reps
            tops = 2.0 * M * N * K / (ms * 1e-3) / 1e12
            nbytes = (M * K * code_bits(pa) + N * K * code_bits(pb)) / 8.0 + (M + N) * K / G + 4.0 * M * N
            gbs = nbytes / (ms * 1e-3) / 1e9
            floor_ms = max(2.0 * M * N * K / (PEAK_INT8_TOPS * 1e12), nbytes / (PEAK_HBM_GBS * 1e9)) * 1e3
            # C converted to BFP in the epilogue, at A's width
            T = fb.BFPTensor.empty(M, N, G, pa, dev)
            fb.gemm_bfp(A, B, pa, out=T)
            torch.cuda.synchronize()
            a.record()
            for _ in range(reps):
                fb.gemm_bfp(A, B, pa, out=T)
            z.record()
            torch.cuda.synchronize()
            fms = a.elapsed_time(z) / reps
            a.record()
            for _ in range(reps):
                fb.gemm(A, B, out=C)
                fb.quantize(C, g=G, m=pa, out=T)
            z.record()
            torch.cuda.synchronize()
            ums = a.elapsed_time(z) / reps
            fbytes = nbytes - 4.0 * M * N + M * N * code_bits(pa) / 8.0 + M * N / G
            ffloor_ms = max(2.0 * M * N * K / (PEAK_INT8_TOPS * 1e12), fbytes / (PEAK_HBM_GBS * 1e9)) * 1e3
            out["%s(%d,%d)" % (name, pa, pb)] = {
                "M": M, "N": N, "K": K, "ms": round(ms, 4), "eff_tops": round(tops, 1),
                "frac_int8_peak": round(tops / PEAK_INT8_TOPS, 4), "min_bytes": int(nbytes),
                "GB_s": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                "roofline_ms": round(floor_ms, 4), "frac_roofline": round(floor_ms / ms, 4),
                "bfp_out": {"m": pa, "fused_ms": round(fms, 4), "unfused_ms": round(ums, 4),
                            "speedup": round(ums / fms, 3), "min_bytes": int(fbytes),
                            "GB_s": round(fbytes / (fms * 1e-3) / 1e9, 1), "roofline_ms": round(ffloor_ms, 4),
                            "frac_roofline": round(ffloor_ms / fms, 4)}}
            log(args, "gemm %s (%d,%d): %.3f ms, %.0f eff TOPS, %.0f GB/s (%.0f%% of the roofline time); "
                "BFP output: %.3f ms fused, %.3f ms unfused (%.0f%% of its roofline time)"
                % (name, pa, pb, ms, tops, gbs, 100.0 * floor_ms / ms, fms, ums, 100.0 * ffloor_ms / fms))
            del A, B, T
        del C, wb
    del act
    return out


def quantize_sweep(torch, fb, synth, dev, args):
    """64M-element quantize (8192 x 8192, g=16, last axis) for each of the
    three distributions separately.  Consecutive launches read three different
    256 MB buffers holding the same values in different rows (the tensor and
    two row rotations of it), so the 256 MB Infinity Cache cannot serve a
    repeated read."""
    out = {}
    n = 8192 * 8192
    dists = (("half_normal", 21), ("weights", 22), ("grads", 23))
    for dist, seed in dists:
        x0 = torch.from_numpy(synth.draw(dist, (8192, 8192), seed)).to(dev)
        xs = [x0, torch.roll(x0, 2731, 0).contiguous(), torch.roll(x0, 5461, 0).contiguous()]
        for m in (2, 4, 6, 8):
            for mode in ("nearest", "stochastic"):
                outs = [fb.BFPTensor.empty(8192, 8192, G, m, dev) for _ in range(3)]
                for i in range(3):
                    fb.quantize(xs[i], g=G, m=m, rounding=mode, seed=1234, out=outs[i])
                torch.cuda.synchronize()
                reps = 12
                a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                for r in range(reps):
                    fb.quantize(xs[r % 3], g=G, m=m, rounding=mode, seed=1234, out=outs[r % 3])
                z.record()
                torch.cuda.synchronize()
                ms = a.elapsed_time(z) / reps
                gbs = q_bytes(n, m) / (ms * 1e-3) / 1e9
                out["%s_m%d_%s" % (dist, m, mode)] = {"us": round(ms * 1e3, 2), "GB_s": round(gbs, 1),
                                                      "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                                                      "bytes": int(q_bytes(n, m))}
                log(args, "quantize %s m=%d %s: %.1f us, %.0f GB/s" % (dist, m, mode, ms * 1e3, gbs))
                del outs
        # The adaptive converter (Algorithm 1, Eq. 2): one pass writes BFP(X,4),
        # the 2-bit tensor left by discarding the low chunk, and the two sums.
        for mode in ("nearest", "stochastic"):
            for r in range(3):
                fb.quantize_adaptive(xs[r], g=G, rounding=mode, seed=1234)
            torch.cuda.synchronize()
            reps = 12
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for r in range(reps):
                fb.quantize_adaptive(xs[r % 3], g=G, rounding=mode, seed=1234)
            z.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(z) / reps
            nbytes = n * (4 + 0.75 + 0.5 + 1.0 / G)
            gbs = nbytes / (ms * 1e-3) / 1e9
            out["%s_adaptive_m4m2_%s" % (dist, mode)] = {"us": round(ms * 1e3, 2), "GB_s": round(gbs, 1),
                                                         "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                                                         "bytes": int(nbytes)}
            log(args, "adaptive %s m=4/2 %s: %.1f us, %.0f GB/s" % (dist, mode, ms * 1e3, gbs))
        del xs, x0
        torch.cuda.empty_cache()
    return out


def epilogue_sweep(torch, fb, synth, dev, args):
    """The GEMM with its output converted to BFP in the epilogue (the layer
    output handed to the next layer as BFP, section V-A) against the same work
    unfused: the FP32 GEMM followed by a separate quantize of C (16384-wide
    rows, groups of 16).  FFN up-projection shape, output at the input's
    width."""
    M, N, K = 8192, 16384, 4096
    X = torch.from_numpy(synth.draw("normal", (M, K), 41)).to(dev)
    W = torch.from_numpy(synth.draw("weights", (N, K), 42)).to(dev)
    C = torch.empty((M, N), dtype=torch.float32, device=dev)
    out = {}

    def timed(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        z.record()
        torch.cuda.synchronize()
        return a.elapsed_time(z) / reps

    for m in (2, 4, 6):
        A, B = fb.quantize(X, g=G, m=m), fb.quantize(W, g=G, m=m)
        T = fb.BFPTensor.empty(M, N, G, m, dev)
        for mode in ("nearest", "stochastic"):
            fused = timed(lambda: fb.gemm_bfp(A, B, m, rounding=mode, seed=77, out=T))
            sep = timed(lambda: (fb.gemm(A, B, out=C), fb.quantize(C, g=G, m=m, rounding=mode, seed=77, out=T)))
            out["ffn_up(%d,%d)->m%d_%s" % (m, m, m, mode)] = {
                "fused_ms": round(fused, 4), "unfused_ms": round(sep, 4), "speedup": round(sep / fused, 3),
                "fused_eff_tops": round(2.0 * M * N * K / (fused * 1e-3) / 1e12, 1)}
            log(args, "gemm_bfp ffn_up m=%d %s: fused %.3f ms, unfused %.3f ms" % (m, mode, fused, sep))
        del A, B, T
    del X, W, C
    return out


def format_sweep(torch, fb, synth, dev, args):
    """The cases the block-scaled kernel does not read as stored: the packed
    storage of section V-D (conversion with its E_max pass), group sizes 8
    and 64, and a GEMM taken below the stored width (stored 4, used at 2;
    stored 6, used at 3), on the out-projection shape (8192 x 4096 x 4096)
    and an 8192 x 8192 conversion.  Each GEMM is timed on both routes: the
    default one (bfp_gemm_ws: the operands repacked into a workspace, then
    the block-scaled kernel; the repack is inside the timed region) and the
    allocation-free general kernel (bfp_gemm / bfp_gemm_packed)."""
    out = {}

    def timed(fn, reps=3):
        fn()
        torch.cuda.synchronize()
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        z.record()
        torch.cuda.synchronize()
        return a.elapsed_time(z) / reps

    n = 8192 * 8192
    x = torch.from_numpy(synth.draw("half_normal", (8192, 8192), 21)).to(dev)
    for m in (2, 4):
        for mode in ("nearest", "stochastic"):
            ms = timed(lambda: fb.quantize_packed(x, m=m, rounding=mode, seed=1234), reps=6)
            mb, eb = fb.packed_sizes(8192, 8192, m)
            moved = 2 * n * 4 + mb + eb  # x read by the E_max pass and by the conversion
            out["packed_quantize_m%d_%s" % (m, mode)] = {
                "us": round(ms * 1e3, 2), "GB_s_moved": round(moved / (ms * 1e-3) / 1e9, 1),
                "frac_hbm": round(moved / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                "bits_per_value": round(8.0 * (mb + eb) / n, 4)}
            log(args, "packed quantize m=%d %s: %.1f us" % (m, mode, ms * 1e3))
    del x
    M, N, K = 8192, 4096, 4096
    X = torch.from_numpy(synth.draw("normal", (M, K), 41)).to(dev)
    W = torch.from_numpy(synth.draw("weights", (N, K), 42)).to(dev)
    C = torch.empty((M, N), dtype=torch.float32, device=dev)
    cases = []
    for m in (2, 4):
        A, B = fb.quantize_packed(X, m=m), fb.quantize_packed(W, m=m)
        cases.append(("packed(%d,%d)" % (m, m), lambda ws, A=A, B=B: fb.gemm_packed(A, B, out=C, workspace=ws)))
    for g in (8, 64):
        A, B = fb.quantize(X, g=g, m=4), fb.quantize(W, g=g, m=4)
        cases.append(("g%d(4,4)" % g, lambda ws, A=A, B=B: fb.gemm(A, B, out=C, workspace=ws)))
    for stored, used in ((4, 2), (6, 3)):
        A, B = fb.quantize(X, g=G, m=stored), fb.quantize(W, g=G, m=stored)
        cases.append(("stored%d_used(%d,%d)" % (stored, used, used),
                      lambda ws, A=A, B=B, u=used: fb.gemm(A, B, u, u, out=C, workspace=ws)))
    tops = lambda ms: 2.0 * M * N * K / (ms * 1e-3) / 1e12
    for name, fn in cases:
        ms = timed(lambda: fn(True))
        ms_general = timed(lambda: fn(False), reps=2)
        out["out_proj_" + name] = {"ms": round(ms, 4), "eff_tops": round(tops(ms), 1),
                                   "frac_int8_peak": round(tops(ms) / PEAK_INT8_TOPS, 4),
                                   "general_kernel_ms": round(ms_general, 3),
                                   "general_kernel_eff_tops": round(tops(ms_general), 1)}
        log(args, "GEMM out_proj %s: %.3f ms repacked, %.3f ms on the general kernel" % (name, ms, ms_general))
    del X, W, C, cases
    return out


def calibration_copy(torch, dev):
    """A plain 256 MiB device copy (torch), three times: its profiler
    counters calibrate the HBM byte counts of the other kernels."""
    src = torch.ones(64 * 1024 * 1024, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    return {"read": src.numel() * 4, "write": dst.numel() * 4}


def measured_traffic(key):
    """HBM bytes per launch of a bench kernel from the committed rocprofv3
    counter runs (profiles/traffic.json), or None if the kernel sources have
    changed since those counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    data = json.load(open(path))
    for fn, sha in data.get("source_sha256", {}).items():
        src = os.path.join(ROOT, "paper_2110_15456_amd", "csrc", fn)
        if not os.path.exists(src) or hashlib.sha256(open(src, "rb").read()).hexdigest() != sha:
            return None
    entry = data.get("bench_keys", {}).get(key)
    return round(entry["bytes_per_launch"]) if entry else None


def host_threads():
    """Threads for the oracle: the cores this process may run on, within the
    CPU share the environment allots (OMP_NUM_THREADS; on a shared GPU host,
    one GPU's share of its cores)."""
    avail = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    share = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    return max(1, min(avail, share) if share > 0 else avail), avail


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(args):
    """The oracle, untuned, on the host cores.  Reported value: one m=4 FFN
    step in the bench's unit -- every conversion and the weight update in
    full, plus the first SAMPLE_ROWS output rows of each GEMM, the GEMM time
    scaled to all rows.  Also: the 64M-element quantize sweep in full for
    every (distribution, m, rounding mode), and each transformer-block and
    ResNet-18 im2col GEMM on a sample of output rows (scaled to all rows)."""
    import numpy as np
    import oracle
    from paper_2110_15456_amd import synth
    threads, avail = host_threads()
    t_all = time.time()
    X = synth.draw("half_normal", (M_TOK, D_IN), 51)
    W = synth.draw("weights", (D_IN, D_FF), 52)
    dY = synth.draw("grads", (M_TOK, D_FF), 53)
    m = 4
    t0 = time.time()
    wk, wb, _ = oracle.quantize_dual(W, g=G, m=m, threads=threads)
    xa, xt, _ = oracle.quantize_dual(X, g=G, m=m, threads=threads)
    dya, dyt, _ = oracle.quantize_dual(dY, g=G, m=m, mode="stochastic", seed_rows=1000, seed_cols=1001,
                                       threads=threads)
    tq = time.time() - t0
    SAMPLE_ROWS = 128
    rows = np.arange(SAMPLE_ROWS)
    t1 = time.time()
    oracle.gemm(xa[0], xa[1], m, wb[0], wb[1], m, g=G, rows=rows, threads=threads)
    oracle.gemm(dya[0], dya[1], m, wk[0], wk[1], m, g=G, rows=rows, threads=threads)
    oracle.gemm(xt[0], xt[1], m, dyt[0], dyt[1], m, g=G, rows=rows, threads=threads)
    tg = time.time() - t1
    # the weight update (on a stand-in gradient of the right shape) and its
    # two-grouping conversion for the next step
    t2 = time.time()
    W2 = oracle.weight_update(W, dY[:D_IN, :D_FF], -LR)
    oracle.quantize_dual(W2, g=G, m=m, threads=threads)
    tq += time.time() - t2
    del X, W, dY, W2, wk, wb, xa, xt, dya, dyt
    # rows sampled: SAMPLE_ROWS of 8192 (fwd, dX) and of 4096 (dW); the three
    # GEMMs have the same N*K per output row, so each took about tg / 3
    full_gemm_s = tg / 3 * (M_TOK + M_TOK + D_IN) / SAMPLE_ROWS
    step_s = tq + full_gemm_s

    # the quantize sweep at full size (8192 x 8192, g = 16 along the last axis)
    quant = {}
    n = 8192 * 8192
    for dist, seed in (("half_normal", 21), ("weights", 22), ("grads", 23)):
        x = synth.draw(dist, (8192, 8192), seed)
        for mq in (2, 4, 6, 8):
            for mode in ("nearest", "stochastic"):
                t = time.time()
                oracle.quantize(x, g=G, m=mq, mode=mode, seed=1234, threads=threads)
                dt = time.time() - t
                quant["%s_m%d_%s" % (dist, mq, mode)] = {"s": round(dt, 3),
                                                         "GB_s": round(q_bytes(n, mq) / dt / 1e9, 3)}
        del x
    # GEMMs on sampled output rows: transformer block at (4,4), ResNet-18
    # im2col at (2,4); the oracle's time per output row does not depend on
    # which rows
    gemms = {}
    shapes = [("qkv", 8192, 12288, 4096, 4, 4), ("out_proj", 8192, 4096, 4096, 4, 4),
              ("ffn_up", 8192, 16384, 4096, 4, 4), ("ffn_down", 8192, 4096, 16384, 4, 4),
              ("conv2_x", 802816, 64, 576, 2, 4), ("conv3_x", 200704, 128, 1152, 2, 4),
              ("conv4_x", 50176, 256, 2304, 2, 4), ("conv5_x", 12544, 512, 4608, 2, 4)]
    for name, Mg, Ng, Kg, pa, pb in shapes:
        rows_g = max(16, min(Mg, (1 << 27) // (Ng * Kg)))  # about 2^27 MACs
        xa_g = synth.draw("half_normal", (rows_g, Kg), 71)
        xb_g = synth.draw("weights", (Ng, Kg), 72)
        qa_g, ea_g, _ = oracle.quantize(xa_g, g=G, m=pa, threads=threads)
        qb_g, eb_g, _ = oracle.quantize(xb_g, g=G, m=pb, threads=threads)
        t = time.time()
        oracle.gemm(qa_g, ea_g, pa, qb_g, eb_g, pb, g=G, threads=threads)
        dt = (time.time() - t) * Mg / rows_g
        gemms["%s(%d,%d)" % (name, pa, pb)] = {"rows_timed": rows_g, "est_s": round(dt, 2),
                                               "eff_gops": round(2.0 * Mg * Ng * Kg / dt / 1e9, 3)}
    return {"value": round(STEP_OPS / step_s / 1e12, 6), "unit": "TOPS", "cores": threads, "kind": "oracle",
            "sample": ("one m=4 FFN step: the conversions of X, dY and W and the weight update in full (%.1f s) and "
                       "the first %d output rows of each GEMM (%.1f s), GEMM time scaled by rows to the full step "
                       "(est. %.0f s per step)" % (tq, SAMPLE_ROWS, tg, step_s)),
            "host": {"cpu_model": cpu_model(), "nproc": os.cpu_count(), "cores_available": avail,
                     "threads_used": threads},
            "quantize_64M": quant, "gemm_sampled": gemms,
            "cpu_seconds": round(time.time() - t_all, 1)}


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (--gpus %d requested)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    if args.cpu_only:
        print(json.dumps({"cpu_baseline": cpu_baseline(args)}), flush=True)
        return
    import torch
    import paper_2110_15456_amd as fb
    from paper_2110_15456_amd import synth
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    fb._lib.load()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    if args.quantize_only:
        res = {"quantize_sweep": quantize_sweep(torch, fb, synth, dev, args)}
        if args.calibrate_copy:
            res["copy_calibration_bytes"] = calibration_copy(torch, dev)
        print(json.dumps(res), flush=True)
        return
    if args.formats_only:
        print(json.dumps({"format_sweep": format_sweep(torch, fb, synth, dev, args)}), flush=True)
        return
    if args.gemm_only:
        if args.gemm_pairs == "resnet":
            print(json.dumps({"resnet_sweep": resnet_sweep(torch, fb, synth, dev, args)}), flush=True)
            return
        print(json.dumps({"gemm_sweep": gemm_sweep(torch, fb, synth, dev, args)}), flush=True)
        return
    step = Step(torch, fb, synth, dev)
    log(args, "inputs generated in %.1f s" % step.gen_s)
    for s in range(args.warmup):
        step.run(s)
    torch.cuda.synchronize()

    events = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for s in range(args.steps):
        step.run(args.warmup + s, events)
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(stop) / args.steps
    value = STEP_OPS / (ms_step * 1e-3) / 1e12

    # per-kernel table from the events recorded inside the timed region
    table = {}
    # algorithmic HBM bytes of the conversions: read the FP32 input(s), write
    # two BFP tensors (and, for the update, the FP32 weights)
    sizes = [M_TOK * D_IN, 0, M_TOK * D_FF, 0, 0, D_IN * D_FF]
    for i, (name, m, a, z) in enumerate(events):
        k = i % 6
        r = table.setdefault("%s_m%d" % (name, m), {"launches": 0, "ms": 0.0, "work": 0.0})
        r["launches"] += 1
        r["ms"] += a.elapsed_time(z)
        if name == "gemm":
            r["work"] += GEMM_OPS
        elif name == "quantize_dual":
            r["work"] += dual_bytes(sizes[k], m)
        else:  # the update converts at the next step's width
            r["work"] += dual_bytes(sizes[k], SCHEDULE[(SCHEDULE.index(m) + 1) % 3]) + 8.0 * sizes[k]
    kernels = {}
    for key, r in table.items():
        avg = r["ms"] / r["launches"]
        per = r["work"] / r["launches"]
        if key.startswith("gemm"):
            ach = per / (avg * 1e-3) / 1e12
            kernels[key] = {"launches": r["launches"], "avg_ms": round(avg, 4), "achieved": round(ach, 1),
                            "unit": "TFLOP/s", "share": 0.0}
        else:
            ach = per / (avg * 1e-3) / 1e9
            kernels[key] = {"launches": r["launches"], "avg_ms": round(avg, 4), "achieved": round(ach, 1),
                            "unit": "GB/s", "frac_hbm": round(ach / PEAK_HBM_GBS, 4), "share": 0.0}
    total = sum(r["ms"] for r in table.values())
    for key, r in table.items():
        kernels[key]["share"] = round(r["ms"] / total, 4)
    dom = max(table, key=lambda k: table[k]["ms"])
    d = kernels[dom]
    if dom.startswith("gemm"):
        mdom = int(dom.split("_m")[1])
        issue = mfma_issue_factor(mdom, mdom)  # chunk passes x zero-padded half blocks
        roof = {"bound": "mfma", "kernel": dom, "achieved": d["achieved"], "peak": PEAK_FP6_TFLOPS,
                "unit": "TFLOP/s", "frac": round(d["achieved"] / PEAK_FP6_TFLOPS, 4), "traffic": measured_traffic(dom),
                "work_per_launch": "2*M*N*K = %.4g FLOP (BFP MACs, algorithmic)" % GEMM_OPS,
                "issued": {"tflops": round(d["achieved"] * issue, 1),
                           "frac": round(d["achieved"] * issue / PEAK_FP6_TFLOPS, 4),
                           "factor": issue,
                           "note": "MFMA work the kernel issues: the algorithmic work x MFMAs per group x 32 / g (a "
                                   "16-value group fills half of a 32-value MFMA block, except an operand split at 2 "
                                   "bits, m = 5, 6, which fills a whole block)"}}
    else:
        roof = {"bound": "hbm", "kernel": dom, "achieved": d["achieved"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(d["achieved"] / PEAK_HBM_GBS, 4), "traffic": measured_traffic(dom)}
    log(args, "step %.3f ms, %.1f eff TOPS, wall %.2f s" % (ms_step, value, wall))

    result = {
        "metric": METRIC, "value": round(value, 2), "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "fp6", "data": "synthetic",
        "config": {"workload": "BFP FFN training step: tokens 8192, 4096->16384, g=16, fwd+dX+dW GEMMs, X and dY "
                               "converted in both groupings from one read (SR on dY), SGD weight update with both "
                               "groupings of W for the next step, mantissa schedule 2->4->6",
                   "M": M_TOK, "d_in": D_IN, "d_ff": D_FF, "g": G, "schedule": list(SCHEDULE)},
        "roofline": roof, "kernels": kernels,
    }
    del step
    torch.cuda.empty_cache()
    if args.calibrate_copy:
        result["copy_calibration_bytes"] = calibration_copy(torch, dev)
    if not args.no_sweeps:
        result["gemm_sweep"] = gemm_sweep(torch, fb, synth, dev, args)
        torch.cuda.empty_cache()
        result["resnet_sweep"] = resnet_sweep(torch, fb, synth, dev, args)
        torch.cuda.empty_cache()
        result["quantize_sweep"] = quantize_sweep(torch, fb, synth, dev, args)
        result["epilogue_sweep"] = epilogue_sweep(torch, fb, synth, dev, args)
        torch.cuda.empty_cache()
        result["format_sweep"] = format_sweep(torch, fb, synth, dev, args)
    if not args.no_cpu:
        log(args, "timing the CPU oracle on a sample ...")
        result["cpu_baseline"] = cpu_baseline(args)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
