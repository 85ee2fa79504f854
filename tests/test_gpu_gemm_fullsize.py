"""GPU parity of bfp_gemm at the full transformer-block and ResNet-18 im2col
sizes, for every mantissa pair of those workloads, on sampled output rows
(the first, the last and 24 random ones) against the oracle:
|C_gpu - C_oracle| <= 1e-6 * sum_G |T_G| for every sampled output.

Transformer block (8192 tokens, hidden 4096, FFN 16384): X ~ N(0, 1) and
W ~ N(0, 0.02), both rounded through bf16, at (2,2), (2,4), (4,4), (4,6),
(6,8) and (8,8).  ResNet-18 convolutions at batch 256 as im2col GEMMs:
half-normal activations and N(0, 0.02) weights at (2,2), (2,4) and (4,4).
Groups of 16 along K, round to nearest."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2110_15456_amd as fb
from paper_2110_15456_amd import synth
from gpu_util import announce, THREADS

pytestmark = pytest.mark.gpu
TRANSFORMER_PAIRS = [(2, 2), (2, 4), (4, 4), (4, 6), (6, 8), (8, 8)]
RESNET_PAIRS = [(2, 2), (2, 4), (4, 4)]


def sampled_rows(M: int, n: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, M - 1], rng.choice(M, n, replace=False)]))


def check_pairs(xa: np.ndarray, xb: np.ndarray, pairs, rows: np.ndarray, label: str):
    M, K = xa.shape
    N = xb.shape[0]
    ta, tb = torch.from_numpy(xa).cuda(), torch.from_numpy(xb).cuda()
    oa, ob = {}, {}
    for pa, pb in pairs:
        if pa not in oa:  # the oracle's A only on the sampled rows
            qa = np.zeros((M, K), np.int16)
            ea = np.zeros((M, K // 16), np.uint8)
            for r in rows:
                q1, e1, _ = oracle.quantize(xa, g=16, m=pa, rows=(int(r), int(r) + 1))
                qa[r], ea[r] = q1[0], e1[0]
            oa[pa] = (qa, ea)
        if pb not in ob:
            qb, eb, _ = oracle.quantize(xb, g=16, m=pb, threads=THREADS)
            ob[pb] = (qb, eb)
        announce("gemm full size %s %dx%dx%d (%d,%d), %d sampled rows" % (label, M, N, K, pa, pb, len(rows)))
        A = fb.quantize(ta, g=16, m=pa)
        B = fb.quantize(tb, g=16, m=pb)
        assert np.array_equal(A.exp.cpu().numpy()[rows], oa[pa][1][rows])
        assert np.array_equal(B.exp.cpu().numpy(), ob[pb][1])
        C = fb.gemm(A, B)
        torch.cuda.synchronize()
        Cg = C.cpu().numpy()[rows].astype(np.float64)
        Co, S = oracle.gemm(oa[pa][0], oa[pa][1], pa, ob[pb][0], ob[pb][1], pb, g=16, rows=rows, threads=THREADS)
        ratio = np.abs(Cg - Co) / np.maximum(S, 1e-300)
        assert np.all(np.abs(Cg - Co) <= 1e-6 * S), "(%d,%d): max err / sum|T| = %.3g" % (pa, pb, ratio.max())
        del A, B, C


@pytest.mark.parametrize("name,shape", [("qkv", (8192, 12288, 4096)), ("out_proj", (8192, 4096, 4096)),
                                        ("ffn_up", (8192, 16384, 4096)), ("ffn_down", (8192, 4096, 16384))])
def test_transformer_block_all_pairs(name, shape):
    M, N, K = shape
    xa = synth.bf16_round(synth.draw("normal", (M, K), 41))
    xb = synth.bf16_round(synth.draw("weights", (N, K), 42))
    check_pairs(xa, xb, TRANSFORMER_PAIRS, sampled_rows(M, 24, 43), name)


@pytest.mark.parametrize("name,shape", [("conv2_x", (802816, 64, 576)), ("conv3_x", (200704, 128, 1152)),
                                        ("conv4_x", (50176, 256, 2304)), ("conv5_x", (12544, 512, 4608))])
def test_resnet18_im2col_all_pairs(name, shape):
    M, N, K = shape
    xa = synth.draw("half_normal", (M, K), 61)
    xb = synth.draw("weights", (N, K), 62)
    check_pairs(xa, xb, RESNET_PAIRS, sampled_rows(M, 24, 63), name)
