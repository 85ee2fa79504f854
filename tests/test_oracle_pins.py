"""Pins of the CPU oracle against the paper and against mathematics, never
against itself: exact rational brute force (fractions), published
known-answer vectors, an independent Philox implementation, the paper's
stochastic-rounding example, closed-form expectations, round-trip and
special-case identities.  CPU only."""
from __future__ import annotations

import math
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2110_15456_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
MODES = ("nearest", "stochastic", "truncate")


# ----------------------------------------------------------------- helpers --
def exp_field(v: float) -> int:
    """Biased FP32 exponent field via frexp (v = f * 2^e, f in [0.5, 1))."""
    v = float(np.float32(v))
    if v == 0.0 or abs(v) < 2.0 ** -126:  # zero or subnormal: field 0
        return 0
    _, e = math.frexp(abs(v))
    return e + 126


def brute_quantize_group(xs, m, mode, noise, emin=0):
    """Definition of section III-A in exact rationals.

    (a) shared exponent = largest exponent field; one LSB is the value of the
    lowest of m magnitude bits whose top bit carries the largest exponent:
    LSB = 2^(E-127-(m-1)).  (b) align: a_k = |x_k| / LSB.  (c)/(d) nearest:
    the nearest multiple of the LSB, ties away from zero (found by comparing
    candidates); stochastic: floor(a + U/256); truncate: floor(a).  Largest
    magnitude 2^m - 1.  Subnormals count as zero."""
    E = max([emin] + [exp_field(v) for v in xs])
    lsb = Fraction(2) ** (E - 127 - (m - 1))
    qmax = 2 ** m - 1
    out = []
    for k, v in enumerate(xs):
        v32 = float(np.float32(v))
        a = Fraction(0) if exp_field(v32) == 0 else abs(Fraction(v32)) / lsb
        if mode == "nearest":
            lo = math.floor(a)
            # candidates lo and lo + 1; the nearer wins, the larger on a tie
            q = lo if (a - lo) < (lo + 1 - a) else lo + 1
        elif mode == "stochastic":
            q = math.floor(a + Fraction(int(noise[k]), 256))
        else:
            q = math.floor(a)
        q = min(q, qmax)
        out.append(-q if (math.copysign(1.0, v32) < 0 and q) else q)
    return out, E


def brute_value(q, E, m):
    return Fraction(int(q)) * Fraction(2) ** (int(E) - 127 - (m - 1))


# ----------------------------------------------------------------- philox --
def _kat():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                w = [int(t, 16) for t in line.split()]
                rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


def test_philox_known_answers():
    for ctr, key, want in _kat():
        assert [int(v) for v in oracle.philox4x32_10(ctr, key)] == want


def test_philox_matches_rocrand_engine(tmp_path):
    """The installed rocRAND Philox4x32-10 engine, compiled for the host, is an
    independent implementation: random counters and keys must agree."""
    hipcc = shutil.which("hipcc") or ("/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else None)
    if hipcc is None or not os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"):
        pytest.skip("hipcc / rocRAND headers not available")
    exe = str(tmp_path / "rocrand_ref")
    subprocess.check_call([hipcc, "-O1", "-x", "c++", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                           os.path.join(GOLDEN, "rocrand_philox_ref.cpp"), "-o", exe],
                          stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
    rng = np.random.default_rng(7)
    cases = rng.integers(0, 2 ** 32, size=(200, 6), dtype=np.uint64)
    text = "\n".join(" ".join("%x" % v for v in row) for row in cases) + "\n"
    out = subprocess.run([exe], input=text, capture_output=True, text=True, check=True).stdout.split("\n")
    for row, line in zip(cases, out):
        want = [int(t, 16) for t in line.split()]
        got = [int(v) for v in oracle.philox4x32_10(row[:4].astype(np.uint32), row[4:].astype(np.uint32))]
        assert got == want


def test_noise_byte_mapping():
    """Byte t of the group is byte (t mod 4) of word (t div 4) mod 4 of the block
    with counter (gid lo, gid hi, t div 16, 0) and key (seed lo, seed hi)."""
    seed, gid = 0x123456789ABCDEF0, (5 << 32) | 77
    for t in range(32):
        ctr = [gid & 0xFFFFFFFF, gid >> 32, t // 16, 0]
        w = oracle.philox4x32_10(ctr, [seed & 0xFFFFFFFF, seed >> 32])
        assert oracle.noise_byte(seed, gid, t) == (int(w[(t // 4) % 4]) >> (8 * (t % 4))) & 0xFF


# --------------------------------------------------------------- quantize --
@pytest.mark.parametrize("m", range(1, 9))
@pytest.mark.parametrize("mode", MODES)
def test_quantize_group_matches_rational_definition(m, mode):
    rng = np.random.default_rng(100 + m)
    for trial in range(60):
        g = int(rng.choice([1, 2, 4, 16, 32]))
        xs = synth.special_values(g, seed=1000 * m + trial) if trial % 3 == 0 else \
            (rng.standard_normal(g) * np.exp2(rng.integers(-8, 8, g))).astype(np.float32)
        noise = rng.integers(0, 256, g)
        q, E, bad = oracle.quantize_group(xs, m, mode, noise)
        want, E_want = brute_quantize_group(list(xs), m, mode, noise)
        assert not bad
        assert E == E_want
        assert [int(v) for v in q] == want


@pytest.mark.parametrize("m", [2, 4, 6, 8])
@pytest.mark.parametrize("mode", MODES)
def test_quantize_floor_matches_rational_definition(m, mode):
    """The packed layout's conversion (section V-D: a few exponent bits above
    a tensor base): a group whose largest exponent lies below the floor is
    converted at the floor -- the same rational definition with E replaced by
    max(E, floor), its values aligned to the coarser LSB."""
    rng = np.random.default_rng(300 + m)
    for trial in range(40):
        xs = (rng.standard_normal(16) * np.exp2(rng.integers(-12, 4, 16))).astype(np.float32)
        emin = int(rng.integers(110, 135))
        noise = rng.integers(0, 256, 16)
        q, E, _ = oracle.quantize_group_floor(xs, m, mode, noise, emin)
        want, E_want = brute_quantize_group(list(xs), m, mode, noise, emin)
        assert E == E_want == max(emin, max(exp_field(v) for v in xs))
        assert [int(v) for v in q] == want


def test_exponent_base_and_packed_groups():
    """The tensor base is the largest exponent field minus 7 (a 3-bit group
    exponent, section V-D), at least 0; every group's exponent then lies in
    base .. base + 7, and a group entirely below the base (1/1024 here, eight
    binades under 4.0) keeps only what its values are worth at the base's LSB:
    1/1024 at m = 2 with E = 122 rounds to 0 (half an LSB is 1/128)."""
    x = np.zeros((3, 16), np.float32)
    x[0, 0] = 4.0           # exponent field 129: base 122
    x[1, :] = 2.0 ** -10    # field 117 < 122
    x[2, 3] = 2.0 ** -6     # field 121 < 122: LSB at m = 2 is 2^(122-127-1) = 2^-6 -> q = 1
    assert oracle.exponent_base(x) == 122
    q, E, base, bad = oracle.quantize_packed(x, m=2)
    assert base == 122 and bad == 0
    assert E.tolist() == [[129], [122], [122]]
    assert not q[1].any() and q[2, 3] == 1 and q[0, 0] == 2
    assert oracle.exponent_base(np.full((1, 16), 1e-30, np.float32)) == 0 + max(0, 27 - 7)
    assert oracle.exponent_base(np.zeros((2, 16), np.float32)) == 0
    # with every group within 7 binades of the largest, the packed conversion is the plain one
    y = (np.random.default_rng(2).standard_normal((8, 64)) * 2.0 ** -3).astype(np.float32)
    y[:, ::16] = 1.0
    qp, Ep, _, _ = oracle.quantize_packed(y, m=4, mode="stochastic", seed=5)
    qn, En, _ = oracle.quantize(y, m=4, mode="stochastic", seed=5)
    assert np.array_equal(qp, qn) and np.array_equal(Ep, En)


def test_quantize_exponent_is_group_max_and_range():
    """Shared exponent = max exponent field; magnitudes within [0, 2^m-1]; the
    element holding the max exponent keeps its leading bit (q >= 2^(m-1))
    unless it rounds to saturation."""
    x = synth.draw("grads", (64, 256), 3)
    for m in range(1, 9):
        q, E, _ = oracle.quantize(x, g=16, m=m)
        ef = ((x.view(np.uint32) >> 23) & 255).reshape(64, 16, 16)
        assert np.array_equal(E, ef.max(axis=2))
        mag = np.abs(q.astype(np.int64)).reshape(64, 16, 16)
        assert mag.max() <= 2 ** m - 1
        lead = np.take_along_axis(mag, ef.argmax(axis=2)[..., None], axis=2)[..., 0]
        assert np.all(lead >= 2 ** (m - 1))


def test_nearest_g1_is_rounding_to_m_significant_bits():
    """g = 1: each value is its own group, so nearest rounding must give the
    nearest number with m significant bits (ties away from zero, saturating at
    the top of the binade).  Checked by properties, on ~260k bit patterns
    covering every exponent."""
    rng = np.random.default_rng(11)
    bits = rng.integers(0, 2 ** 32, 2 ** 18, dtype=np.uint64).astype(np.uint32)
    ex = (bits >> 23) & 255
    bits = bits[ex != 255]
    x = bits.view(np.float32).reshape(1, -1)
    for m in (1, 2, 3, 4, 8):
        q, E, _ = oracle.quantize(x, g=1, m=m)
        q = q[0].astype(np.float64)
        e = E[0].astype(np.int64)
        normal = e > 0
        lsb = np.exp2((e - 127 - (m - 1)).astype(np.float64))
        xv = np.abs(x[0].astype(np.float64))
        deq = np.abs(q) * lsb
        sat = np.abs(q) == 2 ** m - 1
        err = np.abs(deq - xv)
        assert np.all(err[normal & ~sat] <= lsb[normal & ~sat] / 2)
        # a saturated value lies within one LSB below the top of its binade
        assert np.all(xv[normal & sat] >= (2 ** m - 1.5) * lsb[normal & sat])
        # ties: exactly half-way values go up in magnitude
        tie = normal & (np.abs(xv / lsb - np.floor(xv / lsb) - 0.5) == 0)
        assert np.all(np.abs(q[tie]) == np.minimum(np.floor(xv[tie] / lsb[tie]) + 1, 2 ** m - 1))
        assert np.all(q[~normal] == 0)
        assert np.all((np.sign(q) == np.sign(x[0])) | (q == 0))


def test_stochastic_expectation_closed_form():
    """Averaging over all 256 noise bytes, E[q] = floor(256 a) / 256 exactly
    (a = magnitude in LSBs), unless saturated: SR is unbiased with respect to a
    truncated 8 bits below the LSB (Theorem 1 with q = 2^8)."""
    rng = np.random.default_rng(5)
    for trial in range(40):
        g, m = 16, int(rng.integers(1, 9))
        xs = (rng.standard_normal(g) * np.exp2(rng.integers(-6, 6, g))).astype(np.float32)
        total = np.zeros(g, dtype=np.int64)
        for u in range(256):
            q, E, _ = oracle.quantize_group(xs, m, "stochastic", np.full(g, u))
            total += np.abs(q.astype(np.int64))
        lsb = Fraction(2) ** (E - 127 - (m - 1))
        for k in range(g):
            a = Fraction(float(xs[k])).__abs__() / lsb if exp_field(xs[k]) else Fraction(0)
            want = Fraction(math.floor(256 * a), 256)
            if want < 2 ** m - 1:
                assert Fraction(int(total[k]), 256) == want


def test_paper_two_thirds_example():
    """Section III-D: x = 2/3 of an LSB rounds up with probability
    floor(2^bits x) / 2^bits for the paper's 3-bit illustration and the 8-bit
    converter (golden fixture)."""
    with open(os.path.join(GOLDEN, "sr_two_thirds.txt")) as f:
        rows = [tuple(int(t) for t in l.split()) for l in f if l.strip() and not l.startswith("#")]
    # group [2.0, 2/3]: E = 128 and m = 2 give an LSB of exactly 1
    xs = np.array([2.0, 2.0 / 3.0], dtype=np.float32)
    ups = sum(int(oracle.quantize_group(xs, 2, "stochastic", [0, u])[0][1]) for u in range(256))
    bits8 = [r for r in rows if r[0] == 8][0]
    assert Fraction(ups, 256) == Fraction(bits8[1], bits8[2])
    # 3-bit noise = the top 3 bits of an 8-bit byte (U = 32 u3): same rule
    ups3 = sum(int(oracle.quantize_group(xs, 2, "stochastic", [0, 32 * u])[0][1]) for u in range(8))
    bits3 = [r for r in rows if r[0] == 3][0]
    assert Fraction(ups3, 8) == Fraction(bits3[1], bits3[2])
    # and it approaches 2/3 (full-precision noise) from below
    assert Fraction(2, 3) - Fraction(ups, 256) < Fraction(1, 256)


@pytest.mark.parametrize("mode", MODES)
def test_lossless_inputs_round_trip(mode):
    """Values already on their group's m-bit grid quantize exactly, in every
    rounding mode, and dequantize back to themselves."""
    rng = np.random.default_rng(9)
    for m in range(1, 9):
        G, g = 64, 16
        e = rng.integers(100, 140, G)
        mags = rng.integers(0, 2 ** m, (G, g))
        mags[:, 0] = rng.integers(2 ** (m - 1), 2 ** m, G)  # pin the exponent
        sgn = rng.choice([-1, 1], (G, g))
        x = (sgn * mags * np.exp2((e - 127 - (m - 1))[:, None].astype(np.float64))).astype(np.float32)
        x = x.reshape(4, 256)
        q, E, _ = oracle.quantize(x, g=g, m=m, mode=mode, seed=3)
        y = oracle.dequantize(q, E, g, m)
        assert np.array_equal(y, x.astype(np.float64))


def test_transpose_equivalence_bit_exact():
    """quantize along axis 0 == quantize of the transpose along axis 1,
    including stochastic noise (addressed by output group)."""
    x = synth.draw("grads", (96, 40), 4)
    for mode in MODES:
        a = oracle.quantize(x, axis=0, g=16, m=3, mode=mode, seed=99)
        b = oracle.quantize(np.ascontiguousarray(x.T), axis=-1, g=16, m=3, mode=mode, seed=99)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_row_ranges_and_threads_do_not_change_results():
    x = synth.draw("half_normal", (50, 64), 8)
    q, E, _ = oracle.quantize(x, g=16, m=4, mode="stochastic", seed=1, threads=4)
    q2, E2, _ = oracle.quantize(x, g=16, m=4, mode="stochastic", seed=1, rows=(13, 41))
    assert np.array_equal(q[13:41], q2) and np.array_equal(E[13:41], E2)


def test_nonfinite_inputs_are_reported():
    x = np.ones((2, 32), np.float32)
    x[1, 5] = np.inf
    assert oracle.quantize(x, g=16, m=4)[2] == 1
    x[0, 0] = np.nan
    assert oracle.quantize(x, g=16, m=4)[2] == 2


# ------------------------------------------------------------------- gemm --
def brute_gemm(qa, ea, a_m, qb, eb, b_m, g, m_a, m_b):
    """C[i][j] = sum_k value(a[i][k]) * value(b[j][k]) in exact rationals,
    element by element (no grouping), with magnitudes truncated to m_a / m_b
    bits by dropping low-order bits."""
    def lower(v, s):
        return int(math.copysign(abs(int(v)) >> s, v)) if v else 0
    M, K = qa.shape
    N = qb.shape[0]
    C = [[Fraction(0)] * N for _ in range(M)]
    for i in range(M):
        for j in range(N):
            s = Fraction(0)
            for k in range(K):
                va = brute_value(lower(qa[i, k], a_m - m_a), ea[i, k // g], m_a)
                vb = brute_value(lower(qb[j, k], b_m - m_b), eb[j, k // g], m_b)
                s += va * vb
            C[i][j] = s
    return C


@pytest.mark.parametrize("K", [16, 32])
def test_gemm_matches_rational_brute_force(K):
    """The tiny cases: M = N = 4, K = 16 and 32, every stored precision pair,
    each taken at every lower precision too (magnitudes truncated)."""
    x = synth.draw("normal", (4 + 4, K), 20 + K)
    for a_m in range(1, 9):
        for b_m in range(1, 9):
            qa, ea, _ = oracle.quantize(x[:4], g=16, m=a_m)
            qb, eb, _ = oracle.quantize(x[4:], g=16, m=b_m)
            for m_a in range(1, a_m + 1):
                for m_b in range(1, b_m + 1):
                    C, S = oracle.gemm(qa, ea, a_m, qb, eb, b_m, g=16, m_a=m_a, m_b=m_b)
                    want = brute_gemm(qa, ea, a_m, qb, eb, b_m, 16, m_a, m_b)
                    for i in range(4):
                        for j in range(4):
                            # a sum of K/16 <= 2 exact terms in double: exact
                            assert Fraction(C[i, j]) == want[i][j]


def test_gemm_lossless_inputs_equal_float_matmul():
    """Inputs on their groups' grids: the BFP GEMM equals the float64 matmul of
    the inputs exactly (all products and sums are exact in double here)."""
    rng = np.random.default_rng(12)
    M, N, K, g, m = 8, 6, 64, 16, 4
    def grid(rows):
        e = rng.integers(120, 134, (rows, K // g))
        mags = rng.integers(0, 16, (rows, K))
        mags[:, ::g] = rng.integers(8, 16, (rows, K // g))
        sc = np.exp2(np.repeat(e - 127 - (m - 1), g, axis=1).astype(np.float64))
        return (rng.choice([-1, 1], (rows, K)) * mags * sc).astype(np.float32)
    a, b = grid(M), grid(N)
    qa, ea, _ = oracle.quantize(a, g=g, m=m)
    qb, eb, _ = oracle.quantize(b, g=g, m=m)
    C, _ = oracle.gemm(qa, ea, m, qb, eb, m, g=g)
    assert np.array_equal(C, a.astype(np.float64) @ b.astype(np.float64).T)


def test_group_partials_equal_integer_matmul_and_recombine():
    """P[G] is the int64 matmul of the group's magnitude slices (a library
    routine), and sum_G P[G] 2^(ea+eb-254-(m_a-1)-(m_b-1)) reproduces C."""
    x = synth.draw("weights", (12 + 9, 80), 31)
    qa, ea, _ = oracle.quantize(x[:12], g=16, m=6)
    qb, eb, _ = oracle.quantize(x[12:], g=16, m=3)
    P = oracle.group_partials(qa, 6, qb, 3, g=16)
    for G in range(5):
        sl = slice(16 * G, 16 * G + 16)
        assert np.array_equal(P[G], qa[:, sl].astype(np.int64) @ qb[:, sl].astype(np.int64).T)
    C, S = oracle.gemm(qa, ea, 6, qb, eb, 3, g=16)
    sc = np.exp2((ea.T[:, :, None].astype(np.int64) + eb.T[:, None, :] - 254 - 5 - 2).astype(np.float64))
    assert np.allclose(C, (P * sc).sum(axis=0), rtol=1e-15, atol=0)
    assert np.allclose(S, np.abs(P * sc).sum(axis=0), rtol=1e-15, atol=0)


def test_precision_lowering_is_chunk_discard():
    """gemm at m_a = stored m - 4 equals the gemm of magnitudes truncated by 4
    bits, quantized at m - 4 (the low chunk discarded, section V-D)."""
    x = synth.draw("half_normal", (10 + 7, 48), 44)
    qa, ea, _ = oracle.quantize(x[:10], g=16, m=8)
    qb, eb, _ = oracle.quantize(x[10:], g=16, m=4)
    C, _ = oracle.gemm(qa, ea, 8, qb, eb, 4, g=16, m_a=4, m_b=4)
    qa4 = (np.sign(qa) * (np.abs(qa.astype(np.int32)) >> 4)).astype(np.int16)
    C2, _ = oracle.gemm(qa4, ea, 4, qb, eb, 4, g=16)
    assert np.array_equal(C, C2)


def test_relative_improvement_eq2():
    """r(X) of Eq. 2 against its rational definition."""
    x = synth.draw("grads", (3, 64), 17)
    q4, e4, _ = oracle.quantize(x, g=16, m=4)
    q2, e2, _ = oracle.quantize(x, g=16, m=2)
    r = oracle.relative_improvement(q4, e4, q2, e2, g=16)
    num = sum(abs(brute_value(q4[i, k], e4[i, k // 16], 4) - brute_value(q2[i, k], e2[i, k // 16], 2))
              for i in range(3) for k in range(64))
    den = sum(abs(brute_value(q2[i, k], e2[i, k // 16], 2)) for i in range(3) for k in range(64))
    assert abs(r - float(num / den)) <= 1e-12


# ---------------------------------------------------------------------------
# Adaptive precision (Algorithm 1, Eqs. 1-2, section V-D chunk discard)
# ---------------------------------------------------------------------------

def test_low_chunk_drop_equals_direct_truncation():
    """Discarding the low 2-bit chunk of a truncated 4-bit mantissa is the
    truncated 2-bit mantissa of the same value (same shared exponent)."""
    for seed, dist in ((3, "normal"), (4, "grads"), (5, "half_normal")):
        x = synth.draw(dist, (8, 256), seed)
        q4, e4, _ = oracle.quantize(x, g=16, m=4, mode="truncate")
        q2, e2, _ = oracle.quantize(x, g=16, m=2, mode="truncate")
        assert np.array_equal(e4, e2)
        assert np.array_equal(oracle.drop_low_chunk(q4), q2)


def test_improvement_hand_example():
    """One group holding 1.75 and zeros: BFP(1.75, 4) = 14/8 = 1.75, the chunk
    drop keeps 14 >> 2 = 3 at LSB 1/2, i.e. 1.5; r = 0.25 / 1.5 = 1/6."""
    x = np.zeros((1, 16), np.float32)
    x[0, 0] = 1.75
    q4, e4, _ = oracle.quantize(x, g=16, m=4)
    assert q4[0, 0] == 14 and e4[0, 0] == 127
    num, den = oracle.improvement_sums(q4, e4, g=16)
    assert num == 0.25 and den == 1.5
    # sign is carried: -1.75 gives the same sums
    q4n, e4n, _ = oracle.quantize(-x, g=16, m=4)
    assert oracle.improvement_sums(q4n, e4n, g=16) == (0.25, 1.5)


def test_improvement_zero_on_two_bit_grid():
    """Values already on their group's 2-bit grid have no low chunk: r = 0."""
    rng = np.random.default_rng(9)
    k = rng.integers(-3, 4, size=(4, 64)).astype(np.float64)
    k[:, ::16] = 3.0  # each group's maximum sits in the top chunk
    scale = 2.0 ** rng.integers(-20, 20, size=(4, 4)).repeat(16, axis=1)
    x = (k * scale).astype(np.float32)
    q4, e4, _ = oracle.quantize(x, g=16, m=4)
    num, den = oracle.improvement_sums(q4, e4, g=16)
    assert num == 0.0 and den > 0.0


def test_threshold_eq1_and_selection():
    """Eq. 1 endpoints with the paper's alpha = 0.6, beta = 0.3, and the strict
    inequality of Algorithm 1."""
    a, b = 0.6, 0.3
    assert oracle.threshold(a, b, 0, 100, 0, 10) == a
    assert abs(oracle.threshold(a, b, 100, 100, 10, 10) - (a - 2 * b)) < 1e-15
    eps = [oracle.threshold(a, b, i, 100, 3, 10) for i in range(0, 101, 10)]
    assert all(e1 > e2 for e1, e2 in zip(eps, eps[1:]))
    assert oracle.select_mantissa(1.0, 4.0, 0.25) == 4   # r == eps: not below
    assert oracle.select_mantissa(1.0, 4.0, 0.2500001) == 2
    assert oracle.select_mantissa(0.0, 0.0, 0.0) == 4    # r = 0, eps = 0: not below
    assert oracle.select_mantissa(0.0, 0.0, 0.1) == 2


def test_weight_update_rounding_pins():
    """W' = fl32(w + fl32(alpha * dw)): exact cases, a tie, and a case that a
    fused multiply-add would get wrong."""
    f = np.float32
    # exact: small integers, and alpha = -1/2 on dw = w halves w
    assert oracle.weight_update(f([3.0]), f([-5.0]), 1.0)[0] == f(-2.0)
    assert oracle.weight_update(f([6.0]), f([6.0]), -0.5)[0] == f(3.0)
    # 1 + 2^-24 is a tie between 1 and 1 + 2^-23: nearest-even gives 1
    assert oracle.weight_update(f([1.0]), f([2.0 ** -24]), 1.0)[0] == f(1.0)
    # 1 + 1.5 * 2^-24 rounds up to 1 + 2^-23
    assert oracle.weight_update(f([1.0]), f([1.5 * 2.0 ** -24]), 1.0)[0] == f(1.0 + 2.0 ** -23)
    # (1 + 2^-23)^2 = 1 + 2^-22 + 2^-46 rounds to 1 + 2^-22 before the sum, so
    # adding -(1 + 2^-22) gives exactly 0 (a fused multiply-add gives 2^-46)
    a = 1.0 + 2.0 ** -23
    assert oracle.weight_update(f([-(1.0 + 2.0 ** -22)]), f([a]), a)[0] == f(0.0)
    # subnormals are read as, and flushed to, zero of the same sign (and
    # -0 + -0 = -0, -0 + +0 = +0): a negative subnormal gradient, a negative
    # subnormal product, a subnormal weight
    tiny = float(np.finfo(np.float32).tiny)
    r = oracle.weight_update(f([-0.0, -0.0, 0.25 * tiny, -0.0]), f([-0.5 * tiny, -1e-30, 1.0, 0.5 * tiny]), 1e-9)
    assert r[0] == 0.0 and np.signbit(r[0])
    assert r[1] == 0.0 and np.signbit(r[1])
    assert r[2] == np.float32(1e-9)
    assert r[3] == 0.0 and not np.signbit(r[3])


def test_quantize_dual_is_the_two_conversions():
    """Each output of the dual conversion is the single-axis conversion of the
    same matrix (transposed for the column grouping)."""
    rng = np.random.default_rng(7)
    x = rng.standard_normal((48, 32)).astype(np.float32)
    (qr, er), (qc, ec), bad = oracle.quantize_dual(x, m=3, mode="stochastic", seed_rows=5, seed_cols=9)
    assert bad == 0
    q1, e1, _ = oracle.quantize(x, m=3, mode="stochastic", seed=5)
    q2, e2, _ = oracle.quantize(np.ascontiguousarray(x.T), m=3, mode="stochastic", seed=9)
    assert np.array_equal(qr, q1) and np.array_equal(er, e1)
    assert np.array_equal(qc, q2) and np.array_equal(ec, e2)
