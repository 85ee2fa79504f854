"""Pins of the oracle's stochastic-rounding noise against what Theorem 1
(section III-D) needs of it: every noise byte uniform on [0, 256), and the
bytes of different values independent -- across the positions of a group,
across groups (the low and high words of the group index), and across seeds
(the low and high words of the seed).  The converter's random streams
(section V-C) are per value; Philox4x32-10 stands in for its LFSRs.

These are statistical pins: a mapping that reuses one Philox word for several
4-value blocks, ignores the block counter, the group index or a word of the
seed, or loses bits of a byte makes one of them fail by many standard
deviations (the planted-mistake test checks that).  The thresholds are far
in the tails (p < 1e-7), and every input is seeded, so the outcome is fixed.
CPU only."""
from __future__ import annotations

import numpy as np
import pytest
from scipy import stats

import oracle

P_MIN = 1e-7  # smallest acceptable p-value of a chi-square statistic


def chi2_uniform(counts: np.ndarray) -> float:
    """p-value of the chi-square goodness-of-fit of ``counts`` to equal cells."""
    counts = np.asarray(counts, dtype=np.float64).ravel()
    exp = counts.sum() / counts.size
    x2 = float(((counts - exp) ** 2 / exp).sum())
    return float(stats.chi2.sf(x2, counts.size - 1))


def joint_counts(u: np.ndarray, v: np.ndarray, bits: int = 4) -> np.ndarray:
    """2-D histogram of the top ``bits`` bits of two byte arrays."""
    s = 8 - bits
    return np.bincount(((u.astype(np.int64) >> s) << bits) | (v.astype(np.int64) >> s),
                       minlength=1 << (2 * bits))


def test_noise_bytes_are_uniform():
    """2^20 bytes (two seeds, groups of 32): the 256 byte values are equally
    frequent, and each of the 8 bits is set half of the time."""
    u = np.concatenate([oracle.noise_bytes(seed, 0, 1 << 14, 32).ravel() for seed in (1234, 7)])
    assert chi2_uniform(np.bincount(u, minlength=256)) > P_MIN
    n = u.size
    for bit in range(8):
        ones = int(((u >> bit) & 1).sum())
        z = (ones - n / 2) / np.sqrt(n / 4)
        assert abs(z) < 5.5, "bit %d set in %d of %d bytes" % (bit, ones, n)


# Position pairs within a group of 32: neighbours in one Philox word, in
# neighbouring words, the same byte of different words, the two 16-value
# blocks of the group (different counters), and the ends.
POSITION_PAIRS = [(0, 1), (0, 4), (1, 5), (3, 4), (0, 8), (2, 14), (0, 16), (5, 21), (15, 16), (0, 31)]


@pytest.mark.parametrize("p,q", POSITION_PAIRS)
def test_noise_positions_of_a_group_are_independent(p, q):
    """The pair (U_p, U_q) of one group is uniform on the 16 x 16 grid of their
    top nibbles, and U_p = U_q happens about once in 256 groups."""
    u = oracle.noise_bytes(99, 1 << 20, 1 << 16, 32)
    assert chi2_uniform(joint_counts(u[:, p], u[:, q])) > P_MIN
    eq = int((u[:, p] == u[:, q]).sum())
    n = u.shape[0]
    assert abs(eq - n / 256) < 6 * np.sqrt(n / 256), "U_%d == U_%d in %d of %d groups" % (p, q, eq, n)


@pytest.mark.parametrize("delta", [1, 2, 1 << 32])
def test_noise_of_different_groups_is_independent(delta):
    """Group gid and group gid + delta (a neighbour; the high word of the
    index) draw independent bytes at every position."""
    n = 1 << 14
    a = oracle.noise_bytes(5, 3, n, 16)
    b = oracle.noise_bytes(5, 3 + delta, n, 16)
    for p in (0, 7, 15):
        assert chi2_uniform(joint_counts(a[:, p], b[:, p])) > P_MIN
    assert abs(int((a == b).sum()) - a.size / 256) < 6 * np.sqrt(a.size / 256)


@pytest.mark.parametrize("delta", [1, 1 << 32])
def test_noise_of_different_seeds_is_independent(delta):
    """Seed s and seed s + delta (the low and the high word of the key) give
    independent bytes for the same value."""
    n = 1 << 14
    a = oracle.noise_bytes(1234, 0, n, 16)
    b = oracle.noise_bytes(1234 + delta, 0, n, 16)
    for p in (0, 9):
        assert chi2_uniform(joint_counts(a[:, p], b[:, p])) > P_MIN
    assert abs(int((a == b).sum()) - a.size / 256) < 6 * np.sqrt(a.size / 256)


def test_noise_depends_only_on_seed_group_and_position():
    """The same (seed, gid, position) gives the same byte however the groups
    are batched (the noise does not depend on a launch shape)."""
    whole = oracle.noise_bytes(77, 1000, 64, 32)
    parts = np.concatenate([oracle.noise_bytes(77, 1000 + s, 16, 32) for s in range(0, 64, 16)])
    assert np.array_equal(whole, parts)
    assert all(int(whole[5, p]) == oracle.noise_byte(77, 1005, p) for p in range(32))
