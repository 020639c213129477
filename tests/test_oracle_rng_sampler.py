"""Pins for the oracle's random draws and fixed-point sampler (CPU only)."""
import os

import numpy as np
import pytest

from oracle import philox
from oracle.sampling import fixed_point_weights, sample_fixed_point

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat_rows():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        v = [int(x, 16) for x in line.split()]
        rows.append((tuple(v[0:4]), tuple(v[4:6]), tuple(v[6:10])))
    return rows


@pytest.mark.parametrize("ctr,key,out", _kat_rows())
def test_philox_known_answers(ctr, key, out):
    assert philox.philox4x32_10(ctr, key) == out


def test_philox_counter_fields_distinct():
    # Different purposes / indices / steps / sequences give different words.
    words = {philox.draw_u32(2, b, s, p, i) for b in range(3) for s in range(3) for p in range(3) for i in range(4)}
    assert len(words) == 3 * 3 * 3 * 4


def test_uniform_range_and_exactness():
    assert philox.uniform_from_u32(0) == 0.0
    top = philox.uniform_from_u32(0xFFFFFFFF)
    assert top < 1.0 and top == np.float32(1.0 - 2.0 ** -24)
    # 24-bit grid: exact in float32
    x = 0x12345678
    assert float(philox.uniform_from_u32(x)) == (x >> 8) / 2.0 ** 24


def _count_words(r, token):
    """#{x in [0, 2^32): sample_fixed_point(r, x) == token} by bisection on the monotone map."""
    def first_x_reaching(tok):  # smallest x whose sample is >= tok
        lo, hi = 0, 2 ** 32
        while lo < hi:
            mid = (lo + hi) // 2
            if sample_fixed_point(r, mid) >= tok:
                hi = mid
            else:
                lo = mid + 1
        return lo
    return first_x_reaching(token + 1) - first_x_reaching(token)


def test_sampler_exact_probabilities_by_interval_counting():
    # For weights R_j the draw picks j with probability within 2^-32 of R_j / S.
    rng = np.random.default_rng(11)
    for trial in range(5):
        V = int(rng.integers(2, 9))
        r = rng.random(V).astype(np.float32)
        r[rng.random(V) < 0.3] = 0
        if r.sum() == 0:
            r[0] = 0.5
        R = fixed_point_weights(r).astype(object)
        S = sum(R)
        total = 0
        for j in range(V):
            c = _count_words(r, j)
            total += c
            assert abs(c / 2 ** 32 - R[j] / S) <= 2.0 ** -32 + 1e-18
            if R[j] == 0:
                assert c == 0
        assert total == 2 ** 32


def test_sampler_fixed_point_definition_small():
    # r = (0.25, 0.75): R = (2^38, 3*2^38), S = 2^40; t = floor(x*S/2^32) = x*2^8.
    r = np.array([0.25, 0.75], np.float32)
    assert sample_fixed_point(r, 0) == 0
    assert sample_fixed_point(r, 2 ** 30 - 1) == 0   # t = 2^38 - 2^8 < R_0
    assert sample_fixed_point(r, 2 ** 30) == 1       # t = 2^38 = R_0: not > t
    assert sample_fixed_point(r, 2 ** 32 - 1) == 1
    assert sample_fixed_point(np.zeros(4, np.float32), 5) is None


def test_sampler_chi_square():
    from scipy import stats
    rng = np.random.default_rng(3)
    V = 16
    r = rng.random(V).astype(np.float32)
    r /= r.sum()
    words = rng.integers(0, 2 ** 32, size=20000, dtype=np.uint64)
    counts = np.bincount([sample_fixed_point(r, int(w)) for w in words], minlength=V)
    expected = fixed_point_weights(r).astype(np.float64)
    expected = expected / expected.sum() * len(words)
    chi2 = ((counts - expected) ** 2 / expected).sum()
    assert chi2 < stats.chi2.ppf(0.999, V - 1)
