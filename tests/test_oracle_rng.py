"""Pins of the oracle's random draws and sampler against independent sources.

* Philox4x64-10 against numpy's own Philox bit generator (a separate
  implementation of the SC'11 generator).
* uniform_int against the defining property of a multiply-shift range map:
  every output value's preimage is one contiguous run of 32-bit inputs whose
  length is floor or ceil of 2^32 / n.
* Gumbel noise against scipy's Gumbel quantile function.
* Gumbel-max selection against softmax by a chi-square goodness-of-fit test.
"""

import math

import numpy as np
import pytest

from oracle import philox, sampling

M64 = (1 << 64) - 1


def numpy_block(counter, key):
    """Philox4x64-10 block at ``counter`` computed by numpy's generator."""
    c = sum(int(w) << (64 * i) for i, w in enumerate(counter))
    c = (c - 1) % (1 << 256)  # numpy advances the counter before producing a block
    words = np.array([(c >> (64 * i)) & M64 for i in range(4)], dtype=np.uint64)
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64))
    st = bg.state
    st["state"]["counter"] = words
    st["buffer_pos"] = 4
    bg.state = st
    return [int(x) for x in bg.random_raw(4)]


def test_philox_matches_numpy_fixed():
    cases = [
        ((0, 0, 0, 0), (0, 0)),
        ((1, 0, 0, 0), (5, 0)),
        ((M64, M64, M64, M64), (M64, M64)),
        ((7, 128, 513, philox.TAG_ACTION), (12345, 0)),
        ((4095, 49, 0, philox.TAG_RESET), (0xDEADBEEFCAFEF00D, 0)),
    ]
    for ctr, key in cases:
        assert philox.philox4x64_10(ctr, key) == numpy_block(ctr, key)


def test_philox_matches_numpy_random():
    rng = np.random.default_rng(3)
    for _ in range(200):
        ctr = [int(x) for x in rng.integers(0, 1 << 63, size=4, dtype=np.int64)]
        ctr = [c * 2 + int(rng.integers(0, 2)) for c in ctr]
        key = [int(x) for x in rng.integers(0, 1 << 63, size=2, dtype=np.int64)]
        assert philox.philox4x64_10(ctr, key) == numpy_block(ctr, key)


def test_u32_draw_order():
    # draws 0..7 are the halves of block sub=0 (high half first), 8.. of sub=1
    d = philox.u32_draws(9, 3, 11, philox.TAG_RESET, 12)
    b0 = numpy_block((3, 11, 0, philox.TAG_RESET), (9, 0))
    b1 = numpy_block((3, 11, 1, philox.TAG_RESET), (9, 0))
    exp = []
    for w in b0 + b1[:2]:
        exp += [w >> 32, w & 0xFFFFFFFF]
    assert d == exp


def _preimage_start(n, v):
    """Smallest u with uniform_int(u, n) >= v, by bisection (uses only monotonicity)."""
    lo, hi = 0, 1 << 32
    while lo < hi:
        mid = (lo + hi) // 2
        if philox.uniform_int(mid, n) >= v:
            hi = mid
        else:
            lo = mid + 1
    return lo


@pytest.mark.parametrize("n", list(range(1, 145)) + [1000, 65535, 1 << 20, (1 << 32) - 1])
def test_uniform_int_partition(n):
    assert philox.uniform_int(0, n) == 0
    assert philox.uniform_int((1 << 32) - 1, n) == n - 1
    starts = [_preimage_start(n, v) for v in range(min(n, 200))]
    lens = np.diff(starts)
    q = (1 << 32) // n
    assert set(lens.tolist()) <= {q, q + 1}
    # monotone and in range on a random sample
    u = np.random.default_rng(n).integers(0, 1 << 32, size=2000, dtype=np.uint64)
    vals = [philox.uniform_int(int(x), n) for x in np.sort(u)]
    assert all(0 <= v < n for v in vals) and vals == sorted(vals)


def test_gumbel_matches_scipy_quantile():
    from scipy.stats import gumbel_r
    rng = np.random.default_rng(0)
    u = np.concatenate([[0, 1, 2, (1 << 23), (1 << 24) - 2, (1 << 24) - 1],
                        rng.integers(0, 1 << 24, size=5000)])
    q = (u.astype(np.float64) + 0.5) / 2.0 ** 24
    ref = gumbel_r.ppf(q)
    got = np.array([sampling.gumbel_from_u24(int(x)) for x in u], dtype=np.float32)
    # scipy evaluates the same quantile in double; one float32 ulp covers rounding-order
    assert np.all(np.abs(got.astype(np.float64) - ref) <= np.spacing(np.abs(got)).astype(np.float64))
    # the median of the standard Gumbel law is -ln(ln 2)
    assert abs(float(sampling.gumbel_from_u24(1 << 23)) - (-math.log(math.log(2.0)))) < 1e-6


def test_gumbel_table_consistent_and_monotone():
    tab = sampling.gumbel_table()
    assert tab.shape == (1 << 24,) and tab.dtype == np.float32
    assert np.all(np.diff(tab) >= 0)
    idx = np.random.default_rng(1).integers(0, 1 << 24, size=3000)
    for i in idx:
        assert tab[i] == sampling.gumbel_from_u24(int(i))
    assert tab[0] < -2.8 and tab[-1] > 17.0


def test_select_rules():
    # ties go to the lowest index
    assert sampling.select([1.0, 2.0, 2.0], [0.0, 0.0, 0.0]) == 1
    # masked actions are never chosen, even with the largest score
    assert sampling.select([0.0, 9.0, 1.0], [0.0, 0.0, 0.0], [True, False, True]) == 2
    # every action masked -> action 0
    assert sampling.select([0.0, 9.0], [0.0, 0.0], [False, False]) == 0
    # NaN scores count as -inf
    assert sampling.select([float("nan"), -5.0], [0.0, 0.0]) == 1
    assert sampling.select([float("nan"), float("nan")], [0.0, 0.0]) == 0
    # the score is a float32 sum: 1 + 2^-30 rounds to 1, so this is a tie -> index 0
    assert sampling.select([1.0, 1.0], [0.0, 2.0 ** -30]) == 0


def test_sampler_matches_softmax_chi2():
    from scipy.stats import chisquare
    logits = np.array([0.5, -1.0, 2.0, 0.0, 0.3, -0.2], dtype=np.float32)
    p = np.exp(logits.astype(np.float64) - logits.max())
    p /= p.sum()
    n = 30000
    counts = np.zeros(6)
    for k in range(n):
        counts[sampling.sample_action(77, k % 1000, k // 1000, 0, list(logits))] += 1
    stat = chisquare(counts, p * n)
    assert stat.pvalue > 1e-4, (counts, p * n)


def test_sampler_masked_chi2():
    from scipy.stats import chisquare
    logits = np.array([0.0, 1.0, 0.0, -1.0, 0.5, 3.0, 0.0, 0.0, 1.0, 0.0], dtype=np.float32)
    mask = [True, True, False, True, True, False, True, True, True, True]
    legal = np.array(mask)
    p = np.where(legal, np.exp(logits.astype(np.float64)), 0.0)
    p /= p.sum()
    n = 20000
    counts = np.zeros(10)
    for k in range(n):
        counts[sampling.sample_action(5, k, 3, 1, list(logits), mask)] += 1
    assert counts[~legal].sum() == 0
    stat = chisquare(counts[legal], p[legal] * n)
    assert stat.pvalue > 1e-4
