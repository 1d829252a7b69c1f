"""The device orders freeness values F = num / den (Eq. 1 in 1/256 block) by
comparing correctly rounded IEEE doubles; the oracle compares the rationals
by 64-bit cross-multiplication.  Within the library's limits (|num| < 2^30,
1 <= den <= 2048 = largest slot count) the two orders must agree exactly,
ties included, or dispatch (argmax, lowest index on ties) and pairing (sort
by F, then index) would differ.  numpy's float64 division is IEEE
round-to-nearest, the same arithmetic as the device's double division.
"""
import numpy as np

NUM_MAX = 2**30 - 1
DEN_MAX = 2048


def _check(na, da, nb, db):
    exact = np.sign(na.astype(np.int64) * db - nb.astype(np.int64) * da)
    fa = na.astype(np.float64) / da.astype(np.float64)
    fb = nb.astype(np.float64) / db.astype(np.float64)
    approx = np.sign(fa - fb).astype(np.int64)
    bad = np.nonzero(exact != approx)[0]
    assert bad.size == 0, (na[bad[:5]], da[bad[:5]], nb[bad[:5]], db[bad[:5]])


def test_random_pairs_in_range():
    rng = np.random.default_rng(7)
    n = 2_000_000
    na = rng.integers(-NUM_MAX, NUM_MAX + 1, n)
    nb = rng.integers(-NUM_MAX, NUM_MAX + 1, n)
    da = rng.integers(1, DEN_MAX + 1, n)
    db = rng.integers(1, DEN_MAX + 1, n)
    _check(na, da, nb, db)


def test_nearest_neighbours_at_the_largest_magnitudes():
    # for each pair of denominators, the numerator of b closest to a's value
    # (and its two neighbours): the hardest cases, with num near the limit
    rng = np.random.default_rng(11)
    n = 1_000_000
    da = rng.integers(1, DEN_MAX + 1, n)
    db = rng.integers(1, DEN_MAX + 1, n)
    mag = rng.integers(2**29, NUM_MAX + 1, n)
    sgn = rng.choice([-1, 1], n)
    na = sgn * (mag // 1)
    na = np.clip(na, -NUM_MAX, NUM_MAX)
    base = (na.astype(np.int64) * db) // da  # floor of a's value in b's denominator
    for off in (-1, 0, 1, 2):
        nb = np.clip(base + off, -NUM_MAX, NUM_MAX)
        _check(na, da, nb, db)


def test_equal_values_compare_equal():
    rng = np.random.default_rng(13)
    n = 500_000
    d1 = rng.integers(1, 46, n)  # d1 * k <= 2048
    k = rng.integers(1, DEN_MAX // 45, n)
    num = rng.integers(-(NUM_MAX // 46), NUM_MAX // 46, n)
    fa = num.astype(np.float64) / d1
    fb = (num * k).astype(np.float64) / (d1 * k)
    assert np.array_equal(fa, fb)


def test_the_bound_is_needed():
    # far outside the limits two different rationals can round to one double
    # (here numerators beyond 2^53), so the limits are what makes the order exact
    a, b = 2**53 + 1, 2**53
    assert a != b and float(a) / 1.0 == float(b) / 1.0
