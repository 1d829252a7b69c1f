"""Pins of the CPU oracle against what the paper and the mathematics fix.

No GPU.  Each test names the passage or the closed form it checks.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy.stats import norm

import oracle
from exact_sim import exact_headroom
from workloads import preset, scaled

TWO32 = 1 << 32
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ---------------------------------------------------------------------------
# Random numbers: Philox4x64-10 against numpy's independent implementation
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("ctr,key", [
    ([0, 0, 0, 0], [0, 0]),
    ([1, 0, 0, 0], [7, 11]),
    ([12345, 17, 1, 0], [0, 3839]),
    ([2**64 - 1, 2**63, 5, 9], [2**64 - 1, 42]),
])
def test_philox_matches_numpy(ctr, key):
    # numpy's Philox increments its 256-bit counter before each block
    c = [int(v) for v in ctr]
    c0 = (c[0] - 1) % 2**64
    borrow = c[0] == 0
    c1 = (c[1] - borrow) % 2**64
    borrow = borrow and c[1] == 0
    c2 = (c[2] - borrow) % 2**64
    borrow = borrow and c[2] == 0
    c3 = (c[3] - borrow) % 2**64
    g = np.random.Philox(key=np.array(key, np.uint64), counter=np.array([c0, c1, c2, c3], np.uint64))
    assert [int(v) for v in g.random_raw(4)] == [int(v) for v in oracle.philox4x64_10(ctr, key)]


# ---------------------------------------------------------------------------
# Headroom, Eq. 3 and Fig. 3
# ---------------------------------------------------------------------------
def _cfg_one(**over):
    c = preset("tiny")
    c.update(over)
    return c


def _golden(name):
    """key -> list of numbers from a fixture under tests/golden/."""
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if line:
                out[line[0]] = [float(v) for v in line[1:]]
    return out


def test_headroom_matches_fig3_printed_values():
    # Fig. 3 (Section 3.3): the printed per-tier headroom of Eq. 3 as a share
    # of M.  Fig. 3 charges the lowest tier too, so the lowest-tier zeroing is
    # switched off here.
    g = _golden("fig3_headroom.txt")
    K = int(g["K"][0])
    M = 10000
    c = _cfg_one(kv_blocks=M, headroom_base=g["h_max"][0] * M, headroom_decay=math.exp(-g["lambda"][0]),
                 zero_lowest_tier=0)
    c["groups"] = [dict(n_replicas=1, K=K, tiers=dict(kind="uniform"))]
    H = oracle.Oracle(c, 0, 1).headroom(0)[:K]
    pct = [h / 256 / M * 100 for h in H]
    for p in range(K):
        printed, tol = g["H%d_pct" % p]
        assert abs(pct[p] - printed) <= tol, (p, pct[p], printed)
    printed, tol = g["total_pct"]
    assert abs(sum(pct) - printed) <= tol


@pytest.mark.parametrize("name", ["tiny", "enterprise", "gauss10", "sweep", "wide"])
def test_headroom_closed_form_exact_rationals(name):
    # Eq. 3 evaluated in exact rational arithmetic on the binary values of h0
    # and gamma, lowest tier zeroed; the oracle multiplies doubles repeatedly.
    c = scaled(name, replicas_per_group=1)
    o = oracle.Oracle(c, 0, len(c["groups"]))
    for g, grp in enumerate(c["groups"]):
        K = grp["K"]
        want = exact_headroom(c["headroom_base"], c["headroom_decay"], K, 1)
        assert list(o.headroom(g)[:K]) == want
        assert all(v == 0 for v in o.headroom(g)[K:])


def test_single_tier_has_no_headroom():
    # K = 1 is "no differentiation" (Section 5.1): the only tier is the lowest.
    c = _cfg_one()
    c["groups"] = [dict(n_replicas=1, K=1, tiers=dict(kind="uniform"))]
    assert list(oracle.Oracle(c, 0, 1).headroom(0)) == [0] * 10


# ---------------------------------------------------------------------------
# Freeness, Eq. 1 / Eq. 2 / Eq. 4 and the Fig. 2 worked example
# ---------------------------------------------------------------------------
def _fig2_state(extra_running=()):
    """Instance 0 of a 2-instance cluster with M = 2000 blocks of 16 tokens,
    filled as Fig. 2's bar: two tier-0 requests run with half of the physical
    share each, one request waits with the head-of-line share, tier-0
    headroom is the headroom share."""
    g = _golden("fig2_freeness.txt")
    M = 2000
    blocks = lambda key: int(round(g[key][0] / 100 * M))
    phys, hol, head = blocks("phys_pct"), blocks("hol_pct"), blocks("headroom_pct")
    assert phys % 2 == 0
    c = _cfg_one(n_instances=2, kv_blocks=M, headroom_base=float(head), headroom_decay=0.5)
    o = oracle.Oracle(c, 0, 1)
    st = o.export()
    reqs = [(2, 0, phys // 2 * 16, 5, 1), (2, 0, phys // 2 * 16, 5, 2), (1, 0, hol * 16, 5, 3)]
    reqs += list(extra_running)
    held = 0
    for s, (status, tier, length, rem, seq) in enumerate(reqs):
        st["meta"][s] = status | tier << 2 | (1 << 6 if status == 2 else 0)
        st["lr"][s] = length | rem << 16
        st["seq"][s] = seq
        if status == 2:
            held += -(-length // 16)
    st["free"][0] = M - held
    st["next_seq"][0] = 100
    o.import_state(st)
    assert o.check(0) == 0
    return o, c


def test_fig2_worked_example():
    # Fig. 2 (Section 3.2): the bar's free share over B running requests is
    # the freeness, F = free_pct / 100 * M / B.
    g = _golden("fig2_freeness.txt")
    assert sum(g[k][0] for k in ("phys_pct", "hol_pct", "headroom_pct", "free_pct")) == 100
    o, c = _fig2_state()
    num, den = o.freeness(0, 0)
    assert den == 2
    assert Fraction(num, 256 * den) == Fraction(int(g["free_pct"][0]), 100) * c["kv_blocks"] / 2
    # the empty instance: F = M / max(B, 1) (B = 0 read as 1)
    num1, den1 = o.freeness(0, 1)
    assert (num1, den1) == (256 * 2000, 1)


def test_eq4_headroom_charged_once_per_tier():
    # Eq. 4 and the sentence after it: H_p is charged when any request of
    # tier p is present, not per request.  A third tier-0 running request of
    # 10 blocks lowers M - sum V by exactly its 10 physical blocks.
    o, _ = _fig2_state()
    num_a, _ = o.freeness(0, 0)
    o2, _ = _fig2_state(extra_running=[(2, 0, 160, 5, 4)])
    num_b, den_b = o2.freeness(0, 0)
    assert den_b == 3
    assert num_a - num_b == 256 * 10
    # a running request of a new tier (tier 1 is the lowest of K = 2, so it
    # carries no headroom) also costs only its blocks
    o3, _ = _fig2_state(extra_running=[(2, 1, 160, 5, 4)])
    assert num_a - o3.freeness(0, 0)[0] == 256 * 10


def test_eq4_new_tier_adds_its_headroom_once():
    c = _cfg_one(n_instances=2, kv_blocks=2000, headroom_base=400.0, headroom_decay=0.5)
    c["groups"] = [dict(n_replicas=1, K=3, tiers=dict(kind="uniform"))]
    o = oracle.Oracle(c, 0, 1)
    H = o.headroom(0)
    st = o.export()
    for s, (tier, seq) in enumerate([(1, 1), (1, 2)]):
        st["meta"][s] = 2 | tier << 2 | 1 << 6
        st["lr"][s] = 160 | 5 << 16
        st["seq"][s] = seq
    st["free"][0] = 2000 - 20
    o.import_state(st)
    num, den = o.freeness(0, 0)
    # M - 20 physical blocks - one H_1 (two tier-1 requests share it)
    assert num == 256 * (2000 - 20) - H[1]
    assert den == 2


# ---------------------------------------------------------------------------
# Sampling tables: quantised CDFs against closed forms
# ---------------------------------------------------------------------------
def _moments(base, q):
    p = np.diff(np.concatenate([[0], q.astype(np.float64)])) / TWO32
    n = base + np.arange(len(q), dtype=np.float64)
    m = float((p * n).sum())
    return m, float((p * n * n).sum()) - m * m


@pytest.mark.parametrize("name", ["tiny", "enterprise", "gauss10", "sweep", "wide"])
def test_tables_are_monotone_and_complete(name):
    c = scaled(name, replicas_per_group=1)
    o = oracle.Oracle(c, 0, len(c["groups"]))
    tabs = [o.table(w) for w in ("count", "prompt", "output")]
    tabs += [o.table("tier", g) for g in range(len(c["groups"]))]
    for base, q in tabs:
        assert q[-1] == TWO32
        assert np.all(q[:-1] < TWO32)
        assert np.all(np.diff(q.astype(np.int64)) >= 0)
    # the longest request must fit the u16 length field
    (pb, pq), (ob, oq) = tabs[1], tabs[2]
    assert pb + len(pq) - 1 + ob + len(oq) - 1 <= 65535


@pytest.mark.parametrize("name,lam", [("tiny", 2.0), ("enterprise", 6.0), ("sweep", 12.0)])
def test_poisson_count_moments(name, lam):
    base, q = oracle.Oracle(scaled(name, replicas_per_group=1), 0, 1).table("count")
    m, v = _moments(base, q)
    assert abs(m - lam) < 1e-6 and abs(v - lam) < 1e-5


def test_gamma_poisson_count_moments():
    # gamma-mixed Poisson with mean 200, CV 3: mean 200, variance 200 + (3 * 200)^2
    base, q = oracle.Oracle(preset("wide"), 0, 1).table("count")
    m, v = _moments(base, q)
    assert abs(m - 200) < 1e-3
    assert abs(v - (200 + 600.0 ** 2)) / 360200 < 1e-5
    assert abs(q[0] / TWO32 - 1801.0 ** (-1 / 9)) < 1e-9  # P(0) = (1 + scale)^-shape


@pytest.mark.parametrize("name,mean", [("tiny", 128.0), ("enterprise", 256.0), ("gauss10", 200.0)])
def test_geometric_output_moments(name, mean):
    base, q = oracle.Oracle(scaled(name, replicas_per_group=1), 0, 1).table("output")
    assert base == 1
    m, v = _moments(base, q)
    assert abs(m - mean) < 1e-5 * mean
    assert abs(v - mean * (mean - 1)) < 1e-4 * mean * mean


def test_pareto_output_mean():
    # E[min(floor(xmin U^(-1/alpha)), cap)] = xmin + sum_{n=xmin+1}^{cap} (xmin/n)^alpha
    c = preset("wide")
    base, q = oracle.Oracle(c, 0, 1).table("output")
    o = c["output"]
    want = o["min"] + sum((o["min"] / n) ** o["alpha"] for n in range(o["min"] + 1, o["cap"] + 1))
    m, _ = _moments(base, q)
    assert base == o["min"]
    assert abs(m - want) < 1e-6 * want


def test_uniform_prompt_is_exact():
    c = preset("tiny")
    base, q = oracle.Oracle(c, 0, 1).table("prompt")
    lo, hi = c["prompt"]["lo"], c["prompt"]["hi"]
    assert base == lo and len(q) == hi - lo + 1
    n = np.arange(1, hi - lo + 2, dtype=object)
    want = [(int(k) * TWO32) // (hi - lo + 1) for k in n]
    # floor(((n-lo+1)/(hi-lo+1)) * 2^32) in double may sit one below the exact
    # floor when the quotient rounds down
    diff = np.array(want, dtype=np.int64) - q.astype(np.int64)
    assert np.all((diff == 0) | (diff == 1))
    assert q[-1] == TWO32


@pytest.mark.parametrize("name", ["enterprise", "sweep", "wide"])
def test_lognormal_prompt_against_scipy(name):
    c = scaled(name, replicas_per_group=1)
    p = c["prompt"]
    base, q = oracle.Oracle(c, 0, 1).table("prompt")
    n = base + np.arange(len(q) - 1)
    want = norm.cdf((np.log(n + 0.5) - p["mu"]) / p["sigma"])
    assert np.max(np.abs(q[:-1] / TWO32 - want)) < 1e-9


@pytest.mark.parametrize("K", [1, 2, 3, 4, 7, 10])
def test_tier_tables(K):
    c = scaled("sweep", replicas_per_group=1)
    o = oracle.Oracle(c, 0, len(c["groups"]))
    gi = 3 * (K - 1)
    # uniform: P(tier <= k) = (k + 1) / K
    _, q = o.table("tier", gi)
    assert len(q) == K
    for k in range(K - 1):
        assert abs(int(q[k]) - (k + 1) * TWO32 // K) <= 1
    # Gaussian N((K-1)/2, K/4) cut at the half-integers, tails lumped
    _, q = o.table("tier", gi + 1)
    for k in range(K - 1):
        assert abs(q[k] / TWO32 - norm.cdf((k + 0.5 - (K - 1) / 2) / (K / 4))) < 1e-9
    # enterprise: P(k) proportional to 0.5^(K-1-k)
    _, q = o.table("tier", gi + 2)
    w = [Fraction(1, 2) ** (K - 1 - j) for j in range(K)]
    for k in range(K - 1):
        assert abs(int(q[k]) - math.floor(sum(w[:k + 1]) / sum(w) * TWO32)) <= 1


def test_explicit_tier_table():
    c = scaled("enterprise", replicas_per_group=1)
    _, q = oracle.Oracle(c, 0, 1).table("tier", 0)
    cum = np.cumsum([0.05, 0.15, 0.30, 0.50])
    assert np.all(np.abs(q[:3].astype(np.int64) - np.floor(cum[:3] * TWO32).astype(np.int64)) <= 1)


def test_sampled_tier_frequencies_match_the_distribution():
    # whole sampling pipeline (Philox -> uniform -> inverse CDF): per-tier
    # arrival counts of the enterprise mix over 3000 ticks, chi-square test
    c = scaled("enterprise", replicas_per_group=1, ticks=3000)
    c["n_instances"] = 2
    c["slots_per_instance"] = 64
    o = oracle.Oracle(c, 0, 1)
    o.step(3000)
    s = o.export()["stats"].astype(np.int64)
    arrived = np.array([s[p * 8] for p in range(4)])
    n = arrived.sum()
    assert abs(n / 3000 - 6.0) < 4 * math.sqrt(6.0 / 3000)
    exp = n * np.array([0.05, 0.15, 0.30, 0.50])
    chi2 = float(((arrived - exp) ** 2 / exp).sum())
    assert chi2 < 16.27  # 0.999 quantile, 3 degrees of freedom


# ---------------------------------------------------------------------------
# Invariants over whole runs
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name,ticks", [("tiny", 1000), ("enterprise", 300), ("gauss10", 300),
                                        ("sweep", 100), ("wide", 30)])
def test_invariants_hold_every_tick(name, ticks):
    c = scaled(name, replicas_per_group=1)
    R = len(c["groups"])
    o = oracle.Oracle(c, 0, R, check=True)
    o.step(ticks)
    st = o.export()
    stats = st["stats"].reshape(R, oracle.NSTAT).astype(np.int64)
    assert np.all(stats[:, 86] == 0), "block/migration invariants violated"
    assert np.all(stats[:, 87] == ticks)
    I, S = c["n_instances"], c["slots_per_instance"]
    meta = st["meta"].reshape(R, I * S)
    for r in range(R):
        per = stats[r, :80].reshape(10, 8)
        # arrivals are dispatched or rejected
        assert np.array_equal(per[:, 0], per[:, 1] + per[:, 2])
        # dispatched requests have finished or are still live (waiting/running)
        live = np.zeros(10, np.int64)
        for m in meta[r]:
            if (m & 3) in (1, 2):
                live[(m >> 2) & 15] += 1
        assert np.array_equal(per[:, 2], per[:, 4] + live)
        assert np.all(per[:, 3] <= per[:, 2])
        assert st["next_seq"][r] == per[:, 0].sum()


def test_invariant_checker_detects_planted_corruption():
    o = oracle.Oracle(preset("tiny"), 0, 1)
    o.step(200)
    st = o.export()
    assert o.check(0) == 0
    st["free"][1] += 1                     # one block appears from nowhere
    o.import_state(st)
    assert o.check(0) > 0
