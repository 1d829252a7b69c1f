"""Pins of the oracle's Section 6.5 extensions (no GPU): adaptive headroom and
multilevel-feedback promotion of waiting requests.

The paper names both as future work and specifies neither, so what pins the
oracle here is (a) the rule as the library states it, worked by hand on
states built for the purpose (literal expected values, derived in the
comments), (b) the special cases that reduce to the static method, (c) the
exact-rational request-list simulator, which implements both rules from a
different formulation (latency log instead of counter snapshots), over random
overloaded clusters, and (d) invariants of every adaptive run.
"""
import random

import numpy as np
import pytest

import oracle
from test_oracle_exact import _random_cfg, run_pair
from workloads import preset

ADAPT = dict(epoch=25, step_up=512, step_down=128, max=256 * 700, margin=128, slo=[4, 12, 40])
PROMO = dict(period=10, age=[0, 30, 60, 90])


def _tiny(K=3, **kw):
    c = preset("tiny")
    c["groups"] = [dict(n_replicas=1, K=K, tiers=dict(kind="uniform"))]
    c.update(kw)
    return c


# ---------------------------------------------------------------------------
# (a) hand-worked states
# ---------------------------------------------------------------------------
def _blank(o):
    a = o.export()
    for k in ("meta", "lr", "seq", "tarr"):
        a[k][:] = 0
    a["free"][:] = o.cfg["kv_blocks"]
    a["mig"][:] = 0
    a["mig"][0::4] = -1
    return a


def test_promotion_by_hand():
    # one instance of M = 4 blocks of 16 tokens; every request below needs 7
    # blocks, so none is ever admitted and the queue only changes by promotion
    c = _tiny(K=4, n_instances=1, kv_blocks=4, mig_max_pairs=0, promotion=dict(PROMO))
    c["arrival"] = dict(kind="poisson", mean=1e-9)
    o = oracle.Oracle(c)
    a = _blank(o)
    # (tier, arrival tick) of six waiting requests, slots 0..5
    reqs = [(3, 5), (3, 20), (2, 40), (1, 71), (1, 70), (0, 0)]
    for s, (tier, ta) in enumerate(reqs):
        a["meta"][s] = 1 | tier << 2
        a["lr"][s] = 100 | 50 << 16
        a["seq"][s] = s
        a["tarr"][s] = ta
    a["next_seq"][0] = len(reqs)
    o.tick = 100
    o.import_state(a)
    o.step(1)  # tick 100, a promotion pass (100 mod 10 = 0); quotas 30, 60, 90
    # ages 95, 80, 60, 29, 30, 100:
    #   tier 3, age 95 >= 90 -> 2;  tier 3, age 80 < 90 stays;  tier 2, age 60 >= 60 -> 1
    #   tier 1, age 29 < 30 stays;  tier 1, age 30 >= 30 -> 0;   tier 0 stays
    tiers = lambda: list((o.export()["meta"][:6] >> 2) & 15)
    assert tiers() == [2, 3, 1, 1, 0, 0]
    o.step(9)  # ticks 101..109: no pass
    assert tiers() == [2, 3, 1, 1, 0, 0]
    o.step(1)  # tick 110: ages 105, 90, 70, 39, 40, 110
    #   tier 2, age 105 >= 60 -> 1;  tier 3, age 90 >= 90 -> 2;  tier 1, age 70 >= 30 -> 0
    #   tier 1, age 39 >= 30 -> 0;   one tier per pass
    assert tiers() == [1, 2, 0, 0, 0, 0]
    o.step(10)  # tick 120: ages 115, 100
    assert tiers() == [0, 1, 0, 0, 0, 0]
    st = o.export()["stats"]
    assert st[0::8][:4].sum() == 0 and o.check() == 0


def test_promotion_quota_zero_never_promotes():
    c = _tiny(K=3, n_instances=1, kv_blocks=4, mig_max_pairs=0, promotion=dict(period=1, age=[0, 0, 5]))
    c["arrival"] = dict(kind="poisson", mean=1e-9)
    o = oracle.Oracle(c)
    a = _blank(o)
    for s, tier in enumerate([2, 1]):
        a["meta"][s] = 1 | tier << 2
        a["lr"][s] = 100 | 50 << 16
        a["seq"][s] = s
    a["next_seq"][0] = 2
    o.tick = 50
    o.import_state(a)
    o.step(3)
    # tier 2 (quota 5, age 50) moves to 1 and stays there (tier 1 has no quota)
    assert list((o.export()["meta"][:2] >> 2) & 15) == [1, 1]


def test_adaptive_headroom_by_hand():
    # K = 4, zero_lowest: tiers 0..2 adapt.  Static Eq. 3 table (h0 = 78.125
    # blocks, gamma = 0.5): 20000, 10000, 5000, 0 in 1/256 block.  Targets 5,
    # 8, 4 ticks, margin 128 (half the target), steps +1000 / -300, bound 40000.
    ad = dict(epoch=50, step_up=1000, step_down=300, max=40000, margin=128, slo=[5, 8, 4, 9])
    c = _tiny(K=4, adaptive=ad)
    c["headroom_base"], c["headroom_decay"] = 256.0 * 40000 / 65536 / 2, 0.5
    c["arrival"] = dict(kind="poisson", mean=1e-9)
    o = oracle.Oracle(c)
    h0 = list(o.headroom(0)[:4])
    assert h0 == [20000, 10000, 5000, 0]
    a = _blank(o)
    # counters since the last update (snapshots zero):
    #   tier 0: 10 admitted, delay 100: mean 10 > 5              -> up:   21000
    #   tier 1: 10 admitted, delay 40: 256*40 <= 128*8*10         -> down:  9700
    #   tier 2:  4 admitted, delay 20: mean 5 > 4                 -> up:    6000
    #   tier 3: lowest tier, zero_lowest                          -> 0
    for p, (adm, qd) in enumerate([(10, 100), (10, 40), (4, 20), (7, 700)]):
        a["stats"][p * 8 + 3] = adm
        a["stats"][p * 8 + 6] = qd
    a["hq"] = np.array(h0 + [0] * 6, np.int32)
    a["hq_snap"] = np.zeros(20, np.uint64)
    o.tick = 200
    o.import_state(a)
    o.step(1)
    e = o.export()
    assert list(e["hq"][:4]) == [21000, 9700, 6000, 0]
    assert list(e["hq_snap"][:4]) == [10, 10, 4, 7] and list(e["hq_snap"][10:14]) == [100, 40, 20, 700]
    # a hold, the cap and the floor: new counters since the snapshot
    #   tier 0: 10 more, delay 45: mean 4.5, not > 5, 256*45 > 128*5*10 -> hold
    #   tier 1: 1 more, delay 0 -> down 300 (and so on every update, down to 0)
    #   tier 2: none -> hold (later: 2 more, delay 100 each update -> up to
    #           the bound 40000 after 34 updates)
    a = o.export()
    a["stats"][0 * 8 + 3] += 10
    a["stats"][0 * 8 + 6] += 45
    a["stats"][1 * 8 + 3] += 1
    o.import_state(a)
    o.tick = 250
    o.step(1)
    e = o.export()
    assert e["hq"][0] == 21000 and e["hq"][1] == 9700 - 300 and e["hq"][2] == 6000
    for k in range(40):
        a = o.export()
        a["stats"][1 * 8 + 3] += 1
        a["stats"][2 * 8 + 3] += 2
        a["stats"][2 * 8 + 6] += 100
        o.import_state(a)
        o.tick = 300 + 50 * k
        o.step(1)
    e = o.export()
    assert e["hq"][1] == 0 and e["hq"][2] == 40000
    # off-boundary ticks never update
    before = o.export()["hq"].copy()
    o.step(49)
    assert np.array_equal(o.export()["hq"], before)


def test_adaptive_import_validation_and_defaults():
    ad = dict(ADAPT)
    o = oracle.Oracle(_tiny(K=3, adaptive=ad))
    o.step(30)
    a = o.export()
    bad = a.copy()
    bad["hq"] = a["hq"].copy()
    bad["hq"][2] = 5  # the lowest tier under zero_lowest
    with pytest.raises(oracle.OracleError):
        o.import_state(bad)
    bad["hq"] = a["hq"].copy()
    bad["hq"][0] = ad["max"] + 1
    with pytest.raises(oracle.OracleError):
        o.import_state(bad)
    # missing arrays: Eq. 3's table and the current counters as the snapshot
    b = {k: v for k, v in a.items() if k not in ("hq", "hq_snap")}
    o.import_state(b)
    e = o.export()
    assert np.array_equal(e["hq"], o.headroom(0))
    assert list(e["hq_snap"][:3]) == [a["stats"][p * 8 + 3] for p in range(3)]
    # static headroom: the arrays are ignored, zero snapshots
    o2 = oracle.Oracle(_tiny(K=3))
    o2.step(10)
    a2 = o2.export()
    a2["hq"] = a2["hq"] + 7
    o2.import_state(a2)
    assert np.array_equal(o2.export()["hq"], o2.headroom(0)) and not o2.export()["hq_snap"].any()


def test_adaptive_configuration_limits():
    for bad in (dict(ADAPT, margin=257), dict(ADAPT, max=(1 << 29) // 10 + 1), dict(ADAPT, epoch=(1 << 16) + 1),
                dict(ADAPT, slo=[0]), dict(ADAPT, slo=[1 << 21]), dict(ADAPT, max=100)):
        with pytest.raises(oracle.OracleError):
            oracle.Oracle(_tiny(K=3, adaptive=bad))


# ---------------------------------------------------------------------------
# (b) reductions to the static method
# ---------------------------------------------------------------------------
def _same_run(c1, c2, ticks):
    a, b = oracle.Oracle(c1), oracle.Oracle(c2)
    a.step(ticks)
    b.step(ticks)
    ea, eb = a.export(), b.export()
    for k in ("meta", "lr", "seq", "tarr", "free", "mig", "stats", "hist", "hq"):
        assert np.array_equal(ea[k], eb[k]), k


@pytest.mark.parametrize("K", [1, 2, 4])
def test_zero_steps_and_zero_quotas_reduce_to_the_static_method(K):
    c = _tiny(K=K)
    c["arrival"] = dict(kind="poisson", mean=3.0)
    _same_run(c, dict(c, adaptive=dict(ADAPT, step_up=0, step_down=0)), 600)
    _same_run(c, dict(c, promotion=dict(period=1, age=[0] * 10)), 600)
    _same_run(c, dict(c, adaptive=dict(ADAPT, epoch=0), promotion=dict(period=0, age=[1] * 10)), 600)


def test_k1_promotion_has_nothing_to_promote():
    c = _tiny(K=1)
    c["arrival"] = dict(kind="poisson", mean=3.0)
    _same_run(c, dict(c, promotion=dict(period=1, age=[0, 1])), 500)


# ---------------------------------------------------------------------------
# (c) the exact simulator over random overloaded clusters
# ---------------------------------------------------------------------------
def _adaptive_cfg(rng):
    c = _random_cfg(rng)
    K = c["groups"][0]["K"]
    if rng.random() < 0.8:
        c["adaptive"] = dict(epoch=rng.choice([1, 7, 40]), step_up=rng.choice([64, 1000, 40000]),
                             step_down=rng.choice([0, 50, 3000]), max=rng.choice([256 * c["kv_blocks"], 300000]),
                             margin=rng.choice([0, 128, 256]),
                             slo=[rng.choice([1, 3, 10, 50]) for _ in range(rng.randint(1, 10))])
        hb = c["headroom_base"] * 256
        c["adaptive"]["max"] = max(c["adaptive"]["max"], int(hb) + 1)
    if rng.random() < 0.8 and K > 1:
        c["promotion"] = dict(period=rng.choice([1, 5, 30]),
                              age=[0] + [rng.choice([0, 3, 20, 80]) for _ in range(K - 1)])
    return c


@pytest.mark.parametrize("case", range(24))
def test_random_clusters_match_the_exact_simulator(case):
    rng = random.Random(7100 + case)
    c = _adaptive_cfg(rng)
    s = run_pair(c, 250)
    assert s[86] == 0


def test_exact_simulator_reaches_every_branch():
    seen = set()
    for case in range(24):
        rng = random.Random(7100 + case)
        c = _adaptive_cfg(rng)
        o = oracle.Oracle(c)
        prev = o.export()["hq"].copy()
        prev_meta = None
        for t in range(250):
            o.step(1)
            e = o.export()
            d = e["hq"].astype(np.int64) - prev
            if (d > 0).any():
                seen.add("up")
            if (d < 0).any():
                seen.add("down")
            if "adaptive" in c and (e["hq"] == c["adaptive"]["max"]).any():
                seen.add("cap")
            if prev_meta is not None:
                same = (e["seq"] == prev_meta[1]) & ((e["meta"] & 3) == 1) & ((prev_meta[0] & 3) == 1)
                if (((e["meta"] >> 2) & 15)[same] < ((prev_meta[0] >> 2) & 15)[same]).any():
                    seen.add("promoted")
            prev = e["hq"].astype(np.int64)
            prev_meta = (e["meta"].copy(), e["seq"].copy())
    assert seen == {"up", "down", "cap", "promoted"}, seen


# ---------------------------------------------------------------------------
# (d) invariants of adaptive runs
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("K,zero_lowest", [(3, 1), (5, 0), (10, 1)])
def test_headroom_moves_by_one_step_at_epoch_boundaries_within_bounds(K, zero_lowest):
    ad = dict(epoch=13, step_up=700, step_down=90, max=256 * 900, margin=160, slo=[2, 6, 20, 60])
    c = _tiny(K=K, zero_lowest_tier=zero_lowest, adaptive=ad)
    c["arrival"] = dict(kind="poisson", mean=2.5)
    o = oracle.Oracle(c)
    prev = o.export()["hq"].astype(np.int64)
    moved = 0
    for t in range(1, 700):
        o.step(1)  # runs tick t - 1
        h = o.export()["hq"].astype(np.int64)
        d = h - prev
        if (t - 1) % ad["epoch"]:
            assert not d.any()
        for p in range(10):
            assert 0 <= h[p] <= ad["max"]
            if p >= K or (zero_lowest and p == K - 1):
                assert h[p] == 0
            elif d[p]:
                moved += 1
                assert d[p] == ad["step_up"] or d[p] == -ad["step_down"] or h[p] in (0, ad["max"])
        prev = h
    assert moved > 0
    assert o.check() == 0


def test_promotion_never_demotes_and_keeps_requests():
    c = _tiny(K=5, promotion=dict(period=3, age=[0, 4, 8, 12, 16]))
    c["arrival"] = dict(kind="poisson", mean=4.0)
    o = oracle.Oracle(c)
    o.step(1)
    prev = o.export()
    for _ in range(300):
        o.step(1)
        e = o.export()
        keep = (prev["meta"] & 3) == 1
        keep &= (e["meta"] & 3) == 1
        keep &= e["seq"] == prev["seq"]
        assert (((e["meta"] >> 2) & 15)[keep] <= ((prev["meta"] >> 2) & 15)[keep]).all()
        prev = e
    st = o.export()["stats"].astype(np.int64)
    # every arrival is dispatched or rejected, and tiers relabel requests without losing any
    assert st[0:40:8].sum() == st[1:40:8].sum() + st[2:40:8].sum()
    assert o.check() == 0
