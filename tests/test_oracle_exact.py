"""The oracle against the exact-rational per-request simulator (no GPU).

K = 1 must reduce to pure load balancing (no headroom at all, Section 5.1) and
K = 2 to Llumnix's binary headroom h / numHighPriorityRequests (Section 3.3);
the exact simulator implements both literally (per-request headroom shares,
exhaustive argmax over exact fractions).  Random small clusters, overloaded
on purpose, drive every branch: preemption, rejection, queued moves and staged
copies that commit or abort; random draining schedules drive the sentinel,
the all-draining fallback and the auto-scaling counters.
"""
import random

import numpy as np
import pytest

import oracle
from exact_sim import ExactSim
from workloads import preset


def run_pair(cfg, ticks, drain_plan=None):
    """drain_plan: {tick: [(instance, on), ...]} applied before that tick."""
    K = cfg["groups"][0]["K"]
    o = oracle.Oracle(cfg, 0, 1, check=True)
    sim = ExactSim(cfg, K)
    for t in range(ticks):
        for i, on in (drain_plan or {}).get(t, []):
            o.set_drain(0, i, on)
            sim.drain[i] = 1 if on else 0
        o.step(1)
        arrivals = [tuple(int(v) for v in a) for a in o.last_arrivals(0)]
        # dispatch order log invariant: (tier, seq) order is what both use;
        # here check the sampled batch itself is well formed
        assert all(0 <= a[0] < K for a in arrivals)
        sim.tick(arrivals)
        got, want = o.export(), sim.export()
        for k in want:
            if not np.array_equal(got[k], want[k]):
                idx = np.nonzero(got[k] != want[k])[0][:8]
                raise AssertionError("tick %d field %s differs at %s: oracle %s exact %s"
                                     % (t, k, idx, got[k][idx], want[k][idx]))
    # latency histograms: the exact simulator's per-request latencies, binned
    # with the oracle's bin function (itself pinned in test_oracle_pins.py)
    want_h = np.zeros((2, oracle.MAX_TIERS, oracle.HBINS), np.uint32)
    for m in (0, 1):
        for tier, v in sim.latencies[m]:
            want_h[m, tier, oracle.hist_bin(v)] += 1
    got_h = oracle.hist_view(got["hist"], 1)[0]
    assert np.array_equal(got_h, want_h), "latency histograms differ"
    return got["stats"].astype(np.int64)


def test_k2_is_llumnix_binary_headroom():
    s = run_pair(preset("tiny"), 1000)
    assert s[86] == 0
    assert s[80:84].sum() > 0 and s[5::8].sum() > 0  # migrations and preemptions happened


def test_k1_is_pure_load_balancing():
    c = preset("tiny")
    c["groups"] = [dict(n_replicas=1, K=1, tiers=dict(kind="uniform"))]
    s = run_pair(c, 400)
    assert s[86] == 0


def _random_cfg(rng):
    I = rng.choice([1, 2, 3, 4, 6, 8])
    K = rng.randint(1, 5)
    blk = rng.choice([1, 4, 16])
    M = rng.choice([128, 256, 512, 1024])
    kind = rng.choice(["uniform", "gauss", "geometric", "explicit"])
    tiers = dict(kind=kind)
    if kind == "gauss":
        tiers.update(mu=(K - 1) / 2, sigma=max(K / 4, 0.3))
    elif kind == "geometric":
        tiers.update(r=0.5)
    elif kind == "explicit":
        w = [rng.random() + 0.05 for _ in range(K)]
        tiers.update(probs=[v / sum(w) for v in w])
    c = dict(preset("tiny"))
    c.update(
        n_instances=I, slots_per_instance=64, kv_blocks=M, block_tokens=blk,
        headroom_base=rng.choice([0.0, 0.1, 0.25, 0.6, 1.2]) * M, headroom_decay=rng.choice([0.3, 0.5, 0.9]),
        zero_lowest_tier=rng.choice([0, 1]), mig_interval=rng.choice([1, 2, 3]),
        mig_stage_blocks=rng.choice([1, 3, 32]), mig_max_pairs=rng.randint(0, I // 2),
        theta_num=rng.choice([0, 3, 20]), theta_den=10,
        arrival=dict(kind="poisson", mean=rng.choice([0.3, 1.0, 2.0, 5.0])),
        prompt=dict(kind="uniform_int", lo=1, hi=rng.choice([8, 64, 300, 800])),
        output=dict(kind="geometric", mean=rng.choice([4.0, 30.0, 90.0, 200.0])),
        groups=[dict(n_replicas=1, K=K, tiers=tiers)],
        seed=rng.randrange(2**63), replica_id_base=rng.randrange(1000))
    return c


@pytest.mark.parametrize("case", range(20))
def test_random_small_clusters(case):
    rng = random.Random(1000 + case)
    c = _random_cfg(rng)
    s = run_pair(c, 250)
    assert s[86] == 0


def test_random_clusters_reach_every_branch():
    seen = np.zeros(oracle.NSTAT, np.int64)
    for case in range(20):
        c = _random_cfg(random.Random(1000 + case))
        o = oracle.Oracle(c, 0, 1)
        o.step(250)
        seen += o.export()["stats"].astype(np.int64)
    per = seen[:80].reshape(10, 8)
    assert per[:, 1].sum() > 0, "no rejection"
    assert per[:, 5].sum() > 0, "no preemption"
    for k in (80, 81, 82, 83):
        assert seen[k] > 0, "migration counter %d never moved" % k


def _random_drain_plan(rng, I, ticks):
    plan = {}
    for _ in range(rng.randint(1, 6)):
        t = rng.randrange(ticks)
        plan.setdefault(t, []).append((rng.randrange(I), rng.random() < 0.7))
    return plan


@pytest.mark.parametrize("case", range(16))
def test_random_clusters_with_draining(case):
    rng = random.Random(5000 + case)
    c = _random_cfg(rng)
    plan = _random_drain_plan(rng, c["n_instances"], 250)
    s = run_pair(c, 250, plan)
    assert s[86] == 0


def test_every_instance_draining_falls_back_to_the_least_loaded():
    c = preset("tiny")
    plan = {0: [(i, True) for i in range(4)], 200: [(1, False)], 300: [(1, True)]}
    s = run_pair(c, 400, plan)
    assert s[90] > 0  # dispatches went to draining instances
    assert s[86] == 0


def test_draining_branches_are_reached():
    seen = np.zeros(oracle.NSTAT, np.int64)
    for case in range(16):
        rng = random.Random(5000 + case)
        c = _random_cfg(rng)
        plan = _random_drain_plan(rng, c["n_instances"], 250)
        o = oracle.Oracle(c, 0, 1)
        for t in range(250):
            for i, on in plan.get(t, []):
                o.set_drain(0, i, on)
            o.step(1)
        seen += o.export()["stats"].astype(np.int64)
    assert seen[88] > 0, "no scale-out signal"
    assert seen[89] > 0, "no scale-in signal"
    assert seen[80] > 0 and seen[81] > 0
