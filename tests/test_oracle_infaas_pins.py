"""Pins of the oracle's INFaaS-style dispatch policy (no GPU).

The paper's comparison scheduler (Section 3.7) sends each request to the
instance with the smallest cost alpha * q + beta * s + gamma * penalty (queue
depth, a moving-average service-time estimate, a state penalty that is 0 for
ACTIVE and raised for OVERLOADED and INTERFERED) and never migrates.
Pinned here:

* alpha only reduces to join-the-shortest-queue: on a hand-built state whose
  instances cannot admit anything, the queues after one tick are what the
  textbook rule gives when it places that tick's arrivals one by one;
* beta only sends every arrival to the instance with the smallest estimate;
  gamma only avoids the OVERLOADED instance (head of line does not fit);
* no migration ever starts, while Llumnix migrates on the same load;
* whole trajectories (queue depths, estimates, penalties, every counter)
  equal the exact simulator's, with and without draining.
"""
import random

import numpy as np
import pytest

import oracle
from test_oracle_exact import _random_cfg, _random_drain_plan, run_pair
from workloads import preset

INFAAS = dict(policy="infaas", alpha=64, beta=1, gamma=1, pen_overloaded=512, pen_interfered=128, ewma_shift=4)


def _blocked_state(cfg, queues, svc=None):
    """Every instance's KV cache is full with one running request (no growth,
    no finish for the next ticks), so nothing is admitted and each instance
    keeps queues[i] waiting requests."""
    I, S, M, blk = cfg["n_instances"], cfg["slots_per_instance"], cfg["kv_blocks"], cfg["block_tokens"]
    o = oracle.Oracle(cfg, 0, 1)
    st = o.export()
    seq = 1
    for i in range(I):
        base = i * S
        # running: M blocks worth of tokens, length 5 past a block boundary
        length = (M - 1) * blk + 5
        st["meta"][base] = 2 | (1 << 6)
        st["lr"][base] = length | 500 << 16
        st["seq"][base] = seq
        seq += 1
        for q in range(queues[i]):
            st["meta"][base + 1 + q] = 1
            st["lr"][base + 1 + q] = 40 | 20 << 16
            st["seq"][base + 1 + q] = seq
            seq += 1
        st["free"][i] = 0
    st["next_seq"][0] = seq
    if svc is not None:
        st["svc"] = np.asarray(svc, np.int64)
    o.import_state(st)
    o.tick = 7
    return o


def _cfg(**dispatch):
    c = preset("tiny")
    c.update(kv_blocks=256, block_tokens=16)
    c["arrival"] = dict(kind="poisson", mean=5.0)
    c["dispatch"] = dict(INFAAS, **dispatch)
    return c


def _waiting(o):
    a = o.export()
    S = o.S
    return [int(np.sum((a["meta"][i * S:(i + 1) * S] & 3) == 1)) for i in range(o.I)]


@pytest.mark.parametrize("seed", range(6))
def test_alpha_only_is_join_the_shortest_queue(seed):
    c = _cfg(alpha=1, beta=0, gamma=0)
    c["seed"] = seed
    queues = [3, 0, 2, 1]
    o = _blocked_state(c, queues)
    o.step(1)
    n = len(o.last_arrivals(0))
    want = list(queues)
    for _ in range(n):
        j = min(range(len(want)), key=lambda i: (want[i], i))
        want[j] += 1
    assert _waiting(o) == want
    assert n > 0 or seed > 0


def test_beta_only_follows_the_smallest_estimate():
    c = _cfg(alpha=0, beta=1, gamma=0)
    o = _blocked_state(c, [0, 0, 0, 0], svc=[500 * 256, 90 * 256, 300 * 256, 90 * 256 + 1])
    o.step(3)
    q = _waiting(o)
    assert q[1] > 0 and q[0] == q[2] == q[3] == 0


def test_gamma_only_avoids_the_overloaded_instance():
    c = _cfg(alpha=0, beta=0, gamma=1)
    o = _blocked_state(c, [1, 0, 0, 0])
    # instances 1..3 have no head of line: ACTIVE; instance 0's head of line
    # needs blocks it does not have: OVERLOADED
    o.step(1)
    n = len(o.last_arrivals(0))
    q = _waiting(o)
    assert q[0] == 1
    if n:
        # the first arrival goes to instance 1 (lowest index among the ACTIVE);
        # it then becomes OVERLOADED only at the next tick's snapshot
        assert q[1] == n


def test_infaas_never_migrates():
    c = preset("tiny")
    c["arrival"] = dict(kind="poisson", mean=3.0)
    o = oracle.Oracle(c, 0, 1)
    o.step(600)
    assert o.export()["stats"][80:84].sum() > 0  # Llumnix does migrate here
    c["dispatch"] = dict(INFAAS)
    o = oracle.Oracle(c, 0, 1)
    o.step(600)
    s = o.export()["stats"]
    assert s[80:84].sum() == 0 and s[86] == 0
    assert np.any(o.export()["svc"] > 0)


def test_infaas_trajectory_matches_the_exact_simulator():
    c = preset("tiny")
    c["dispatch"] = dict(INFAAS)
    s = run_pair(c, 600)
    assert s[86] == 0 and s[5::8].sum() > 0  # preemptions: INTERFERED states happened


@pytest.mark.parametrize("case", range(10))
def test_random_infaas_clusters(case):
    rng = random.Random(7000 + case)
    c = _random_cfg(rng)
    c["dispatch"] = dict(policy="infaas", alpha=rng.choice([0, 1, 64, 300]), beta=rng.choice([0, 1, 3]),
                         gamma=rng.choice([0, 1, 5]), pen_overloaded=rng.choice([0, 40, 512]),
                         pen_interfered=rng.choice([0, 20, 128]), ewma_shift=rng.choice([0, 2, 4, 16]))
    plan = _random_drain_plan(rng, c["n_instances"], 250) if case % 2 else None
    s = run_pair(c, 250, plan)
    assert s[86] == 0 and s[80:84].sum() == 0


# ---------------------------------------------------------------------------
# tier-blind scheduling: the priority-blind local scheduler of the paper's
# INFaaS baseline (Section 5.3)
# ---------------------------------------------------------------------------
def _strip_tiers(a):
    """State with the tier label removed from every slot's meta."""
    b = dict(a)
    b["meta"] = a["meta"] & np.uint8(~(15 << 2) & 0xFF)
    return b


@pytest.mark.parametrize("mix", ["uniform", "gauss", "explicit"])
def test_tier_blind_infaas_is_the_single_tier_system(mix):
    # INFaaS never looks at tiers and a tier-blind local scheduler does not
    # either, so K tiers behave like one: same slots, same request order,
    # same estimates; the per-tier counters add up to the single tier's
    c = preset("tiny")
    c["arrival"] = dict(kind="poisson", mean=3.0)
    c["dispatch"] = dict(INFAAS)
    c["tier_blind"] = 1
    tiers = dict(kind=mix)
    if mix == "gauss":
        tiers.update(mu=1.5, sigma=1.0)
    if mix == "explicit":
        tiers.update(probs=[0.1, 0.2, 0.3, 0.4])
    c["groups"] = [dict(n_replicas=1, K=4, tiers=tiers)]
    one = dict(c)
    one["groups"] = [dict(n_replicas=1, K=1, tiers=dict(kind="uniform"))]
    a, b = oracle.Oracle(c), oracle.Oracle(one)
    a.step(800)
    b.step(800)
    sa, sb = a.export(), b.export()
    for k in ("lr", "seq", "tarr", "free", "mig", "next_seq", "svc"):
        assert np.array_equal(sa[k], sb[k]), k
    assert np.array_equal(_strip_tiers(sa)["meta"], sb["meta"])
    per_a = sa["stats"][:80].reshape(10, 8).astype(np.int64).sum(axis=0)
    per_b = sb["stats"][:80].reshape(10, 8).astype(np.int64)[0]
    assert np.array_equal(per_a, per_b)
    assert np.array_equal(sa["stats"][80:], sb["stats"][80:])
    assert len(set(int(v) for v in (sa["meta"][(sa["meta"] & 3) != 0] >> 2) & 15)) > 1


def test_tier_aware_infaas_is_not_the_single_tier_system():
    # the same run with the priority-ordered local queue differs
    c = preset("tiny")
    c["arrival"] = dict(kind="poisson", mean=3.0)
    c["dispatch"] = dict(INFAAS)
    c["groups"] = [dict(n_replicas=1, K=4, tiers=dict(kind="uniform"))]
    one = dict(c)
    one["groups"] = [dict(n_replicas=1, K=1, tiers=dict(kind="uniform"))]
    a, b = oracle.Oracle(c), oracle.Oracle(one)
    a.step(800)
    b.step(800)
    assert not np.array_equal(a.export()["seq"], b.export()["seq"])


@pytest.mark.parametrize("case", range(8))
def test_random_tier_blind_clusters(case):
    rng = random.Random(9000 + case)
    c = _random_cfg(rng)
    c["tier_blind"] = 1
    if case % 2:
        c["dispatch"] = dict(INFAAS)
    plan = _random_drain_plan(rng, c["n_instances"], 250) if case % 3 == 0 else None
    s = run_pair(c, 250, plan)
    assert s[86] == 0
