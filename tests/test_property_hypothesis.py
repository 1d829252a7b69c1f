"""Property-based tests (hypothesis) over the space of small configurations.

CPU: the oracle against the exact-rational per-request simulator
(tests/exact_sim.py), tick by tick, over configurations hypothesis draws from
the whole parameter space the oracle accepts: instance and tier counts,
block sizes, capacities, headroom schedules (Eq. 3, both readings of the
lowest tier), migration interval, stage size, pair cap and threshold
(Section 3.5), loads from idle to overloaded, both global policies (Section
3.4 freeness, Section 3.7 cost), tier-blind queues, draining schedules and
the Section 6.5 extensions.  The examples are derandomised, so every run
checks the same cases; a failure is shrunk to a small configuration.

GPU: the HIP path against the oracle, bit-exact, over the same kind of
configurations with wider clusters (up to 256 instances, up to 2048 slots)
and queue-cache depths; several replicas per configuration.
"""
import numpy as np
import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import given, settings, HealthCheck, strategies as st  # noqa: E402

import oracle  # noqa: E402
from workloads import preset  # noqa: E402


def _tiers(draw, K):
    kind = draw(st.sampled_from(["uniform", "gauss", "geometric", "explicit"]))
    t = dict(kind=kind)
    if kind == "gauss":
        t.update(mu=draw(st.floats(-1.0, K + 0.5)), sigma=draw(st.floats(0.2, 3.0)))
    elif kind == "geometric":
        t.update(r=draw(st.sampled_from([0.25, 0.5, 0.8])))
    elif kind == "explicit":
        w = draw(st.lists(st.integers(0, 9), min_size=K, max_size=K).filter(lambda v: sum(v) > 0))
        t.update(probs=[v / sum(w) for v in w])
    return t


@st.composite
def configs(draw, max_instances=8, slot_choices=(64,), extensions=True):
    I = draw(st.integers(1, max_instances))
    K = draw(st.integers(1, 10))
    blk = draw(st.sampled_from([1, 2, 4, 16, 64]))
    M = draw(st.sampled_from([8, 64, 256, 1024, 4096]))
    c = dict(preset("tiny"))
    c.update(
        n_instances=I, slots_per_instance=draw(st.sampled_from(slot_choices)), kv_blocks=M, block_tokens=blk,
        headroom_base=draw(st.sampled_from([0.0, 0.05, 0.3, 1.0, 2.5])) * M,
        headroom_decay=draw(st.sampled_from([0.1, 0.5, 0.7, 0.99])),
        zero_lowest_tier=draw(st.integers(0, 1)), mig_interval=draw(st.integers(1, 4)),
        mig_stage_blocks=draw(st.sampled_from([1, 2, 7, 32, 1000])), mig_max_pairs=draw(st.integers(0, I // 2)),
        theta_num=draw(st.sampled_from([0, 1, 3, 50])), theta_den=draw(st.sampled_from([1, 10])),
        arrival=dict(kind="poisson", mean=draw(st.sampled_from([0.1, 0.8, 2.0, 6.0, 20.0]))),
        prompt=dict(kind="uniform_int", lo=1, hi=draw(st.sampled_from([1, 16, 200, 1500]))),
        output=dict(kind="geometric", mean=draw(st.sampled_from([1.0, 3.0, 40.0, 300.0]))),
        groups=[dict(n_replicas=1, K=K, tiers=_tiers(draw, K))],
        seed=draw(st.integers(0, 2**63 - 1)), replica_id_base=draw(st.integers(0, 10**6)))
    if draw(st.booleans()):
        c["dispatch"] = dict(policy="infaas", alpha=draw(st.sampled_from([0, 1, 64])), beta=draw(st.integers(0, 2)),
                             gamma=draw(st.integers(0, 2)), pen_overloaded=draw(st.sampled_from([0, 256, 4096])),
                             pen_interfered=draw(st.sampled_from([0, 64])), ewma_shift=draw(st.integers(0, 6)))
    if draw(st.integers(0, 3)) == 0:
        c["tier_blind"] = 1
    if extensions and draw(st.integers(0, 2)) == 0:
        c["adaptive"] = dict(epoch=draw(st.sampled_from([1, 5, 30])), step_up=draw(st.sampled_from([64, 2000])),
                             step_down=draw(st.sampled_from([0, 100])), max=max(256 * M, int(c["headroom_base"] * 256) + 1),
                             margin=draw(st.sampled_from([0, 128, 256])),
                             slo=[draw(st.sampled_from([1, 4, 30])) for _ in range(K)])
    if extensions and K > 1 and draw(st.integers(0, 2)) == 0:
        c["promotion"] = dict(period=draw(st.sampled_from([1, 4, 25])),
                              age=[0] + [draw(st.sampled_from([0, 2, 15, 60])) for _ in range(K - 1)])
    return c


@st.composite
def drain_plans(draw, I, ticks):
    n = draw(st.integers(0, 4))
    plan = {}
    for _ in range(n):
        t = draw(st.integers(0, ticks - 1))
        plan.setdefault(t, []).append((draw(st.integers(0, I - 1)), draw(st.booleans())))
    return plan


# ---------------------------------------------------------------------------
# CPU: oracle = exact-rational simulator, tick by tick
# ---------------------------------------------------------------------------
@settings(max_examples=150, deadline=None, derandomize=True, suppress_health_check=list(HealthCheck))
@given(data=st.data())
def test_oracle_equals_exact_simulator(data):
    from test_oracle_exact import run_pair
    c = data.draw(configs())
    plan = data.draw(drain_plans(c["n_instances"], 60))
    s = run_pair(c, 60, plan)
    assert s[86] == 0
    # request conservation (counted per tier): every arrival is dispatched or rejected
    per = s[:80].reshape(10, 8)
    assert (per[:, 0] == per[:, 1] + per[:, 2]).all()


# ---------------------------------------------------------------------------
# GPU: HIP path = oracle, bit-exact
# ---------------------------------------------------------------------------
@pytest.mark.gpu
@settings(max_examples=120, deadline=None, derandomize=True, suppress_health_check=list(HealthCheck))
@given(data=st.data())
def test_gpu_equals_oracle(data):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2608_16336_amd import Scheduler
    c = data.draw(configs(max_instances=256, slot_choices=(64, 128, 256, 2048)))
    c["groups"][0]["n_replicas"] = data.draw(st.integers(1, 3))
    ticks = data.draw(st.integers(1, 150))
    depth = data.draw(st.sampled_from([None, 0, 1, 7]))
    g = Scheduler(c)
    if depth is not None:
        g.queue_cache = depth
    g.step(ticks)
    torch.cuda.synchronize()
    for r in range(g.R):
        o = oracle.Oracle(c, r, 1)
        o.step(ticks)
        a, b = g.export(r, 1), o.export()
        for k in b:
            if not np.array_equal(a[k], b[k]):
                idx = np.nonzero(a[k] != b[k])[0][:8]
                raise AssertionError("replica %d field %s differs at %s: gpu %s oracle %s"
                                     % (r, k, idx, a[k][idx], b[k][idx]))
        assert np.array_equal(g.digests(r, 1), o.digests())
        o.close()
    assert g.stats()["raw"][86] == 0
    g.close()
