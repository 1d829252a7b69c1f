"""GPU parity: the HIP path against the CPU oracle, bit-exact.

Every comparison is element by element over the canonical state (slot meta,
len/rem, seq, arrival tick, free blocks, migration records, sequence counter)
and the per-replica counters, all integers.  Calls go through the C ABI via
the ctypes binding.
"""
import random

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from workloads import preset, scaled  # noqa: E402

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only hosts, never run there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2608_16336_amd import Scheduler  # noqa: E402
from paper_2608_16336_amd.mts import MtsError  # noqa: E402


def assert_same(gpu, ref, what=""):
    for k in ref:
        a, b = gpu[k], ref[k]
        if not np.array_equal(a, b):
            idx = np.nonzero(a != b)[0][:8]
            raise AssertionError("%s field %s differs at %s: gpu %s oracle %s" % (what, k, idx, a[idx], b[idx]))


def run_both(cfg, ticks, r_sample=None):
    g = Scheduler(cfg)
    g.step(ticks)
    torch.cuda.synchronize()
    R = g.R
    picks = range(R) if r_sample is None else r_sample
    for r in picks:
        o = oracle.Oracle(cfg, r, 1)
        o.step(ticks)
        assert_same(g.export(r, 1), o.export(), "replica %d" % r)
        assert np.array_equal(g.digests(r, 1), o.digests())
    return g


@pytest.mark.parametrize("name", ["tiny", "enterprise", "gauss10", "sweep", "wide"])
def test_tables_match_oracle(name):
    c = scaled(name, replicas_per_group=1)
    g = Scheduler(c)
    o = oracle.Oracle(c, 0, len(c["groups"]))
    for w in ("count", "prompt", "output"):
        bg, qg = g.table(w)
        bo, qo = o.table(w)
        assert bg == bo and np.array_equal(qg, qo), w
    for gi in range(len(c["groups"])):
        bg, qg = g.table("tier", gi)
        bo, qo = o.table("tier", gi)
        assert bg == bo and np.array_equal(qg, qo)
        assert np.array_equal(g.headroom(gi), o.headroom(gi))


def test_tiny_full_state_every_tick():
    cfg = preset("tiny")
    g = Scheduler(cfg)
    o = oracle.Oracle(cfg)
    for t in range(cfg["ticks"]):
        g.step(1)
        o.step(1)
        assert_same(g.export(), o.export(), "tick %d" % t)
    s = g.stats()
    assert s["raw"][86] == 0 and s["raw"][87] == cfg["ticks"]


@pytest.mark.parametrize("name,rpg,ticks", [
    ("enterprise", 12, 600),
    ("gauss10", 12, 600),
    ("sweep", 1, 400),
    ("wide", 2, 150),
])
def test_presets_reduced(name, rpg, ticks):
    cfg = scaled(name, replicas_per_group=rpg)
    g = Scheduler(cfg)
    g.step(ticks)
    o = oracle.Oracle(cfg)
    o.step(ticks)
    assert_same(g.export(), o.export(), name)
    assert np.array_equal(g.digests(), o.digests())
    assert g.stats()["raw"][86] == 0


def _random_cfg(case):
    from test_oracle_exact import _random_cfg as rc
    return rc(random.Random(1000 + case))


@pytest.mark.parametrize("case", range(20))
def test_random_small_clusters(case):
    cfg = _random_cfg(case)
    cfg["groups"][0]["n_replicas"] = 3
    run_both(cfg, 250)


def test_chunking_invariance():
    cfg = scaled("sweep", replicas_per_group=1)
    a = Scheduler(cfg)
    a.step(137)
    a.step(263)
    b = Scheduler(cfg)
    b.step(400)
    assert_same(a.export(), b.export(), "chunked")


@pytest.mark.parametrize("blocks", [1, 7, 29])
def test_launch_shape_does_not_change_results(blocks):
    # fewer waves than replicas: each wave runs several replicas in turn
    cfg = scaled("sweep", replicas_per_group=1)
    ref = Scheduler(cfg)
    ref.step(300)
    g = Scheduler(cfg)
    g.set_launch(64, blocks)
    g.step(300)
    assert_same(g.export(), ref.export(), "%d blocks" % blocks)


def test_replica_alone_equals_replica_in_batch():
    cfg = scaled("gauss10", replicas_per_group=16)
    batch = Scheduler(cfg)
    batch.step(300)
    for r in (0, 7, 15):
        one = scaled("gauss10", replicas_per_group=1)
        one["replica_id_base"] = r
        alone = Scheduler(one)
        alone.step(300)
        assert_same(alone.export(), batch.export(r, 1), "replica %d" % r)


def test_zero_ticks_is_a_noop():
    cfg = preset("tiny")
    g = Scheduler(cfg)
    g.step(0)
    assert g.tick == 0
    assert g.stats()["raw"].sum() == 0


def test_export_import_roundtrip_resumes_exactly():
    cfg = scaled("enterprise", replicas_per_group=4)
    a = Scheduler(cfg)
    a.step(300)
    st = a.export()
    b = Scheduler(cfg)
    b.import_state(st)
    b.tick = 300
    a.step(200)
    b.step(200)
    assert_same(b.export(), a.export(), "resumed vs uninterrupted")
    o = oracle.Oracle(cfg)
    o.import_state(st)
    o.tick = 300
    o.step(200)
    assert_same(a.export(), o.export(), "resumed oracle")


def test_moving_the_clock_keeps_the_canonical_state():
    cfg = scaled("enterprise", replicas_per_group=2)
    g = Scheduler(cfg)
    g.step(150)
    before = g.export()
    g.tick = 777
    assert_same(g.export(), before, "after set_tick")
    g.tick = 150
    g.step(50)
    o = oracle.Oracle(cfg)
    o.step(200)
    assert_same(g.export(), o.export(), "clock moved back and forth")


def test_corrupted_state_is_reported():
    cfg = preset("tiny")
    g = Scheduler(cfg)
    g.step(100)
    st = g.export()
    st["free"][2] += 1  # a block appears from nowhere
    g.import_state(st)
    g.step(1)
    with pytest.raises(MtsError) as e:
        g.stats()
    assert e.value.code == -4


def test_out_of_range_import_is_rejected():
    cfg = preset("tiny")
    g = Scheduler(cfg)
    st = g.export()
    st["mig"][0:4] = [7, 0, 0, 0]  # destination instance 7 of 4
    with pytest.raises(MtsError) as e:
        g.import_state(st)
    assert e.value.code == -1


def test_single_instance_and_no_pairs():
    for over in (dict(n_instances=1, mig_max_pairs=0), dict(mig_max_pairs=0)):
        cfg = preset("tiny")
        cfg.update(over)
        run_both(cfg, 300)


def test_near_zero_arrivals():
    cfg = preset("tiny")
    cfg["arrival"] = dict(kind="poisson", mean=1e-3)
    run_both(cfg, 500)


def test_overloaded_rejections():
    cfg = preset("tiny")
    cfg["slots_per_instance"] = 64
    cfg["arrival"] = dict(kind="poisson", mean=9.0)
    g = run_both(cfg, 400)
    assert g.stats()["raw"][1:80:8].sum() > 0


def test_largest_instance_table():
    # I = 256 instances of S = 2048 slots: the widest replica this build serves
    cfg = scaled("wide", replicas_per_group=1)
    run_both(cfg, 60)


def test_kernel_timing_counts_launches_and_changes_nothing():
    cfg = scaled("sweep", replicas_per_group=1)
    g = Scheduler(cfg)
    g.set_timing(True)
    g.step(700)
    st, ar, n = g.timing()
    assert n >= 1 and st > 0.0 and ar > 0.0
    assert g.timing() == (0.0, 0.0, 0)
    ref = Scheduler(cfg)
    ref.step(700)
    assert_same(g.export(), ref.export(), "timed vs untimed")
    assert g.launch()[1] == min(g.R, g.launch()[1])


# ---------------------------------------------------------------------------
# draining (Sections 3.4, 3.5) and auto-scaling signals (Section 3.6)
# ---------------------------------------------------------------------------
def run_plan_both(cfg, ticks, plan, replicas=None):
    """plan: {tick: [(instance, on), ...]} applied to every replica before that tick."""
    g = Scheduler(cfg)
    R, I = g.R, cfg["n_instances"]
    picks = range(R) if replicas is None else replicas
    orc = {r: oracle.Oracle(cfg, r, 1) for r in picks}
    flags = np.zeros((R, I), np.uint8)
    t = 0
    for stop in sorted([k for k in plan if k < ticks]) + [ticks]:
        if stop > t:
            g.step(stop - t)
            for o in orc.values():
                o.step(stop - t)
            t = stop
        if stop in plan:
            for i, on in plan[stop]:
                flags[:, i] = 1 if on else 0
                for o in orc.values():
                    o.set_drain(0, i, on)
            g.set_draining(flags)
    for r, o in orc.items():
        assert_same(g.export(r, 1), o.export(), "replica %d" % r)
        assert np.array_equal(g.digests(r, 1), o.digests())
    return g


@pytest.mark.parametrize("case", range(12))
def test_random_clusters_with_draining(case):
    from test_oracle_exact import _random_cfg as rc, _random_drain_plan
    rng = random.Random(5000 + case)
    cfg = rc(rng)
    plan = _random_drain_plan(rng, cfg["n_instances"], 250)
    cfg["groups"][0]["n_replicas"] = 3
    run_plan_both(cfg, 250, plan)


def test_every_instance_draining_falls_back_to_the_least_loaded():
    cfg = preset("tiny")
    plan = {0: [(i, True) for i in range(4)], 200: [(1, False)], 300: [(1, True)]}
    g = run_plan_both(cfg, 400, plan)
    s = g.stats()["raw"]
    assert s[90] > 0 and s[86] == 0


def test_drain_empties_an_instance_and_signals_are_counted():
    cfg = scaled("enterprise", replicas_per_group=6)
    plan = {100: [(0, True), (5, True)], 400: [(5, False)]}
    g = run_plan_both(cfg, 600, plan)
    s = g.stats()["raw"]
    assert s[86] == 0 and s[88] + s[89] > 0
    st = g.export()
    S, I = cfg["slots_per_instance"], cfg["n_instances"]
    meta = st["meta"].reshape(g.R, I, S)
    assert not np.any(meta[:, 0, :] & 3), "a draining instance still holds requests"
    assert np.all(st["drain"].reshape(g.R, I)[:, 0] == 1)


def test_draining_flags_are_validated():
    g = Scheduler(preset("tiny"))
    with pytest.raises(MtsError) as e:
        g.set_draining(np.array([0, 2, 0, 0], np.uint8))
    assert e.value.code == -1


# ---------------------------------------------------------------------------
# per-tier latency histograms (Section 5.1) and the differentiation study
# ---------------------------------------------------------------------------
def test_histogram_export_matches_full_export():
    cfg = scaled("enterprise", replicas_per_group=8)
    g = Scheduler(cfg)
    g.step(500)
    full = g.export()
    h = g.histograms(2, 5)
    assert np.array_equal(h.ravel(), full["hist"].reshape(g.R, -1)[2:7].ravel())
    st = g.replica_stats()
    assert np.array_equal(st.ravel(), full["stats"])
    # bins add up to the admitted / finished counters per tier
    hh = g.histograms().astype(np.int64)
    s = st.astype(np.int64)
    for p in range(4):
        assert np.array_equal(hh[:, 0, p].sum(axis=1), s[:, p * 8 + 3])
        assert np.array_equal(hh[:, 1, p].sum(axis=1), s[:, p * 8 + 4])
    assert hh[:, 1].sum() > 0


def test_differentiation_study_small_run_matches_oracle():
    from paper_2608_16336_amd import study
    cfg = study.sweep_cfg(30.0, 1, 500)
    g = Scheduler(cfg)
    g.step(500)
    torch.cuda.synchronize()
    for r in (0, 13, 29):  # K = 1 uniform, K = 5 gauss, K = 10 enterprise
        o = oracle.Oracle(cfg, r, 1)
        o.step(500)
        assert_same(g.export(r, 1), o.export(), "study replica %d" % r)
        o.close()
    g.close()
    _, rows = study.run(30.0, 1, 500)
    assert len(rows) == 3 * sum(range(1, 11))
    k1 = [x for x in rows if x["K"] == 1]
    assert len(k1) == 3 and all(x["tier"] == 0 for x in k1)
    assert sum(x["admitted"] for x in rows) > 0


# ---------------------------------------------------------------------------
# INFaaS-style cost dispatch (Section 3.7), the alternative global policy
# ---------------------------------------------------------------------------
INFAAS = dict(policy="infaas", alpha=64, beta=1, gamma=1, pen_overloaded=512, pen_interfered=128, ewma_shift=4)


@pytest.mark.parametrize("case", range(12))
def test_random_infaas_clusters(case):
    from test_oracle_exact import _random_cfg as rc, _random_drain_plan
    rng = random.Random(7000 + case)
    cfg = rc(rng)
    cfg["dispatch"] = dict(policy="infaas", alpha=rng.choice([0, 1, 64, 300]), beta=rng.choice([0, 1, 3]),
                           gamma=rng.choice([0, 1, 5]), pen_overloaded=rng.choice([0, 40, 512]),
                           pen_interfered=rng.choice([0, 20, 128]), ewma_shift=rng.choice([0, 2, 4, 16]))
    cfg["groups"][0]["n_replicas"] = 3
    if case % 2:
        g = run_plan_both(cfg, 250, _random_drain_plan(rng, cfg["n_instances"], 250))
    else:
        g = run_both(cfg, 250)
    s = g.stats()["raw"]
    assert s[80:84].sum() == 0 and s[86] == 0


@pytest.mark.parametrize("name,rpg,ticks", [
    ("tiny", 1, 1000),
    ("enterprise", 8, 600),
    ("gauss10", 8, 600),
    ("sweep", 1, 300),
    ("wide", 1, 100),
])
def test_infaas_presets_reduced(name, rpg, ticks):
    cfg = scaled(name, replicas_per_group=rpg)
    cfg["dispatch"] = dict(INFAAS)
    g = Scheduler(cfg)
    g.step(ticks)
    o = oracle.Oracle(cfg)
    o.step(ticks)
    assert_same(g.export(), o.export(), name)
    assert np.array_equal(g.digests(), o.digests())
    s = g.stats()["raw"]
    assert s[86] == 0 and s[80:84].sum() == 0
    assert np.any(g.export()["svc"] > 0)


def test_infaas_export_import_resumes_exactly():
    cfg = scaled("enterprise", replicas_per_group=4)
    cfg["dispatch"] = dict(INFAAS)
    a = Scheduler(cfg)
    a.step(300)
    st = a.export()
    b = Scheduler(cfg)
    b.import_state(st)
    b.tick = a.tick
    a.step(200)
    b.step(200)
    assert_same(b.export(), a.export(), "resumed")


def test_infaas_estimate_is_validated():
    cfg = preset("tiny")
    cfg["dispatch"] = dict(INFAAS)
    g = Scheduler(cfg)
    st = g.export()
    st["svc"][1] = -5
    with pytest.raises(MtsError) as e:
        g.import_state(st)
    assert e.value.code == -1


# ---------------------------------------------------------------------------
# queue cache (the waiting requests behind each head of line, kept in LDS):
# a performance setting that must never change a result
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("depth", [0, 1, 3, 7, 15])
def test_queue_cache_depth_does_not_change_results(depth):
    cfg = scaled("gauss10", replicas_per_group=6)
    g = Scheduler(cfg)
    g.queue_cache = depth
    assert g.queue_cache == depth
    g.step(700)
    o = oracle.Oracle(cfg)
    o.step(700)
    assert_same(g.export(), o.export(), "gauss10 depth %d" % depth)
    for case in (3, 8, 14):
        c = _random_cfg(case)
        c["groups"][0]["n_replicas"] = 2
        h = Scheduler(c)
        h.queue_cache = depth
        h.step(250)
        o = oracle.Oracle(c)
        o.step(250)
        assert_same(h.export(), o.export(), "random %d depth %d" % (case, depth))


def test_queue_cache_depth_is_validated():
    g = Scheduler(preset("tiny"))
    # the automatic depth: at most 7, 15 for 128 or more instances
    assert 0 <= g.queue_cache <= (15 if g.I >= 128 else 7)
    with pytest.raises(MtsError):
        g.queue_cache = 16


# ---------------------------------------------------------------------------
# tier-blind scheduling (the priority-blind local scheduler of the paper's
# INFaaS baseline, Section 5.3)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("case", range(10))
def test_random_tier_blind_clusters(case):
    from test_oracle_exact import _random_cfg as rc, _random_drain_plan
    rng = random.Random(9000 + case)
    cfg = rc(rng)
    cfg["tier_blind"] = 1
    if case % 2:
        cfg["dispatch"] = dict(INFAAS)
    cfg["groups"][0]["n_replicas"] = 3
    if case % 3 == 0:
        run_plan_both(cfg, 250, _random_drain_plan(rng, cfg["n_instances"], 250))
    else:
        run_both(cfg, 250)


@pytest.mark.parametrize("name,rpg,ticks,policy", [
    ("enterprise", 6, 600, "infaas"),
    ("gauss10", 6, 600, "infaas"),
    ("sweep", 1, 300, "llumnix"),
    ("wide", 1, 80, "infaas"),
])
def test_tier_blind_presets_reduced(name, rpg, ticks, policy):
    cfg = scaled(name, replicas_per_group=rpg)
    cfg["tier_blind"] = 1
    if policy == "infaas":
        cfg["dispatch"] = dict(INFAAS)
    g = Scheduler(cfg)
    g.step(ticks)
    o = oracle.Oracle(cfg)
    o.step(ticks)
    assert_same(g.export(), o.export(), name)
    assert g.stats()["raw"][86] == 0


# ---------------------------------------------------------------------------
# wider random clusters: several 64-slot chunks per instance, every knob
# ---------------------------------------------------------------------------
def _wide_random_cfg(rng):
    I = rng.choice([2, 3, 5, 8, 16, 33])
    S = rng.choice([128, 192, 256, 512, 1024])
    K = rng.randint(1, 10)
    blk = rng.choice([1, 2, 16, 64])
    M = rng.choice([64, 300, 2048, 8192])
    kind = rng.choice(["uniform", "gauss", "geometric", "explicit"])
    tiers = dict(kind=kind)
    if kind == "gauss":
        tiers.update(mu=(K - 1) / 2, sigma=max(K / 4, 0.3))
    elif kind == "geometric":
        tiers.update(r=0.5)
    elif kind == "explicit":
        w = [rng.choice([0.0, 0.2, 1.0]) + (0.05 if j == 0 else 0.0) for j in range(K)]
        tiers.update(probs=[v / sum(w) for v in w])
    c = preset("tiny")
    c.update(
        n_instances=I, slots_per_instance=S, kv_blocks=M, block_tokens=blk,
        headroom_base=rng.choice([0.0, 0.2, 0.7]) * M, headroom_decay=rng.choice([0.4, 0.8]),
        zero_lowest_tier=rng.choice([0, 1]), mig_interval=rng.choice([1, 2, 5]),
        mig_stage_blocks=rng.choice([1, 8, 64]), mig_max_pairs=rng.randint(0, I // 2),
        theta_num=rng.choice([0, 3, 40]), theta_den=10,
        arrival=rng.choice([dict(kind="poisson", mean=rng.choice([1.0, 6.0, 30.0])),
                            dict(kind="gamma_poisson", mean=rng.choice([5.0, 40.0]), cv=2.0)]),
        prompt=rng.choice([dict(kind="uniform_int", lo=1, hi=rng.choice([100, 2000])),
                           dict(kind="lognormal", mu=5.0, sigma=1.0, lo=8, hi=6000)]),
        output=rng.choice([dict(kind="geometric", mean=rng.choice([20.0, 150.0])),
                           dict(kind="pareto", alpha=1.5, min=4, cap=3000)]),
        groups=[dict(n_replicas=2, K=K, tiers=tiers)],
        seed=rng.randrange(2**63), replica_id_base=rng.randrange(1000))
    c["mig_max_pairs"] = min(c["mig_max_pairs"], I // 2)
    if rng.random() < 0.3:
        c["dispatch"] = dict(policy="infaas", alpha=rng.choice([0, 64]), beta=rng.choice([0, 1]), gamma=1,
                             pen_overloaded=256, pen_interfered=64, ewma_shift=rng.choice([0, 4]))
    if rng.random() < 0.25:
        c["tier_blind"] = 1
    return c


@pytest.mark.parametrize("case", range(40))
def test_wide_random_clusters(case):
    from test_oracle_exact import _random_drain_plan
    rng = random.Random(11000 + case)
    cfg = _wide_random_cfg(rng)
    depth = rng.choice([None, 0, 3, 15])
    plan = _random_drain_plan(rng, cfg["n_instances"], 200) if rng.random() < 0.4 else {}
    g = Scheduler(cfg)
    if depth is not None:
        g.queue_cache = depth
    orc = [oracle.Oracle(cfg, r, 1) for r in range(g.R)]
    flags = np.zeros((g.R, cfg["n_instances"]), np.uint8)
    t = 0
    for stop in sorted([k for k in plan if k < 200]) + [200]:
        if stop > t:
            g.step(stop - t)
            for o in orc:
                o.step(stop - t)
            t = stop
        if stop in plan:
            for i, on in plan[stop]:
                flags[:, i] = 1 if on else 0
                for o in orc:
                    o.set_drain(0, i, on)
            g.set_draining(flags)
    for r, o in enumerate(orc):
        assert_same(g.export(r, 1), o.export(), "case %d replica %d" % (case, r))
        assert np.array_equal(g.digests(r, 1), o.digests())
    assert g.stats()["raw"][86] == 0


@pytest.mark.parametrize("probs", [[0.4, 0.0, 0.6], [0.5, 0.5, 0.0], [0.0, 0.3, 0.7, 0.0], [0.2, 0.3, 0.5, 0.0, 0.0]])
def test_zero_probability_tiers(probs):
    # a tier of probability 0 makes a cumulative table entry exactly 2^32;
    # no request may ever carry such a tier
    cfg = preset("tiny")
    cfg["groups"] = [dict(n_replicas=3, K=len(probs), tiers=dict(kind="explicit", probs=probs))]
    g = run_both(cfg, 300)
    s = g.stats()["raw"]
    for p, w in enumerate(probs):
        if w == 0.0:
            assert s[p * 8] == 0


# ---------------------------------------------------------------------------
# clock wrap of the running word's finish field (14 bits), limits, groups
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("t0", [16300, 32700, 65500, (1 << 31) - 150, (1 << 32) - (1 << 16) - 700])
def test_runs_across_finish_field_wraps(t0):
    cfg = preset("tiny")
    cfg["output"] = dict(kind="pareto", alpha=1.2, min=50, cap=16000)
    cfg["groups"][0]["n_replicas"] = 2
    g = Scheduler(cfg)
    g.tick = t0
    o = oracle.Oracle(cfg)
    o.tick = t0
    for n in (120, 250, 230):
        g.step(n)
        o.step(n)
        assert_same(g.export(), o.export(), "t0 %d" % t0)
    assert g.stats()["raw"][86] == 0


def test_extreme_lengths_and_tiny_kv():
    cfg = preset("tiny")
    cfg.update(kv_blocks=3, block_tokens=64)
    cfg["prompt"] = dict(kind="uniform_int", lo=1, hi=49000)
    cfg["output"] = dict(kind="pareto", alpha=0.8, min=1, cap=16383)
    cfg["groups"][0]["n_replicas"] = 2
    run_both(cfg, 400)
    cfg = preset("tiny")
    cfg.update(kv_blocks=1, block_tokens=1)
    cfg["prompt"] = dict(kind="uniform_int", lo=1, hi=1)
    cfg["output"] = dict(kind="geometric", mean=3.0)
    cfg["groups"][0]["n_replicas"] = 2
    run_both(cfg, 300)


def test_several_groups_with_different_tier_counts():
    cfg = preset("tiny")
    cfg.update(n_instances=6, slots_per_instance=128, kv_blocks=512, mig_max_pairs=3)
    cfg["arrival"] = dict(kind="poisson", mean=4.0)
    cfg["groups"] = [dict(n_replicas=2, K=1, tiers=dict(kind="uniform")),
                     dict(n_replicas=1, K=10, tiers=dict(kind="gauss", mu=4.5, sigma=0.05)),
                     dict(n_replicas=2, K=7, tiers=dict(kind="geometric", r=0.2)),
                     dict(n_replicas=1, K=3, tiers=dict(kind="explicit", probs=[0.0, 0.0, 1.0]))]
    g = run_both(cfg, 400)
    assert g.stats()["raw"][86] == 0


# ---------------------------------------------------------------------------
# arrival sampling: counts across the dense path's limits, bursts, tier order
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("arrival,K,blind", [
    (dict(kind="poisson", mean=7.9), 10, 0),        # about 506 arrivals per 64 ticks: segments cut near the LDS stage size
    (dict(kind="poisson", mean=60.0), 10, 0),       # a third of the ticks hold 64 or more arrivals
    (dict(kind="poisson", mean=60.0), 6, 1),
    (dict(kind="gamma_poisson", mean=10.0, cv=3.0), 7, 0),   # mostly empty ticks and rare large bursts
    (dict(kind="gamma_poisson", mean=150.0, cv=0.3), 3, 0),  # every tick above the dense limit
    (dict(kind="poisson", mean=0.3), 4, 0),
])
def test_arrival_bursts_and_tier_order(arrival, K, blind):
    cfg = preset("tiny")
    cfg.update(n_instances=3, slots_per_instance=64, kv_blocks=1024, mig_max_pairs=1, arrival=arrival,
               tier_blind=blind)
    cfg["groups"] = [dict(n_replicas=3, K=K, tiers=dict(kind="gauss", mu=(K - 1) / 2, sigma=K / 3)),
                     dict(n_replicas=2, K=K, tiers=dict(kind="uniform"))]
    g = Scheduler(cfg)
    orc = [oracle.Oracle(cfg, r, 1) for r in range(g.R)]
    for n in (37, 150, 64):   # chunks that do not fill whole waves: waves straddle replicas
        g.step(n)
        for o in orc:
            o.step(n)
    for r, o in enumerate(orc):
        assert_same(g.export(r, 1), o.export(), "replica %d" % r)
        assert np.array_equal(g.digests(r, 1), o.digests())
    s = g.stats()["raw"]
    assert sum(int(s[p * 8]) for p in range(K)) > 0


# ---------------------------------------------------------------------------
# Section 6.5 extensions: adaptive headroom, promotion of waiting requests
# ---------------------------------------------------------------------------
def _with_extensions(rng, c):
    K = max(g["K"] for g in c["groups"])
    hmax = int(c["headroom_base"] * 256) + 1
    c["adaptive"] = dict(epoch=rng.choice([1, 9, 64]), step_up=rng.choice([100, 4000, 60000]),
                         step_down=rng.choice([0, 300, 9000]), max=max(hmax, rng.choice([256 * 64, 256 * c["kv_blocks"]])),
                         margin=rng.choice([0, 100, 256]),
                         slo=[rng.choice([1, 4, 30, 400]) for _ in range(rng.randint(1, 10))])
    if rng.random() < 0.85:
        c["promotion"] = dict(period=rng.choice([1, 4, 37]),
                              age=[0] + [rng.choice([0, 2, 15, 90]) for _ in range(max(K - 1, 0))])
    if rng.random() < 0.2:
        del c["adaptive"]
    return c


def _compare(g, orc, what):
    for r, o in enumerate(orc):
        assert_same(g.export(r, 1), o.export(), "%s replica %d" % (what, r))
        assert np.array_equal(g.digests(r, 1), o.digests())


@pytest.mark.parametrize("case", range(24))
def test_random_clusters_with_adaptive_headroom_and_promotion(case):
    rng = random.Random(13000 + case)
    cfg = _with_extensions(rng, _wide_random_cfg(rng))
    g = Scheduler(cfg)
    depth = rng.choice([None, 0, 1, 7])
    if depth is not None:
        g.queue_cache = depth
    orc = [oracle.Oracle(cfg, r, 1) for r in range(g.R)]
    for n in (1, 70, 129):  # launches start on and off the update ticks
        g.step(n)
        for o in orc:
            o.step(n)
    _compare(g, orc, "case %d" % case)
    assert g.stats()["raw"][86] == 0


@pytest.mark.parametrize("case", range(8))
def test_large_random_clusters_with_adaptive_headroom_and_promotion(case):
    # 65..256 instances: the eight-wave kernels, whose queue cache continues
    # in HBM, under promotion (which drops that cache) and adaptive headroom;
    # queue-cache depths from none to the deepest
    rng = random.Random(15000 + case)
    cfg = _wide_random_cfg(rng)
    cfg["n_instances"] = rng.choice([65, 128, 200, 256])
    cfg["slots_per_instance"] = rng.choice([128, 256, 512])
    cfg["mig_max_pairs"] = rng.randint(0, cfg["n_instances"] // 2)
    cfg["arrival"] = dict(kind="gamma_poisson", mean=rng.choice([20.0, 80.0]), cv=2.0)
    cfg = _with_extensions(rng, cfg)
    g = Scheduler(cfg)
    depth = rng.choice([None, 0, 1, 7, 15])
    if depth is not None:
        g.queue_cache = depth
    orc = [oracle.Oracle(cfg, r, 1) for r in range(g.R)]
    for n in (1, 70, 129):  # launches start on and off the update ticks
        g.step(n)
        for o in orc:
            o.step(n)
    _compare(g, orc, "case %d" % case)
    assert g.stats()["raw"][86] == 0


def test_wide_with_adaptive_headroom_and_promotion():
    cfg = scaled("wide", replicas_per_group=2)
    cfg["adaptive"] = dict(epoch=25, step_up=2048, step_down=512, max=256 * cfg["kv_blocks"] // 4, margin=128,
                           slo=[2, 6, 15, 40, 100])
    cfg["promotion"] = dict(period=5, age=[0] + [40 + 10 * p for p in range(1, 10)])
    g = run_both(cfg, 400)
    assert g.stats()["raw"][86] == 0


@pytest.mark.parametrize("name,rpg,ticks", [("gauss10", 3, 500), ("sweep", 1, 300), ("enterprise", 4, 400)])
def test_extension_presets_reduced(name, rpg, ticks):
    cfg = scaled(name, replicas_per_group=rpg)
    K = max(gr["K"] for gr in cfg["groups"])
    cfg["adaptive"] = dict(epoch=25, step_up=2048, step_down=512, max=256 * cfg["kv_blocks"] // 4, margin=128,
                           slo=[2, 6, 15, 40, 100])
    cfg["promotion"] = dict(period=5, age=[0] + [40 + 10 * p for p in range(1, K)])
    g = run_both(cfg, ticks)
    assert g.stats()["raw"][86] == 0


@pytest.mark.parametrize("policy,blind", [("infaas", 0), ("llumnix", 1), ("infaas", 1)])
def test_promotion_under_other_policies(policy, blind):
    cfg = scaled("gauss10", replicas_per_group=2)
    cfg["tier_blind"] = blind
    if policy == "infaas":
        cfg["dispatch"] = dict(policy="infaas", alpha=64, beta=1, gamma=1, pen_overloaded=512,
                               pen_interfered=128, ewma_shift=4)
    cfg["promotion"] = dict(period=3, age=[0] + [20] * 9)
    cfg["adaptive"] = dict(epoch=10, step_up=1000, step_down=200, max=256 * 2048, margin=200, slo=[5, 50])
    run_both(cfg, 400)


def test_extension_state_export_import_resumes_exactly():
    cfg = scaled("gauss10", replicas_per_group=3)
    cfg["adaptive"] = dict(epoch=7, step_up=3000, step_down=700, max=256 * 4096, margin=180, slo=[3, 20])
    cfg["promotion"] = dict(period=4, age=[0] + [25] * 9)
    g = Scheduler(cfg)
    g.step(213)
    a = g.export()
    assert (a["hq"].reshape(g.R, 10) != g.headroom(0)).any()  # the headroom moved
    h = Scheduler(cfg)
    h.tick = 213
    h.import_state(a)
    g.step(150)
    h.step(150)
    for k, v in g.export().items():
        assert np.array_equal(v, h.export()[k]), k
    # defaults for missing arrays (Eq. 3's table, the imported counters) match the oracle's
    b = {k: v for k, v in a.items() if k not in ("hq", "hq_snap")}
    h2 = Scheduler(cfg)
    h2.tick = 213
    h2.import_state(b)
    o = oracle.Oracle(cfg)
    o.tick = 213
    o.import_state(b)
    h2.step(90)
    o.step(90)
    assert_same(h2.export(), o.export(), "defaults")
    # out-of-range headroom is rejected
    bad = dict(a)
    bad["hq"] = a["hq"].copy()
    bad["hq"][3] = cfg["adaptive"]["max"] + 1
    with pytest.raises(MtsError):
        h2.import_state(bad)
    bad["hq"] = a["hq"].copy()
    bad["hq"][9] = 5  # the lowest of 10 tiers under zero_lowest_tier
    with pytest.raises(MtsError):
        h2.import_state(bad)


@pytest.mark.parametrize("case", range(12))
def test_large_clusters_pairing_ends(case):
    # Clusters of 65..256 instances, overloaded so that many instances are
    # below zero freeness: pairing reads only the two ends of the (F, index)
    # order, which the kernels for 128+ instances take by wave minima and
    # maxima when they are disjoint (Section 3.5); pair caps from 1 to I/2,
    # thresholds 0 and 3/10, some instances draining.
    rng = random.Random(12000 + case)
    I = [65, 96, 128, 129, 200, 256][case % 6]
    c = preset("tiny")
    c.update(n_instances=I, slots_per_instance=rng.choice([64, 128]), kv_blocks=rng.choice([64, 256]),
             block_tokens=16, headroom_base=rng.choice([0.0, 40.0]), headroom_decay=0.6,
             mig_interval=1, mig_stage_blocks=rng.choice([2, 32]),
             mig_max_pairs=rng.choice([1, 2, I // 4, I // 2]), theta_num=rng.choice([0, 3]), theta_den=10,
             arrival=dict(kind="poisson", mean=float(rng.choice([I // 2, 2 * I]))),
             prompt=dict(kind="uniform_int", lo=16, hi=rng.choice([400, 2000])),
             output=dict(kind="geometric", mean=rng.choice([30.0, 120.0])),
             groups=[dict(n_replicas=2, K=rng.randint(1, 10), tiers=dict(kind="uniform"))],
             seed=rng.randrange(2**63), replica_id_base=rng.randrange(1000))
    g = Scheduler(c)
    orc = [oracle.Oracle(c, r, 1) for r in range(g.R)]
    g.step(60)
    for o in orc:
        o.step(60)
    if case % 3 == 0:
        flags = np.zeros((g.R, I), np.uint8)
        drained = rng.sample(range(I), 5)
        flags[:, drained] = 1
        g.set_draining(flags)
        for o in orc:
            for i in drained:
                o.set_drain(0, i, True)
    g.step(90)
    for o in orc:
        o.step(90)
    moved = 0
    for r, o in enumerate(orc):
        e = o.export()
        assert_same(g.export(r, 1), e, "case %d replica %d" % (case, r))
        assert np.array_equal(g.digests(r, 1), o.digests())
        moved += int(e["stats"][80:82].sum())
    assert moved > 0, "no migration started"
    assert g.stats()["raw"][86] == 0


@pytest.mark.parametrize("name,rpg,ticks", [("gauss10", 3, 300), ("enterprise", 3, 300), ("wide", 2, 150)])
def test_waiting_seqs_spanning_more_than_2_27(name, rpg, ticks):
    # The rescans rank on 32-bit keys (tier rank << 27 | seq - lowest seq)
    # only when the candidates' seqs span less than 2^27, and on the 64-bit
    # (tier, seq) keys otherwise.  Moving the seqs of the live requests in odd
    # slots up by 2^28 puts both ranges in every queue (seqs stay distinct;
    # next_seq moves past them); the imported state then runs as the oracle
    # runs it.
    cfg = scaled(name, replicas_per_group=rpg)
    g = Scheduler(cfg)
    g.step(ticks)
    st = g.export()
    R, I, S = g.R, cfg["n_instances"], cfg["slots_per_instance"]
    seq = st["seq"].reshape(R, I, S).astype(np.int64)
    live = (st["meta"].reshape(R, I, S) & 3) != 0
    odd = (np.arange(S) % 2 == 1)[None, None, :]
    assert ((st["meta"].reshape(R, I, S) & 3) == 1).sum() > 0, "no request waits"
    seq = np.where(live & odd, seq + (1 << 28), seq)
    st["seq"] = seq.reshape(-1).astype(np.uint32)
    st["next_seq"] = (seq.reshape(R, -1).max(axis=1) + 1).astype(np.uint32)
    g.import_state(st)
    o = oracle.Oracle(cfg)
    o.import_state(st)
    o.tick = g.tick
    g.step(200)
    o.step(200)
    assert_same(g.export(), o.export(), "%s with seqs spanning 2^28" % name)
    assert np.array_equal(g.digests(), o.digests())
    assert g.stats()["raw"][86] == 0
    g.close()
