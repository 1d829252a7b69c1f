"""GPU parity at the workloads' full sizes, in the launch shape bench.py times.

Every replica of the full configuration runs on the device with the automatic
launch (all replicas resident, one wave each).  The oracle then replays a
sample of replicas spread over the groups, one by one, and their canonical
state and digests must match bit for bit; over all replicas the device's own
per-tick checks (block conservation, free >= 0) must report nothing.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from workloads import preset  # noqa: E402

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only hosts, never run there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2608_16336_amd import Scheduler  # noqa: E402


def assert_same(gpu, ref, what=""):
    for k in ref:
        a, b = gpu[k], ref[k]
        if not np.array_equal(a, b):
            idx = np.nonzero(a != b)[0][:8]
            raise AssertionError("%s field %s differs at %s: gpu %s oracle %s" % (what, k, idx, a[idx], b[idx]))


def sample_replicas(cfg, per_group_picks):
    """First and last replica of evenly spaced groups, plus the very last replica."""
    picks, base = [], 0
    groups = cfg["groups"]
    step = max(1, len(groups) // per_group_picks)
    for gi, g in enumerate(groups):
        if gi % step == 0:
            picks += [base, base + g["n_replicas"] - 1]
        base += g["n_replicas"]
    picks.append(base - 1)
    return sorted(set(picks))


@pytest.mark.parametrize("name,ticks,groups_sampled", [
    ("enterprise", 1200, 1),
    ("gauss10", 1200, 1),
    ("sweep", 1000, 5),
    ("wide", 120, 1),
])
def test_full_size_sampled_replicas(name, ticks, groups_sampled):
    cfg = preset(name)
    g = Scheduler(cfg)
    threads, blocks = g.launch()
    # one wave per replica; a workgroup of eight for 128 or more instances
    assert threads == (512 if cfg["n_instances"] >= 128 else 64) and 1 <= blocks <= g.R
    g.step(ticks)
    torch.cuda.synchronize()
    s = g.stats()  # raises on a device invariant violation
    assert s["raw"][86] == 0 and s["raw"][87] == g.R * ticks
    picks = sample_replicas(cfg, groups_sampled)
    if name == "wide":
        picks = [0, g.R - 1]
    for r in picks:
        o = oracle.Oracle(cfg, r, 1)
        o.step(ticks)
        assert_same(g.export(r, 1), o.export(), "%s replica %d" % (name, r))
        assert np.array_equal(g.digests(r, 1), o.digests()), "%s replica %d digest" % (name, r)
        o.close()
    g.close()


def test_full_sweep_is_deterministic_across_launch_shapes():
    # the bench's launch and a quarter of it (each wave then runs four replicas)
    cfg = preset("sweep")
    a = Scheduler(cfg)
    _, blocks = a.launch()
    a.step(300)
    da = a.digests()
    a.close()
    b = Scheduler(cfg)
    b.set_launch(64, max(1, blocks // 4))
    b.step(300)
    db = b.digests()
    b.close()
    assert np.array_equal(da, db)


def test_full_sweep_with_draining_instances():
    # two instances of every replica drain from tick 200 on, one returns at 600
    cfg = preset("sweep")
    g = Scheduler(cfg)
    R, I = g.R, cfg["n_instances"]
    g.step(200)
    flags = np.zeros((R, I), np.uint8)
    flags[:, 3] = 1
    flags[:, 17] = 1
    g.set_draining(flags)
    g.step(400)
    flags[:, 17] = 0
    g.set_draining(flags)
    g.step(200)
    torch.cuda.synchronize()
    s = g.stats()
    assert s["raw"][86] == 0
    for r in sample_replicas(cfg, 3):
        o = oracle.Oracle(cfg, r, 1)
        o.step(200)
        o.set_drain(0, 3, True)
        o.set_drain(0, 17, True)
        o.step(400)
        o.set_drain(0, 17, False)
        o.step(200)
        assert_same(g.export(r, 1), o.export(), "sweep replica %d with draining" % r)
        assert np.array_equal(g.digests(r, 1), o.digests())
        o.close()
    g.close()


@pytest.mark.parametrize("name,ticks,picks", [
    ("enterprise", 5000, [0, 517, 1023]),
    ("gauss10", 10000, [0, 4095]),
    ("sweep", 10000, [5, 1930, 3839]),
])
def test_full_length_runs_sampled(name, ticks, picks):
    # the workloads' whole runs, as the bench times them, in launches of 1000 ticks
    cfg = preset(name)
    g = Scheduler(cfg)
    for _ in range(ticks // 1000):
        g.step(1000)
    torch.cuda.synchronize()
    s = g.stats()
    assert s["raw"][86] == 0 and s["raw"][87] == g.R * ticks
    for r in picks:
        o = oracle.Oracle(cfg, r, 1, check=False)
        o.step(ticks)
        assert_same(g.export(r, 1), o.export(), "%s replica %d after %d ticks" % (name, r, ticks))
        assert np.array_equal(g.digests(r, 1), o.digests())
        o.close()
    g.close()
