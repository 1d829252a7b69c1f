"""The allocation-free entry point against mts_step, through the C ABI.

mts_step_noalloc stages each chunk's arrivals in the library's static device
scratch instead of the handle's buffer; its results must equal mts_step's bit
for bit.  Two calls in a row on the same GPU, the second with a smaller
input: the scratch keeps the first call's contents, and nothing of it may
leak into the second.  The first workload's arrival records need several
launches per call (its chunk is bounded by the scratch, not by the handle's
buffer).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads import preset, scaled  # noqa: E402

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only hosts, never run there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2608_16336_amd import Scheduler  # noqa: E402
from paper_2608_16336_amd.mts import MtsError  # noqa: E402


def assert_same(a, b, what=""):
    for k in b:
        if not np.array_equal(a[k], b[k]):
            idx = np.nonzero(a[k] != b[k])[0][:8]
            raise AssertionError("%s field %s differs at %s: noalloc %s step %s" % (what, k, idx, a[k][idx], b[k][idx]))


def run_pair(cfg, ticks, calls):
    ref = Scheduler(cfg)
    new = Scheduler(cfg)
    for n in calls:
        ref.step(n)
        new.step_noalloc(n)
    torch.cuda.synchronize()
    assert_same(new.export(), ref.export(), cfg["name"])
    assert np.array_equal(new.digests(), ref.digests())
    assert new.tick == ref.tick == ticks
    s = new.stats()
    assert s["raw"][86] == 0 and s["digest"] == ref.stats()["digest"]
    ref.close()
    new.close()


def test_noalloc_equals_step_twice_second_smaller():
    # first: two wide replicas (about 500 KB of arrival records per tick, so
    # about 128 ticks per launch), 300 ticks in two calls
    run_pair(scaled("wide", replicas_per_group=2), 300, [170, 130])
    # second, smaller: the tiny cluster, 200 ticks
    run_pair(preset("tiny"), 200, [200])


def test_noalloc_rejects_a_tick_beyond_the_scratch():
    # 80 replicas whose largest arrival count is about 110,000: one tick's
    # records need about 70 MB, more than the 64 MiB scratch
    cfg = preset("tiny")
    cfg.update(n_instances=1, slots_per_instance=64, mig_max_pairs=0,
               arrival=dict(kind="gamma_poisson", mean=700.0, cv=3.0),
               groups=[dict(n_replicas=80, K=2, tiers=dict(kind="uniform"))])
    g = Scheduler(cfg)
    with pytest.raises(MtsError) as e:
        g.step_noalloc(1)
    assert e.value.code == -2  # MTS_ENOMEM
    assert g.tick == 0
    g.close()
