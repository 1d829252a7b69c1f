"""Pins of the oracle's draining, F_normal and auto-scaling (no GPU).

* Section 3.4: F_normal is the freeness without any priority headroom; the
  difference to the full freeness is exactly the Eq. 4 headroom term, and at
  K = 1 the two coincide.
* Section 3.6: scale-out when the cluster average of F_normal is below -0.5,
  scale-in when it is above 1.5 (strict), checked on hand-built states whose
  averages sit exactly on and just beyond the thresholds.
* Section 3.5 (draining): a draining instance receives no dispatch while other
  instances have room, and its requests are migrated off continuously -- it
  empties long before its running requests would have finished.
"""
import numpy as np
import pytest

import oracle
from workloads import preset


def _cfg(I=2, S=64, M=2048, K=2):
    c = preset("tiny")
    c.update(n_instances=I, slots_per_instance=S, kv_blocks=M, mig_max_pairs=I // 2)
    c["groups"] = [dict(n_replicas=1, K=K, tiers=dict(kind="uniform"))]
    return c


def _state(c, per_instance):
    """per_instance[i]: list of (status, tier, blocks, rem); len = 16 * blocks."""
    o = oracle.Oracle(c, 0, 1)
    st = o.export()
    S, M = c["slots_per_instance"], c["kv_blocks"]
    seq = 1
    for i, reqs in enumerate(per_instance):
        held = 0
        for s, (status, tier, nblk, rem) in enumerate(reqs):
            o_ = i * S + s
            st["meta"][o_] = status | tier << 2 | (1 << 6 if status == 2 else 0)
            st["lr"][o_] = (16 * nblk) | rem << 16
            st["seq"][o_] = seq
            seq += 1
            if status == 2:
                held += nblk
        st["free"][i] = M - held
    st["next_seq"][0] = seq
    o.import_state(st)
    assert o.check(0) == 0
    return o


def test_fnormal_differs_from_full_freeness_by_the_headroom_term():
    c = preset("tiny")
    c["groups"] = [dict(n_replicas=1, K=4, tiers=dict(kind="uniform"))]
    c["headroom_base"] = 300.0
    o = oracle.Oracle(c, 0, 1)
    H = o.headroom(0)
    checked = 0
    for _ in range(40):
        o.step(7)
        st = o.export()
        for i in range(c["n_instances"]):
            nf, df = o.freeness(0, i)
            nn, dn = o.freeness_normal(0, i)
            meta = st["meta"].reshape(c["n_instances"], -1)[i]
            tiers = {int(m >> 2) & 15 for m in meta if m & 3 == 2}
            assert dn == df
            assert nn - nf == sum(int(H[p]) for p in tiers)
            checked += 1
    assert checked == 160


def test_fnormal_equals_full_freeness_for_one_tier():
    c = preset("tiny")
    c["groups"] = [dict(n_replicas=1, K=1, tiers=dict(kind="uniform"))]
    o = oracle.Oracle(c, 0, 1)
    for _ in range(30):
        o.step(9)
        for i in range(c["n_instances"]):
            assert o.freeness(0, i) == o.freeness_normal(0, i)


# F_normal = (free - HoL demand) / max(B, 1) blocks per running request
RUN, WAIT = 2, 1


def test_scale_out_threshold_is_strict_at_minus_one_half():
    c = _cfg()
    # instance 0: two running requests of 512 blocks, a waiting one needing
    # 1026 > 1024 free blocks: F = (1024 - 1026) / 2 = -1
    inst0 = [(RUN, 0, 512, 50), (RUN, 0, 512, 50), (WAIT, 0, 1026, 5)]
    # instance 1: one request holding all 2048 blocks: F = 0; average -1/2
    o = _state(c, [inst0, [(RUN, 1, 2048, 50)]])
    assert o.autoscale()[0] == 0
    # instance 1 with 32 running requests of 64 blocks and a waiting request
    # of one block: F = -1/32, average below -1/2
    inst1 = [(RUN, 1, 64, 50)] * 32 + [(WAIT, 1, 1, 5)]
    o = _state(c, [inst0, inst1])
    assert o.autoscale()[0] == -1


def test_scale_in_threshold_is_strict_at_three_halves():
    c = _cfg()
    # F = (2048 - 1022 - 1023) / 2 = 3/2 on both instances: average exactly 3/2
    three_halves = [(RUN, 0, 1022, 50), (RUN, 1, 1023, 50)]
    o = _state(c, [three_halves, three_halves])
    assert o.autoscale()[0] == 0
    # F = 4 / 2 = 2 on instance 1: average 7/4
    o = _state(c, [three_halves, [(RUN, 0, 1022, 50), (RUN, 1, 1022, 50)]])
    assert o.autoscale()[0] == 1


def test_empty_instances_signal_scale_in():
    # an idle cluster: F_normal = M per instance
    o = _state(_cfg(), [[], []])
    assert o.autoscale()[0] == 1


def test_drain_flag_is_part_of_the_state():
    c = preset("tiny")
    o = oracle.Oracle(c, 0, 1)
    o.step(50)
    o.set_drain(0, 2, True)
    st = o.export()
    assert list(st["drain"]) == [0, 0, 1, 0]
    p = oracle.Oracle(c, 0, 1)
    p.import_state(st)
    p.tick = 50
    o.step(100)
    p.step(100)
    for k, v in o.export().items():
        assert np.array_equal(v, p.export()[k]), k
    assert np.array_equal(o.digests(), p.digests())


def test_draining_instance_gets_no_dispatch_and_is_emptied_by_migration():
    c = preset("tiny")
    c["arrival"] = dict(kind="poisson", mean=0.8)  # room on the other instances
    o = oracle.Oracle(c, 0, 1, check=True)
    o.step(150)
    S = c["slots_per_instance"]
    st = o.export()
    lr0 = st["lr"][:S]
    meta0 = st["meta"][:S]
    rem_max = max(int(v >> 16) for v, m in zip(lr0, meta0) if m & 3 == 2)
    busy_before = int(np.count_nonzero(meta0 & 3))
    assert busy_before > 3 and rem_max > 60
    moved_before = st["stats"][80] + st["stats"][82]
    o.set_drain(0, 0, True)
    emptied = None
    for t in range(300):
        seq0 = int(o.export()["next_seq"][0])
        o.step(1)
        st = o.export()
        seq = st["seq"][:S]
        meta = st["meta"][:S]
        # nothing sampled this tick landed on instance 0
        assert not np.any((meta & 3 != 0) & (seq >= seq0)), "tick %d dispatched to a draining instance" % t
        if emptied is None and not np.any(meta & 3):
            emptied = t
    assert emptied is not None and emptied < rem_max, (emptied, rem_max)
    assert st["stats"][80] + st["stats"][82] > moved_before  # by migration
    assert st["stats"][86] == 0
