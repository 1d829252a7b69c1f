"""Pins of the oracle's per-tier latency histograms (no GPU).

The histograms count every request's queue delay (arrival to first
admission) and end-to-end time (arrival to its last token) per tier, in
ticks -- the per-tier latency distributions the paper's evaluation reads
(Section 5.1, Section 6.2).  Pinned here:

* the bin function partitions the integers into contiguous ranges: one value
  per bin below 16, then eight equal ranges per octave [2^e, 2^(e+1));
* the bin counts add up to the independent admitted / finished counters, and
  the binned values bracket the independent queue-delay / end-to-end sums;
* what is counted, request by request, equals the exact simulator's
  per-request latencies (``test_oracle_exact.py``);
* under overload, strict tier order gives tier 0 the shortest queue delays
  and the lowest tier the longest, while K = 1 has a single tier
  (Section 5.1: tier 0 stays fast, the lowest tier takes the longest tail).
"""
import numpy as np
import pytest

import oracle
from workloads import preset, scaled


def bin_ranges(limit):
    """(lo, hi) of every bin reached by the values 0 .. limit - 1."""
    bins = np.array([oracle.hist_bin(v) for v in range(limit)])
    assert np.all(np.diff(bins) >= 0) and np.all(np.diff(bins) <= 1), "bins not contiguous and monotone"
    lo, hi = {}, {}
    for v, b in enumerate(bins):
        lo.setdefault(int(b), v)
        hi[int(b)] = v
    return lo, hi


def test_bins_partition_the_integers():
    lo, hi = bin_ranges(1 << 16)
    assert sorted(lo) == list(range(len(lo)))
    for b in range(16):
        assert lo[b] == hi[b] == b
    # eight equal ranges per octave above 16
    for e in range(4, 16):
        octave = [b for b in lo if lo[b] >= 1 << e and hi[b] < 1 << (e + 1)]
        assert len(octave) == 8, e
        widths = {hi[b] - lo[b] + 1 for b in octave}
        assert widths == {1 << (e - 3)}, (e, widths)
    # the octaves up to 2^32 continue the pattern: boundaries of sub-ranges
    for e in range(16, 32):
        first = oracle.hist_bin(1 << e)
        assert first == oracle.hist_bin((1 << e) - 1) + 1
        for k in range(8):
            a = (1 << e) + k * (1 << (e - 3))
            assert oracle.hist_bin(a) == first + k == oracle.hist_bin(a + (1 << (e - 3)) - 1)
    assert oracle.hist_bin((1 << 32) - 1) == oracle.HBINS - 1


@pytest.mark.parametrize("name,ticks", [("tiny", 1000), ("enterprise", 600)])
def test_bin_counts_match_the_counters(name, ticks):
    cfg = preset("tiny") if name == "tiny" else scaled(name, replicas_per_group=2)
    o = oracle.Oracle(cfg)
    o.step(ticks)
    a = o.export()
    nr = o.r_count
    h = oracle.hist_view(a["hist"], nr).astype(np.int64)
    s = a["stats"].reshape(nr, oracle.NSTAT).astype(np.int64)
    lo, hi = bin_ranges(1 << 14)
    lo_v = np.array([lo.get(b, 0) for b in range(oracle.HBINS)])
    hi_v = np.array([hi.get(b, 0) for b in range(oracle.HBINS)])
    assert ticks < 1 << 14
    for r in range(nr):
        for p in range(oracle.MAX_TIERS):
            for m, (cnt, total) in enumerate(((3, 6), (4, 7))):
                n = h[r, m, p]
                assert n.sum() == s[r, p * 8 + cnt]
                assert (n * lo_v).sum() <= s[r, p * 8 + total] <= (n * hi_v).sum()
    assert h[:, 0].sum() > 0 and h[:, 1].sum() > 0


def _tier_means(cfg, ticks):
    o = oracle.Oracle(cfg)
    o.step(ticks)
    s = o.export()["stats"].reshape(o.r_count, oracle.NSTAT).astype(np.int64).sum(axis=0)
    K = cfg["groups"][0]["K"]
    return [s[p * 8 + 6] / max(1, s[p * 8 + 3]) for p in range(K)], s


def test_overload_orders_queue_delay_by_tier():
    cfg = preset("tiny")
    cfg["arrival"] = dict(kind="poisson", mean=3.0)  # well above capacity
    cfg["groups"] = [dict(n_replicas=1, K=3, tiers=dict(kind="uniform"))]
    means, s = _tier_means(cfg, 1500)
    assert s[86] == 0
    assert means[0] < means[1] < means[2], means
    assert means[2] > 4 * means[0]
