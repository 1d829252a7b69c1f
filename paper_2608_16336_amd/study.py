"""Per-tier latency differentiation across tier counts K = 1..10.

The paper's evaluation (Section 5.1, Section 6.1) asks how well K tiers
separate their latencies and what the finer granularity costs.  This study
asks the same question of the scheduling step alone, in ticks: it runs the
K = 1..10 x {uniform, Gaussian, enterprise} sweep on the GPU at a chosen
arrival rate and reads, per (tier mix, K, tier), the queue-delay (arrival to
first admission: the scheduler's share of the time to first token) and
end-to-end (arrival to last token) distributions from the library's
per-replica latency histograms, summed over the seeds of each group.

The results are in scheduler ticks on synthetic loads; they are not
comparable with the paper's simulated seconds.

    python -m paper_2608_16336_amd.study --arrival-mean 24 --ticks 4000
"""
import argparse
import json
import os
import sys

import numpy as np

from .mts import HIST_BINS, MAX_TIERS, Scheduler

MIXES = ("uniform", "gauss", "enterprise")


def bin_edges():
    """(lo, hi) value range of every histogram bin, as arrays: bins below 16
    hold one value; above, each octave [2^e, 2^(e+1)) has eight equal bins."""
    lo = np.zeros(HIST_BINS, np.float64)
    hi = np.zeros(HIST_BINS, np.float64)
    for b in range(HIST_BINS):
        if b < 16:
            lo[b] = hi[b] = b
        else:
            e, k = 4 + (b - 16) // 8, (b - 16) % 8
            w = 2.0 ** (e - 3)
            lo[b] = 2.0 ** e + k * w
            hi[b] = lo[b] + w - 1
    return lo, hi


def percentile(counts, q):
    """Upper edge of the bin holding the q-quantile of a histogram (None if empty)."""
    n = int(counts.sum())
    if n == 0:
        return None
    c = np.cumsum(counts)
    b = int(np.searchsorted(c, q * n - 1e-9, side="left"))
    return float(bin_edges()[1][min(b, HIST_BINS - 1)])


INFAAS = dict(policy="infaas", alpha=64, beta=1, gamma=1, pen_overloaded=512, pen_interfered=128, ewma_shift=4)


def sweep_cfg(arrival_mean, replicas_per_group, ticks, policy="llumnix", tier_blind=False, extensions=()):
    from workloads import preset, with_extensions
    cfg = preset("sweep")
    if extensions:
        cfg = with_extensions(cfg, adaptive="adaptive" in extensions, promotion="promotion" in extensions)
    if policy == "infaas":
        cfg["dispatch"] = dict(INFAAS)
    if tier_blind:
        cfg["tier_blind"] = 1
    cfg["arrival"] = dict(kind="poisson", mean=float(arrival_mean))
    for g in cfg["groups"]:
        g["n_replicas"] = replicas_per_group
    cfg["ticks"] = ticks
    cfg["name"] = "differentiation study: sweep groups x %d, Poisson %g/tick, %s dispatch%s%s" % (
        replicas_per_group, arrival_mean, policy, ", tier-blind queues" if tier_blind else "",
        "".join(", " + label for key, label in (("adaptive", "adaptive headroom"), ("promotion", "promotion"))
                if key in extensions))
    return cfg


def run(arrival_mean=24.0, replicas_per_group=128, ticks=4000, device="cuda", policy="llumnix",
        tier_blind=False, extensions=()):
    """Run the sweep and return one row per (tier mix, K, tier)."""
    import torch
    cfg = sweep_cfg(arrival_mean, replicas_per_group, ticks, policy, tier_blind, extensions)
    g = Scheduler(cfg, device=device)
    g.step(ticks)
    torch.cuda.synchronize()
    hist = g.histograms().astype(np.int64)
    st = g.replica_stats().astype(np.int64)
    g.close()
    rows = []
    r0 = 0
    for grp in cfg["groups"]:
        n = grp["n_replicas"]
        K = grp["K"]
        mix = {"uniform": "uniform", "gauss": "gauss", "geometric": "enterprise"}[grp["tiers"]["kind"]]
        h = hist[r0:r0 + n].sum(axis=0)
        s = st[r0:r0 + n].sum(axis=0)
        for p in range(K):
            adm, fin = int(s[p * 8 + 3]), int(s[p * 8 + 4])
            rows.append(dict(mix=mix, K=K, tier=p, arrived=int(s[p * 8 + 0]), rejected=int(s[p * 8 + 1]),
                             admitted=adm, finished=fin, preempted=int(s[p * 8 + 5]),
                             qdelay_mean=s[p * 8 + 6] / adm if adm else None,
                             e2e_mean=s[p * 8 + 7] / fin if fin else None,
                             qdelay_p50=percentile(h[0, p], 0.50), qdelay_p90=percentile(h[0, p], 0.90),
                             qdelay_p99=percentile(h[0, p], 0.99),
                             e2e_p50=percentile(h[1, p], 0.50), e2e_p90=percentile(h[1, p], 0.90),
                             e2e_p99=percentile(h[1, p], 0.99)))
        r0 += n
    return cfg, rows


def _fmt(v):
    return "-" if v is None else ("%.1f" % v if isinstance(v, float) else str(v))


def markdown(rows):
    out = ["| mix | K | tier | admitted | queue delay mean | p50 | p90 | p99 | end-to-end mean | p50 | p90 | p99 |",
           "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append("| %s | %d | %d | %d | %s | %s | %s | %s | %s | %s | %s | %s |" % (
            r["mix"], r["K"], r["tier"], r["admitted"], _fmt(r["qdelay_mean"]), _fmt(r["qdelay_p50"]),
            _fmt(r["qdelay_p90"]), _fmt(r["qdelay_p99"]), _fmt(r["e2e_mean"]), _fmt(r["e2e_p50"]),
            _fmt(r["e2e_p90"]), _fmt(r["e2e_p99"])))
    return "\n".join(out)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--arrival-mean", type=float, default=24.0)
    ap.add_argument("--replicas-per-group", type=int, default=128)
    ap.add_argument("--ticks", type=int, default=4000)
    ap.add_argument("--policy", choices=("llumnix", "infaas"), default="llumnix")
    ap.add_argument("--tier-blind", action="store_true",
                    help="first-come-first-served queues and arrival-order dispatch (the paper's INFaaS+vLLM baseline)")
    ap.add_argument("--adaptive", action="store_true", help="adaptive headroom (Section 6.5 extension)")
    ap.add_argument("--promotion", action="store_true", help="promotion of long-waiting requests (Section 6.5 extension)")
    ap.add_argument("--json", help="also write the rows to this file")
    a = ap.parse_args(argv)
    ext = tuple(e for e in ("adaptive", "promotion") if getattr(a, e))
    cfg, rows = run(a.arrival_mean, a.replicas_per_group, a.ticks, policy=a.policy, tier_blind=a.tier_blind,
                    extensions=ext)
    print("# %s, %d ticks\n" % (cfg["name"], a.ticks))
    print(markdown(rows))
    if a.json:
        with open(a.json, "w") as f:
            json.dump(dict(config=cfg["name"], ticks=a.ticks, rows=rows), f)


if __name__ == "__main__":
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    main()
