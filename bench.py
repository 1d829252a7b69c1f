"""Benchmark of the multi-tier scheduling step on one MI355X.

A step is one ``mts_step`` call advancing every replica of the workload by
``--ticks-per-step`` ticks (all phases of the tick: decode/KV accounting,
admission, freeness, tier-ordered dispatch, migration).  The default workload
is the K = 1..10 sweep (3840 replicas x 32 instances x 512 slots); 10 timed
steps of 1000 ticks cover its full 10,000-tick run from an empty cluster.
Warm-up steps run on a separate handle of the same workload.

Prints one JSON line: replica-ticks/s (wall clock over the timed steps),
slot-updates/s, the roofline of the step kernel (its launches timed by the
library with HIP events on the launch stream) and the CPU oracle timed on a
bounded sample on this host, one process per core.  The step kernel is bound
by instruction issue: its roofline is VALU wave instructions per second
against the chip's issue peak, with the instructions per replica-tick from
rocprofv3 counters of this exact kernel source; next to it the HBM side:
the event-byte floor of the run (its own counters), the measured traffic and
a measured device copy rate.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
# VALU issue peak of MI355X: 256 compute units x 4 SIMDs of 16 lanes; one
# wave64 VALU instruction occupies a SIMD for 4 cycles, so a compute unit
# issues one wave instruction per cycle: 256 x 2.4 GHz = 614.4 G wave
# instructions/s (39.3 T lane operations/s)
VALU_PEAK_GINST = 256 * 2.4

# Counters of k_step from rocprofv3 on the default bench run (the sweep, one
# launch per 1000-tick step), keyed by the SHA-256 prefix of the step-kernel
# source they were taken on; any other kernel source reports null for them.
#   valu_per_rt   SQ_INSTS_VALU per replica-tick (wave instructions)
#   lane_util     SQ_THREAD_CYCLES_VALU / (64 SQ_ACTIVE_INST_VALU)
#   read, write   HBM bytes per launch from TCC_EA0_RDREQ_{32B,64B,128B} and
#                 TCC_EA0_WRREQ{,_64B} (requests times their sizes)
PROFILED = {
    'e7eb6393498a72f8': {"valu_per_rt": 869.2, "lane_util": 0.3756, "read": 9133853824, "write": 7667387645},
}


def kernel_source_hash():
    import hashlib
    with open(os.path.join(ROOT, "paper_2608_16336_amd", "csrc", "mts_kernels.hip"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def dense_bytes(cfg, R, ticks, d):
    """Bytes a dense per-slot pass would move per the state layout (status 1 B
    per slot per tick; len/rem 8 B read+write per running slot-tick; seq 4 B per
    waiting slot-tick; 13 B per placed or moved request; 1 B per status
    change).  The event-driven kernel does not move these; their rate is
    reported only as the effective bandwidth a dense kernel would need."""
    n_slots = R * cfg["n_instances"] * cfg["slots_per_instance"]
    per = d[:80].reshape(10, 8)
    dispatched = int(per[:, 2].sum())
    admitted = int(per[:, 3].sum())
    finished = int(per[:, 4].sum())
    preempted = int(per[:, 5].sum())
    mq, ms, mc, ma = (int(v) for v in d[80:84])
    run, wait = int(d[84]), int(d[85])
    placed = dispatched + mq + mc
    changes = dispatched + admitted + finished + 2 * preempted + 2 * (mq + ms + mc + ma)
    return n_slots * ticks + 8 * run + 4 * wait + 13 * placed + changes


# Bytes each event of the tick must move at the state layout's field widths
# (slot word 4, meta 1, seq 4, arrival tick 4; wheel entry 4; histogram bin
# read and written 8), with every field touched once and no cache line
# granularity: the floor of an event-driven tick.
EVENT_BYTES = {
    "arrival": 8,        # the sampled record, read by the step kernel
    "placement": 13,     # a dispatched request's word, meta, seq, arrival tick
    "admission": 21,     # word + meta written, arrival tick read, wheel entry, queue-delay bin
    "finish": 25,        # wheel entry, word + meta + arrival tick read, word cleared, end-to-end bin
    "preemption": 22,    # victim's word, meta, seq, arrival tick read, word + meta written, wheel entry
    "queued_move": 30,   # 13 B read, 13 B written, source word cleared
    "mig_start": 6,      # inbound word + meta, source meta
    "mig_commit": 34,    # 13 B read, 13 B written, source word cleared, wheel entry
    "mig_abort": 5,      # inbound word + meta cleared
}


def event_counts(d):
    per = d[:80].reshape(10, 8)
    mq, ms, mc, ma = (int(v) for v in d[80:84])
    return {"arrival": int(per[:, 0].sum()), "placement": int(per[:, 2].sum()),
            "admission": int(per[:, 3].sum()), "finish": int(per[:, 4].sum()),
            "preemption": int(per[:, 5].sum()), "queued_move": mq, "mig_start": ms,
            "mig_commit": mc, "mig_abort": ma}


def event_bytes(R, ticks, d):
    """The event-byte floor of the run (its own counters) plus 4 B per
    replica-tick for the arrival count."""
    n = event_counts(d)
    return sum(EVENT_BYTES[k] * v for k, v in n.items()) + 4 * R * ticks


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _cpu_worker(args):
    """One oracle process: replicas one after the other, each from an empty
    cluster for the given ticks (returns replica-ticks and seconds)."""
    cfg, picks, ticks = args
    import oracle
    t0 = time.perf_counter()
    for r in picks:
        o = oracle.Oracle(cfg, r, 1, check=False)
        o.step(ticks)
        o.close()
    return len(picks) * ticks, time.perf_counter() - t0


def cpu_baseline(cfg, single_replicas, per_core_replicas, sample_ticks):
    """The oracle on this host's cores: one thread, then one process per core
    over disjoint replicas spread over the workload's groups."""
    import multiprocessing as mp
    R = sum(g["n_replicas"] for g in cfg["groups"])
    spread = lambda n: [int(k * R // n) for k in range(n)] if n < R else list(range(R))  # noqa: E731
    rt1, dt1 = _cpu_worker((cfg, spread(single_replicas), sample_ticks))
    single = rt1 / dt1
    P = min(16, len(os.sched_getaffinity(0)))
    picks = spread(P * per_core_replicas)
    parts = [(cfg, picks[k::P], sample_ticks) for k in range(P)]
    with mp.get_context("spawn").Pool(P) as pool:
        res = pool.map(_cpu_worker, parts)
    rtp = sum(r for r, _ in res)
    dtp = max(dt for _, dt in res)
    multi = rtp / dtp
    slots = cfg["n_instances"] * cfg["slots_per_instance"]
    return {"value": multi, "unit": "replica-ticks/s", "cores": P, "kind": "oracle",
            "cpu": cpu_model(), "slot_updates_per_s": multi * slots,
            "single_core_value": single,
            "sample": "%d replicas spread over the groups x %d ticks from an empty cluster, one oracle process "
                      "per core on %d cores (%.1f s); single thread: %d replicas, %.1f s"
                      % (len(picks), sample_ticks, P, dtp, len(spread(single_replicas)), dt1)}


def copy_bandwidth(torch, nbytes=1 << 30, reps=5):
    """Device-to-device copy rate (bytes read + written per second): the
    practical HBM peak of this GPU."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    del src, dst
    return 2.0 * nbytes * reps / (ms / 1e3) / 1e9


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="sweep")
    ap.add_argument("--ticks-per-step", type=int, default=1000)
    ap.add_argument("--blocks", type=int, default=0, help="blocks of the step kernel (0: automatic)")
    ap.add_argument("--cpu-replicas", type=int, default=16, help="oracle replicas of the single-thread run")
    ap.add_argument("--cpu-replicas-per-core", type=int, default=12,
                    help="oracle replicas per process of the one-process-per-core run")
    ap.add_argument("--cpu-ticks", type=int, default=10000)
    ap.add_argument("--no-copy-bandwidth", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0,
                    help="MiB copied device-to-device once before timing (counter calibration)")
    ap.add_argument("--policy", choices=("llumnix", "infaas"), default="llumnix",
                    help="global dispatch policy (infaas: cost-based dispatch without migration)")
    ap.add_argument("--tier-blind", action="store_true",
                    help="first-come-first-served queues and arrival-order dispatch")
    ap.add_argument("--extensions", action="store_true",
                    help="adaptive headroom and promotion of waiting requests at the workloads package's settings")
    ap.add_argument("--drain-instances", type=int, default=0,
                    help="mark the first n instances of every replica draining after the first timed step")
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py measures one GPU only: the replicas are independent, so a multi-GPU run "
              "is R/N replicas per GPU with no communication; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2608_16336_amd import Scheduler
    from workloads import preset, with_extensions

    cfg = preset(args.workload)
    if args.extensions:
        cfg = with_extensions(cfg)
    if args.policy == "infaas":
        cfg["dispatch"] = dict(policy="infaas", alpha=64, beta=1, gamma=1, pen_overloaded=512,
                               pen_interfered=128, ewma_shift=4)
    if args.tier_blind:
        cfg["tier_blind"] = 1
    R = sum(g["n_replicas"] for g in cfg["groups"])
    T, K, W = args.ticks_per_step, args.steps, args.warmup
    torch.cuda.set_device(0)

    if W > 0:
        warm = Scheduler(cfg)
        if args.blocks:
            warm.set_launch(0, args.blocks)
        for _ in range(W):
            warm.step(T)
        torch.cuda.synchronize()
        warm.close()
        del warm

    if args.calibrate_copy:
        src = torch.ones(args.calibrate_copy << 18, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    sch = Scheduler(cfg)
    if args.blocks:
        sch.set_launch(0, args.blocks)
    torch.cuda.synchronize()
    s0 = sch.stats()["raw"].astype(np.int64)
    stream = torch.cuda.current_stream()
    sch.set_timing(True)  # HIP events around every kernel launch, on the launch stream
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        if k == 1 and args.drain_instances:
            # host decision between steps (synchronous, inside the timed region)
            flags = np.zeros((R, cfg["n_instances"]), np.uint8)
            flags[:, :args.drain_instances] = 1
            sch.set_draining(flags)
        sch.step(T, stream=stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms, arr_ms, launches = sch.timing()
    s1 = sch.stats()
    d = s1["raw"].astype(np.int64) - s0
    if d[86] != 0:
        print("device invariant checks failed: %d" % d[86], file=sys.stderr)
        sys.exit(1)

    rticks = R * T * K
    value = rticks / wall
    slots = cfg["n_instances"] * cfg["slots_per_instance"]
    avg_launch_s = step_ms / 1e3 / launches
    rt_per_launch = rticks / launches
    default_run = (args.workload, T, args.policy, args.drain_instances, args.tier_blind, args.extensions) == (
        "sweep", 1000, "llumnix", 0, False, False)
    prof = PROFILED.get(kernel_source_hash()) if default_run else None
    # HBM: the event-byte floor of this run, the measured traffic, the copy rate
    b_ev = event_bytes(R, T * K, d) / launches
    traffic = None if prof is None else prof["read"] + prof["write"]
    copy_gbs = None if args.no_copy_bandwidth else copy_bandwidth(torch)
    hbm = {"algorithmic_event_bytes_per_launch": b_ev,
           "event_bytes": EVENT_BYTES, "events": event_counts(d),
           "achieved_GBps": b_ev / avg_launch_s / 1e9,
           "frac": b_ev / avg_launch_s / 1e9 / HBM_PEAK_GBS,
           "measured_bytes_per_launch": traffic,
           "measured_GBps": None if traffic is None else traffic / avg_launch_s / 1e9,
           "measured_frac": None if traffic is None else traffic / avg_launch_s / 1e9 / HBM_PEAK_GBS,
           "measured_over_event_bytes": None if traffic is None else traffic / b_ev,
           "copy_kernel_GBps": copy_gbs,
           "effective_dense_GBps": dense_bytes(cfg, R, T * K, d) / launches / avg_launch_s / 1e9}
    # issue: VALU wave instructions per replica-tick (profile of this source)
    inst = None if prof is None else prof["valu_per_rt"] * rt_per_launch / avg_launch_s / 1e9
    issue_frac = None if inst is None else inst / VALU_PEAK_GINST
    roofline = {"bound": "alu", "achieved": inst, "peak": VALU_PEAK_GINST, "unit": "G wave64 VALU inst/s",
                "frac": issue_frac, "traffic": traffic,
                "kernel": "k_step", "launches": launches, "avg_launch_ms": avg_launch_s * 1e3,
                "replica_ticks_per_launch": rt_per_launch,
                "valu_inst_per_replica_tick": None if prof is None else prof["valu_per_rt"],
                "valu_lane_utilization": None if prof is None else prof["lane_util"],
                "hbm": hbm}
    if issue_frac is not None and hbm["measured_frac"] is not None and hbm["measured_frac"] > issue_frac:
        roofline["bound"] = "hbm"

    out = {
        "metric": "replica-ticks/s and request-slot updates/s at 1 MI355X; % of HBM roofline",
        "value": value,
        "unit": "replica-ticks/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": wall / K * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic (seeded Philox arrivals, on-device sampling)",
        "config": {"workload": cfg["name"], "replicas": R, "instances": cfg["n_instances"],
                   "slots_per_instance": cfg["slots_per_instance"], "ticks_per_step": T,
                   "ticks_timed": T * K, "parallelism": "replicas across workgroups",
                   "policy": args.policy, "tier_blind": args.tier_blind, "draining_instances": args.drain_instances,
                   "adaptive_headroom_and_promotion": args.extensions,
                   "blocks": sch.launch()[1], "threads_per_block": sch.launch()[0]},
        "slot_updates_per_s": value * slots,
        "roofline": roofline,
        "arrivals_kernel_ms_per_step": arr_ms / K,
        "kernel_source": kernel_source_hash(),
        "digest": "%016x" % int(s1["digest"]),
    }
    sch.close()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_replicas, args.cpu_replicas_per_core, args.cpu_ticks)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
