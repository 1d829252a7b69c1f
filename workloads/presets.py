"""Workload presets for the multi-tier scheduling step.

Each preset is a plain ``dict``.  Keys:

``n_instances``        serving instances per replica (the paper's "replicas")
``slots_per_instance`` request slots per instance (multiple of 64)
``kv_blocks``          KV-cache capacity M of one instance, in blocks
``block_tokens``       tokens per KV block
``headroom_base``      h0: headroom of tier 0, in blocks (h0 = M * h_max)
``headroom_decay``     gamma: per-tier decay factor (gamma = e^-lambda)
``zero_lowest_tier``   1: the lowest tier K-1 gets no headroom
``mig_interval``       migration rounds happen on ticks t with t % interval == 0
``mig_stage_blocks``   KV blocks copied per migration stage (one stage per tick)
``mig_max_pairs``      at most this many (source, destination) pairs per round
``theta_num/den``      freeness-gap threshold theta = num/den
``arrival``            per-tick arrival count: poisson(mean) | gamma_poisson(mean, cv)
``prompt``             prompt length: uniform_int(lo, hi) | lognormal(mu, sigma, lo, hi)
``output``             output length: geometric(mean) | pareto(alpha, min, cap)
``groups``             list of {n_replicas, K, tiers}; replicas are the
                       concatenation of the groups in order.
                       tiers: uniform | gauss(mu, sigma) | geometric(r) | explicit(probs)
``seed``               64-bit seed; replica g draws from key (seed, replica_id_base + g)
``replica_id_base``    global id of the first replica
``ticks``              ticks of the full run

The five presets are the synthetic stand-ins for the paper's workloads
(Section 4.2-4.4): Poisson arrivals, right-skewed request lengths and the
uniform / Gaussian / enterprise tier mixes.
"""
import copy

_COMMON = dict(zero_lowest_tier=1, mig_interval=1, mig_stage_blocks=32,
               theta_num=3, theta_den=10, seed=0, replica_id_base=0)


def _cfg(**kw):
    d = dict(_COMMON)
    d.update(kw)
    if "mig_max_pairs" not in d:
        d["mig_max_pairs"] = d["n_instances"] // 2
    return d


TINY = _cfg(
    name="tiny: R=1 I=4 S=64 K=2 uniform, M=2048, Poisson 2/tick",
    n_instances=4, slots_per_instance=64, kv_blocks=2048, block_tokens=16,
    headroom_base=256.0, headroom_decay=0.5,
    arrival=dict(kind="poisson", mean=2.0),
    prompt=dict(kind="uniform_int", lo=64, hi=1024),
    output=dict(kind="geometric", mean=128.0),
    groups=[dict(n_replicas=1, K=2, tiers=dict(kind="uniform"))],
    ticks=1000)

ENTERPRISE = _cfg(
    name="enterprise: R=1024 I=16 S=256 K=4 (.05/.15/.30/.50), M=8192, Poisson 6/tick",
    n_instances=16, slots_per_instance=256, kv_blocks=8192, block_tokens=16,
    headroom_base=512.0, headroom_decay=0.5,
    arrival=dict(kind="poisson", mean=6.0),
    prompt=dict(kind="lognormal", mu=6.2, sigma=0.8, lo=32, hi=8192),
    output=dict(kind="geometric", mean=256.0),
    groups=[dict(n_replicas=1024, K=4,
                 tiers=dict(kind="explicit", probs=[0.05, 0.15, 0.30, 0.50]))],
    ticks=5000)

GAUSS10 = _cfg(
    name="gauss10: R=4096 I=16 S=256 K=10 N(4.5,2.0), M=8192, Poisson 6/tick",
    n_instances=16, slots_per_instance=256, kv_blocks=8192, block_tokens=16,
    headroom_base=512.0, headroom_decay=0.7,
    arrival=dict(kind="poisson", mean=6.0),
    prompt=dict(kind="uniform_int", lo=128, hi=4096),
    output=dict(kind="geometric", mean=200.0),
    groups=[dict(n_replicas=4096, K=10, tiers=dict(kind="gauss", mu=4.5, sigma=2.0))],
    ticks=10000)


def _sweep_groups(per_group):
    groups = []
    for K in range(1, 11):
        groups.append(dict(n_replicas=per_group, K=K, tiers=dict(kind="uniform")))
        groups.append(dict(n_replicas=per_group, K=K,
                           tiers=dict(kind="gauss", mu=(K - 1) / 2.0, sigma=K / 4.0)))
        groups.append(dict(n_replicas=per_group, K=K,
                           tiers=dict(kind="geometric", r=0.5)))
    return groups


SWEEP = _cfg(
    name="sweep: K=1..10 x {uniform, gauss, enterprise} x 128 = 3840 replicas, I=32 S=512, M=16384, Poisson 12/tick",
    n_instances=32, slots_per_instance=512, kv_blocks=16384, block_tokens=16,
    headroom_base=1024.0, headroom_decay=0.6,
    arrival=dict(kind="poisson", mean=12.0),
    prompt=dict(kind="lognormal", mu=6.5, sigma=1.0, lo=32, hi=16384),
    output=dict(kind="geometric", mean=256.0),
    groups=_sweep_groups(128),
    ticks=10000)

WIDE = _cfg(
    name="wide: R=8 I=256 S=2048 K=10 uniform, M=32768, gamma-Poisson mean 200 CV 3",
    n_instances=256, slots_per_instance=2048, kv_blocks=32768, block_tokens=16,
    headroom_base=2048.0, headroom_decay=0.6,
    arrival=dict(kind="gamma_poisson", mean=200.0, cv=3.0),
    prompt=dict(kind="lognormal", mu=7.0, sigma=1.2, lo=32, hi=32768),
    output=dict(kind="pareto", alpha=1.5, min=16, cap=8192),
    groups=[dict(n_replicas=8, K=10, tiers=dict(kind="uniform"))],
    ticks=20000)

PRESETS = {"tiny": TINY, "enterprise": ENTERPRISE, "gauss10": GAUSS10,
           "sweep": SWEEP, "wide": WIDE}


def preset(name):
    """Deep copy of a named preset."""
    return copy.deepcopy(PRESETS[name])


def with_extensions(cfg, adaptive=True, promotion=True):
    """The Section 6.5 extensions at the settings the benchmark and the study
    use (a copy of cfg): headroom updated every 50 ticks, up 8 blocks when the
    tier's mean queue delay since the last update exceeds 2^(p+1) ticks for
    tier p, down 2 blocks when it stays at or below half of that, never above
    a quarter of M; a promotion pass every 10 ticks with a quota of 50 p
    ticks for tier p."""
    d = copy.deepcopy(cfg)
    if adaptive:
        d["adaptive"] = dict(epoch=50, step_up=8 * 256, step_down=2 * 256, max=d["kv_blocks"] * 256 // 4,
                             margin=128, slo=[2 << p for p in range(10)])
    if promotion:
        d["promotion"] = dict(period=10, age=[50 * p for p in range(10)])
    return d


def n_replicas(cfg):
    return sum(g["n_replicas"] for g in cfg["groups"])


def scaled(name, replicas_per_group=None, ticks=None, **over):
    """A preset with fewer replicas per group and/or fewer ticks.

    ``replicas_per_group`` caps every group's replica count, so a reduced
    sweep still covers every (K, tier distribution) group.
    """
    d = preset(name)
    if replicas_per_group is not None:
        for g in d["groups"]:
            g["n_replicas"] = min(g["n_replicas"], replicas_per_group)
    if ticks is not None:
        d["ticks"] = ticks
    d.update(over)
    return d
