"""CPU oracle for the multi-tier scheduling step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or runs anything from here.

The C source ``mts_oracle.c`` is a plain single-threaded implementation of the
tick written from the paper (Eq. 1-4, Sections 3.1-3.5).  This module builds
it with gcc and marshals the workload dictionaries of :mod:`workloads` into its
own configuration struct (it shares no struct, header or code with the HIP
library).
"""
import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mts_oracle.c")
# MTS_ORACLE_LIB lets the mutation test point the wrapper at a deliberately
# broken build of the oracle
LIB = os.environ.get("MTS_ORACLE_LIB") or os.path.join(HERE, "_build", "libmts_oracle.so")

NSTAT = 96
MAX_TIERS = 10
HBINS = 240  # latency histogram bins per (metric, tier)
STAT_FIELDS = ("arrived", "rejected", "dispatched", "admitted", "finished",
               "preempted", "qdelay_sum", "e2e_sum")
STAT_GLOBALS = ("mig_queued", "mig_started", "mig_committed", "mig_aborted",
                "run_slot_ticks", "wait_slot_ticks", "invariant_violations", "ticks",
                "scale_out_ticks", "scale_in_ticks", "drain_fallback_dispatches")

_TIER_KIND = {"uniform": 0, "gauss": 1, "geometric": 2, "explicit": 3}
_ARR_KIND = {"poisson": 0, "gamma_poisson": 1}
_PROMPT_KIND = {"uniform_int": 0, "lognormal": 1}
_OUT_KIND = {"geometric": 0, "pareto": 1}
_POLICY = {"llumnix": 0, "infaas": 1}


def build(force=True):
    """Compile the oracle with gcc (-O2, no FP contraction)."""
    os.makedirs(os.path.dirname(LIB), exist_ok=True)
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared",
                           "-Wall", "-o", tmp, SRC, "-lm"])
    os.replace(tmp, LIB)
    return LIB


class _Group(ctypes.Structure):
    _fields_ = [("n_replicas", ctypes.c_uint32), ("K", ctypes.c_uint32),
                ("kind", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("a", ctypes.c_double), ("b", ctypes.c_double),
                ("probs", ctypes.c_double * MAX_TIERS)]


class _Cfg(ctypes.Structure):
    _fields_ = [("n_instances", ctypes.c_uint32), ("slots", ctypes.c_uint32),
                ("kv_blocks", ctypes.c_uint32), ("block_tokens", ctypes.c_uint32),
                ("h0", ctypes.c_double), ("gamma", ctypes.c_double),
                ("zero_lowest", ctypes.c_uint32), ("mig_interval", ctypes.c_uint32),
                ("mig_stage", ctypes.c_uint32), ("mig_max_pairs", ctypes.c_uint32),
                ("theta_num", ctypes.c_int32), ("theta_den", ctypes.c_int32),
                ("arr_kind", ctypes.c_int32), ("prompt_kind", ctypes.c_int32),
                ("out_kind", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("arr_mean", ctypes.c_double), ("arr_cv", ctypes.c_double),
                ("prompt_mu", ctypes.c_double), ("prompt_sigma", ctypes.c_double),
                ("prompt_lo", ctypes.c_uint32), ("prompt_hi", ctypes.c_uint32),
                ("out_a", ctypes.c_double),
                ("out_min", ctypes.c_uint32), ("out_cap", ctypes.c_uint32),
                ("seed", ctypes.c_uint64), ("replica_id_base", ctypes.c_uint64),
                ("n_groups", ctypes.c_uint32), ("pad2", ctypes.c_uint32),
                ("groups", ctypes.POINTER(_Group)),
                ("policy", ctypes.c_uint32), ("ewma_shift", ctypes.c_uint32),
                ("alpha", ctypes.c_int32), ("beta", ctypes.c_int32), ("gamma_w", ctypes.c_int32),
                ("pen_over", ctypes.c_uint32), ("pen_intf", ctypes.c_uint32), ("tier_blind", ctypes.c_uint32),
                ("adapt_epoch", ctypes.c_uint32), ("adapt_up", ctypes.c_uint32), ("adapt_down", ctypes.c_uint32),
                ("adapt_max", ctypes.c_uint32), ("adapt_margin", ctypes.c_uint32),
                ("adapt_slo", ctypes.c_uint32 * MAX_TIERS),
                ("promote_period", ctypes.c_uint32), ("promote_age", ctypes.c_uint32 * MAX_TIERS)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        vp, u32, u64, i32 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32
        L.or_create.restype = vp
        L.or_create.argtypes = [ctypes.POINTER(_Cfg), u32, u32, ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
        L.or_destroy.argtypes = [vp]
        L.or_step.argtypes = [vp, u64]
        L.or_tick_now.restype = u64
        L.or_tick_now.argtypes = [vp]
        L.or_set_tick.argtypes = [vp, u64]
        L.or_export.restype = ctypes.c_int
        L.or_export.argtypes = [vp, u32, u32] + [vp] * 9
        L.or_import.restype = ctypes.c_int
        L.or_import.argtypes = [vp, u32, u32] + [vp] * 9
        L.or_digest.argtypes = [vp, vp]
        L.or_table.restype = ctypes.c_int
        L.or_table.argtypes = [vp, ctypes.c_int, u32, vp, u32, ctypes.POINTER(u32)]
        L.or_headroom.argtypes = [vp, u32, vp]
        L.or_freeness.argtypes = [vp, u32, u32, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]
        L.or_last_arrivals.restype = ctypes.c_int
        L.or_last_arrivals.argtypes = [vp, u32, vp, u32]
        L.or_check.restype = u64
        L.or_check.argtypes = [vp, u32]
        L.or_philox4x64_10.argtypes = [vp, vp, vp]
        L.or_set_drain.restype = ctypes.c_int
        L.or_set_drain.argtypes = [vp, u32, u32, ctypes.c_int]
        L.or_freeness_normal.argtypes = [vp, u32, u32, ctypes.POINTER(ctypes.c_int64),
                                         ctypes.POINTER(ctypes.c_int64)]
        L.or_autoscale.restype = ctypes.c_int
        L.or_autoscale.argtypes = [vp, u32, ctypes.POINTER(ctypes.c_int64)]
        L.or_hist_get.restype = ctypes.c_int
        L.or_hist_get.argtypes = [vp, u32, u32, vp]
        L.or_hist_set.restype = ctypes.c_int
        L.or_hist_set.argtypes = [vp, u32, u32, vp]
        L.or_hist_bin.restype = u32
        L.or_hist_bin.argtypes = [u64]
        L.or_svc_get.restype = ctypes.c_int
        L.or_svc_get.argtypes = [vp, u32, u32, vp]
        L.or_svc_set.restype = ctypes.c_int
        L.or_svc_set.argtypes = [vp, u32, u32, vp]
        L.or_adapt_get.restype = ctypes.c_int
        L.or_adapt_get.argtypes = [vp, u32, u32, vp, vp]
        L.or_adapt_set.restype = ctypes.c_int
        L.or_adapt_set.argtypes = [vp, u32, u32, vp, vp]
        _lib = L
    return _lib


def philox4x64_10(ctr, key):
    """The oracle's Philox4x64-10 block function (for pinning against numpy)."""
    c = np.asarray(ctr, dtype=np.uint64)
    k = np.asarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().or_philox4x64_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def _ptr(a):
    return a.ctypes.data


def make_cfg(cfg):
    """Marshal a workload dict into the oracle's own C struct."""
    groups = (_Group * len(cfg["groups"]))()
    for j, g in enumerate(cfg["groups"]):
        t = g["tiers"]
        groups[j].n_replicas = g["n_replicas"]
        groups[j].K = g["K"]
        groups[j].kind = _TIER_KIND[t["kind"]]
        if t["kind"] == "gauss":
            groups[j].a, groups[j].b = t["mu"], t["sigma"]
        elif t["kind"] == "geometric":
            groups[j].a = t["r"]
        elif t["kind"] == "explicit":
            for p, v in enumerate(t["probs"]):
                groups[j].probs[p] = v
    c = _Cfg()
    c.n_instances = cfg["n_instances"]
    c.slots = cfg["slots_per_instance"]
    c.kv_blocks = cfg["kv_blocks"]
    c.block_tokens = cfg["block_tokens"]
    c.h0 = cfg["headroom_base"]
    c.gamma = cfg["headroom_decay"]
    c.zero_lowest = cfg["zero_lowest_tier"]
    c.mig_interval = cfg["mig_interval"]
    c.mig_stage = cfg["mig_stage_blocks"]
    c.mig_max_pairs = cfg["mig_max_pairs"]
    c.theta_num = cfg["theta_num"]
    c.theta_den = cfg["theta_den"]
    a = cfg["arrival"]
    c.arr_kind = _ARR_KIND[a["kind"]]
    c.arr_mean = a["mean"]
    c.arr_cv = a.get("cv", 0.0)
    p = cfg["prompt"]
    c.prompt_kind = _PROMPT_KIND[p["kind"]]
    c.prompt_mu = p.get("mu", 0.0)
    c.prompt_sigma = p.get("sigma", 0.0)
    c.prompt_lo, c.prompt_hi = p["lo"], p["hi"]
    o = cfg["output"]
    c.out_kind = _OUT_KIND[o["kind"]]
    if o["kind"] == "geometric":
        c.out_a = o["mean"]
    else:
        c.out_a, c.out_min, c.out_cap = o["alpha"], o["min"], o["cap"]
    c.seed = cfg["seed"]
    c.replica_id_base = cfg["replica_id_base"]
    c.n_groups = len(cfg["groups"])
    c.groups = groups
    d = cfg.get("dispatch", {"policy": "llumnix"})
    c.policy = _POLICY[d["policy"]]
    c.tier_blind = 1 if cfg.get("tier_blind") else 0
    if d["policy"] == "infaas":
        c.alpha, c.beta, c.gamma_w = d["alpha"], d["beta"], d["gamma"]
        c.pen_over, c.pen_intf = d["pen_overloaded"], d["pen_interfered"]
        c.ewma_shift = d["ewma_shift"]
    ad = cfg.get("adaptive")
    if ad:
        c.adapt_epoch, c.adapt_up, c.adapt_down = ad["epoch"], ad["step_up"], ad["step_down"]
        c.adapt_max, c.adapt_margin = ad["max"], ad["margin"]
        slo = list(ad["slo"])
        for p in range(MAX_TIERS):
            c.adapt_slo[p] = slo[min(p, len(slo) - 1)]
    pr = cfg.get("promotion")
    if pr:
        c.promote_period = pr["period"]
        for p, v in enumerate(pr["age"]):
            c.promote_age[p] = v
    return c, groups


class OracleError(RuntimeError):
    pass


class Oracle:
    """A set of replicas [r_begin, r_begin + r_count) of a workload, simulated
    on the CPU one tick at a time."""

    def __init__(self, cfg, r_begin=0, r_count=None, check=True):
        self.cfg = cfg
        self.R_total = sum(g["n_replicas"] for g in cfg["groups"])
        if r_count is None:
            r_count = self.R_total - r_begin
        self.r_begin, self.r_count = r_begin, r_count
        self.I, self.S = cfg["n_instances"], cfg["slots_per_instance"]
        self._c, self._groups = make_cfg(cfg)
        err = ctypes.c_int(0)
        self._h = lib().or_create(ctypes.byref(self._c), r_begin, r_count, 1 if check else 0, ctypes.byref(err))
        if not self._h:
            raise OracleError("oracle rejected the configuration (code %d)" % err.value)

    def close(self):
        if self._h:
            lib().or_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def tick(self):
        return lib().or_tick_now(self._h)

    @tick.setter
    def tick(self, t):
        lib().or_set_tick(self._h, t)

    def step(self, n=1):
        lib().or_step(self._h, n)

    def _arrays(self, nr):
        IS = self.I * self.S
        return dict(meta=np.zeros(nr * IS, np.uint8), lr=np.zeros(nr * IS, np.uint32),
                    seq=np.zeros(nr * IS, np.uint32), tarr=np.zeros(nr * IS, np.uint32),
                    free=np.zeros(nr * self.I, np.int32), mig=np.zeros(nr * self.I * 4, np.int32),
                    next_seq=np.zeros(nr, np.uint32), stats=np.zeros(nr * NSTAT, np.uint64),
                    drain=np.zeros(nr * self.I, np.uint8),
                    hist=np.zeros(nr * 2 * MAX_TIERS * HBINS, np.uint32),
                    svc=np.zeros(nr * self.I, np.int64),
                    hq=np.zeros(nr * MAX_TIERS, np.int32), hq_snap=np.zeros(nr * 2 * MAX_TIERS, np.uint64))

    _ORDER = ("meta", "lr", "seq", "tarr", "free", "mig", "next_seq", "stats", "drain")

    def export(self, r0=0, nr=None):
        """Canonical state of local replicas [r0, r0+nr) as flat numpy arrays."""
        if nr is None:
            nr = self.r_count - r0
        a = self._arrays(nr)
        rc = lib().or_export(self._h, r0, nr, *[_ptr(a[k]) for k in self._ORDER])
        if rc or lib().or_hist_get(self._h, r0, nr, _ptr(a["hist"])) or lib().or_svc_get(self._h, r0, nr, _ptr(a["svc"])):
            raise OracleError("export range")
        if lib().or_adapt_get(self._h, r0, nr, _ptr(a["hq"]), _ptr(a["hq_snap"])):
            raise OracleError("export range")
        return a

    def import_state(self, a, r0=0, nr=None):
        if nr is None:
            nr = len(a["next_seq"])
        b = {k: np.ascontiguousarray(a[k], dtype=v.dtype) if k in a else v for k, v in self._arrays(nr).items()}
        for k in ("hist", "svc"):
            if k not in a:
                b[k][:] = 0
        rc = lib().or_import(self._h, r0, nr, *[_ptr(b[k]) for k in self._ORDER])
        if rc or lib().or_hist_set(self._h, r0, nr, _ptr(b["hist"])) or lib().or_svc_set(self._h, r0, nr, _ptr(b["svc"])):
            raise OracleError("import range")
        # adaptive headroom state: a missing array takes its default (Eq. 3's
        # table; the current counters as the last update's)
        if lib().or_adapt_set(self._h, r0, nr, _ptr(b["hq"]) if "hq" in a else None,
                              _ptr(b["hq_snap"]) if "hq_snap" in a else None):
            raise OracleError("import: adaptive headroom state out of range")

    def digests(self):
        out = np.zeros(self.r_count, np.uint64)
        lib().or_digest(self._h, _ptr(out))
        return out

    def table(self, which, g=0):
        """(base, quantised CDF) of table ``which`` in {'tier', 'count', 'prompt', 'output'}."""
        w = {"tier": 0, "count": 1, "prompt": 2, "output": 3}[which]
        cap = 1 << 17
        out = np.zeros(cap, np.uint64)
        base = ctypes.c_uint32(0)
        n = lib().or_table(self._h, w, g, _ptr(out), cap, ctypes.byref(base))
        if n < 0:
            raise OracleError("table")
        return base.value, out[:n].copy()

    def headroom(self, g=0):
        out = np.zeros(MAX_TIERS, np.int32)
        lib().or_headroom(self._h, g, _ptr(out))
        return out

    def set_drain(self, r, i, on=True):
        """Mark instance i of local replica r as draining (or not)."""
        if lib().or_set_drain(self._h, r, i, 1 if on else 0):
            raise OracleError("set_drain range")

    def freeness_normal(self, r, i):
        """(num, den): F_normal = num / (256 den) blocks per running request, no headroom."""
        n, d = ctypes.c_int64(0), ctypes.c_int64(0)
        lib().or_freeness_normal(self._h, r, i, ctypes.byref(n), ctypes.byref(d))
        return n.value, d.value

    def autoscale(self, r=0):
        """(signal, fixed-point sum): -1 scale out, +1 scale in, 0 none, for the current state."""
        v = ctypes.c_int64(0)
        sig = lib().or_autoscale(self._h, r, ctypes.byref(v))
        return sig, v.value

    def freeness(self, r, i):
        num, den = ctypes.c_int64(0), ctypes.c_int64(0)
        lib().or_freeness(self._h, r, i, ctypes.byref(num), ctypes.byref(den))
        return num.value, den.value

    def last_arrivals(self, r=0):
        cap = 1 << 16
        out = np.zeros(cap * 3, np.uint32)
        n = lib().or_last_arrivals(self._h, r, _ptr(out), cap)
        return out[: 3 * n].reshape(n, 3)

    def check(self, r=0):
        return int(lib().or_check(self._h, r))


def stat_index(tier, field):
    return tier * 8 + STAT_FIELDS.index(field)


def stat_global(name):
    return 80 + STAT_GLOBALS.index(name)


def hist_bin(v):
    """The oracle's histogram bin of a latency of v ticks."""
    return int(lib().or_hist_bin(int(v)))


def hist_view(h, nr):
    """Flat histogram array -> [replica][metric (0 queue delay, 1 end-to-end)][tier][bin]."""
    return np.asarray(h).reshape(nr, 2, MAX_TIERS, HBINS)
