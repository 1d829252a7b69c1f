"""ctypes binding of libmts (include/mts.h): argument marshalling only.

Every step of the scheduling tick runs in the HIP kernels of libmts.so.
PyTorch only provides the device buffer and the stream.  If the library is
missing the binding raises instead of falling back to anything else.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_lib", "libmts.so")

ABI_VERSION = 6
MAX_TIERS = 10
NSTAT = 96
HIST_BINS = 240  # latency histogram bins per (metric, tier)

TIER_KINDS = {"uniform": 0, "gauss": 1, "geometric": 2, "explicit": 3}
POLICIES = {"llumnix": 0, "infaas": 1}
ARRIVAL_KINDS = {"poisson": 0, "gamma_poisson": 1}
PROMPT_KINDS = {"uniform_int": 0, "lognormal": 1}
OUTPUT_KINDS = {"geometric": 0, "pareto": 1}

ERRORS = {0: "MTS_OK", -1: "MTS_EINVAL", -2: "MTS_ENOMEM", -3: "MTS_EDEVICE",
          -4: "MTS_ESTATE", -5: "MTS_ERANGE"}


class MtsError(RuntimeError):
    def __init__(self, func, code):
        self.code = code
        super().__init__("%s failed: %s (%d)" % (func, ERRORS.get(code, "?"), code))


class mts_group(ctypes.Structure):
    _fields_ = [("n_replicas", ctypes.c_uint32), ("K", ctypes.c_uint32),
                ("tier_kind", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("p0", ctypes.c_double), ("p1", ctypes.c_double),
                ("probs", ctypes.c_double * MAX_TIERS)]


class mts_cfg(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_uint32), ("n_instances", ctypes.c_uint32),
                ("slots_per_instance", ctypes.c_uint32), ("kv_blocks", ctypes.c_uint32),
                ("block_tokens", ctypes.c_uint32), ("zero_lowest_tier", ctypes.c_uint32),
                ("headroom_base", ctypes.c_double), ("headroom_decay", ctypes.c_double),
                ("mig_interval", ctypes.c_uint32), ("mig_stage_blocks", ctypes.c_uint32),
                ("mig_max_pairs", ctypes.c_uint32),
                ("theta_num", ctypes.c_int32), ("theta_den", ctypes.c_int32),
                ("arrival_kind", ctypes.c_uint32), ("prompt_kind", ctypes.c_uint32),
                ("output_kind", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("arrival_mean", ctypes.c_double), ("arrival_cv", ctypes.c_double),
                ("prompt_mu", ctypes.c_double), ("prompt_sigma", ctypes.c_double),
                ("prompt_lo", ctypes.c_uint32), ("prompt_hi", ctypes.c_uint32),
                ("output_param", ctypes.c_double),
                ("output_min", ctypes.c_uint32), ("output_cap", ctypes.c_uint32),
                ("seed", ctypes.c_uint64), ("replica_id_base", ctypes.c_uint64),
                ("n_groups", ctypes.c_uint32), ("reserved2", ctypes.c_uint32),
                ("groups", ctypes.POINTER(mts_group)),
                ("dispatch_policy", ctypes.c_uint32), ("infaas_ewma_shift", ctypes.c_uint32),
                ("infaas_alpha", ctypes.c_int32), ("infaas_beta", ctypes.c_int32), ("infaas_gamma", ctypes.c_int32),
                ("infaas_pen_overloaded", ctypes.c_uint32), ("infaas_pen_interfered", ctypes.c_uint32),
                ("tier_blind", ctypes.c_uint32),
                ("adapt_epoch", ctypes.c_uint32), ("adapt_up", ctypes.c_uint32), ("adapt_down", ctypes.c_uint32),
                ("adapt_max", ctypes.c_uint32), ("adapt_margin", ctypes.c_uint32),
                ("adapt_slo", ctypes.c_uint32 * MAX_TIERS),
                ("promote_period", ctypes.c_uint32), ("promote_age", ctypes.c_uint32 * MAX_TIERS)]


class mts_stats_t(ctypes.Structure):
    _fields_ = [("per_tier", (ctypes.c_uint64 * 8) * MAX_TIERS),
                ("mig_queued", ctypes.c_uint64), ("mig_started", ctypes.c_uint64),
                ("mig_committed", ctypes.c_uint64), ("mig_aborted", ctypes.c_uint64),
                ("run_slot_ticks", ctypes.c_uint64), ("wait_slot_ticks", ctypes.c_uint64),
                ("invariant_violations", ctypes.c_uint64), ("ticks", ctypes.c_uint64),
                ("scale_out_ticks", ctypes.c_uint64), ("scale_in_ticks", ctypes.c_uint64),
                ("drain_fallback_dispatches", ctypes.c_uint64),
                ("replicas", ctypes.c_uint64), ("digest", ctypes.c_uint64)]


class mts_state_view(ctypes.Structure):
    _fields_ = [(k, ctypes.c_void_p) for k in
                ("meta", "lr", "seq", "tarr", "free", "mig", "next_seq", "stats", "drain", "hist", "svc",
                 "hq", "hq_snap")]


EXPORTED = ("mts_state_bytes", "mts_create", "mts_step", "mts_stats", "mts_digest",
            "mts_export_state", "mts_import_state", "mts_get_table", "mts_get_headroom",
            "mts_tick", "mts_set_tick", "mts_set_launch", "mts_get_launch", "mts_set_timing",
            "mts_get_timing", "mts_set_draining", "mts_set_queue_cache", "mts_get_queue_cache",
            "mts_set_wheel_cap", "mts_get_wheel", "mts_step_noalloc", "mts_destroy", "mts_strerror")

_lib = None


def load_library(path=LIB_PATH):
    """Load libmts.so; raises OSError when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise OSError("libmts.so not built (%s); run __graft_entry__.build()" % path)
    L = ctypes.CDLL(path)
    vp, u32, u64, i32 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32
    ci = ctypes.c_int
    L.mts_state_bytes.argtypes = [ctypes.POINTER(mts_cfg), ctypes.POINTER(ctypes.c_size_t)]
    L.mts_create.argtypes = [ctypes.POINTER(mts_cfg), vp, ctypes.c_size_t, vp, ctypes.POINTER(vp)]
    L.mts_step.argtypes = [vp, u64, vp]
    L.mts_step_noalloc.argtypes = [vp, u64, vp]
    L.mts_stats.argtypes = [vp, ctypes.POINTER(mts_stats_t)]
    L.mts_digest.argtypes = [vp, u32, u32, vp]
    L.mts_export_state.argtypes = [vp, u32, u32, ctypes.POINTER(mts_state_view)]
    L.mts_import_state.argtypes = [vp, u32, u32, ctypes.POINTER(mts_state_view)]
    L.mts_get_table.argtypes = [vp, ci, u32, vp, u32, ctypes.POINTER(u32), ctypes.POINTER(u32)]
    L.mts_get_headroom.argtypes = [vp, u32, vp]
    L.mts_tick.argtypes = [vp]
    L.mts_tick.restype = u64
    L.mts_set_tick.argtypes = [vp, u64]
    L.mts_set_tick.restype = ci
    L.mts_set_launch.argtypes = [vp, u32, u32]
    L.mts_get_launch.argtypes = [vp, ctypes.POINTER(u32), ctypes.POINTER(u32)]
    L.mts_set_timing.argtypes = [vp, ci]
    L.mts_set_draining.argtypes = [vp, u32, u32, vp]
    L.mts_set_queue_cache.argtypes = [vp, u32]
    L.mts_get_queue_cache.argtypes = [vp, ctypes.POINTER(u32)]
    L.mts_set_wheel_cap.argtypes = [vp, u32]
    L.mts_get_wheel.argtypes = [vp, ctypes.POINTER(u32), ctypes.POINTER(u32), ctypes.POINTER(u64)]
    L.mts_get_timing.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                 ctypes.POINTER(u32)]
    L.mts_destroy.argtypes = [vp]
    L.mts_destroy.restype = None
    L.mts_strerror.argtypes = [ci]
    L.mts_strerror.restype = ctypes.c_char_p
    for f in ("mts_state_bytes", "mts_create", "mts_step", "mts_step_noalloc", "mts_stats", "mts_digest", "mts_export_state",
              "mts_import_state", "mts_get_table", "mts_get_headroom", "mts_set_launch", "mts_get_launch",
              "mts_set_timing", "mts_get_timing", "mts_set_draining", "mts_set_queue_cache",
              "mts_get_queue_cache", "mts_set_wheel_cap", "mts_get_wheel"):
        getattr(L, f).restype = ci
    _lib = L
    return L


def _check(func, rc):
    if rc != 0:
        raise MtsError(func, rc)


def make_cfg(cfg):
    """Marshal a workload dict into (mts_cfg, groups array)."""
    groups = (mts_group * len(cfg["groups"]))()
    for j, g in enumerate(cfg["groups"]):
        t = g["tiers"]
        groups[j].n_replicas = g["n_replicas"]
        groups[j].K = g["K"]
        groups[j].tier_kind = TIER_KINDS[t["kind"]]
        if t["kind"] == "gauss":
            groups[j].p0, groups[j].p1 = t["mu"], t["sigma"]
        elif t["kind"] == "geometric":
            groups[j].p0 = t["r"]
        elif t["kind"] == "explicit":
            for p, v in enumerate(t["probs"]):
                groups[j].probs[p] = v
    c = mts_cfg()
    c.abi_version = ABI_VERSION
    c.n_instances = cfg["n_instances"]
    c.slots_per_instance = cfg["slots_per_instance"]
    c.kv_blocks = cfg["kv_blocks"]
    c.block_tokens = cfg["block_tokens"]
    c.zero_lowest_tier = cfg["zero_lowest_tier"]
    c.headroom_base = cfg["headroom_base"]
    c.headroom_decay = cfg["headroom_decay"]
    c.mig_interval = cfg["mig_interval"]
    c.mig_stage_blocks = cfg["mig_stage_blocks"]
    c.mig_max_pairs = cfg["mig_max_pairs"]
    c.theta_num = cfg["theta_num"]
    c.theta_den = cfg["theta_den"]
    a, p, o = cfg["arrival"], cfg["prompt"], cfg["output"]
    c.arrival_kind = ARRIVAL_KINDS[a["kind"]]
    c.arrival_mean = a["mean"]
    c.arrival_cv = a.get("cv", 0.0)
    c.prompt_kind = PROMPT_KINDS[p["kind"]]
    c.prompt_mu = p.get("mu", 0.0)
    c.prompt_sigma = p.get("sigma", 0.0)
    c.prompt_lo, c.prompt_hi = p["lo"], p["hi"]
    c.output_kind = OUTPUT_KINDS[o["kind"]]
    if o["kind"] == "geometric":
        c.output_param = o["mean"]
    else:
        c.output_param, c.output_min, c.output_cap = o["alpha"], o["min"], o["cap"]
    c.seed = cfg["seed"]
    c.replica_id_base = cfg["replica_id_base"]
    c.n_groups = len(cfg["groups"])
    c.groups = groups
    d = cfg.get("dispatch", {"policy": "llumnix"})
    c.dispatch_policy = POLICIES[d["policy"]]
    c.tier_blind = 1 if cfg.get("tier_blind") else 0
    if d["policy"] == "infaas":
        c.infaas_alpha, c.infaas_beta, c.infaas_gamma = d["alpha"], d["beta"], d["gamma"]
        c.infaas_pen_overloaded, c.infaas_pen_interfered = d["pen_overloaded"], d["pen_interfered"]
        c.infaas_ewma_shift = d["ewma_shift"]
    # Section 6.5 extensions: {"epoch", "step_up", "step_down", "max", "margin",
    # "slo"} (headroom amounts in 1/256 block; slo lists per-tier targets in
    # ticks, the last one repeated for the tiers it does not reach) and
    # {"period", "age"} (per-tier quotas in ticks, missing tiers 0 = never)
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


def mts_state_bytes(cfg):
    """Device bytes a handle for this workload needs (host-only call)."""
    c, _g = make_cfg(cfg)
    n = ctypes.c_size_t(0)
    _check("mts_state_bytes", load_library().mts_state_bytes(ctypes.byref(c), ctypes.byref(n)))
    return n.value


def _stream_handle(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Scheduler:
    """R replicas of a workload on one GPU, advanced by ``step``."""

    _ORDER = ("meta", "lr", "seq", "tarr", "free", "mig", "next_seq", "stats", "drain", "hist", "svc", "hq",
              "hq_snap")

    def __init__(self, cfg, device="cuda", stream=None):
        import torch
        L = load_library()
        if not torch.cuda.is_available():
            raise RuntimeError("libmts needs a GPU")
        self.cfg = cfg
        self.R = sum(g["n_replicas"] for g in cfg["groups"])
        self.I, self.S = cfg["n_instances"], cfg["slots_per_instance"]
        self._c, self._groups = make_cfg(cfg)
        self.nbytes = mts_state_bytes(cfg)
        # torch's caching allocator hands out 512-byte aligned blocks
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
        h = ctypes.c_void_p(0)
        _check("mts_create", L.mts_create(ctypes.byref(self._c), ctypes.c_void_p(self.buf.data_ptr()),
                                          self.nbytes, _stream_handle(stream), ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            load_library().mts_destroy(self._h)
            self._h = ctypes.c_void_p(0)
            self.buf = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def tick(self):
        return load_library().mts_tick(self._h)

    @tick.setter
    def tick(self, t):
        _check("mts_set_tick", load_library().mts_set_tick(self._h, t))

    def step(self, n_ticks, stream=None):
        _check("mts_step", load_library().mts_step(self._h, n_ticks, _stream_handle(stream)))

    def step_noalloc(self, n_ticks, stream=None):
        """step() with the arrival staging in the library's static device
        scratch: allocates nothing (mts_step_noalloc)."""
        _check("mts_step_noalloc", load_library().mts_step_noalloc(self._h, n_ticks, _stream_handle(stream)))

    def set_launch(self, threads=0, blocks=0):
        _check("mts_set_launch", load_library().mts_set_launch(self._h, threads, blocks))

    def set_timing(self, on=True):
        """Record HIP events around every kernel launch of later steps."""
        _check("mts_set_timing", load_library().mts_set_timing(self._h, 1 if on else 0))

    def timing(self):
        """(step-kernel ms, arrival-kernel ms, step-kernel launches) since the last call."""
        st, ar, n = ctypes.c_double(0), ctypes.c_double(0), ctypes.c_uint32(0)
        _check("mts_get_timing", load_library().mts_get_timing(self._h, ctypes.byref(st), ctypes.byref(ar),
                                                               ctypes.byref(n)))
        return st.value, ar.value, n.value

    def launch(self):
        """(threads, blocks) of the step kernel as mts_step launches it."""
        th, bl = ctypes.c_uint32(0), ctypes.c_uint32(0)
        _check("mts_get_launch", load_library().mts_get_launch(self._h, ctypes.byref(th), ctypes.byref(bl)))
        return th.value, bl.value

    def stats(self, allow_violations=False):
        st = mts_stats_t()
        rc = load_library().mts_stats(self._h, ctypes.byref(st))
        if rc != 0 and not (allow_violations and rc == -4):
            raise MtsError("mts_stats", rc)
        raw = np.zeros(NSTAT, np.uint64)
        for p in range(MAX_TIERS):
            for f in range(8):
                raw[p * 8 + f] = st.per_tier[p][f]
        raw[80:91] = [st.mig_queued, st.mig_started, st.mig_committed, st.mig_aborted,
                      st.run_slot_ticks, st.wait_slot_ticks, st.invariant_violations, st.ticks,
                      st.scale_out_ticks, st.scale_in_ticks, st.drain_fallback_dispatches]
        return dict(raw=raw, replicas=st.replicas, digest=st.digest)

    def digests(self, r0=0, nr=None):
        nr = self.R - r0 if nr is None else nr
        out = np.zeros(nr, np.uint64)
        _check("mts_digest", load_library().mts_digest(self._h, r0, nr, out.ctypes.data))
        return out

    def _arrays(self, nr):
        IS = self.I * self.S
        return dict(meta=np.zeros(nr * IS, np.uint8), lr=np.zeros(nr * IS, np.uint32),
                    seq=np.zeros(nr * IS, np.uint32), tarr=np.zeros(nr * IS, np.uint32),
                    free=np.zeros(nr * self.I, np.int32), mig=np.zeros(nr * self.I * 4, np.int32),
                    next_seq=np.zeros(nr, np.uint32), stats=np.zeros(nr * NSTAT, np.uint64),
                    drain=np.zeros(nr * self.I, np.uint8),
                    hist=np.zeros(nr * 2 * MAX_TIERS * HIST_BINS, np.uint32),
                    svc=np.zeros(nr * self.I, np.int64),
                    hq=np.zeros(nr * MAX_TIERS, np.int32), hq_snap=np.zeros(nr * 2 * MAX_TIERS, np.uint64))

    @property
    def queue_cache(self):
        """Queue-cache entries per instance behind the head of line (LDS)."""
        d = ctypes.c_uint32(0)
        _check("mts_get_queue_cache", load_library().mts_get_queue_cache(self._h, ctypes.byref(d)))
        return d.value

    @queue_cache.setter
    def queue_cache(self, depth):
        _check("mts_set_queue_cache", load_library().mts_set_queue_cache(self._h, depth))

    def set_wheel_cap(self, cap):
        """Entries per finish-wheel bucket from the next step on (test hook)."""
        _check("mts_set_wheel_cap", load_library().mts_set_wheel_cap(self._h, cap))

    def wheel(self):
        """(capacity in use, reserved capacity, bucket rebuilds so far)."""
        c, m, n = ctypes.c_uint32(0), ctypes.c_uint32(0), ctypes.c_uint64(0)
        _check("mts_get_wheel", load_library().mts_get_wheel(self._h, ctypes.byref(c), ctypes.byref(m),
                                                             ctypes.byref(n)))
        return c.value, m.value, n.value

    def set_draining(self, flags, r0=0, nr=None):
        """flags: 0/1 per (replica, instance) of replicas [r0, r0 + nr)."""
        f = np.ascontiguousarray(flags, dtype=np.uint8).ravel()
        nr = len(f) // self.I if nr is None else nr
        if len(f) != nr * self.I:
            raise ValueError("need %d flags" % (nr * self.I))
        _check("mts_set_draining", load_library().mts_set_draining(self._h, r0, nr, f.ctypes.data))

    def export(self, r0=0, nr=None):
        nr = self.R - r0 if nr is None else nr
        a = self._arrays(nr)
        v = mts_state_view(*[a[k].ctypes.data for k in self._ORDER])
        _check("mts_export_state", load_library().mts_export_state(self._h, r0, nr, ctypes.byref(v)))
        return a

    def histograms(self, r0=0, nr=None):
        """Latency histograms of replicas [r0, r0 + nr) as
        [replica][metric (0 queue delay, 1 end-to-end)][tier][bin] (u32)."""
        nr = self.R - r0 if nr is None else nr
        h = np.zeros(nr * 2 * MAX_TIERS * HIST_BINS, np.uint32)
        ptrs = [None] * len(self._ORDER)
        ptrs[self._ORDER.index("hist")] = h.ctypes.data
        v = mts_state_view(*ptrs)
        _check("mts_export_state", load_library().mts_export_state(self._h, r0, nr, ctypes.byref(v)))
        return h.reshape(nr, 2, MAX_TIERS, HIST_BINS)

    def replica_stats(self, r0=0, nr=None):
        """Per-replica counters of replicas [r0, r0 + nr) as [replica][MTS_NSTAT] (u64)."""
        nr = self.R - r0 if nr is None else nr
        st = np.zeros(nr * NSTAT, np.uint64)
        ptrs = [None] * len(self._ORDER)
        ptrs[self._ORDER.index("stats")] = st.ctypes.data
        v = mts_state_view(*ptrs)
        _check("mts_export_state", load_library().mts_export_state(self._h, r0, nr, ctypes.byref(v)))
        return st.reshape(nr, NSTAT)

    def import_state(self, a, r0=0, nr=None):
        """Overwrite replicas [r0, r0 + nr); a missing "drain", "hist" or "svc"
        clears it, a missing "hq" / "hq_snap" takes its default (mts.h)."""
        nr = len(a["next_seq"]) if nr is None else nr
        b = {k: np.ascontiguousarray(a[k], dtype=v.dtype) for k, v in self._arrays(nr).items() if k in a}
        v = mts_state_view(*[b[k].ctypes.data if k in b else None for k in self._ORDER])
        _check("mts_import_state", load_library().mts_import_state(self._h, r0, nr, ctypes.byref(v)))

    def table(self, which, g=0):
        w = {"tier": 0, "count": 1, "prompt": 2, "output": 3}[which]
        n, base = ctypes.c_uint32(0), ctypes.c_uint32(0)
        L = load_library()
        _check("mts_get_table", L.mts_get_table(self._h, w, g, None, 0, ctypes.byref(n), ctypes.byref(base)))
        out = np.zeros(n.value, np.uint64)
        _check("mts_get_table", L.mts_get_table(self._h, w, g, out.ctypes.data, n.value,
                                                ctypes.byref(n), ctypes.byref(base)))
        return base.value, out

    def headroom(self, g=0):
        out = np.zeros(MAX_TIERS, np.int32)
        _check("mts_get_headroom", load_library().mts_get_headroom(self._h, g, out.ctypes.data))
        return out
