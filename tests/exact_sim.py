"""Exact-rational, per-request reference simulator for tiny inputs (tests only).

This is a second formulation of the scheduling tick.  It is deliberately
different from the C oracle's: it shares no code with it, it sums the virtual
usage V(r) of Eq. 2 request by request, splits each tier's headroom evenly
over that tier's running requests (H_p / n_p, so a tier with two running
requests charges H_p / 2 to each -- for K = 2 this is exactly Llumnix's
binary rule h / numHighPriorityRequests, Section 3.3), keeps every freeness
value as an exact ``Fraction`` and picks every argmax/argmin by exhaustive
search.  The headroom table is derived here in exact rational arithmetic from
Eq. 3 instead of the oracle's repeated double multiplication.

The arrivals of each tick are inputs: the caller passes the (tier, prompt,
output) triples the oracle sampled, so this simulator covers the scheduling
decisions and the accounting, not the sampler.

Draining (Sections 3.4, 3.5) is modelled literally: a draining instance's
full freeness is ``-inf`` (the infinite-usage sentinel), dispatch takes the
argmax over the non-draining instances with room and, only when there is
none, the least loaded draining one; pairing sorts draining instances first
and never uses one as a destination.  The INFaaS-style policy (Section 3.7) is written out literally too: the
cost alpha * q + beta * s + gamma * penalty of every candidate instance, its
queue depth q counted from the request list, its state penalty from the head
of line against the free blocks (OVERLOADED) or this tick's preemptions
(INTERFERED), the service-time estimate s as a moving average of the per-tick
mean end-to-end time (1/256 tick, floors as the policy defines them), the
minimum by exhaustive search, and no migration at all.

Tier-blind scheduling (the priority-blind local scheduler of the paper's
INFaaS baseline, Section 5.3) replaces the tier by a constant in every
ordering -- dispatch order, queue order, preemption victim, migration
candidate -- and nowhere else.

Adaptive headroom and multilevel-feedback promotion (Section 6.5, future
work; the readings are the library's) are written from the request list: the
headroom update at an epoch boundary takes the queue delays of the requests
first admitted since the previous boundary from the per-request latency log
and compares their exact mean with the tier's target; promotion walks the
waiting requests and compares each one's age with its tier's quota.

The auto-scaling signal (Section 3.6)
averages F_normal -- Eq. 1 with no headroom at all -- in fixed point with
floor(F * 2^20) per instance.
"""
import math
from fractions import Fraction

EMPTY, WAITING, RUNNING, INBOUND = 0, 1, 2, 3
NSTAT = 96
F_ARRIVED, F_REJECTED, F_DISPATCHED, F_ADMITTED, F_FINISHED, F_PREEMPTED, F_QDELAY, F_E2E = range(8)
MIG_QUEUED, MIG_STARTED, MIG_COMMITTED, MIG_ABORTED, RUN_TICKS, WAIT_TICKS, INVARIANT, TICKS = range(80, 88)
SCALE_OUT, SCALE_IN, DRAIN_FALLBACK = range(88, 91)


def exact_headroom(h0, gamma, K, zero_lowest):
    """Eq. 3, H_p = h0 * gamma^p, in 1/256 block with round-half-even,
    evaluated on the exact binary values of h0 and gamma."""
    out = []
    for p in range(K):
        x = Fraction(h0) * Fraction(gamma) ** p * 256
        out.append(round(x))  # Fraction.__round__ rounds half to even
    if zero_lowest:
        out[K - 1] = 0
    return out


class Request:
    __slots__ = ("st", "tier", "len", "rem", "seq", "tarr", "admitted", "migrating")

    def __init__(self, st, tier, length, rem, seq, tarr, admitted=0, migrating=0):
        self.st, self.tier, self.len, self.rem = st, tier, length, rem
        self.seq, self.tarr, self.admitted, self.migrating = seq, tarr, admitted, migrating

    def copy(self):
        return Request(self.st, self.tier, self.len, self.rem, self.seq, self.tarr,
                       self.admitted, self.migrating)


class ExactSim:
    def __init__(self, cfg, K):
        self.cfg = cfg
        self.I, self.S = cfg["n_instances"], cfg["slots_per_instance"]
        self.M, self.blk = cfg["kv_blocks"], cfg["block_tokens"]
        self.K = K
        self.Hint = exact_headroom(cfg["headroom_base"], cfg["headroom_decay"], K, cfg["zero_lowest_tier"])
        self.H = [Fraction(h, 256) for h in self.Hint]
        self.adapt = cfg.get("adaptive") or {}
        self.promo = cfg.get("promotion") or {}
        self.epoch_mark = 0  # first entry of the latency log since the last headroom update
        self.theta = Fraction(cfg["theta_num"], cfg["theta_den"])
        self.slots = [[None] * self.S for _ in range(self.I)]
        self.free = [self.M] * self.I
        self.mig = [None] * self.I  # per source: [dst, src_slot, dst_slot, copied]
        self.drain = [0] * self.I
        self.next_seq = 0
        self.stats = [0] * NSTAT
        # every request's (tier, queue delay) at its first admission and
        # (tier, end-to-end time) at its finish, in ticks
        self.latencies = ([], [])
        d = cfg.get("dispatch", {"policy": "llumnix"})
        self.infaas = d["policy"] == "infaas"
        self.dsp = d
        self.svc = [0] * self.I  # INFaaS service-time estimate, 1/256 tick
        self.blind = bool(cfg.get("tier_blind"))
        self.t = 0

    # -- helpers --------------------------------------------------------
    def blocks(self, n):
        return -(-n // self.blk)

    def requests(self, i, st):
        return [(s, r) for s, r in enumerate(self.slots[i]) if r is not None and r.st == st]

    def rank(self, tier):
        """What a tier counts for in an ordering."""
        return 0 if self.blind else tier

    def hol(self, i):
        w = self.requests(i, WAITING)
        return min(w, key=lambda sr: (self.rank(sr[1].tier), sr[1].seq))[0] if w else None

    def lowest_empty(self, i):
        for s, r in enumerate(self.slots[i]):
            if r is None:
                return s
        return None

    def freeness(self, i):
        """Eq. 1 with V(r) of Eq. 2 summed request by request."""
        running = self.requests(i, RUNNING)
        n_tier = {}
        for _, r in running:
            n_tier[r.tier] = n_tier.get(r.tier, 0) + 1
        V = Fraction(0)
        for _, r in running:
            V += self.blocks(r.len) + self.H[r.tier] / n_tier[r.tier]
        h = self.hol(i)
        if h is not None:
            V += self.blocks(self.slots[i][h].len)
        for m in self.mig:
            if m is not None and m[0] == i:
                V += m[3]
        return (self.M - V) / max(len(running), 1)

    def freeness_normal(self, i):
        """Eq. 1 without headroom: physical usage and head-of-line demand only."""
        running = self.requests(i, RUNNING)
        V = sum(self.blocks(r.len) for _, r in running)
        h = self.hol(i)
        if h is not None:
            V += self.blocks(self.slots[i][h].len)
        for m in self.mig:
            if m is not None and m[0] == i:
                V += m[3]
        return Fraction(self.M - V, max(len(running), 1))

    def full_freeness(self, i):
        return -math.inf if self.drain[i] else self.freeness(i)

    def autoscale(self):
        total = sum(math.floor(self.freeness_normal(i) * 2**20) for i in range(self.I))
        if total < -self.I * 2**19:
            return -1, total
        if total > 3 * self.I * 2**19:
            return 1, total
        return 0, total

    # -- the tick ---------------------------------------------------------
    def promote(self, t):
        period = self.promo.get("period", 0)
        if not period or t % period:
            return
        age = list(self.promo["age"]) + [0] * 10
        for i in range(self.I):
            for _, r in self.requests(i, WAITING):
                if r.tier >= 1 and age[r.tier] and t - r.tarr >= age[r.tier]:
                    r.tier -= 1

    def adapt_headroom(self, t):
        epoch = self.adapt.get("epoch", 0)
        if not epoch or t % epoch:
            return
        fresh = self.latencies[0][self.epoch_mark:]
        self.epoch_mark = len(self.latencies[0])
        ad = self.adapt
        slo = list(ad["slo"])
        for p in range(self.K):
            if self.cfg["zero_lowest_tier"] and p == self.K - 1:
                continue
            lat = [v for tier, v in fresh if tier == p]
            if not lat:
                continue
            mean = Fraction(sum(lat), len(lat))
            target = slo[min(p, len(slo) - 1)]
            h = self.Hint[p]
            if mean > target:
                h = min(h + ad["step_up"], ad["max"])
            elif mean <= Fraction(ad["margin"] * target, 256):
                h = max(h - ad["step_down"], 0)
            self.Hint[p] = h
            self.H[p] = Fraction(h, 256)

    def tick(self, arrivals):
        t = self.t
        st = self.stats
        self.promote(t)
        self.adapt_headroom(t)
        aborted = set()
        finished = [[] for _ in range(self.I)]  # end-to-end ticks of this tick's finishes
        interfered = set()
        # A: decode, growth, preemption, finish
        for i in range(self.I):
            row = self.slots[i]
            need = sum(1 for _, r in self.requests(i, RUNNING) if r.len % self.blk == 0)
            while need > self.free[i]:
                run = self.requests(i, RUNNING)
                v, rv = max(run, key=lambda sr: (self.rank(sr[1].tier), sr[1].seq))
                if rv.migrating:
                    rv.migrating = 0
                    aborted.add(i)
                self.free[i] += self.blocks(rv.len)
                if rv.len % self.blk == 0:
                    need -= 1
                rv.st = WAITING
                st[rv.tier * 8 + F_PREEMPTED] += 1
                interfered.add(i)
            self.free[i] -= need
            for s, r in self.requests(i, RUNNING):
                r.len += 1
                r.rem -= 1
                if r.rem == 0:
                    self.free[i] += self.blocks(r.len)
                    st[r.tier * 8 + F_FINISHED] += 1
                    st[r.tier * 8 + F_E2E] += t - r.tarr
                    self.latencies[1].append((r.tier, t - r.tarr))
                    finished[i].append(t - r.tarr)
                    if r.migrating:
                        aborted.add(i)
                    row[s] = None
        # A2: release reservations of aborted migrations
        for i in sorted(aborted):
            dst, _, ds, copied = self.mig[i]
            self.free[dst] += copied
            self.slots[dst][ds] = None
            self.mig[i] = None
            st[MIG_ABORTED] += 1
        # B: admission
        for i in range(self.I):
            while True:
                h = self.hol(i)
                if h is None:
                    break
                r = self.slots[i][h]
                if self.blocks(r.len) > self.free[i]:
                    break
                self.free[i] -= self.blocks(r.len)
                r.st = RUNNING
                if not r.admitted:
                    r.admitted = 1
                    st[r.tier * 8 + F_ADMITTED] += 1
                    st[r.tier * 8 + F_QDELAY] += t - r.tarr
                    self.latencies[0].append((r.tier, t - r.tarr))
        # INFaaS: estimates from this tick's finishes, states after admission
        if self.infaas:
            for i in range(self.I):
                if finished[i]:
                    mean = 256 * sum(finished[i]) // len(finished[i])
                    self.svc[i] += (mean - self.svc[i]) // 2 ** self.dsp["ewma_shift"]
            penalty = {}
            for i in range(self.I):
                h = self.hol(i)
                if h is not None and self.blocks(self.slots[i][h].len) > self.free[i]:
                    penalty[i] = self.dsp["pen_overloaded"]
                elif i in interfered:
                    penalty[i] = self.dsp["pen_interfered"]
                else:
                    penalty[i] = 0
        # C': auto-scaling signal
        sig, _ = self.autoscale()
        if sig < 0:
            st[SCALE_OUT] += 1
        elif sig > 0:
            st[SCALE_IN] += 1
        # D: dispatch in (tier, seq) order to the freest instance with room
        seq0 = self.next_seq
        self.next_seq += len(arrivals)
        for tier, _, _ in arrivals:
            st[tier * 8 + F_ARRIVED] += 1
        order = sorted(range(len(arrivals)), key=lambda k: (self.rank(arrivals[k][0]), k))
        for k in order:
            tier, prompt, out = arrivals[k]
            room = [i for i in range(self.I) if self.lowest_empty(i) is not None]
            if not room:
                st[tier * 8 + F_REJECTED] += 1
                continue
            cands = [i for i in room if not self.drain[i]]
            if not cands:
                cands = room  # all draining: the least loaded one
                st[DRAIN_FALLBACK] += 1
            if self.infaas:
                d = self.dsp
                cost = {j: d["alpha"] * 256 * len(self.requests(j, WAITING)) + d["beta"] * self.svc[j]
                        + d["gamma"] * 256 * penalty[j] for j in cands}
                low = min(cost.values())
                i = min(j for j in cands if cost[j] == low)
            else:
                F = {i: self.freeness(i) for i in cands}
                best = max(F.values())
                i = min(j for j in cands if F[j] == best)
            self.slots[i][self.lowest_empty(i)] = Request(WAITING, tier, prompt, out, seq0 + k, t)
            st[tier * 8 + F_DISPATCHED] += 1
        # E1: staged copies
        for i in range(self.I):
            m = self.mig[i]
            if m is None:
                continue
            dst, ss, ds, copied = m
            r = self.slots[i][ss]
            b = self.blocks(r.len)
            w = min(self.cfg["mig_stage_blocks"], b - copied)
            if w > self.free[dst]:
                self.free[dst] += copied
                self.slots[dst][ds] = None
                r.migrating = 0
                st[MIG_ABORTED] += 1
                self.mig[i] = None
                continue
            self.free[dst] -= w
            m[3] += w
            if m[3] == b:
                moved = r.copy()
                moved.st, moved.migrating = RUNNING, 0
                self.slots[dst][ds] = moved
                self.slots[i][ss] = None
                self.free[i] += b
                st[MIG_COMMITTED] += 1
                self.mig[i] = None
        # E2: pairing (INFaaS never migrates)
        if t % self.cfg["mig_interval"] == 0 and not self.infaas:
            busy = set()
            for i, m in enumerate(self.mig):
                if m is not None:
                    busy.add(i)
                    busy.add(m[0])
            L = [i for i in range(self.I) if i not in busy]
            F = {i: self.full_freeness(i) for i in L}
            L.sort(key=lambda i: (F[i], i))
            n = len(L)
            for k in range(n):
                if k >= self.cfg["mig_max_pairs"] or k >= n - 1 - k:
                    break
                src, dst = L[k], L[n - 1 - k]
                if self.drain[dst]:
                    break
                if F[src] >= 0 or F[dst] - F[src] < self.theta:
                    break
                ds = self.lowest_empty(dst)
                if ds is None:
                    continue
                h = self.hol(src)
                if h is not None:
                    self.slots[dst][ds] = self.slots[src][h]
                    self.slots[src][h] = None
                    st[MIG_QUEUED] += 1
                else:
                    run = [(s, r) for s, r in self.requests(src, RUNNING) if not r.migrating]
                    if not run:  # an empty draining source: nothing to move
                        continue
                    c, rc = max(run, key=lambda sr: (self.rank(sr[1].tier), -self.blocks(sr[1].len), sr[1].seq))
                    self.slots[dst][ds] = Request(INBOUND, 0, 0, 0, 0, 0)
                    rc.migrating = 1
                    self.mig[src] = [dst, c, ds, 0]
                    st[MIG_STARTED] += 1
        # stats
        for i in range(self.I):
            st[RUN_TICKS] += len(self.requests(i, RUNNING))
            st[WAIT_TICKS] += len(self.requests(i, WAITING))
        st[TICKS] += 1
        self.t += 1

    # -- canonical state ------------------------------------------------
    def export(self):
        import numpy as np
        IS = self.I * self.S
        meta = np.zeros(IS, np.uint8)
        lr = np.zeros(IS, np.uint32)
        seq = np.zeros(IS, np.uint32)
        tarr = np.zeros(IS, np.uint32)
        for i in range(self.I):
            for s, r in enumerate(self.slots[i]):
                if r is None:
                    continue
                o = i * self.S + s
                meta[o] = r.st | r.tier << 2 | r.admitted << 6 | r.migrating << 7
                lr[o] = r.len | r.rem << 16
                seq[o] = r.seq
                tarr[o] = r.tarr
        mig = np.zeros(self.I * 4, np.int32)
        for i, m in enumerate(self.mig):
            mig[4 * i:4 * i + 4] = m if m is not None else [-1, 0, 0, 0]
        return dict(meta=meta, lr=lr, seq=seq, tarr=tarr,
                    free=np.array(self.free, np.int32), mig=mig,
                    next_seq=np.array([self.next_seq], np.uint32),
                    stats=np.array(self.stats, np.uint64), drain=np.array(self.drain, np.uint8),
                    svc=np.array(self.svc, np.int64),
                    hq=np.array(self.Hint + [0] * (10 - self.K), np.int32))
