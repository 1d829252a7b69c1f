/*
 * mts_oracle.c -- plain, slow, single-threaded CPU oracle for the multi-tier
 * Llumnix scheduling step.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this file's library.  It shares no
 * code, header, table builder or constant with the HIP library; the two are
 * compared element by element.
 *
 * What it computes (per replica, per tick t; replicas are independent):
 *   A  decode: one token per running request, KV-block growth, preemption
 *      under memory pressure, finish.  (Section 2.1 block-based KV cache;
 *      Section 2.2 preemption; Section 3.1 Llumlet block-level KV management)
 *   A2 release of migration reservations whose source request was preempted
 *      or finished in A.  (Section 3.5)
 *   B  admission of the head-of-line request while its blocks fit.
 *      (Section 3.1 priority-ordered queue; Eq. 2 head-of-line demand)
 *   C  freeness F = (M - sum_r V(r)) / B.  (Eq. 1, Eq. 2, Eq. 3, Eq. 4)
 *   D  arrival sampling and tier-ordered dispatch to argmax F.  (Section 3.4)
 *   E  migration: staged copies, then pairing of low-F sources with high-F
 *      destinations.  (Section 3.5, Fig. 4)
 * Draining (Section 3.5, last paragraph; Section 3.4): a draining instance
 * carries an infinite-virtual-usage sentinel, so its full freeness is minus
 * infinity: it receives no dispatch while another instance can take the
 * request, it is the first migration source and never a destination; when
 * every instance with a free slot is draining, dispatch falls back to the
 * least loaded of them (largest freeness without the sentinel).
 * Latency histograms (the per-tier latency distributions of Section 5.1,
 * in ticks): each request's queue delay (arrival to first admission, the
 * scheduler's share of the time to first token) and end-to-end time
 * (arrival to the tick of its last token) is counted per tier in a
 * log-linear histogram: values 0..15 have a bin each; a larger value v with
 * 2^e <= v < 2^(e+1) falls into one of eight equal sub-ranges of that
 * octave, bin 16 + 8 (e - 4) + (floor(v / 2^(e-3)) - 8), up to bin 239.
 * INFaaS-style dispatch (Section 3.7), the paper's comparison policy, as an
 * alternative global scheduler: each arrival goes to the instance with the
 * smallest cost alpha * q + beta * s + gamma * penalty, where q is the
 * instance's queue depth (waiting requests, updated after every placement),
 * s an exponentially weighted moving average of the end-to-end time of the
 * requests that finished on it (updated once per tick, after admission,
 * from that tick's finishes), and penalty the state penalty: OVERLOADED when
 * its head of line does not fit its free blocks after admission, else
 * INTERFERED when it preempted a request in this tick, else ACTIVE (0).  It
 * keeps no freeness for dispatch and never migrates.
 * Tier-blind scheduling (the priority-blind vLLM local scheduler the paper
 * pairs with INFaaS, Section 5.3): when set, tiers no longer order anything
 * -- arrivals are dispatched in arrival order, each instance's queue is
 * served first come first served, preemption takes the newest running
 * request and the migration candidate is chosen by size and age alone --
 * while tiers still label requests in the counters and histograms and still
 * enter the headroom of Eq. 4.
 * Auto-scaling (Section 3.6): every tick, after admission, the cluster
 * average of the normal-priority freeness F_normal (Eq. 1 without headroom)
 * is compared with the scale-out (-0.5) and scale-in (1.5) thresholds; the
 * ticks that signal either are counted.
 * Adaptive headroom and multilevel-feedback promotion (Section 6.5, future
 * work the paper leaves unspecified; the readings below are this oracle's):
 *   - every adapt_epoch ticks each tier's headroom H_p moves up by a step
 *     when the mean queue delay of the tier's requests first admitted since
 *     the previous update exceeds the tier's target, down by a step when that
 *     mean is at most a margin fraction of the target (the headroom went
 *     unused), within [0, adapt_max];
 *   - every promote_period ticks each waiting request of tier p >= 1 whose
 *     age since arrival has reached the tier's quota moves up to tier p - 1.
 * Every quantity is an integer.  The headroom H_p is quantised to 1/256 block
 * and freeness values are compared by exact 64-bit cross-multiplication.
 *
 * Random draws: Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC 2011), keyed by (seed, global replica id),
 * turned into samples through 32-bit inverse-CDF tables built here in double
 * precision.
 *
 * Parity pins live in the test suite (printed values of Fig. 2 and Fig. 3,
 * the Eq. 4 indicator statement, K=1 load balancing, K=2 binary headroom,
 * exhaustive search on tiny inputs, conservation invariants, sampling
 * moments, Philox against an independent library).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_MAX_TIERS 10
#define OR_NSTAT 96
#define OR_TABLE_CAP (1u << 17)
#define OR_HBINS 240
enum { H_QDELAY = 0, H_E2E = 1 };

/* per-tier counters: stats[tier * 8 + field] */
enum { F_ARRIVED = 0, F_REJECTED, F_DISPATCHED, F_ADMITTED, F_FINISHED,
       F_PREEMPTED, F_QDELAY, F_E2E };
/* replica-wide counters */
enum { S_MIG_QUEUED = 80, S_MIG_STARTED, S_MIG_COMMITTED, S_MIG_ABORTED,
       S_RUN_SLOT_TICKS, S_WAIT_SLOT_TICKS, S_INVARIANT, S_TICKS,
       S_SCALE_OUT, S_SCALE_IN, S_DRAIN_FALLBACK };

enum { ST_EMPTY = 0, ST_WAITING = 1, ST_RUNNING = 2, ST_INBOUND = 3 };

enum { TIER_UNIFORM = 0, TIER_GAUSS = 1, TIER_GEOMETRIC = 2, TIER_EXPLICIT = 3 };
enum { ARR_POISSON = 0, ARR_GAMMA_POISSON = 1 };
enum { PROMPT_UNIFORM_INT = 0, PROMPT_LOGNORMAL = 1 };
enum { OUT_GEOMETRIC = 0, OUT_PARETO = 1 };

typedef struct {
    uint32_t n_replicas, K;
    int32_t kind;
    int32_t pad;
    double a, b;                 /* gauss: mu, sigma; geometric: r */
    double probs[OR_MAX_TIERS];  /* explicit */
} or_group;

typedef struct {
    uint32_t n_instances, slots, kv_blocks, block_tokens;
    double h0, gamma;
    uint32_t zero_lowest, mig_interval, mig_stage, mig_max_pairs;
    int32_t theta_num, theta_den;
    int32_t arr_kind, prompt_kind, out_kind, pad;
    double arr_mean, arr_cv;
    double prompt_mu, prompt_sigma;
    uint32_t prompt_lo, prompt_hi;
    double out_a;                /* geometric: mean; pareto: alpha */
    uint32_t out_min, out_cap;   /* pareto */
    uint64_t seed, replica_id_base;
    uint32_t n_groups, pad2;
    const or_group *groups;
    /* global policy: 0 Llumnix freeness, 1 INFaaS cost */
    uint32_t policy, ewma_shift;
    int32_t alpha, beta, gamma_w;
    uint32_t pen_over, pen_intf;
    uint32_t tier_blind;         /* 1: tiers order nothing (priority-blind local scheduler) */
    /* adaptive headroom: 0 epoch keeps Eq. 3's static table */
    uint32_t adapt_epoch, adapt_up, adapt_down, adapt_max, adapt_margin;
    uint32_t adapt_slo[OR_MAX_TIERS];     /* mean queue-delay target per tier, ticks */
    /* promotion: 0 period promotes nothing; promote_age[p] = 0 never promotes tier p */
    uint32_t promote_period;
    uint32_t promote_age[OR_MAX_TIERS];
} or_cfg;

enum { POLICY_LLUMNIX = 0, POLICY_INFAAS = 1 };

typedef struct {
    uint8_t st, tier, admitted, migrating;
    uint32_t len, rem, seq, tarr;
} slot_t;

/* one record per source instance; dst < 0 means no migration */
typedef struct { int32_t dst, src_slot, dst_slot, copied; } mig_t;

typedef struct {
    uint64_t *q;      /* q[j] = floor(2^32 * CDF(base + j)); last entry 2^32 */
    uint32_t n, base;
} table_t;

typedef struct {
    uint64_t gid;
    uint32_t group;
    slot_t *slot;     /* [I][S] */
    int64_t *freeb;   /* [I] free KV blocks */
    mig_t *mig;       /* [I] */
    uint8_t *drain;   /* [I] 1: the instance is draining */
    int64_t *svc;     /* [I] INFaaS service-time estimate, 1/256 tick */
    uint64_t *fsum;   /* [I] end-to-end ticks of this tick's finishes */
    uint32_t *fcnt;   /* [I] number of this tick's finishes */
    uint8_t *intf;    /* [I] preempted a request in this tick */
    uint32_t next_seq;
    int32_t hq[OR_MAX_TIERS];           /* headroom H_p in 1/256 block (Eq. 3, then adapted) */
    uint64_t snap_adm[OR_MAX_TIERS];    /* admitted / queue-delay counters at the last update */
    uint64_t snap_qd[OR_MAX_TIERS];
    uint64_t stats[OR_NSTAT];
    uint32_t (*hist)[OR_MAX_TIERS][OR_HBINS];  /* [2]: queue delay, end-to-end */
    uint32_t n_arr, cap_arr;
    uint32_t *arr;    /* last tick's arrivals in sampling order: tier, prompt, out */
} replica_t;

typedef struct or_ctx {
    or_cfg cfg;
    or_group *groups;
    uint32_t I, S, r_begin, r_count;
    uint64_t tick;
    int check;
    int32_t (*Hq)[OR_MAX_TIERS];
    table_t *tier_tab;
    table_t count_tab, prompt_tab, out_tab;
    replica_t *rep;
} or_ctx;

/* ------------------------------------------------------------------ */
/* Random numbers: Philox4x64-10 from its published definition.        */
/* ------------------------------------------------------------------ */
static void mulhilo64(uint64_t a, uint64_t b, uint64_t *hi, uint64_t *lo)
{
    unsigned __int128 p = (unsigned __int128)a * (unsigned __int128)b;
    *hi = (uint64_t)(p >> 64);
    *lo = (uint64_t)p;
}

void or_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t hi0, lo0, hi1, lo1;
        mulhilo64(0xD2E7470EE14C6C93ULL, x0, &hi0, &lo0);
        mulhilo64(0xCA5A826395121157ULL, x2, &hi1, &lo1);
        uint64_t n0 = hi1 ^ x1 ^ k0, n1 = lo1, n2 = hi0 ^ x3 ^ k1, n3 = lo0;
        x0 = n0; x1 = n1; x2 = n2; x3 = n3;
        k0 += 0x9E3779B97F4A7C15ULL;  /* Weyl key schedule */
        k1 += 0xBB67AE8584CAA73BULL;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* ------------------------------------------------------------------ */
/* Inverse-CDF tables (all distribution math happens here, on the host) */
/* ------------------------------------------------------------------ */
static const double TWO32 = 4294967296.0;

/* standard normal CDF, Phi(z) = erfc(-z / sqrt 2) / 2 */
static double std_normal_cdf(double z) { return 0.5 * erfc(-z * 0.70710678118654752440); }

/* quantise a CDF value; the caller decides when the table ends */
static uint64_t quant(double c)
{
    if (!(c > 0.0)) return 0;
    double x = floor(c * TWO32);
    if (x >= TWO32) return (uint64_t)1 << 32;
    return (uint64_t)x;
}

/* a CDF value is "complete" when the remaining tail is below 2^-32 */
static int tail_done(double c) { return (1.0 - c) * TWO32 < 1.0; }

static int table_alloc(table_t *t, uint32_t cap)
{
    t->q = (uint64_t *)calloc(cap, sizeof(uint64_t));
    t->n = 0;
    return t->q ? 0 : -2;
}

/* Tier distributions, Section 4.2: uniform 1/K; Gaussian discretised at the
 * half-integers with both tails lumped into tiers 0 and K-1; enterprise as
 * P(k) proportional to r^(K-1-k); or explicit probabilities. */
static int build_tier_table(const or_group *g, table_t *t)
{
    uint32_t K = g->K;
    if (table_alloc(t, OR_MAX_TIERS)) return -2;
    t->base = 0;
    double w[OR_MAX_TIERS], total = 0.0, cum = 0.0;
    if (g->kind == TIER_GEOMETRIC) {
        w[K - 1] = 1.0;
        for (int j = (int)K - 2; j >= 0; --j) w[j] = w[j + 1] * g->a;
    } else if (g->kind == TIER_EXPLICIT) {
        for (uint32_t j = 0; j < K; ++j) w[j] = g->probs[j];
    }
    if (g->kind == TIER_GEOMETRIC || g->kind == TIER_EXPLICIT)
        for (uint32_t j = 0; j < K; ++j) total += w[j];
    for (uint32_t k = 0; k + 1 < K; ++k) {
        double c;
        switch (g->kind) {
        case TIER_UNIFORM: c = (double)(k + 1) / (double)K; break;
        case TIER_GAUSS: c = std_normal_cdf(((double)k + 0.5 - g->a) / g->b); break;
        default: cum += w[k]; c = cum / total; break;
        }
        t->q[k] = quant(c);
    }
    t->q[K - 1] = (uint64_t)1 << 32;
    t->n = K;
    return 0;
}

/* Per-tick arrival count: Poisson(mean) (Section 4.4), or a gamma-mixed
 * Poisson (negative binomial with shape 1/cv^2, scale mean*cv^2). */
static int build_count_table(const or_cfg *c, table_t *t)
{
    if (table_alloc(t, OR_TABLE_CAP)) return -2;
    t->base = 0;
    double p, cum, ratio = 0.0, shape = 0.0;
    if (c->arr_kind == ARR_POISSON) {
        p = exp(-c->arr_mean);
    } else {
        shape = 1.0 / (c->arr_cv * c->arr_cv);
        double scale = c->arr_mean * c->arr_cv * c->arr_cv;
        p = exp(-shape * log1p(scale));
        ratio = scale / (1.0 + scale);
    }
    cum = p;
    for (uint32_t n = 0;; ++n) {
        if (n > 0) {
            if (c->arr_kind == ARR_POISSON) p = p * c->arr_mean / (double)n;
            else p = p * (((double)n - 1.0 + shape) / (double)n) * ratio;
            cum += p;
        }
        if (tail_done(cum)) { t->q[n] = (uint64_t)1 << 32; t->n = n + 1; return 0; }
        if (n + 1 >= OR_TABLE_CAP) return -1;
        t->q[n] = quant(cum);
    }
}

/* Prompt length: uniform integers on [lo, hi], or a log-normal discretised
 * at the half-integers and clipped to [lo, hi] (tails lumped at the ends). */
static int build_prompt_table(const or_cfg *c, table_t *t)
{
    uint32_t lo = c->prompt_lo, hi = c->prompt_hi;
    if (hi < lo || hi - lo + 1 > OR_TABLE_CAP) return -1;
    if (table_alloc(t, hi - lo + 1)) return -2;
    t->base = lo;
    for (uint32_t n = lo;; ++n) {
        uint32_t j = n - lo;
        double cdf;
        if (c->prompt_kind == PROMPT_UNIFORM_INT)
            cdf = (double)(n - lo + 1) / (double)(hi - lo + 1);
        else
            cdf = std_normal_cdf((log((double)n + 0.5) - c->prompt_mu) / c->prompt_sigma);
        if (n == hi || tail_done(cdf)) { t->q[j] = (uint64_t)1 << 32; t->n = j + 1; return 0; }
        t->q[j] = quant(cdf);
    }
}

/* Output length: geometric on {1, 2, ...} with the given mean, or
 * min(floor(xmin * U^(-1/alpha)), cap) (Pareto, capped). */
static int build_output_table(const or_cfg *c, table_t *t)
{
    if (table_alloc(t, OR_TABLE_CAP)) return -2;
    if (c->out_kind == OUT_GEOMETRIC) {
        double q = 1.0 - 1.0 / c->out_a, surv = 1.0;
        t->base = 1;
        for (uint32_t n = 1;; ++n) {
            surv = surv * q;
            uint32_t j = n - 1;
            if (surv * TWO32 < 1.0) { t->q[j] = (uint64_t)1 << 32; t->n = j + 1; return 0; }
            if (j + 1 >= OR_TABLE_CAP) return -1;
            t->q[j] = quant(1.0 - surv);
        }
    } else {
        uint32_t lo = c->out_min, hi = c->out_cap;
        if (hi < lo || hi - lo + 1 > OR_TABLE_CAP) return -1;
        t->base = lo;
        for (uint32_t n = lo;; ++n) {
            uint32_t j = n - lo;
            double surv = pow((double)lo / ((double)n + 1.0), c->out_a);
            if (n == hi || surv * TWO32 < 1.0) { t->q[j] = (uint64_t)1 << 32; t->n = j + 1; return 0; }
            t->q[j] = quant(1.0 - surv);
        }
    }
}

/* smallest j with u < q[j] */
static uint32_t sample(const table_t *t, uint32_t u)
{
    uint32_t lo = 0, hi = t->n - 1;
    while (lo < hi) {
        uint32_t mid = lo + (hi - lo) / 2;
        if ((uint64_t)u < t->q[mid]) hi = mid; else lo = mid + 1;
    }
    return lo;
}

/* Eq. 3 with h0 = M * h_max and gamma = e^-lambda, in 1/256 block:
 * H_q[p] = round-half-even(256 * h0 * gamma^p), gamma^p by repeated
 * multiplication; the lowest tier gets none when zero_lowest is set. */
static void build_headroom(const or_cfg *c, uint32_t K, int32_t out[OR_MAX_TIERS])
{
    double base = c->h0 * 256.0, g = 1.0;
    for (uint32_t p = 0; p < OR_MAX_TIERS; ++p) {
        out[p] = p < K ? (int32_t)rint(base * g) : 0;
        g = g * c->gamma;
    }
    if (c->zero_lowest) out[K - 1] = 0;
}

/* ------------------------------------------------------------------ */
/* helpers                                                             */
/* ------------------------------------------------------------------ */
static uint32_t blocks(const or_ctx *x, uint32_t len)
{
    return (len + x->cfg.block_tokens - 1) / x->cfg.block_tokens;
}

static slot_t *inst_slots(const or_ctx *x, replica_t *rp, uint32_t i) { return rp->slot + (size_t)i * x->S; }

static int lowest_empty(const or_ctx *x, replica_t *rp, uint32_t i)
{
    slot_t *sl = inst_slots(x, rp, i);
    for (uint32_t s = 0; s < x->S; ++s) if (sl[s].st == ST_EMPTY) return (int)s;
    return -1;
}

/* head of line: the waiting request with the smallest (tier, seq) */
/* the rank a tier gives in every ordering: the tier itself, or 0 for all
 * when scheduling is tier-blind */
static uint32_t prio(const or_ctx *x, uint32_t tier) { return x->cfg.tier_blind ? 0 : tier; }

static int head_of_line(const or_ctx *x, replica_t *rp, uint32_t i)
{
    slot_t *sl = inst_slots(x, rp, i);
    int h = -1;
    for (uint32_t s = 0; s < x->S; ++s) {
        if (sl[s].st != ST_WAITING) continue;
        uint32_t ps = prio(x, sl[s].tier);
        if (h < 0 || ps < prio(x, sl[h].tier) || (ps == prio(x, sl[h].tier) && sl[s].seq < sl[h].seq)) h = (int)s;
    }
    return h;
}

static void clear_slot(slot_t *s) { memset(s, 0, sizeof(*s)); }

/* Freeness of instance i from its definition, Eq. 1: F = (M - sum_r V(r)) / B,
 * returned as num / (256 * den).  V(r) per Eq. 2: the head-of-line request
 * contributes its block demand, other queued requests nothing, a running
 * request its physical blocks plus headroom.  Headroom per Eq. 4: H_p once
 * for every tier p with at least one running request.  Blocks already copied
 * into an inbound reservation are physical usage of the destination.  B = 0
 * is read as B = 1. */
static void freeness(const or_ctx *x, replica_t *rp, uint32_t i, int64_t *num, int64_t *den)
{
    slot_t *sl = inst_slots(x, rp, i);
    int64_t phys = 0, running = 0;
    int present[OR_MAX_TIERS] = {0};
    for (uint32_t s = 0; s < x->S; ++s) {
        if (sl[s].st == ST_RUNNING) {
            phys += blocks(x, sl[s].len);
            running += 1;
            present[sl[s].tier] = 1;
        }
    }
    for (uint32_t j = 0; j < x->I; ++j)
        if (rp->mig[j].dst == (int32_t)i) phys += rp->mig[j].copied;
    int h = head_of_line(x, rp, i);
    int64_t demand = h >= 0 ? blocks(x, sl[h].len) : 0;
    int64_t v256 = 256 * (phys + demand);
    for (int p = 0; p < OR_MAX_TIERS; ++p)
        if (present[p]) v256 += rp->hq[p];
    *num = 256 * (int64_t)x->cfg.kv_blocks - v256;
    *den = running > 0 ? running : 1;
}

/* F_a > F_b, exact */
static int f_greater(int64_t na, int64_t da, int64_t nb, int64_t db) { return na * db > nb * da; }

/* Normal-priority freeness (Section 3.4): Eq. 1 with the virtual usage of
 * Eq. 2 but without any headroom term -- physical blocks of the running
 * requests, blocks copied into inbound reservations, the head of line's
 * demand.  num / (256 den) as for freeness(); the draining sentinel does not
 * enter it. */
static void freeness_normal(const or_ctx *x, replica_t *rp, uint32_t i, int64_t *num, int64_t *den)
{
    slot_t *sl = inst_slots(x, rp, i);
    int64_t phys = 0, running = 0;
    for (uint32_t s = 0; s < x->S; ++s) {
        if (sl[s].st == ST_RUNNING) {
            phys += blocks(x, sl[s].len);
            running += 1;
        }
    }
    for (uint32_t j = 0; j < x->I; ++j)
        if (rp->mig[j].dst == (int32_t)i) phys += rp->mig[j].copied;
    int h = head_of_line(x, rp, i);
    int64_t demand = h >= 0 ? blocks(x, sl[h].len) : 0;
    *num = 256 * ((int64_t)x->cfg.kv_blocks - phys - demand);
    *den = running > 0 ? running : 1;
}

/* floor(a / b) for b > 0 */
static int64_t floor_div(int64_t a, int64_t b)
{
    int64_t q = a / b;
    if (a % b != 0 && a < 0) q -= 1;
    return q;
}

/* Auto-scaling signal (Section 3.6) of the current state: the cluster
 * average of F_normal against -1/2 (scale out) and 3/2 (scale in).  Each
 * instance's F_normal = num / (256 den) enters in fixed point as
 * floor(F_normal * 2^20); the sum over the instances is exact.  Returns -1
 * (scale out), +1 (scale in) or 0; *sum receives the fixed-point sum. */
static int autoscale_signal(const or_ctx *x, replica_t *rp, int64_t *sum)
{
    int64_t acc = 0;
    for (uint32_t i = 0; i < x->I; ++i) {
        int64_t num, den;
        freeness_normal(x, rp, i, &num, &den);
        acc += floor_div(num * 4096, den);  /* num * 2^20 / (256 den) */
    }
    *sum = acc;
    const int64_t half = (int64_t)x->I << 19;  /* I * 2^20 / 2 */
    if (acc < -half) return -1;
    if (acc > 3 * half) return 1;
    return 0;
}

/* Histogram bin of a latency of v ticks: v itself below 16; above, the
 * octave [2^e, 2^(e+1)) is split into eight sub-ranges of width 2^(e-3). */
static uint32_t hist_bin(uint64_t v)
{
    if (v < 16) return (uint32_t)v;
    uint32_t e = 4;
    while (e < 63 && (v >> (e + 1)) != 0) e++;
    uint64_t sub = (v >> (e - 3)) - 8;  /* 0..7 */
    uint64_t b = 16 + 8 * (uint64_t)(e - 4) + sub;
    return b < OR_HBINS ? (uint32_t)b : OR_HBINS - 1;
}

static void hist_add(replica_t *rp, int which, uint32_t tier, uint64_t v)
{
    rp->hist[which][tier][hist_bin(v)]++;
}

/* ------------------------------------------------------------------ */
/* Phase A: decode one token per running request                      */
/* ------------------------------------------------------------------ */
static void phase_decode(or_ctx *x, replica_t *rp, uint64_t t, uint8_t *abort_pending)
{
    const uint32_t blk = x->cfg.block_tokens;
    for (uint32_t i = 0; i < x->I; ++i) {
        slot_t *sl = inst_slots(x, rp, i);
        /* requests whose next token starts a new block */
        int64_t grow = 0;
        for (uint32_t s = 0; s < x->S; ++s)
            if (sl[s].st == ST_RUNNING && sl[s].len % blk == 0) grow++;
        /* memory pressure: preempt the lowest-priority running request
         * (largest tier, then newest) until the growth fits; recompute
         * semantics -- the request keeps its tokens and goes back to the
         * queue without KV blocks */
        while (grow > rp->freeb[i]) {
            int v = -1;
            for (uint32_t s = 0; s < x->S; ++s) {
                if (sl[s].st != ST_RUNNING) continue;
                if (v < 0) { v = (int)s; continue; }
                uint32_t ps = prio(x, sl[s].tier), pv = prio(x, sl[v].tier);
                if (ps > pv || (ps == pv && sl[s].seq > sl[v].seq)) v = (int)s;
            }
            if (v < 0) break;  /* only reachable from an inconsistent imported state */
            if (sl[v].migrating) { sl[v].migrating = 0; abort_pending[i] = 1; }
            rp->freeb[i] += blocks(x, sl[v].len);
            if (sl[v].len % blk == 0) grow--;
            sl[v].st = ST_WAITING;
            rp->stats[sl[v].tier * 8 + F_PREEMPTED]++;
            rp->intf[i] = 1;
        }
        rp->freeb[i] -= grow;
        for (uint32_t s = 0; s < x->S; ++s) {
            if (sl[s].st != ST_RUNNING) continue;
            sl[s].len += 1;
            sl[s].rem -= 1;
            if (sl[s].rem == 0) {
                rp->freeb[i] += blocks(x, sl[s].len);
                rp->stats[sl[s].tier * 8 + F_FINISHED]++;
                rp->stats[sl[s].tier * 8 + F_E2E] += t - sl[s].tarr;
                hist_add(rp, H_E2E, sl[s].tier, t - sl[s].tarr);
                rp->fsum[i] += t - sl[s].tarr;
                rp->fcnt[i] += 1;
                if (sl[s].migrating) abort_pending[i] = 1;
                clear_slot(&sl[s]);
            }
        }
    }
}

/* Phase A2: a migration whose source request left the running state gives
 * its destination reservation back. */
static void phase_release(or_ctx *x, replica_t *rp, const uint8_t *abort_pending)
{
    for (uint32_t i = 0; i < x->I; ++i) {
        if (!abort_pending[i]) continue;
        mig_t *m = &rp->mig[i];
        if (m->dst < 0) continue;
        rp->freeb[m->dst] += m->copied;
        clear_slot(&inst_slots(x, rp, (uint32_t)m->dst)[m->dst_slot]);
        m->dst = -1; m->src_slot = 0; m->dst_slot = 0; m->copied = 0;
        rp->stats[S_MIG_ABORTED]++;
    }
}

/* Phase B: admit the head-of-line request while its blocks fit (strict
 * (tier, seq) order, head-of-line blocking). */
static void phase_admit(or_ctx *x, replica_t *rp, uint64_t t)
{
    for (uint32_t i = 0; i < x->I; ++i) {
        slot_t *sl = inst_slots(x, rp, i);
        for (;;) {
            int h = head_of_line(x, rp, i);
            if (h < 0) break;
            int64_t need = blocks(x, sl[h].len);
            if (need > rp->freeb[i]) break;
            rp->freeb[i] -= need;
            sl[h].st = ST_RUNNING;
            if (!sl[h].admitted) {
                sl[h].admitted = 1;
                rp->stats[sl[h].tier * 8 + F_ADMITTED]++;
                rp->stats[sl[h].tier * 8 + F_QDELAY] += t - sl[h].tarr;
                hist_add(rp, H_QDELAY, sl[h].tier, t - sl[h].tarr);
            }
        }
    }
}

/* floor(v / 2^k) */
static int64_t floor_shift(int64_t v, uint32_t k)
{
    int64_t d = (int64_t)1 << k;
    return floor_div(v, d);
}

/* INFaaS service-time estimate: once per tick, from the mean end-to-end
 * time of the requests that finished on the instance in this tick,
 * s += (256 * sum / count - s) / 2^shift, both divisions rounded down. */
static void infaas_update_estimates(const or_ctx *x, replica_t *rp)
{
    for (uint32_t i = 0; i < x->I; ++i) {
        if (rp->fcnt[i] == 0) continue;
        int64_t mean = (int64_t)((rp->fsum[i] * 256) / rp->fcnt[i]);
        rp->svc[i] += floor_shift(mean - rp->svc[i], x->cfg.ewma_shift);
    }
}

/* the INFaaS state penalty of instance i in ticks: OVERLOADED (head of line
 * does not fit the free blocks) before INTERFERED (preempted this tick) */
static int64_t infaas_penalty(const or_ctx *x, replica_t *rp, uint32_t i)
{
    int h = head_of_line(x, rp, i);
    if (h >= 0 && (int64_t)blocks(x, inst_slots(x, rp, i)[h].len) > rp->freeb[i]) return x->cfg.pen_over;
    if (rp->intf[i]) return x->cfg.pen_intf;
    return 0;
}

static int64_t waiting_count(const or_ctx *x, replica_t *rp, uint32_t i)
{
    slot_t *sl = inst_slots(x, rp, i);
    int64_t q = 0;
    for (uint32_t s = 0; s < x->S; ++s) q += sl[s].st == ST_WAITING;
    return q;
}

/* cost in 1/256 tick: alpha * q + beta * s + gamma * penalty */
static int64_t infaas_cost(const or_ctx *x, replica_t *rp, uint32_t i, int64_t pen)
{
    return (int64_t)x->cfg.alpha * waiting_count(x, rp, i) * 256 + (int64_t)x->cfg.beta * rp->svc[i] +
           (int64_t)x->cfg.gamma_w * pen * 256;
}

/* ------------------------------------------------------------------ */
/* Phase D: sample this tick's arrivals, dispatch in tier order        */
/* ------------------------------------------------------------------ */
static void phase_dispatch(or_ctx *x, replica_t *rp, uint64_t t)
{
    const uint32_t K = x->groups[rp->group].K;
    uint64_t key[2] = {x->cfg.seed, rp->gid};
    uint64_t ctr[4] = {t, 0, 0, 0}, r[4];
    or_philox4x64_10(ctr, key, r);
    uint32_t n = x->count_tab.base + sample(&x->count_tab, (uint32_t)r[0]);
    if (n > rp->cap_arr) {
        rp->cap_arr = n;
        rp->arr = (uint32_t *)realloc(rp->arr, (size_t)n * 3 * sizeof(uint32_t));
    }
    rp->n_arr = n;
    for (uint32_t k = 0; k < n; ++k) {
        uint64_t c2[4] = {t, k, 1, 0};
        or_philox4x64_10(c2, key, r);
        uint32_t *a = rp->arr + 3 * (size_t)k;
        a[0] = x->tier_tab[rp->group].base + sample(&x->tier_tab[rp->group], (uint32_t)r[0]);
        a[1] = x->prompt_tab.base + sample(&x->prompt_tab, (uint32_t)r[1]);
        a[2] = x->out_tab.base + sample(&x->out_tab, (uint32_t)r[2]);
        rp->stats[a[0] * 8 + F_ARRIVED]++;
    }
    uint32_t seq0 = rp->next_seq;
    rp->next_seq += n;

    int64_t *num = (int64_t *)malloc(x->I * sizeof(int64_t));
    int64_t *den = (int64_t *)malloc(x->I * sizeof(int64_t));
    int64_t *nempty = (int64_t *)malloc(x->I * sizeof(int64_t));
    int64_t *pen = (int64_t *)malloc(x->I * sizeof(int64_t));
    const int infaas = x->cfg.policy == POLICY_INFAAS;
    for (uint32_t i = 0; i < x->I; ++i) {
        /* INFaaS states are taken once per tick, before dispatch */
        pen[i] = infaas ? infaas_penalty(x, rp, i) : 0;
        freeness(x, rp, i, &num[i], &den[i]);
        nempty[i] = 0;
        slot_t *sl = inst_slots(x, rp, i);
        for (uint32_t s = 0; s < x->S; ++s) nempty[i] += sl[s].st == ST_EMPTY;
    }
    /* strict tier order (tier 0 first), FCFS within a tier; arrival order
     * when tier-blind */
    for (uint32_t p = 0; p < (x->cfg.tier_blind ? 1 : K); ++p) {
        for (uint32_t k = 0; k < n; ++k) {
            const uint32_t *a = rp->arr + 3 * (size_t)k;
            if (prio(x, a[0]) != p) continue;
            int best = -1, fallback = 0;
            if (infaas) {
                /* argmin cost over the non-draining instances with a free
                 * slot, else over every instance with a free slot */
                for (int pass = 0; pass < 2 && best < 0; ++pass) {
                    int64_t bc = 0;
                    for (uint32_t i = 0; i < x->I; ++i) {
                        if (nempty[i] == 0 || (pass == 0 && rp->drain[i])) continue;
                        int64_t c = infaas_cost(x, rp, i, pen[i]);
                        if (best < 0 || c < bc) { best = (int)i; bc = c; }
                    }
                    fallback = pass == 1 && best >= 0;
                }
            } else {
                /* argmax F over the instances with a free slot; a draining
                 * instance's F is minus infinity */
                for (uint32_t i = 0; i < x->I; ++i) {
                    if (nempty[i] == 0 || rp->drain[i]) continue;
                    if (best < 0 || f_greater(num[i], den[i], num[best], den[best])) best = (int)i;
                }
                if (best < 0) {
                    /* every instance that can take the request is draining: the
                     * least loaded of them, by freeness without the sentinel */
                    for (uint32_t j = 0; j < x->I; ++j) {
                        if (nempty[j] == 0) continue;
                        if (best < 0 || f_greater(num[j], den[j], num[best], den[best])) best = (int)j;
                    }
                    fallback = best >= 0;
                }
            }
            if (best < 0) { rp->stats[a[0] * 8 + F_REJECTED]++; continue; }
            if (fallback) rp->stats[S_DRAIN_FALLBACK]++;
            int s = lowest_empty(x, rp, (uint32_t)best);
            slot_t *sl = &inst_slots(x, rp, (uint32_t)best)[s];
            sl->st = ST_WAITING; sl->tier = (uint8_t)a[0]; sl->admitted = 0; sl->migrating = 0;
            sl->len = a[1]; sl->rem = a[2]; sl->seq = seq0 + k; sl->tarr = (uint32_t)t;
            nempty[best]--;
            rp->stats[a[0] * 8 + F_DISPATCHED]++;
            freeness(x, rp, (uint32_t)best, &num[best], &den[best]);
        }
    }
    free(num); free(den); free(nempty); free(pen);
}

/* ------------------------------------------------------------------ */
/* Phase E: migration                                                  */
/* ------------------------------------------------------------------ */
static int in_migration(const or_ctx *x, const replica_t *rp, uint32_t i)
{
    if (rp->mig[i].dst >= 0) return 1;
    for (uint32_t j = 0; j < x->I; ++j) if (rp->mig[j].dst == (int32_t)i) return 1;
    return 0;
}

static void phase_migrate(or_ctx *x, replica_t *rp, uint64_t t)
{
    /* E1: every active migration copies one stage of up to B_stage blocks
     * into its destination; when all blocks of the (still decoding) request
     * are there, the request commits to the destination (Fig. 4).  A stage
     * that does not fit aborts the migration. */
    for (uint32_t i = 0; i < x->I; ++i) {
        mig_t *m = &rp->mig[i];
        if (m->dst < 0) continue;
        slot_t *src = &inst_slots(x, rp, i)[m->src_slot];
        slot_t *dst = &inst_slots(x, rp, (uint32_t)m->dst)[m->dst_slot];
        int64_t b = blocks(x, src->len);
        int64_t w = b - m->copied;
        if (w > (int64_t)x->cfg.mig_stage) w = x->cfg.mig_stage;
        if (w > rp->freeb[m->dst]) {
            rp->freeb[m->dst] += m->copied;
            clear_slot(dst);
            src->migrating = 0;
            rp->stats[S_MIG_ABORTED]++;
        } else {
            rp->freeb[m->dst] -= w;
            m->copied += (int32_t)w;
            if (m->copied < b) continue;
            *dst = *src;
            dst->st = ST_RUNNING; dst->migrating = 0;
            clear_slot(src);
            rp->freeb[i] += b;
            rp->stats[S_MIG_COMMITTED]++;
        }
        m->dst = -1; m->src_slot = 0; m->dst_slot = 0; m->copied = 0;
    }

    /* E2: on interval ticks, rank the instances not in a migration by F and
     * pair the k-th lowest (which must be overloaded, F < 0) with the k-th
     * highest while the freeness gap is at least theta.  The source gives
     * its head-of-line queued request if it has one (moved at once, no KV
     * state), else its lowest-priority running request with the smallest
     * KV footprint, which starts a staged copy. */
    if (t % x->cfg.mig_interval != 0 || x->cfg.policy == POLICY_INFAAS) return;
    uint32_t I = x->I, n = 0;
    uint32_t *L = (uint32_t *)malloc(I * sizeof(uint32_t));
    int64_t *num = (int64_t *)malloc(I * sizeof(int64_t));
    int64_t *den = (int64_t *)malloc(I * sizeof(int64_t));
    for (uint32_t i = 0; i < I; ++i) {
        freeness(x, rp, i, &num[i], &den[i]);
        if (!in_migration(x, rp, i)) L[n++] = i;
    }
    /* insertion sort by (F ascending, index ascending); a draining
     * instance's F is minus infinity, so draining instances come first */
    for (uint32_t a = 1; a < n; ++a) {
        uint32_t v = L[a];
        int b = (int)a - 1;
        for (; b >= 0; --b) {
            uint32_t u = L[b];
            int after = rp->drain[u] != rp->drain[v] ? !rp->drain[u]
                      : (!rp->drain[u] && f_greater(num[u], den[u], num[v], den[v]));
            if (!after) break;
            L[b + 1] = L[b];
        }
        L[b + 1] = v;
    }
    for (uint32_t k = 0; k < x->cfg.mig_max_pairs && k + 1 + k < n; ++k) {
        uint32_t src = L[k], dst = L[n - 1 - k];
        /* a draining destination means every instance left is draining */
        if (rp->drain[dst]) break;
        if (!rp->drain[src]) {
            /* a draining source has F = minus infinity: overloaded, and any
             * destination is more than theta freer */
            if (num[src] >= 0) break;
            /* F_dst - F_src >= theta_num / theta_den with F = num / (256 den) */
            __int128 lhs = (__int128)x->cfg.theta_den * ((__int128)num[dst] * den[src] - (__int128)num[src] * den[dst]);
            __int128 rhs = (__int128)x->cfg.theta_num * 256 * den[src] * den[dst];
            if (lhs < rhs) break;
        }
        int ds = lowest_empty(x, rp, dst);
        if (ds < 0) continue;
        slot_t *dsl = &inst_slots(x, rp, dst)[ds];
        int h = head_of_line(x, rp, src);
        if (h >= 0) {
            slot_t *ssl = &inst_slots(x, rp, src)[h];
            *dsl = *ssl;
            clear_slot(ssl);
            rp->stats[S_MIG_QUEUED]++;
        } else {
            slot_t *sl = inst_slots(x, rp, src);
            int c = -1;
            for (uint32_t s = 0; s < x->S; ++s) {
                if (sl[s].st != ST_RUNNING || sl[s].migrating) continue;
                if (c < 0) { c = (int)s; continue; }
                uint32_t bs = blocks(x, sl[s].len), bc = blocks(x, sl[c].len);
                uint32_t ps = prio(x, sl[s].tier), pc = prio(x, sl[c].tier);
                if (ps > pc || (ps == pc && (bs < bc || (bs == bc && sl[s].seq > sl[c].seq))))
                    c = (int)s;
            }
            /* nothing to move: only a draining source can be empty; its pair
             * is skipped like one with a full destination */
            if (c < 0) continue;
            clear_slot(dsl);
            dsl->st = ST_INBOUND;
            sl[c].migrating = 1;
            rp->mig[src].dst = (int32_t)dst; rp->mig[src].src_slot = c;
            rp->mig[src].dst_slot = ds; rp->mig[src].copied = 0;
            rp->stats[S_MIG_STARTED]++;
        }
    }
    free(L); free(num); free(den);
}

/* ------------------------------------------------------------------ */
/* invariants                                                          */
/* ------------------------------------------------------------------ */
static uint64_t check_invariants(const or_ctx *x, replica_t *rp)
{
    uint64_t bad = 0;
    uint32_t K = x->groups[rp->group].K;
    for (uint32_t i = 0; i < x->I; ++i) {
        slot_t *sl = inst_slots(x, rp, i);
        int64_t held = 0;
        int inbound_slots = 0;
        for (uint32_t s = 0; s < x->S; ++s) {
            if (sl[s].st == ST_RUNNING) held += blocks(x, sl[s].len);
            if (sl[s].st == ST_INBOUND) inbound_slots++;
            if (sl[s].st == ST_WAITING || sl[s].st == ST_RUNNING) {
                if (sl[s].tier >= K || sl[s].rem == 0 || sl[s].len == 0 || sl[s].len > 65535) bad++;
            }
            if (sl[s].migrating && sl[s].st != ST_RUNNING) bad++;
            if (sl[s].migrating && !(rp->mig[i].dst >= 0 && rp->mig[i].src_slot == (int32_t)s)) bad++;
        }
        int roles = 0, inbound_refs = 0;
        if (rp->mig[i].dst >= 0) roles++;
        for (uint32_t j = 0; j < x->I; ++j) {
            if (rp->mig[j].dst == (int32_t)i) {
                roles++; inbound_refs++;
                held += rp->mig[j].copied;
                if (sl[rp->mig[j].dst_slot].st != ST_INBOUND) bad++;
            }
        }
        if (roles > 1 || inbound_refs != inbound_slots) bad++;
        if (rp->mig[i].dst >= 0) {
            const mig_t *m = &rp->mig[i];
            if ((uint32_t)m->dst >= x->I || (uint32_t)m->dst == i) bad++;
            else {
                const slot_t *v = &sl[m->src_slot];
                if (v->st != ST_RUNNING || !v->migrating || m->copied < 0 || m->copied > (int32_t)blocks(x, v->len)) bad++;
            }
        }
        if (rp->freeb[i] < 0) bad++;
        if (rp->freeb[i] + held != (int64_t)x->cfg.kv_blocks) bad++;
    }
    return bad;
}

/* ------------------------------------------------------------------ */
/* Section 6.5 extensions, at the start of a tick                      */
/* ------------------------------------------------------------------ */
/* Adaptive headroom: at a tick t with t mod adapt_epoch = 0, tier p (every
 * tier but the lowest when zero_lowest is set) takes the a requests of tier p
 * first admitted since the previous update, with summed queue delay d:
 *   d > slo_p * a                     the mean delay misses the target:
 *                                     H_p = min(H_p + adapt_up, adapt_max)
 *   256 d <= adapt_margin * slo_p * a the target is met with margin, the
 *                                     headroom sat unused:
 *                                     H_p = max(H_p - adapt_down, 0)
 * and H_p stays otherwise, also when a = 0. */
static void adapt_headroom(const or_ctx *x, replica_t *rp, uint64_t t)
{
    const or_cfg *c = &x->cfg;
    if (c->adapt_epoch == 0 || t % c->adapt_epoch != 0) return;
    const uint32_t K = x->groups[rp->group].K;
    for (uint32_t p = 0; p < K; ++p) {
        const uint64_t adm = rp->stats[p * 8 + F_ADMITTED], qd = rp->stats[p * 8 + F_QDELAY];
        const unsigned __int128 a = adm - rp->snap_adm[p], d = qd - rp->snap_qd[p];
        rp->snap_adm[p] = adm;
        rp->snap_qd[p] = qd;
        if ((c->zero_lowest && p == K - 1) || a == 0) continue;
        const unsigned __int128 slo = c->adapt_slo[p];
        int64_t h = rp->hq[p];
        if (d > slo * a) h = h + c->adapt_up > c->adapt_max ? c->adapt_max : h + c->adapt_up;
        else if (256 * d <= c->adapt_margin * slo * a) h = h < c->adapt_down ? 0 : h - c->adapt_down;
        rp->hq[p] = (int32_t)h;
    }
}

/* Multilevel-feedback promotion: at a tick t with t mod promote_period = 0,
 * every waiting request of tier p >= 1 whose age t - tarr has reached
 * promote_age[p] (> 0) moves to tier p - 1; later counters and histograms
 * label it with the tier it holds then. */
static void promote_waiting(const or_ctx *x, replica_t *rp, uint64_t t)
{
    const or_cfg *c = &x->cfg;
    if (c->promote_period == 0 || t % c->promote_period != 0) return;
    for (size_t s = 0; s < (size_t)x->I * x->S; ++s) {
        slot_t *sl = &rp->slot[s];
        if (sl->st != ST_WAITING || sl->tier == 0) continue;
        const uint32_t age = (uint32_t)t - sl->tarr;
        if (c->promote_age[sl->tier] != 0 && age >= c->promote_age[sl->tier]) sl->tier -= 1;
    }
}

static void tick_replica(or_ctx *x, replica_t *rp, uint64_t t, uint8_t *abort_pending)
{
    promote_waiting(x, rp, t);
    adapt_headroom(x, rp, t);
    memset(abort_pending, 0, x->I);
    memset(rp->fsum, 0, x->I * sizeof(uint64_t));
    memset(rp->fcnt, 0, x->I * sizeof(uint32_t));
    memset(rp->intf, 0, x->I);
    phase_decode(x, rp, t, abort_pending);
    phase_release(x, rp, abort_pending);
    phase_admit(x, rp, t);
    if (x->cfg.policy == POLICY_INFAAS) infaas_update_estimates(x, rp);
    if (x->check) rp->stats[S_INVARIANT] += check_invariants(x, rp);
    int64_t fsum;
    int sig = autoscale_signal(x, rp, &fsum);
    if (sig < 0) rp->stats[S_SCALE_OUT]++;
    if (sig > 0) rp->stats[S_SCALE_IN]++;
    phase_dispatch(x, rp, t);
    phase_migrate(x, rp, t);
    uint64_t run = 0, wait = 0;
    for (size_t s = 0; s < (size_t)x->I * x->S; ++s) {
        run += rp->slot[s].st == ST_RUNNING;
        wait += rp->slot[s].st == ST_WAITING;
    }
    rp->stats[S_RUN_SLOT_TICKS] += run;
    rp->stats[S_WAIT_SLOT_TICKS] += wait;
    rp->stats[S_TICKS]++;
    if (x->check) rp->stats[S_INVARIANT] += check_invariants(x, rp);
}

/* ------------------------------------------------------------------ */
/* exported API (consumed by the test suite through ctypes)            */
/* ------------------------------------------------------------------ */
void or_destroy(or_ctx *x);

or_ctx *or_create(const or_cfg *cfg, uint32_t r_begin, uint32_t r_count, int check, int *err)
{
    *err = -1;
    if (!cfg || cfg->n_groups == 0 || !cfg->groups) return NULL;
    if (cfg->n_instances == 0 || cfg->n_instances > 256 || cfg->slots == 0) return NULL;
    if (cfg->block_tokens == 0 || cfg->kv_blocks == 0 || cfg->mig_interval == 0 || cfg->theta_den <= 0) return NULL;
    if (cfg->policy > POLICY_INFAAS || cfg->ewma_shift > 16 || cfg->tier_blind > 1) return NULL;
    if (cfg->adapt_margin > 256 || cfg->adapt_max > (1u << 29) / OR_MAX_TIERS) return NULL;
    uint32_t R = 0;
    for (uint32_t g = 0; g < cfg->n_groups; ++g) {
        if (cfg->groups[g].K == 0 || cfg->groups[g].K > OR_MAX_TIERS) return NULL;
        R += cfg->groups[g].n_replicas;
    }
    if (r_begin > R || r_count > R - r_begin) return NULL;

    or_ctx *x = (or_ctx *)calloc(1, sizeof(or_ctx));
    if (!x) { *err = -2; return NULL; }
    x->cfg = *cfg;
    x->groups = (or_group *)calloc(cfg->n_groups, sizeof(or_group));
    memcpy(x->groups, cfg->groups, cfg->n_groups * sizeof(or_group));
    x->cfg.groups = x->groups;
    x->I = cfg->n_instances; x->S = cfg->slots;
    x->r_begin = r_begin; x->r_count = r_count;
    x->check = check;
    x->Hq = calloc(cfg->n_groups, sizeof(*x->Hq));
    x->tier_tab = (table_t *)calloc(cfg->n_groups, sizeof(table_t));
    int rc = 0;
    for (uint32_t g = 0; g < cfg->n_groups && !rc; ++g) {
        build_headroom(cfg, cfg->groups[g].K, x->Hq[g]);
        rc = build_tier_table(&cfg->groups[g], &x->tier_tab[g]);
    }
    if (!rc && cfg->adapt_epoch) {
        if (cfg->adapt_epoch > (1u << 16)) rc = -1;
        for (uint32_t p = 0; p < OR_MAX_TIERS && !rc; ++p)
            if (cfg->adapt_slo[p] == 0 || cfg->adapt_slo[p] > (1u << 20)) rc = -1;
        for (uint32_t g = 0; g < cfg->n_groups && !rc; ++g)
            for (uint32_t p = 0; p < OR_MAX_TIERS; ++p)
                if ((uint32_t)x->Hq[g][p] > cfg->adapt_max) rc = -1;
    }
    if (!rc) rc = build_count_table(cfg, &x->count_tab);
    if (!rc) rc = build_prompt_table(cfg, &x->prompt_tab);
    if (!rc) rc = build_output_table(cfg, &x->out_tab);
    if (!rc) {
        uint64_t maxlen = (uint64_t)x->prompt_tab.base + x->prompt_tab.n - 1 +
                          (uint64_t)x->out_tab.base + x->out_tab.n - 1;
        if (maxlen > 65535) rc = -1;
    }
    if (rc) { *err = rc; or_destroy(x); return NULL; }

    x->rep = (replica_t *)calloc(r_count ? r_count : 1, sizeof(replica_t));
    for (uint32_t r = 0; r < r_count; ++r) {
        replica_t *rp = &x->rep[r];
        uint32_t gr = r_begin + r, g = 0, acc = 0;
        while (gr >= acc + cfg->groups[g].n_replicas) { acc += cfg->groups[g].n_replicas; ++g; }
        rp->gid = cfg->replica_id_base + gr;
        rp->group = g;
        rp->slot = (slot_t *)calloc((size_t)x->I * x->S, sizeof(slot_t));
        rp->freeb = (int64_t *)calloc(x->I, sizeof(int64_t));
        rp->mig = (mig_t *)calloc(x->I, sizeof(mig_t));
        rp->drain = (uint8_t *)calloc(x->I, 1);
        rp->hist = calloc(2, sizeof(*rp->hist));
        rp->svc = (int64_t *)calloc(x->I, sizeof(int64_t));
        rp->fsum = (uint64_t *)calloc(x->I, sizeof(uint64_t));
        rp->fcnt = (uint32_t *)calloc(x->I, sizeof(uint32_t));
        rp->intf = (uint8_t *)calloc(x->I, 1);
        if (!rp->slot || !rp->freeb || !rp->mig || !rp->drain || !rp->hist || !rp->svc || !rp->fsum || !rp->fcnt || !rp->intf) {
            *err = -2; or_destroy(x); return NULL;
        }
        for (uint32_t i = 0; i < x->I; ++i) { rp->freeb[i] = cfg->kv_blocks; rp->mig[i].dst = -1; }
        memcpy(rp->hq, x->Hq[g], sizeof(rp->hq));
    }
    *err = 0;
    return x;
}

void or_destroy(or_ctx *x)
{
    if (!x) return;
    if (x->rep)
        for (uint32_t r = 0; r < x->r_count; ++r) {
            free(x->rep[r].slot); free(x->rep[r].freeb); free(x->rep[r].mig); free(x->rep[r].arr);
            free(x->rep[r].drain); free(x->rep[r].hist);
            free(x->rep[r].svc); free(x->rep[r].fsum); free(x->rep[r].fcnt); free(x->rep[r].intf);
        }
    free(x->rep);
    if (x->tier_tab) for (uint32_t g = 0; g < x->cfg.n_groups; ++g) free(x->tier_tab[g].q);
    free(x->tier_tab);
    free(x->count_tab.q); free(x->prompt_tab.q); free(x->out_tab.q);
    free(x->Hq); free(x->groups); free(x);
}

/* advance every replica by n ticks */
void or_step(or_ctx *x, uint64_t n)
{
    uint8_t *ap = (uint8_t *)malloc(x->I);
    for (uint64_t k = 0; k < n; ++k) {
        for (uint32_t r = 0; r < x->r_count; ++r) tick_replica(x, &x->rep[r], x->tick, ap);
        x->tick++;
    }
    free(ap);
}

uint64_t or_tick_now(const or_ctx *x) { return x->tick; }
void or_set_tick(or_ctx *x, uint64_t t) { x->tick = t; }

/* canonical state export/import for replicas [r0, r0+nr) of this context.
 * meta = status | tier << 2 | admitted << 6 | migrating << 7
 * lr   = len | rem << 16
 * mig  = dst, src_slot, dst_slot, copied (dst = -1: none) */
int or_export(const or_ctx *x, uint32_t r0, uint32_t nr, uint8_t *meta, uint32_t *lr, uint32_t *seq,
              uint32_t *tarr, int32_t *freeb, int32_t *mig, uint32_t *next_seq, uint64_t *stats, uint8_t *drain)
{
    if (r0 > x->r_count || nr > x->r_count - r0) return -1;
    size_t IS = (size_t)x->I * x->S;
    for (uint32_t r = 0; r < nr; ++r) {
        const replica_t *rp = &x->rep[r0 + r];
        for (size_t s = 0; s < IS; ++s) {
            const slot_t *sl = &rp->slot[s];
            size_t o = (size_t)r * IS + s;
            meta[o] = (uint8_t)(sl->st | sl->tier << 2 | sl->admitted << 6 | sl->migrating << 7);
            lr[o] = sl->len | sl->rem << 16;
            seq[o] = sl->seq;
            tarr[o] = sl->tarr;
        }
        for (uint32_t i = 0; i < x->I; ++i) {
            freeb[(size_t)r * x->I + i] = (int32_t)rp->freeb[i];
            int32_t *m = mig + ((size_t)r * x->I + i) * 4;
            m[0] = rp->mig[i].dst; m[1] = rp->mig[i].src_slot; m[2] = rp->mig[i].dst_slot; m[3] = rp->mig[i].copied;
            drain[(size_t)r * x->I + i] = rp->drain[i];
        }
        next_seq[r] = rp->next_seq;
        memcpy(stats + (size_t)r * OR_NSTAT, rp->stats, sizeof(rp->stats));
    }
    return 0;
}

int or_import(or_ctx *x, uint32_t r0, uint32_t nr, const uint8_t *meta, const uint32_t *lr, const uint32_t *seq,
              const uint32_t *tarr, const int32_t *freeb, const int32_t *mig, const uint32_t *next_seq,
              const uint64_t *stats, const uint8_t *drain)
{
    if (r0 > x->r_count || nr > x->r_count - r0) return -1;
    size_t IS = (size_t)x->I * x->S;
    for (uint32_t r = 0; r < nr; ++r) {
        replica_t *rp = &x->rep[r0 + r];
        for (size_t s = 0; s < IS; ++s) {
            slot_t *sl = &rp->slot[s];
            size_t o = (size_t)r * IS + s;
            sl->st = meta[o] & 3; sl->tier = (meta[o] >> 2) & 15;
            sl->admitted = (meta[o] >> 6) & 1; sl->migrating = (meta[o] >> 7) & 1;
            sl->len = lr[o] & 0xFFFF; sl->rem = lr[o] >> 16;
            sl->seq = seq[o]; sl->tarr = tarr[o];
        }
        for (uint32_t i = 0; i < x->I; ++i) {
            rp->freeb[i] = freeb[(size_t)r * x->I + i];
            const int32_t *m = mig + ((size_t)r * x->I + i) * 4;
            rp->mig[i].dst = m[0]; rp->mig[i].src_slot = m[1]; rp->mig[i].dst_slot = m[2]; rp->mig[i].copied = m[3];
            rp->drain[i] = drain[(size_t)r * x->I + i] ? 1 : 0;
        }
        rp->next_seq = next_seq[r];
        memcpy(rp->stats, stats + (size_t)r * OR_NSTAT, sizeof(rp->stats));
    }
    return 0;
}

/* Order-independent digest of one replica's state: a wrapping sum of the
 * SplitMix64 finaliser (Steele, Lea, Flood, OOPSLA 2014) over the non-empty
 * slots and every instance record. */
static uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

void or_digest(const or_ctx *x, uint64_t *out)
{
    size_t IS = (size_t)x->I * x->S;
    for (uint32_t r = 0; r < x->r_count; ++r) {
        const replica_t *rp = &x->rep[r];
        uint64_t g = mix64(rp->gid), d = 0;
        for (size_t s = 0; s < IS; ++s) {
            const slot_t *sl = &rp->slot[s];
            if (sl->st == ST_EMPTY) continue;
            uint64_t meta = (uint64_t)(sl->st | sl->tier << 2 | sl->admitted << 6 | sl->migrating << 7);
            uint64_t a = (uint64_t)(sl->len | sl->rem << 16) | (uint64_t)sl->seq << 32;
            uint64_t b = (uint64_t)sl->tarr | meta << 32;
            uint64_t p = mix64(g + 2 * (uint64_t)s + 1);
            d += mix64(p ^ a) + mix64(p ^ b);
        }
        for (uint32_t i = 0; i < x->I; ++i) {
            const mig_t *m = &rp->mig[i];
            uint64_t p = mix64(g + 2 * ((uint64_t)IS + i) + 1);
            uint64_t c = (uint64_t)(uint32_t)rp->freeb[i] | (uint64_t)(uint32_t)m->dst << 32;
            uint64_t e = (uint64_t)(uint32_t)m->src_slot | (uint64_t)(uint32_t)m->dst_slot << 32;
            d += mix64(p ^ c) + mix64(p ^ e) + mix64(p ^ ((uint64_t)(uint32_t)m->copied | (uint64_t)rp->drain[i] << 32));
        }
        out[r] = d;
    }
}

/* tables, for comparison with the library's own (which: 0 tier of group g,
 * 1 count, 2 prompt, 3 output).  Returns the length, writes base. */
int or_table(const or_ctx *x, int which, uint32_t g, uint64_t *out, uint32_t cap, uint32_t *base)
{
    const table_t *t = which == 0 ? &x->tier_tab[g] : which == 1 ? &x->count_tab :
                       which == 2 ? &x->prompt_tab : &x->out_tab;
    if (which == 0 && g >= x->cfg.n_groups) return -1;
    *base = t->base;
    for (uint32_t j = 0; j < t->n && j < cap; ++j) out[j] = t->q[j];
    return (int)t->n;
}

void or_headroom(const or_ctx *x, uint32_t g, int32_t out[OR_MAX_TIERS])
{
    memcpy(out, x->Hq[g], sizeof(int32_t) * OR_MAX_TIERS);
}

void or_freeness(const or_ctx *x, uint32_t r, uint32_t i, int64_t *num, int64_t *den)
{
    freeness(x, &x->rep[r], i, num, den);
}

/* the arrivals sampled in the last tick of local replica r (tier, prompt,
 * output triples in sampling order; seq = next_seq_before + index) */
int or_last_arrivals(const or_ctx *x, uint32_t r, uint32_t *out, uint32_t cap)
{
    const replica_t *rp = &x->rep[r];
    for (uint32_t k = 0; k < rp->n_arr && k < cap; ++k) memcpy(out + 3 * (size_t)k, rp->arr + 3 * (size_t)k, 12);
    return (int)rp->n_arr;
}

uint64_t or_check(or_ctx *x, uint32_t r) { return check_invariants(x, &x->rep[r]); }

/* draining flag of instance i of local replica r (a host decision: scale-in
 * or graceful shutdown) */
int or_set_drain(or_ctx *x, uint32_t r, uint32_t i, int on)
{
    if (r >= x->r_count || i >= x->I) return -1;
    x->rep[r].drain[i] = on ? 1 : 0;
    return 0;
}

void or_freeness_normal(const or_ctx *x, uint32_t r, uint32_t i, int64_t *num, int64_t *den)
{
    freeness_normal(x, &x->rep[r], i, num, den);
}

/* auto-scaling signal of the current state of local replica r */
int or_autoscale(const or_ctx *x, uint32_t r, int64_t *sum)
{
    return autoscale_signal(x, &x->rep[r], sum);
}

/* latency histograms of local replicas [r0, r0 + nr): out[r][which][tier][bin],
 * which 0 = queue delay, 1 = end-to-end; or_hist_set restores them */
int or_hist_get(const or_ctx *x, uint32_t r0, uint32_t nr, uint32_t *out)
{
    if (r0 > x->r_count || nr > x->r_count - r0) return -1;
    const size_t per = 2 * OR_MAX_TIERS * OR_HBINS;
    for (uint32_t r = 0; r < nr; ++r) memcpy(out + r * per, x->rep[r0 + r].hist, per * sizeof(uint32_t));
    return 0;
}

int or_hist_set(or_ctx *x, uint32_t r0, uint32_t nr, const uint32_t *in)
{
    if (r0 > x->r_count || nr > x->r_count - r0) return -1;
    const size_t per = 2 * OR_MAX_TIERS * OR_HBINS;
    for (uint32_t r = 0; r < nr; ++r) memcpy(x->rep[r0 + r].hist, in + r * per, per * sizeof(uint32_t));
    return 0;
}

uint32_t or_hist_bin(uint64_t v) { return hist_bin(v); }

/* INFaaS service-time estimates of local replicas [r0, r0 + nr), [r][I] in
 * 1/256 tick; or_svc_set restores them */
int or_svc_get(const or_ctx *x, uint32_t r0, uint32_t nr, int64_t *out)
{
    if (r0 > x->r_count || nr > x->r_count - r0) return -1;
    for (uint32_t r = 0; r < nr; ++r) memcpy(out + (size_t)r * x->I, x->rep[r0 + r].svc, x->I * sizeof(int64_t));
    return 0;
}

int or_svc_set(or_ctx *x, uint32_t r0, uint32_t nr, const int64_t *in)
{
    if (r0 > x->r_count || nr > x->r_count - r0) return -1;
    for (uint32_t r = 0; r < nr; ++r) memcpy(x->rep[r0 + r].svc, in + (size_t)r * x->I, x->I * sizeof(int64_t));
    return 0;
}

/* adaptive headroom state of replicas [r0, r0+nr): hq[nr][10] in 1/256
 * block; snap[nr][2][10] the admitted and queue-delay counters at the last
 * update.  With a static headroom (adapt_epoch 0) or_adapt_set ignores both
 * arrays and restores Eq. 3's table with zero counters; otherwise hq NULL
 * restores Eq. 3's table, snap NULL takes the current counters, and an H_p
 * outside [0, adapt_max], for a tier >= K or for the lowest tier when
 * zero_lowest is set, other than 0, is rejected (-1, nothing changed). */
int or_adapt_get(const or_ctx *x, uint32_t r0, uint32_t nr, int32_t *hq, uint64_t *snap)
{
    if (r0 > x->r_count || nr > x->r_count - r0) return -1;
    for (uint32_t r = 0; r < nr; ++r) {
        const replica_t *rp = &x->rep[r0 + r];
        memcpy(hq + (size_t)r * OR_MAX_TIERS, rp->hq, sizeof(rp->hq));
        memcpy(snap + (size_t)r * 2 * OR_MAX_TIERS, rp->snap_adm, sizeof(rp->snap_adm));
        memcpy(snap + (size_t)r * 2 * OR_MAX_TIERS + OR_MAX_TIERS, rp->snap_qd, sizeof(rp->snap_qd));
    }
    return 0;
}

int or_adapt_set(or_ctx *x, uint32_t r0, uint32_t nr, const int32_t *hq, const uint64_t *snap)
{
    if (r0 > x->r_count || nr > x->r_count - r0) return -1;
    const or_cfg *c = &x->cfg;
    for (uint32_t r = 0; r < nr; ++r) {
        replica_t *rp = &x->rep[r0 + r];
        const uint32_t K = x->groups[rp->group].K;
        if (c->adapt_epoch && hq)
            for (uint32_t p = 0; p < OR_MAX_TIERS; ++p) {
                const int32_t v = hq[(size_t)r * OR_MAX_TIERS + p];
                if (v < 0 || (uint32_t)v > c->adapt_max || (p >= K && v != 0) || (c->zero_lowest && p == K - 1 && v != 0))
                    return -1;
            }
    }
    for (uint32_t r = 0; r < nr; ++r) {
        replica_t *rp = &x->rep[r0 + r];
        if (c->adapt_epoch && hq) memcpy(rp->hq, hq + (size_t)r * OR_MAX_TIERS, sizeof(rp->hq));
        else memcpy(rp->hq, x->Hq[rp->group], sizeof(rp->hq));
        for (int p = 0; p < OR_MAX_TIERS; ++p) {
            if (c->adapt_epoch && snap) {
                rp->snap_adm[p] = snap[(size_t)r * 2 * OR_MAX_TIERS + p];
                rp->snap_qd[p] = snap[(size_t)r * 2 * OR_MAX_TIERS + OR_MAX_TIERS + p];
            } else {
                rp->snap_adm[p] = c->adapt_epoch ? rp->stats[p * 8 + F_ADMITTED] : 0;
                rp->snap_qd[p] = c->adapt_epoch ? rp->stats[p * 8 + F_QDELAY] : 0;
            }
        }
    }
    return 0;
}
