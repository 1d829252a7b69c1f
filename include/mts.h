/*
 * mts.h -- multi-tier Llumnix scheduling step on MI355X (gfx950).
 *
 * A handle owns R independent simulated clusters ("replicas").  Each replica
 * has I serving instances with KV capacity M blocks and S request slots each.
 * mts_step advances every replica by n scheduling ticks on the GPU.  One tick
 * of one replica:
 *   A  decode one token per running request; a request whose length is a
 *      multiple of the block size needs a new KV block; when an instance
 *      cannot grant every new block it preempts its lowest-priority running
 *      requests (largest tier, then newest) back to its queue; a request
 *      whose output is complete finishes and frees its blocks
 *      (Section 2.1 block-based KV cache, Section 2.2 preemption, Section 3.1)
 *   A2 a migration whose source request was preempted or finished returns
 *      its destination reservation (Section 3.5)
 *   B  each instance admits its head-of-line request (smallest (tier, seq))
 *      while its blocks fit (Section 3.1; Eq. 2 head-of-line demand)
 *   C  freeness F = (M - sum_r V(r)) / B with per-tier headroom
 *      H_p = h0 * gamma^p charged once per present tier (Eq. 1-4)
 *   D  this tick's arrivals are sampled and dispatched tier 0 first, FCFS
 *      within a tier, each to the instance with the largest F that has a
 *      free slot (Section 3.4)
 *   E  in-flight migrations copy one stage of KV blocks (commit when all are
 *      copied, abort when a stage does not fit); on interval ticks
 *      instances are ranked by F and low-F sources (F < 0) are paired with
 *      high-F destinations while the gap is at least theta; each source
 *      moves its head-of-line queued request, else starts a staged copy of
 *      its lowest-priority, smallest running request (Section 3.5, Fig. 4)
 * Optional, at the start of a tick (Section 6.5 future work, see mts_cfg):
 *   the headroom of each tier adapts to its observed queue delay, and
 *   waiting requests that waited past their tier's quota are promoted.
 * All scheduler state and arithmetic is integer; headroom is fixed point at
 * 1/256 block and freeness values are compared exactly.
 *
 * Conventions: every function returns MTS_OK (0) or a negative MTS_E* code
 * and never throws.  Host pointers are plain CPU memory; the device buffer
 * passed to mts_create is device memory owned by the caller.  A handle is not
 * thread-safe; calls on one handle must not overlap.
 */
#ifndef MTS_H
#define MTS_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MTS_ABI_VERSION 6
#define MTS_MAX_TIERS 10
#define MTS_NSTAT 96
/* Latency histogram bins per (metric, tier); see mts_state_view.hist */
#define MTS_HIST_BINS 240

enum {
    MTS_OK = 0,
    MTS_EINVAL = -1,  /* bad argument or configuration outside the limits below */
    MTS_ENOMEM = -2,  /* device buffer too small, or host allocation failed */
    MTS_EDEVICE = -3, /* a HIP call failed */
    MTS_ESTATE = -4,  /* a device-side invariant check failed (see mts_stats) */
    MTS_ERANGE = -5   /* replica range or table index out of range; tick/seq counter would overflow */
};

/* tier distributions (Section 4.2) */
enum { MTS_TIERS_UNIFORM = 0,   /* P(k) = 1/K */
       MTS_TIERS_GAUSS = 1,     /* P(tier <= k) = Phi((k + 1/2 - p0) / p1), tails lumped */
       MTS_TIERS_GEOMETRIC = 2, /* P(k) proportional to p0^(K-1-k) */
       MTS_TIERS_EXPLICIT = 3 };/* P(k) proportional to probs[k] */
/* per-tick arrival count (Section 4.4) */
enum { MTS_ARRIVAL_POISSON = 0,       /* Poisson(arrival_mean) */
       MTS_ARRIVAL_GAMMA_POISSON = 1 };/* gamma-mixed Poisson: mean, coefficient of variation */
/* prompt length in tokens */
enum { MTS_PROMPT_UNIFORM_INT = 0,    /* uniform on [prompt_lo, prompt_hi] */
       MTS_PROMPT_LOGNORMAL = 1 };    /* P(len <= n) = Phi((ln(n + 1/2) - mu) / sigma), clipped */
/* output length in tokens */
enum { MTS_OUTPUT_GEOMETRIC = 0,      /* support {1, 2, ...}, mean output_param */
       MTS_OUTPUT_PARETO = 1 };       /* min(floor(output_min * U^(-1/output_param)), output_cap) */

/* A group of consecutive replicas sharing a tier count and tier mix. */
typedef struct mts_group {
    uint32_t n_replicas;  /* >= 1 */
    uint32_t K;           /* tiers, 1..10; tier 0 is the highest priority */
    uint32_t tier_kind;   /* MTS_TIERS_* */
    uint32_t reserved;    /* must be 0 */
    double p0, p1;        /* GAUSS: mu, sigma > 0; GEOMETRIC: ratio in (0, 1] */
    double probs[MTS_MAX_TIERS]; /* EXPLICIT: K non-negative weights, positive sum */
} mts_group;

typedef struct mts_cfg {
    uint32_t abi_version;        /* MTS_ABI_VERSION */
    uint32_t n_instances;        /* I: 1..256 */
    uint32_t slots_per_instance; /* S: multiple of 64, 64..2048 */
    uint32_t kv_blocks;          /* M: 1..2^21 blocks per instance */
    uint32_t block_tokens;       /* tokens per KV block: power of two, 1..64 */
    uint32_t zero_lowest_tier;   /* 1: the lowest tier K-1 gets no headroom */
    double headroom_base;        /* h0 in blocks (Eq. 3: h0 = M * h_max), >= 0 */
    double headroom_decay;       /* gamma = e^-lambda, in [0, 1] */
    uint32_t mig_interval;       /* pairing happens on ticks t with t % interval == 0; >= 1 */
    uint32_t mig_stage_blocks;   /* B_stage: blocks copied per stage (one stage per tick); >= 1 */
    uint32_t mig_max_pairs;      /* pairs per round, <= I / 2 */
    int32_t theta_num, theta_den;/* theta = num/den in blocks per running request; 0 <= num < 2^20, 1 <= den <= 1024 */
    uint32_t arrival_kind;       /* MTS_ARRIVAL_* */
    uint32_t prompt_kind;        /* MTS_PROMPT_* */
    uint32_t output_kind;        /* MTS_OUTPUT_* */
    uint32_t reserved;           /* must be 0 */
    double arrival_mean;         /* > 0 */
    double arrival_cv;           /* GAMMA_POISSON: > 0 */
    double prompt_mu, prompt_sigma; /* LOGNORMAL */
    uint32_t prompt_lo, prompt_hi;  /* 1 <= lo <= hi */
    double output_param;         /* GEOMETRIC: mean >= 1; PARETO: alpha > 0 */
    uint32_t output_min, output_cap; /* PARETO: 1 <= min <= cap; every output length <= 16383 */
    uint64_t seed;               /* Philox key word 0 */
    uint64_t replica_id_base;    /* replica r draws with Philox key (seed, replica_id_base + r) */
    uint32_t n_groups;           /* >= 1 */
    uint32_t reserved2;          /* must be 0 */
    const mts_group* groups;     /* n_groups entries, copied by mts_create */
    /* Global dispatch policy.  MTS_POLICY_LLUMNIX (0): tier-ordered dispatch
     * to the largest freeness and migration (Sections 3.4, 3.5).
     * MTS_POLICY_INFAAS (1), the paper's comparison scheduler (Section 3.7):
     * each arrival goes to the instance with the smallest
     *   cost = alpha * q + beta * s + gamma * penalty      (1/256 tick)
     * with q the instance's waiting requests (updated after every placement,
     * weighted as 256 each), s its service-time estimate in 1/256 tick and
     * penalty in ticks (weighted as 256 each): pen_overloaded when its head of
     * line does not fit its free blocks after admission, else pen_interfered
     * when it preempted a request in this tick, else 0; ties go to the lowest
     * index; no migration starts.  s is updated once per tick after
     * admission from that tick's finishes on the instance:
     *   s += floor((floor(256 * sum / count) - s) / 2^infaas_ewma_shift)
     * with sum the end-to-end ticks of the count requests that finished. */
    uint32_t dispatch_policy;    /* MTS_POLICY_* */
    uint32_t infaas_ewma_shift;  /* 0..16 */
    int32_t infaas_alpha;        /* 0..65536 */
    int32_t infaas_beta;         /* 0..1024 */
    int32_t infaas_gamma;        /* 0..65536 */
    uint32_t infaas_pen_overloaded, infaas_pen_interfered; /* ticks, 0..2^20 */
    /* 1: tier-blind scheduling, the priority-blind local scheduler the paper
     * pairs with INFaaS (Section 5.3): arrivals are dispatched in arrival
     * order, queues are served first come first served, preemption takes the
     * newest running request and the migration candidate ignores tiers.
     * Tiers still label the counters and histograms and still enter Eq. 4's
     * headroom.  0: tier order everywhere (Sections 3.1, 3.4). */
    uint32_t tier_blind;
    /* Adaptive headroom (Section 6.5 names it as future work and leaves the
     * controller open; this is the library's reading).  adapt_epoch = 0
     * keeps Eq. 3's static table.  Otherwise each replica carries its own
     * table, starting from Eq. 3's, and at the start of every tick t with
     * t % adapt_epoch == 0 each tier p < K (but the lowest when
     * zero_lowest_tier is set) takes the a requests of tier p first admitted
     * since the previous update and their summed queue delay d (ticks):
     *   d > adapt_slo[p] * a                 the mean misses the target:
     *        H_p = min(H_p + adapt_up, adapt_max)
     *   256 d <= adapt_margin * adapt_slo[p] * a
     *                                        met with margin, the headroom
     *                                        sat unused: H_p = max(H_p - adapt_down, 0)
     * and H_p stays otherwise, also when a = 0.  H_p, adapt_up, adapt_down
     * and adapt_max are in 1/256 block; exact for any counter values. */
    uint32_t adapt_epoch;        /* 0..65536 ticks */
    uint32_t adapt_up, adapt_down;/* any */
    uint32_t adapt_max;          /* >= every static H_p, <= 2^29 / MTS_MAX_TIERS */
    uint32_t adapt_margin;       /* 0..256 (fraction of the target in 1/256) */
    uint32_t adapt_slo[MTS_MAX_TIERS]; /* mean queue-delay target per tier, 1..2^20 ticks (epoch > 0) */
    /* Multilevel-feedback promotion (Section 6.5 future work; the library's
     * reading).  promote_period = 0 promotes nothing.  Otherwise at the start
     * of every tick t with t % promote_period == 0 each waiting request of
     * tier p >= 1 whose age t - tarr (mod 2^32) is at least promote_age[p]
     * moves to tier p - 1 (one tier per pass; promote_age[p] = 0: tier p is
     * never promoted; promote_age[0] is ignored).  A promoted request keeps
     * its new tier: admission, preemption, finish, the queue order, Eq. 4's
     * tier mask, the counters and the histograms all see the tier it holds. */
    uint32_t promote_period;
    uint32_t promote_age[MTS_MAX_TIERS];
} mts_cfg;

enum { MTS_POLICY_LLUMNIX = 0, MTS_POLICY_INFAAS = 1 };

/* Counters summed over all replicas (mts_stats) or per replica
 * (mts_export_state).  Index layout of the raw arrays: per_tier[p][f] is
 * element p * 8 + f, the scalar counters follow at 80..90 in the order of
 * the fields below, 91..95 are zero in the canonical state (the device keeps
 * a diagnostic at 91, see mts_get_wheel). */
enum { MTS_F_ARRIVED = 0, MTS_F_REJECTED, MTS_F_DISPATCHED, MTS_F_ADMITTED,
       MTS_F_FINISHED, MTS_F_PREEMPTED, MTS_F_QDELAY_SUM, MTS_F_E2E_SUM };
typedef struct mts_stats_t {
    uint64_t per_tier[MTS_MAX_TIERS][8];
    uint64_t mig_queued, mig_started, mig_committed, mig_aborted;
    uint64_t run_slot_ticks, wait_slot_ticks;  /* running / waiting requests summed over ticks */
    uint64_t invariant_violations;             /* device-side checks that failed */
    uint64_t ticks;                            /* replica-ticks executed */
    /* Section 3.6: replica-ticks whose cluster-average normal-priority
     * freeness (Eq. 1 without headroom, fixed point floor(F * 2^20) per
     * instance) is below -1/2 (scale out) or above 3/2 (scale in); evaluated
     * after admission */
    uint64_t scale_out_ticks, scale_in_ticks;
    /* Section 3.4: arrivals placed on a draining instance because every
     * instance with a free slot was draining */
    uint64_t drain_fallback_dispatches;
    uint64_t replicas;
    uint64_t digest;  /* wrapping sum of the per-replica state digests */
} mts_stats_t;

/* Host views of the canonical state of replicas [r0, r0 + nr), all arrays
 * dense in (replica, instance, slot) order:
 *   meta[nr*I*S]  status | tier << 2 | admitted-once << 6 | migrating-out << 7,
 *                 status 0 empty, 1 waiting, 2 running, 3 inbound reservation
 *   lr[nr*I*S]    len | rem << 16 (tokens so far, output tokens left)
 *   seq[nr*I*S]   per-replica arrival sequence number
 *   tarr[nr*I*S]  arrival tick
 *   free[nr*I]    free KV blocks
 *   mig[nr*I*4]   per source instance: dst (-1 none), src slot, dst slot, blocks copied
 *   next_seq[nr], stats[nr*MTS_NSTAT]
 *   drain[nr*I]   1 if the instance is draining (see mts_set_draining)
 *   hist[nr*2*MTS_MAX_TIERS*MTS_HIST_BINS]
 *                 per-tier latency histograms in ticks (the per-tier latency
 *                 distributions of Section 5.1), index
 *                 ((r * 2 + metric) * MTS_MAX_TIERS + tier) * MTS_HIST_BINS + bin;
 *                 metric 0 = queue delay (arrival to first admission, counted
 *                 when admitted), 1 = end-to-end (arrival to the tick of the
 *                 last token, counted at finish).  Bin of a value v: v for
 *                 v < 16; otherwise, with 2^e <= v < 2^(e+1),
 *                 16 + 8 (e - 4) + floor(v / 2^(e-3)) - 8 (eight equal
 *                 sub-ranges per octave; at most 239)
 *   svc[nr*I]     INFaaS service-time estimate s of each instance, 1/256 tick
 *                 (0 under MTS_POLICY_LLUMNIX)
 *   hq[nr*MTS_MAX_TIERS]
 *                 headroom H_p in 1/256 block the replica uses now (Eq. 3's
 *                 table unless the headroom adapts; 0 for p >= K)
 *   hq_snap[nr*2*MTS_MAX_TIERS]
 *                 adaptive headroom: the per-tier admitted (first 10) and
 *                 queue-delay-sum (next 10) counters at the last update
 *                 (zeros when the headroom is static)
 * Empty slots are all-zero.  Export skips every NULL array.  Import needs
 * every array but drain, hist, svc, hq and hq_snap; a NULL drain clears the
 * flags, a NULL hist empties the histograms, a NULL svc zeroes the
 * estimates; an estimate outside 0..2^40 is MTS_EINVAL.  With a static
 * headroom hq and hq_snap are ignored.  With an adaptive one a NULL hq
 * restores Eq. 3's table, a NULL hq_snap takes the imported counters, and an
 * H_p outside 0..adapt_max, or other than 0 for p >= K or for the lowest
 * tier under zero_lowest_tier, is MTS_EINVAL. */
typedef struct mts_state_view {
    uint8_t* meta;
    uint32_t* lr;
    uint32_t* seq;
    uint32_t* tarr;
    int32_t* free;
    int32_t* mig;
    uint32_t* next_seq;
    uint64_t* stats;
    uint8_t* drain;
    uint32_t* hist;
    int64_t* svc;
    int32_t* hq;
    uint64_t* hq_snap;
} mts_state_view;

typedef struct mts_ctx* mts_handle;

/* Validate cfg and report the device bytes mts_create needs.
 * Returns MTS_EINVAL for a configuration outside the limits above. */
int mts_state_bytes(const mts_cfg* cfg, size_t* bytes);

/* Validate cfg, build the sampling and headroom tables (host, double
 * precision), copy them into dev_buf and initialise every replica to an
 * empty cluster (all slots empty, free = M, tick 0).  dev_buf is device
 * memory of at least mts_state_bytes bytes, 256-byte aligned, owned by the
 * caller and kept alive until mts_destroy.  The initialisation is enqueued
 * on stream.  On success *out receives the handle. */
int mts_create(const mts_cfg* cfg, void* dev_buf, size_t bytes, hipStream_t stream, mts_handle* out);

/* Enqueue n_ticks ticks of every replica on stream and return after the
 * launch (asynchronous).  n_ticks = 0 is a no-op.  MTS_ERANGE if the tick
 * would pass 2^32 - 2^16, or a replica's sequence counter could pass 2^32
 * (the library bounds it by the largest imported counter plus the ticks
 * stepped since, times the most arrivals one tick can hold). */
int mts_step(mts_handle h, uint64_t n_ticks, hipStream_t stream);

/* For callers that cannot allocate device memory while stepping (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * mts_step with the arrival staging (per-tick counts and tier-sorted records
 * of a chunk of ticks) in a static device array of 64 MiB per GPU instead of
 * the handle's buffer.  It calls no allocating routine and records no timing
 * events; results are identical to mts_step's.  The array's device address is
 * looked up once per device by mts_create.  Ticks run in launches of as many
 * ticks as fit the array (at most 1024): MTS_ENOMEM when even one tick's
 * records (replicas x the largest arrival count x 8 bytes) do not fit, and
 * nothing is launched.  MTS_EDEVICE if the lookup failed.  Every call on one
 * GPU shares that GPU's array: calls on different handles that overlap on one
 * GPU (other streams, other threads) race and must be serialised by the
 * caller.  Otherwise as mts_step. */
int mts_step_noalloc(mts_handle h, uint64_t n_ticks, hipStream_t stream);

/* Synchronise with the last stream used on h, sum the per-replica counters
 * and compute the state digest.  Returns MTS_ESTATE (with *out filled) when
 * a device-side invariant check failed. */
int mts_stats(mts_handle h, mts_stats_t* out);

/* Per-replica state digests of replicas [r0, r0 + nr) into out[nr]
 * (wrapping sum of SplitMix64-mixed slot and instance records). */
int mts_digest(mts_handle h, uint32_t r0, uint32_t nr, uint64_t* out);

/* Copy the canonical state of replicas [r0, r0 + nr) to host arrays
 * (synchronises with the last stream used). */
int mts_export_state(mts_handle h, uint32_t r0, uint32_t nr, const mts_state_view* out);

/* Overwrite the state of replicas [r0, r0 + nr) from host arrays in the
 * canonical layout (synchronous).  The state is taken as given at the
 * handle's current tick; the device invariant checks report inconsistencies
 * at the next mts_step.  MTS_EINVAL for indices out of range, a tier >= K, a
 * live request with len or rem 0, rem > 16383 or len + rem > 65535. */
int mts_import_state(mts_handle h, uint32_t r0, uint32_t nr, const mts_state_view* in);

/* Mark instances as draining (scale-in or graceful shutdown; Section 3.5):
 * flags[nr*I], 1 = draining, for replicas [r0, r0 + nr).  A draining
 * instance carries an infinite virtual-usage sentinel: its full freeness is
 * minus infinity, so it receives no dispatch while any other instance has a
 * free slot (when every instance with a free slot drains, the least loaded
 * of them -- largest freeness without the sentinel -- takes the arrival),
 * it is paired first as a migration source and never as a destination, and
 * its requests leave by migration.  It keeps decoding and admitting its own
 * queue.  Synchronous; applies from the next tick.  MTS_ERANGE for a
 * replica range outside the handle, MTS_EINVAL for a flag other than 0 or 1. */
int mts_set_draining(mts_handle h, uint32_t r0, uint32_t nr, const uint8_t* flags);

/* The library's own tables, for comparison with an independent build:
 * which = 0 tier CDF of group g, 1 arrival count, 2 prompt length, 3 output
 * length.  out[j] = floor(2^32 * CDF(base + j)), last entry 2^32; *len is
 * the table length (written even when cap is smaller), *base its first value. */
int mts_get_table(mts_handle h, int which, uint32_t g, uint64_t* out, uint32_t cap,
                  uint32_t* len, uint32_t* base);

/* Headroom of group g in 1/256 block (Eq. 3 with the lowest tier rule). */
int mts_get_headroom(mts_handle h, uint32_t g, int32_t out[MTS_MAX_TIERS]);

/* Next tick to execute (ticks done so far). */
uint64_t mts_tick(mts_handle h);

/* Set the next tick to execute, e.g. after mts_import_state of a state saved
 * at that tick.  The canonical state (every request's length and remaining
 * output) is unchanged; only the clock moves (synchronous).  MTS_ERANGE if
 * the tick does not fit the 32-bit tick fields. */
int mts_set_tick(mts_handle h, uint64_t tick);

/* Force the launch shape of the step kernel: threads per block (0, or the
 * block size mts_get_launch reports: one 64-lane wave per replica, eight
 * waves per replica for 128 or more instances) and number of blocks (0:
 * automatic, else at most the replica count; each block runs replicas r,
 * r + blocks, ...). */
int mts_set_launch(mts_handle h, uint32_t threads, uint32_t blocks);

/* Launch shape mts_step uses now: *threads = the block size (64, or 512 for
 * 128 or more instances) and *blocks = the forced count, or the automatic one
 * (replicas, capped at the step-kernel blocks the device holds at once).
 * Queries the current device's occupancy. */
int mts_get_launch(mts_handle h, uint32_t* threads, uint32_t* blocks);

/* Queue cache of the step kernel: per instance, the waiting requests that
 * follow the head of line in (tier, seq) order are kept in LDS, so that
 * admitting or moving the head does not rescan the instance's slots.
 * mts_create picks the deepest of 7, 3, 1 (15, 11, 7, 3, 1 for 128 or more
 * instances; else 0) entries that keeps the step kernel's blocks per compute
 * unit.  For more than 64 instances the cache continues in the state buffer
 * (up to 64 further requests per instance).  Results never depend on the
 * depth (a performance setting, also a test hook).  mts_set_queue_cache takes effect at the next
 * mts_step; MTS_EINVAL for a depth above 15 or one whose LDS does not fit. */
int mts_set_queue_cache(mts_handle h, uint32_t depth);
int mts_get_queue_cache(mts_handle h, uint32_t* depth);

/* Finish wheel of the step kernel (a test hook): every running request is
 * filed under its finish tick in a per-replica wheel of buckets holding up to
 * `cap` entries each; a bucket that fills is rebuilt at its visit by an exact
 * scan of the slots, so results never depend on the capacity.  mts_create
 * picks cap_max from the arrival rate; mts_set_wheel_cap lowers it (1 ..
 * cap_max, else MTS_EINVAL) from the next mts_step on, so that tests reach the
 * rebuild.  mts_get_wheel reports the capacity in use, the reserved one and
 * the number of bucket rebuilds summed over the replicas (a device counter
 * kept at index 91 of the per-replica counters; it is not part of the
 * canonical state: mts_export_state reports it as 0 and mts_import_state
 * resets it).  Any pointer may be NULL. */
int mts_set_wheel_cap(mts_handle h, uint32_t cap);
int mts_get_wheel(mts_handle h, uint32_t* cap, uint32_t* cap_max, uint64_t* rebuilds);

/* Kernel timing with HIP events recorded on the launch stream (off by
 * default; costs three events per chunk of ticks).  With on = 1, every later
 * mts_step records the duration of each arrival-kernel and step-kernel
 * launch.  mts_get_timing waits for the recorded launches, returns the
 * summed durations in milliseconds and the number of step-kernel launches,
 * and starts a new sum.  Any pointer may be NULL. */
int mts_set_timing(mts_handle h, int on);
int mts_get_timing(mts_handle h, double* step_ms, double* arrivals_ms, uint32_t* step_launches);

/* Free the handle's host memory.  dev_buf stays with the caller. */
void mts_destroy(mts_handle h);

const char* mts_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif /* MTS_H */
