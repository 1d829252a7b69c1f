// Internal declarations shared by the libmts translation units.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include <hip/hip_runtime_api.h>

#include "mts.h"

namespace mts {

constexpr uint32_t kMaxInstances = 256;
constexpr uint32_t kMaxSlots = 2048;
constexpr uint32_t kMaxBlockTokens = 64;
constexpr uint32_t kMaxOutput = 16383;
constexpr uint32_t kMaxBlocks = 1u << 21;
constexpr uint32_t kMaxGroups = 4096;
constexpr uint64_t kMaxReplicas = 1u << 20;
constexpr uint32_t kMaxTable = 1u << 17;
// words of the device table of the Section 6.5 extensions
#define MTS_EXT_WORDS 32

// slot status and meta flags (canonical layout, see mts.h)
constexpr uint32_t kEmpty = 0, kWaiting = 1, kRunning = 2, kInbound = 3;
constexpr uint32_t kAdmitted = 0x40, kMigrating = 0x80;

// counter indices
constexpr int kArrived = 0, kRejected = 1, kDispatched = 2, kAdmittedCnt = 3, kFinished = 4,
              kPreempted = 5, kQdelay = 6, kE2e = 7;
constexpr int kMigQueued = 80, kMigStarted = 81, kMigCommitted = 82, kMigAborted = 83,
              kRunSlotTicks = 84, kWaitSlotTicks = 85, kInvariant = 86, kTicks = 87,
              kScaleOut = 88, kScaleIn = 89, kDrainFallback = 90;
// device diagnostic, not part of the canonical state: finish-wheel buckets
// rebuilt by a scan after they overflowed
constexpr int kWheelRebuilds = 91;
// latency histograms: queue delay and end-to-end, per tier
constexpr int kHistQdelay = 0, kHistE2e = 1;
constexpr size_t kHistPerReplica = size_t(2) * MTS_MAX_TIERS * MTS_HIST_BINS;

struct Table {
    uint32_t base = 0;
    std::vector<uint64_t> q;  // last entry is 2^32
};

struct Tables {
    std::vector<Table> tier;     // per group
    std::vector<int32_t> hq;     // [group][MTS_MAX_TIERS], 1/256 block
    Table count, prompt, output;
};

int validate(const mts_cfg& c);
int build_tables(const mts_cfg& c, Tables& T);

// Device buffer layout: byte offsets of every array inside dev_buf.
struct Layout {
    size_t tier_q, hq, group_K, count_q, prompt_q, output_q, group_of;  // tables
    size_t count_g, prompt_g, output_g;                                 // guide tables
    size_t slot;                                                        // [R][I][S] uint4 records
    size_t freeb, mig, drain;                                           // [R][I], [R][I][4], [R][I] u8
    size_t hist;                                                        // [R][2][10][MTS_HIST_BINS] u32
    size_t svc;                                                         // [R][I] i64 INFaaS estimate
    size_t ext;                                                         // u32 adapt_slo[10], promote_age[10]
    size_t hqr, hsnap;                                                  // adaptive: [R][10] i32, [R][2][10] u64
    size_t next_seq, stats, digest;                                     // [R], [R][NSTAT], [R]
    size_t arr_cnt, arr_rec;                                            // [R][chunk], [R][chunk][cap]
    size_t wheel;                                                       // [R][wsz][wcap]
    size_t qx;                                                          // [R][I][kQxDepth] uint4 (I > 64 only)
    size_t total;
};

// The kernels for more than 64 instances keep, behind each instance's queue
// cache in LDS, up to this many further waiting requests in order in HBM.
constexpr uint32_t kQxDepth = 64;

// Everything a kernel launch needs, passed by value.
struct Params {
    uint32_t R, I, S, W;           // W = S / 64 occupancy words per instance
    uint32_t M, blk_shift, RB;     // RB = block_tokens growth residues
    uint32_t mig_interval, mig_stage, mig_max_pairs;
    int32_t theta_num, theta_den;
    uint32_t count_n, prompt_n, output_n;  // table lengths (entries incl. the implicit 2^32)
    uint32_t count_base, prompt_base, output_base;
    uint32_t count_gs, prompt_gs, output_gs;  // guide shift: bucket = u >> shift
    uint32_t chunk, arr_cap;       // ticks per arrival batch, records per tick
    uint32_t wsz, wcap;            // finish wheel: buckets (power of two), entries per bucket
    uint64_t seed, id_base;
    uint32_t policy, ewma_shift;   // MTS_POLICY_*, INFaaS moving-average shift
    long long alpha256, beta, gamma256;  // INFaaS weights (alpha and gamma times 256)
    uint32_t pen_over, pen_intf;   // INFaaS state penalties in ticks
    uint32_t qdepth;               // queue-cache entries behind each head of line (LDS)
    uint32_t blind;                // 1: tiers order nothing (tier-blind scheduling)
    uint32_t zero_lowest;          // 1: the lowest tier carries no headroom
    // adaptive headroom (epoch 0: static) and promotion (period 0: none)
    uint32_t adapt_epoch, adapt_up, adapt_down, adapt_max, adapt_margin;
    uint32_t promo_period;
    const uint32_t* ext;           // extension table, MTS_EXT_WORDS u32 (mts_api.cpp builds it)
    int32_t* hqr;                  // [R][10] per-replica headroom (adaptive only)
    unsigned long long* hsnap;     // [R][2][10] admitted / queue-delay counters at the last update
    const unsigned long long* tier_q;  // [group][MTS_MAX_TIERS] floor(2^32 CDF), up to 2^32
    const int32_t* hq;             // [group][MTS_MAX_TIERS]
    const uint32_t* group_K32;     // [group] tier count
    const uint32_t* count_q;
    const uint32_t* prompt_q;
    const uint32_t* output_q;
    const uint32_t* count_g;       // guide tables, 2^(32 - shift) + 1 entries
    const uint32_t* prompt_g;
    const uint32_t* output_g;
    const uint16_t* group_of;      // [R]
    uint4* slot;                   // [R][I][S] {slot word, meta, seq, arrival tick}
    int32_t* freeb;
    int32_t* mig;
    uint8_t* drain;
    uint32_t* hist;
    long long* svc;
    uint32_t* next_seq;
    unsigned long long* stats;
    unsigned long long* digest;
    uint32_t* arr_cnt;
    unsigned long long* arr_rec;
    uint32_t* wheel;
    uint4* qx;                     // [R][I][kQxDepth] queue cache extension (I > 64; null otherwise)
};

// LDS bytes of one wave (one replica) of the step kernel
// (ext: the adaptive-headroom or promotion state is kept in LDS)
size_t lds_bytes(uint32_t I, uint32_t S, uint32_t RB, uint32_t wsz, uint32_t policy, uint32_t qdepth, bool ext);

// kernel launches (mts_kernels.hip, mts_arrivals.hip); return hipError_t as int
int launch_init(const Params& p, hipStream_t stream);
int launch_arrivals(const Params& p, unsigned long long t0, uint32_t nt, hipStream_t stream);
int launch_step(const Params& p, unsigned long long t0, uint32_t nt, uint32_t blocks, hipStream_t stream);
// resident step-kernel blocks per CU (0 if the runtime cannot tell); threads
// per block (one wave per replica, or eight for 128 or more instances)
int step_blocks_per_cu(const Params& p);
int step_threads(const Params& p);
int launch_digest(const Params& p, uint32_t r0, uint32_t nr, uint32_t tick, hipStream_t stream);
int launch_shift_clock(const Params& p, uint32_t delta, hipStream_t stream);

// static device scratch of mts_step_noalloc (mts_noalloc.hip): its size, the
// once-per-device lookup of its address (with that device current) and the
// address found (null before the lookup or after it failed)
constexpr size_t kNoallocScratchBytes = size_t(64) << 20;
int scratch_setup(int device);
char* scratch_ptr(int device);

}  // namespace mts
