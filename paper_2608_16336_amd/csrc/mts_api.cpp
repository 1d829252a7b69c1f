// libmts C ABI: handle management, device buffer layout, launches, state
// export/import and counter reduction.  See include/mts.h for the contract.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

#include "mts_internal.h"

using namespace mts;

struct mts_ctx {
    mts_cfg cfg{};
    std::vector<mts_group> groups;
    Tables tables;
    Layout lay{};
    char* dev = nullptr;
    size_t bytes = 0;
    uint32_t R = 0, I = 0, S = 0;
    uint64_t tick = 0;
    uint32_t arr_cap = 0;              // arrival records per (replica, tick)
    uint64_t seq_bound = 0;            // no replica's sequence counter exceeds this
    uint32_t chunk = 0;                // ticks per arrival batch
    uint32_t wsz = 0, wcap = 0;        // finish wheel: buckets, entries per bucket
    uint32_t wcap_max = 0;             // entries per bucket the layout reserves
    uint32_t blocks = 0;               // step-kernel blocks (one wave each); 0 = automatic
    uint32_t qdepth = 0;               // queue-cache entries per instance (chosen at create)
    int device = 0;
    hipStream_t last = nullptr;
    std::vector<uint16_t> group_of;
    std::vector<uint32_t> group_K;
    bool timing = false;
    std::vector<hipEvent_t> ev;        // 3 per timed chunk: before arrivals, before step, after step
    ~mts_ctx()
    {
        for (hipEvent_t e : ev) (void)hipEventDestroy(e);
    }
};

namespace {

size_t up256(size_t x) { return (x + 255) & ~size_t(255); }

uint32_t total_replicas(const mts_cfg& c)
{
    uint64_t R = 0;
    for (uint32_t g = 0; g < c.n_groups; ++g) R += c.groups[g].n_replicas;
    return uint32_t(R);
}

// device bytes reserved for pre-sampled arrivals; sets the ticks per batch
constexpr size_t kArrivalBudget = size_t(2048) << 20;

uint32_t chunk_for(uint32_t R, uint32_t cap)
{
    const size_t per_tick = size_t(R) * cap * 8 + size_t(R) * 4;
    return uint32_t(std::max<size_t>(1, std::min<size_t>(1024, kArrivalBudget / per_tick)));
}

// Guide table of an inverse-CDF table q (Chen and Asau's indexed search):
// bucket j of the 32-bit uniforms, [j 2^shift, (j+1) 2^shift), holds samples in
// [g[j], g[j+1]], where g[j] = min{n : j 2^shift < q[n]} and g[G] = n - 1.  The
// device searches only that range, so it returns exactly min{n : u < q[n]}.
uint32_t guide_shift(const Table& t)
{
    uint32_t lg = 1;
    while ((size_t(1) << lg) < t.q.size() && lg < 16) ++lg;
    return 32 - lg;
}

std::vector<uint32_t> guide_table(const Table& t)
{
    const uint32_t sh = guide_shift(t);
    const size_t G = size_t(1) << (32 - sh);
    std::vector<uint32_t> g(G + 1);
    size_t n = 0;
    for (size_t j = 0; j < G; ++j) {
        const uint64_t thr = uint64_t(j) << sh;
        while (t.q[n] <= thr) ++n;
        g[j] = uint32_t(n);
    }
    g[G] = uint32_t(t.q.size() - 1);
    return g;
}

size_t guide_bytes(const Table& t) { return ((size_t(1) << (32 - guide_shift(t))) + 1) * 4; }

// Finish wheel of one replica: a running request is filed under bucket
// fin mod wsz.  Buckets hold the finishes of one tick plus the few longer
// requests that share the bucket and are carried to its next visit; entries
// per bucket give a wide margin over the arrival rate, and a bucket that
// overflows is rebuilt by an exact scan.
void wheel_size(const mts_cfg& c, const Tables& T, uint32_t& wsz, uint32_t& wcap)
{
    const uint32_t maxout = T.output.base + uint32_t(T.output.q.size()) - 1;
    wsz = 1;
    while (wsz <= maxout && wsz < 512) wsz <<= 1;
    const double cv = c.arrival_kind == MTS_ARRIVAL_GAMMA_POISSON ? c.arrival_cv : 0.0;
    const double want = 2.0 * c.arrival_mean * (1.0 + cv) + 24.0;
    wcap = uint32_t(std::min(2048.0, std::ceil(want / 16.0) * 16.0));
}

Layout make_layout(const mts_cfg& c, const Tables& T, uint32_t R, uint32_t chunk, uint32_t cap,
                   uint32_t wsz, uint32_t wcap)
{
    Layout L{};
    const size_t I = c.n_instances, S = c.slots_per_instance;
    const size_t N = size_t(R) * I * S;
    size_t o = 0;
    L.tier_q = o;   o = up256(o + size_t(c.n_groups) * MTS_MAX_TIERS * 8);
    L.hq = o;       o = up256(o + size_t(c.n_groups) * MTS_MAX_TIERS * 4);
    L.group_K = o;  o = up256(o + size_t(c.n_groups) * 4);
    L.count_q = o;  o = up256(o + T.count.q.size() * 4);
    L.prompt_q = o; o = up256(o + T.prompt.q.size() * 4);
    L.output_q = o; o = up256(o + T.output.q.size() * 4);
    L.count_g = o;  o = up256(o + guide_bytes(T.count));
    L.prompt_g = o; o = up256(o + guide_bytes(T.prompt));
    L.output_g = o; o = up256(o + guide_bytes(T.output));
    L.group_of = o; o = up256(o + size_t(R) * 2);
    L.slot = o;     o = up256(o + N * 16);
    L.freeb = o;    o = up256(o + size_t(R) * I * 4);
    L.mig = o;      o = up256(o + size_t(R) * I * 16);
    L.drain = o;    o = up256(o + size_t(R) * I);
    L.hist = o;     o = up256(o + size_t(R) * kHistPerReplica * 4);
    L.svc = o;      o = up256(o + size_t(R) * I * 8);
    L.ext = o;      o = up256(o + MTS_EXT_WORDS * 4);
    const bool adapt = c.adapt_epoch != 0;
    L.hqr = o;      o = up256(o + (adapt ? size_t(R) * MTS_MAX_TIERS * 4 : 0));
    L.hsnap = o;    o = up256(o + (adapt ? size_t(R) * 2 * MTS_MAX_TIERS * 8 : 0));
    L.next_seq = o; o = up256(o + size_t(R) * 4);
    L.stats = o;    o = up256(o + size_t(R) * MTS_NSTAT * 8);
    L.digest = o;   o = up256(o + size_t(R) * 8);
    L.arr_cnt = o;  o = up256(o + size_t(R) * chunk * 4);
    L.arr_rec = o;  o = up256(o + size_t(R) * chunk * cap * 8);
    L.wheel = o;    o = up256(o + size_t(R) * wsz * wcap * 4);
    // the queue cache's extension, for the kernels of more than 64 instances
    L.qx = o;       o = up256(o + (I > 64 ? size_t(R) * I * kQxDepth * 16 : 0));
    L.total = o;
    return L;
}

Params make_params(const mts_ctx* h)
{
    Params p{};
    char* d = h->dev;
    const mts_cfg& c = h->cfg;
    p.R = h->R; p.I = h->I; p.S = h->S; p.W = h->S / 64;
    p.M = c.kv_blocks;
    uint32_t sh = 0;
    while ((1u << sh) < c.block_tokens) ++sh;
    p.blk_shift = sh;
    p.RB = c.block_tokens;
    p.mig_interval = c.mig_interval; p.mig_stage = c.mig_stage_blocks; p.mig_max_pairs = c.mig_max_pairs;
    p.theta_num = c.theta_num; p.theta_den = c.theta_den;
    p.count_n = uint32_t(h->tables.count.q.size());
    p.prompt_n = uint32_t(h->tables.prompt.q.size());
    p.output_n = uint32_t(h->tables.output.q.size());
    p.count_base = h->tables.count.base;
    p.prompt_base = h->tables.prompt.base;
    p.output_base = h->tables.output.base;
    p.count_gs = guide_shift(h->tables.count);
    p.prompt_gs = guide_shift(h->tables.prompt);
    p.output_gs = guide_shift(h->tables.output);
    p.chunk = h->chunk;
    p.arr_cap = h->arr_cap;
    p.wsz = h->wsz;
    p.wcap = h->wcap;
    p.seed = c.seed;
    p.id_base = c.replica_id_base;
    p.policy = c.dispatch_policy;
    p.ewma_shift = c.infaas_ewma_shift;
    p.alpha256 = static_cast<long long>(c.infaas_alpha) * 256;
    p.beta = c.infaas_beta;
    p.gamma256 = static_cast<long long>(c.infaas_gamma) * 256;
    p.pen_over = c.infaas_pen_overloaded;
    p.pen_intf = c.infaas_pen_interfered;
    p.qdepth = h->qdepth;
    p.blind = c.tier_blind;
    p.zero_lowest = c.zero_lowest_tier;
    p.adapt_epoch = c.adapt_epoch;
    p.adapt_up = c.adapt_up;
    p.adapt_down = c.adapt_down;
    p.adapt_max = c.adapt_max;
    p.adapt_margin = c.adapt_margin;
    p.promo_period = c.promote_period;
    const Layout& L = h->lay;
    p.ext = reinterpret_cast<const uint32_t*>(d + L.ext);
    p.hqr = c.adapt_epoch ? reinterpret_cast<int32_t*>(d + L.hqr) : nullptr;
    p.hsnap = c.adapt_epoch ? reinterpret_cast<unsigned long long*>(d + L.hsnap) : nullptr;
    p.tier_q = reinterpret_cast<const unsigned long long*>(d + L.tier_q);
    p.hq = reinterpret_cast<const int32_t*>(d + L.hq);
    p.group_K32 = reinterpret_cast<const uint32_t*>(d + L.group_K);
    p.count_q = reinterpret_cast<const uint32_t*>(d + L.count_q);
    p.prompt_q = reinterpret_cast<const uint32_t*>(d + L.prompt_q);
    p.output_q = reinterpret_cast<const uint32_t*>(d + L.output_q);
    p.count_g = reinterpret_cast<const uint32_t*>(d + L.count_g);
    p.prompt_g = reinterpret_cast<const uint32_t*>(d + L.prompt_g);
    p.output_g = reinterpret_cast<const uint32_t*>(d + L.output_g);
    p.group_of = reinterpret_cast<const uint16_t*>(d + L.group_of);
    p.slot = reinterpret_cast<uint4*>(d + L.slot);
    p.freeb = reinterpret_cast<int32_t*>(d + L.freeb);
    p.mig = reinterpret_cast<int32_t*>(d + L.mig);
    p.drain = reinterpret_cast<uint8_t*>(d + L.drain);
    p.hist = reinterpret_cast<uint32_t*>(d + L.hist);
    p.svc = reinterpret_cast<long long*>(d + L.svc);
    p.next_seq = reinterpret_cast<uint32_t*>(d + L.next_seq);
    p.stats = reinterpret_cast<unsigned long long*>(d + L.stats);
    p.digest = reinterpret_cast<unsigned long long*>(d + L.digest);
    p.arr_cnt = reinterpret_cast<uint32_t*>(d + L.arr_cnt);
    p.arr_rec = reinterpret_cast<unsigned long long*>(d + L.arr_rec);
    p.wheel = reinterpret_cast<uint32_t*>(d + L.wheel);
    p.qx = h->I > 64 ? reinterpret_cast<uint4*>(d + L.qx) : nullptr;
    return p;
}

// u32 device image of a table: its first n-1 entries (the last, 2^32, is implicit)
std::vector<uint32_t> device_table(const Table& t, size_t pad_to = 0)
{
    std::vector<uint32_t> v(std::max(t.q.size() - 1, pad_to), 0);
    for (size_t j = 0; j + 1 < t.q.size(); ++j) v[j] = uint32_t(t.q[j]);
    return v;
}

int hip_rc(hipError_t e) { return e == hipSuccess ? MTS_OK : MTS_EDEVICE; }

// the step kernel keeps adaptive-headroom or promotion state in LDS
bool ext_state(const mts_cfg& c) { return c.adapt_epoch != 0 || c.promote_period != 0; }

int prepare(const mts_cfg* cfg, mts_ctx& x)
{
    if (!cfg) return MTS_EINVAL;
    int rc = validate(*cfg);
    if (rc) return rc;
    x.cfg = *cfg;
    x.groups.assign(cfg->groups, cfg->groups + cfg->n_groups);
    x.cfg.groups = x.groups.data();
    rc = build_tables(x.cfg, x.tables);
    if (rc) return rc;
    x.R = total_replicas(x.cfg);
    x.I = cfg->n_instances;
    x.S = cfg->slots_per_instance;
    x.arr_cap = uint32_t(x.tables.count.base + x.tables.count.q.size());
    x.chunk = chunk_for(x.R, x.arr_cap);
    wheel_size(x.cfg, x.tables, x.wsz, x.wcap);
    x.wcap_max = x.wcap;
    x.lay = make_layout(x.cfg, x.tables, x.R, x.chunk, x.arr_cap, x.wsz, x.wcap);
    return MTS_OK;
}

}  // namespace

extern "C" {

const char* mts_strerror(int code)
{
    switch (code) {
    case MTS_OK: return "ok";
    case MTS_EINVAL: return "invalid argument or configuration";
    case MTS_ENOMEM: return "buffer too small or out of memory";
    case MTS_EDEVICE: return "HIP runtime error";
    case MTS_ESTATE: return "device invariant check failed";
    case MTS_ERANGE: return "index or counter out of range";
    default: return "unknown error";
    }
}

int mts_state_bytes(const mts_cfg* cfg, size_t* bytes)
{
    if (!bytes) return MTS_EINVAL;
    mts_ctx x;
    int rc = prepare(cfg, x);
    if (rc) return rc;
    *bytes = x.lay.total;
    return MTS_OK;
}

int mts_create(const mts_cfg* cfg, void* dev_buf, size_t bytes, hipStream_t stream, mts_handle* out)
{
    if (!out || !dev_buf || (reinterpret_cast<uintptr_t>(dev_buf) & 255)) return MTS_EINVAL;
    *out = nullptr;
    mts_ctx* x = new (std::nothrow) mts_ctx;
    if (!x) return MTS_ENOMEM;
    int rc = prepare(cfg, *x);
    if (rc) { delete x; return rc; }
    if (bytes < x->lay.total) { delete x; return MTS_ENOMEM; }
    x->dev = static_cast<char*>(dev_buf);
    x->bytes = bytes;
    if (hipGetDevice(&x->device) != hipSuccess) { delete x; return MTS_EDEVICE; }
    int max_lds = 0;
    if (hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, x->device) != hipSuccess) {
        delete x;
        return MTS_EDEVICE;
    }
    if (lds_bytes(x->I, x->S, x->cfg.block_tokens, x->wsz, x->cfg.dispatch_policy, 0, ext_state(x->cfg)) > size_t(max_lds)) { delete x; return MTS_EINVAL; }
    // queue cache depth: the deepest of 7, 3, 1 (15, 11, 7, 3, 1 for 128 or
    // more instances, whose long burst queues it spares rescans of 2048
    // slots) that keeps the step kernel's blocks per CU (the cache only saves
    // rescans; a lost block per CU costs more: with no spare room per CU the
    // dispatcher cannot place every block at once; and for small instances a
    // deeper cache costs more in insertions than it saves)
    {
        Params p = make_params(x);
        p.qdepth = 0;
        const int base = step_blocks_per_cu(p);
        for (uint32_t d : {15u, 11u, 7u, 3u, 1u}) {
            if (d > 7 && x->I < 128) continue;
            p.qdepth = d;
            if (lds_bytes(x->I, x->S, x->cfg.block_tokens, x->wsz, x->cfg.dispatch_policy, d, ext_state(x->cfg)) > size_t(max_lds)) continue;
            if (step_blocks_per_cu(p) >= base) { x->qdepth = d; break; }
        }
    }

    // tables and per-replica group index
    const uint32_t G = x->cfg.n_groups;
    // tier tables keep 64-bit entries: a tier of probability 0 at the top
    // makes an earlier entry exactly 2^32
    std::vector<uint64_t> tier(size_t(G) * MTS_MAX_TIERS, 0);
    for (uint32_t g = 0; g < G; ++g) {
        const Table& t = x->tables.tier[g];
        for (size_t j = 0; j + 1 < t.q.size(); ++j) tier[size_t(g) * MTS_MAX_TIERS + j] = t.q[j];
        x->group_K.push_back(x->groups[g].K);
    }
    for (uint32_t g = 0; g < G; ++g)
        for (uint32_t k = 0; k < x->groups[g].n_replicas; ++k) x->group_of.push_back(uint16_t(g));
    // the count, prompt and output tables end where the CDF reaches 1, so
    // every entry but their last fits 32 bits; checked, as the sampler relies on it
    for (const Table* t : {&x->tables.count, &x->tables.prompt, &x->tables.output})
        for (size_t j = 0; j + 1 < t->q.size(); ++j)
            if (t->q[j] > 0xFFFFFFFFull) { delete x; return MTS_EINVAL; }
    const std::vector<uint32_t> cq = device_table(x->tables.count, 1), pq = device_table(x->tables.prompt, 1),
                                oq = device_table(x->tables.output, 1);
    const Layout& L = x->lay;
    hipError_t e = hipSuccess;
    auto up = [&](size_t off, const void* src, size_t n) {
        if (e == hipSuccess && n) e = hipMemcpyAsync(x->dev + off, src, n, hipMemcpyHostToDevice, stream);
    };
    up(L.tier_q, tier.data(), tier.size() * 8);
    up(L.hq, x->tables.hq.data(), x->tables.hq.size() * 4);
    up(L.group_K, x->group_K.data(), x->group_K.size() * 4);
    up(L.count_q, cq.data(), cq.size() * 4);
    up(L.prompt_q, pq.data(), pq.size() * 4);
    up(L.output_q, oq.data(), oq.size() * 4);
    const std::vector<uint32_t> cg = guide_table(x->tables.count), pg = guide_table(x->tables.prompt),
                                og = guide_table(x->tables.output);
    up(L.count_g, cg.data(), cg.size() * 4);
    up(L.prompt_g, pg.data(), pg.size() * 4);
    up(L.output_g, og.data(), og.size() * 4);
    up(L.group_of, x->group_of.data(), x->group_of.size() * 2);
    // extension table: per-tier targets and quotas, the smallest non-zero
    // quota of tiers 1..9 (2^32 - 1: none), period, epoch, up, down, max,
    // margin, zero_lowest_tier, then the device addresses of the per-replica
    // headroom and snapshot arrays (0 when the headroom is static)
    uint32_t ext[MTS_EXT_WORDS] = {0};
    {
        const mts_cfg& c = x->cfg;
        std::memcpy(ext, c.adapt_slo, sizeof(c.adapt_slo));
        std::memcpy(ext + MTS_MAX_TIERS, c.promote_age, sizeof(c.promote_age));
        uint32_t qmin = 0xFFFFFFFFu;
        for (uint32_t q = 1; q < MTS_MAX_TIERS; ++q)
            if (c.promote_age[q] != 0 && c.promote_age[q] < qmin) qmin = c.promote_age[q];
        const uint32_t words[8] = {qmin, c.promote_period, c.adapt_epoch, c.adapt_up, c.adapt_down, c.adapt_max,
                                   c.adapt_margin, c.zero_lowest_tier};
        std::memcpy(ext + 2 * MTS_MAX_TIERS, words, sizeof(words));
        const uint64_t addr[2] = {c.adapt_epoch ? uint64_t(reinterpret_cast<uintptr_t>(x->dev + L.hqr)) : 0,
                                  c.adapt_epoch ? uint64_t(reinterpret_cast<uintptr_t>(x->dev + L.hsnap)) : 0};
        std::memcpy(ext + 28, addr, sizeof(addr));
    }
    up(L.ext, ext, sizeof(ext));
    // adaptive headroom starts from each replica's group table
    std::vector<int32_t> hqr;
    if (x->cfg.adapt_epoch) {
        hqr.resize(size_t(x->R) * MTS_MAX_TIERS);
        for (uint32_t r = 0; r < x->R; ++r)
            std::memcpy(&hqr[size_t(r) * MTS_MAX_TIERS], &x->tables.hq[size_t(x->group_of[r]) * MTS_MAX_TIERS],
                        MTS_MAX_TIERS * 4);
        up(L.hqr, hqr.data(), hqr.size() * 4);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(stream);  // host vectors go out of scope
    if (e != hipSuccess) { delete x; return MTS_EDEVICE; }
    const Params p = make_params(x);
    if (launch_init(p, stream) != 0) { delete x; return MTS_EDEVICE; }
    // address of this device's static scratch for mts_step_noalloc; a failed
    // lookup leaves that entry point unavailable (MTS_EDEVICE), not the handle
    (void)scratch_setup(x->device);
    x->last = stream;
    *out = x;
    return MTS_OK;
}

int mts_set_launch(mts_handle h, uint32_t threads, uint32_t blocks)
{
    if (!h) return MTS_EINVAL;
    // the block is the replica's waves: its size is fixed by the instance count
    if (threads != 0 && int(threads) != step_threads(make_params(h))) return MTS_EINVAL;
    if (blocks > h->R) return MTS_EINVAL;
    h->blocks = blocks;
    return MTS_OK;
}

namespace {

int auto_blocks(mts_handle h, const Params& p, uint32_t* blocks)
{
    if (h->blocks) { *blocks = h->blocks; return MTS_OK; }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device) != hipSuccess) return MTS_EDEVICE;
    // every replica resident at once when the CUs hold them all; else one
    // full wave of resident blocks striding over the replicas
    const uint32_t per_cu = uint32_t(std::max(1, step_blocks_per_cu(p)));
    *blocks = std::min<uint32_t>(h->R, uint32_t(cus) * per_cu);
    return MTS_OK;
}

}  // namespace

int mts_set_queue_cache(mts_handle h, uint32_t depth)
{
    if (!h || depth > 15) return MTS_EINVAL;
    int max_lds = 0;
    if (hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device) != hipSuccess)
        return MTS_EDEVICE;
    if (lds_bytes(h->I, h->S, h->cfg.block_tokens, h->wsz, h->cfg.dispatch_policy, depth, ext_state(h->cfg)) > size_t(max_lds))
        return MTS_EINVAL;
    hipError_t e = hipStreamSynchronize(h->last);
    if (e != hipSuccess) return MTS_EDEVICE;
    h->qdepth = depth;
    return MTS_OK;
}

int mts_get_queue_cache(mts_handle h, uint32_t* depth)
{
    if (!h || !depth) return MTS_EINVAL;
    *depth = h->qdepth;
    return MTS_OK;
}

int mts_get_launch(mts_handle h, uint32_t* threads, uint32_t* blocks)
{
    if (!h || !threads || !blocks) return MTS_EINVAL;
    const Params p = make_params(h);
    *threads = uint32_t(step_threads(p));
    return auto_blocks(h, p, blocks);
}

int mts_step(mts_handle h, uint64_t n_ticks, hipStream_t stream)
{
    if (!h) return MTS_EINVAL;
    if (n_ticks == 0) return MTS_OK;
    // ticks are 32-bit on the device and the sequence counters grow by at
    // most arr_cap - 1 per tick
    const uint64_t end = h->tick + n_ticks;
    const uint64_t seq_end = h->seq_bound + n_ticks * uint64_t(h->arr_cap);
    if (end > 0xFFFF0000ull || seq_end > 0xFFFFFFFFull) return MTS_ERANGE;
    const Params p = make_params(h);
    uint32_t blocks = 0;
    const int rc = auto_blocks(h, p, &blocks);
    if (rc) return rc;
    for (uint64_t t = h->tick; t < end; t += h->chunk) {
        const uint32_t nt = uint32_t(std::min<uint64_t>(h->chunk, end - t));
        hipEvent_t e[3] = {nullptr, nullptr, nullptr};
        if (h->timing) {
            for (hipEvent_t& x : e)
                if (hipEventCreate(&x) != hipSuccess) return MTS_EDEVICE;
            h->ev.insert(h->ev.end(), e, e + 3);
            if (hipEventRecord(e[0], stream) != hipSuccess) return MTS_EDEVICE;
        }
        if (launch_arrivals(p, t, nt, stream) != 0) return MTS_EDEVICE;
        if (h->timing && hipEventRecord(e[1], stream) != hipSuccess) return MTS_EDEVICE;
        if (launch_step(p, t, nt, blocks, stream) != 0) return MTS_EDEVICE;
        if (h->timing && hipEventRecord(e[2], stream) != hipSuccess) return MTS_EDEVICE;
    }
    h->tick = end;
    h->seq_bound = seq_end;
    h->last = stream;
    return MTS_OK;
}

int mts_step_noalloc(mts_handle h, uint64_t n_ticks, hipStream_t stream)
{
    if (!h) return MTS_EINVAL;
    if (n_ticks == 0) return MTS_OK;
    char* base = scratch_ptr(h->device);
    if (!base) return MTS_EDEVICE;
    // ticks per launch: the counts [R][c] (u32) and records [R][c][cap] (u64)
    // of c ticks must fit the static scratch
    const size_t R = h->R, cap = h->arr_cap;
    auto need = [&](size_t c) { return up256(R * c * 4) + R * c * cap * 8; };
    size_t c = std::min<size_t>(1024, kNoallocScratchBytes / (R * cap * 8 + R * 4));
    while (c > 0 && need(c) > kNoallocScratchBytes) --c;
    if (c == 0) return MTS_ENOMEM;
    const uint64_t end = h->tick + n_ticks;
    const uint64_t seq_end = h->seq_bound + n_ticks * uint64_t(h->arr_cap);
    if (end > 0xFFFF0000ull || seq_end > 0xFFFFFFFFull) return MTS_ERANGE;
    Params p = make_params(h);
    p.chunk = uint32_t(c);
    p.arr_cnt = reinterpret_cast<uint32_t*>(base);
    p.arr_rec = reinterpret_cast<unsigned long long*>(base + up256(R * c * 4));
    uint32_t blocks = 0;
    const int rc = auto_blocks(h, p, &blocks);
    if (rc) return rc;
    for (uint64_t t = h->tick; t < end; t += c) {
        const uint32_t nt = uint32_t(std::min<uint64_t>(c, end - t));
        if (launch_arrivals(p, t, nt, stream) != 0) return MTS_EDEVICE;
        if (launch_step(p, t, nt, blocks, stream) != 0) return MTS_EDEVICE;
    }
    h->tick = end;
    h->seq_bound = seq_end;
    h->last = stream;
    return MTS_OK;
}

int mts_digest(mts_handle h, uint32_t r0, uint32_t nr, uint64_t* out)
{
    if (!h || !out) return MTS_EINVAL;
    if (r0 > h->R || nr > h->R - r0) return MTS_ERANGE;
    const Params p = make_params(h);
    if (launch_digest(p, r0, nr, uint32_t(h->tick), h->last) != 0) return MTS_EDEVICE;
    hipError_t e = hipMemcpyAsync(out, h->dev + h->lay.digest + size_t(r0) * 8, size_t(nr) * 8, hipMemcpyDeviceToHost, h->last);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last);
    return hip_rc(e);
}

int mts_stats(mts_handle h, mts_stats_t* out)
{
    if (!h || !out) return MTS_EINVAL;
    std::vector<uint64_t> st(size_t(h->R) * MTS_NSTAT), dg(h->R);
    hipError_t e = hipStreamSynchronize(h->last);
    if (e == hipSuccess)
        e = hipMemcpy(st.data(), h->dev + h->lay.stats, st.size() * 8, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return MTS_EDEVICE;
    int rc = mts_digest(h, 0, h->R, dg.data());
    if (rc) return rc;
    uint64_t sum[MTS_NSTAT] = {0};
    for (uint32_t r = 0; r < h->R; ++r)
        for (int k = 0; k < MTS_NSTAT; ++k) sum[k] += st[size_t(r) * MTS_NSTAT + k];
    std::memset(out, 0, sizeof(*out));
    std::memcpy(out->per_tier, sum, 80 * 8);
    out->mig_queued = sum[kMigQueued];
    out->mig_started = sum[kMigStarted];
    out->mig_committed = sum[kMigCommitted];
    out->mig_aborted = sum[kMigAborted];
    out->run_slot_ticks = sum[kRunSlotTicks];
    out->wait_slot_ticks = sum[kWaitSlotTicks];
    out->invariant_violations = sum[kInvariant];
    out->ticks = sum[kTicks];
    out->scale_out_ticks = sum[kScaleOut];
    out->scale_in_ticks = sum[kScaleIn];
    out->drain_fallback_dispatches = sum[kDrainFallback];
    out->replicas = h->R;
    uint64_t d = 0;
    for (uint64_t v : dg) d += v;
    out->digest = d;
    return out->invariant_violations ? MTS_ESTATE : MTS_OK;
}

namespace {

// canonical len | rem << 16 of a slot word at the next tick to run
uint32_t word_to_lr(uint32_t w, uint64_t tick)
{
    const uint32_t st = w >> 30, lo = w & 0xFFFFu, mid = (w >> 16) & 0x3FFFu;
    if (st == kWaiting) return lo | (mid << 16);
    if (st == kRunning) {
        const uint32_t rem = (mid - uint32_t(tick) + 1u) & 0x3FFFu;
        return (lo - rem) | (rem << 16);
    }
    return 0;
}

}  // namespace

int mts_export_state(mts_handle h, uint32_t r0, uint32_t nr, const mts_state_view* v)
{
    if (!h || !v) return MTS_EINVAL;
    if (r0 > h->R || nr > h->R - r0) return MTS_ERANGE;
    const size_t IS = size_t(h->I) * h->S, I = h->I;
    const Layout& L = h->lay;
    hipError_t e = hipStreamSynchronize(h->last);
    auto get = [&](void* dst, size_t off, size_t n) {
        if (e == hipSuccess && dst && n) e = hipMemcpy(dst, h->dev + off, n, hipMemcpyDeviceToHost);
    };
    // slot records {word, meta, seq, arrival tick}; the device marks an empty
    // slot by its word alone, and an inbound reservation by its word and
    // meta; their other fields are zero in the canonical state
    if (v->lr || v->meta || v->seq || v->tarr) {
        std::vector<uint32_t> rec(size_t(nr) * IS * 4);
        get(rec.data(), L.slot + size_t(r0) * IS * 16, rec.size() * 4);
        if (e == hipSuccess)
            for (size_t k = 0; k < size_t(nr) * IS; ++k) {
                const uint32_t w = rec[4 * k], st = w >> 30;
                const bool gone = w == 0 || st == kInbound;
                if (v->lr) v->lr[k] = word_to_lr(w, h->tick);
                if (v->meta) v->meta[k] = w == 0 ? 0 : uint8_t(rec[4 * k + 1]);
                if (v->seq) v->seq[k] = gone ? 0 : rec[4 * k + 2];
                if (v->tarr) v->tarr[k] = gone ? 0 : rec[4 * k + 3];
            }
    }
    get(v->free, L.freeb + size_t(r0) * I * 4, size_t(nr) * I * 4);
    get(v->mig, L.mig + size_t(r0) * I * 16, size_t(nr) * I * 16);
    get(v->next_seq, L.next_seq + size_t(r0) * 4, size_t(nr) * 4);
    get(v->stats, L.stats + size_t(r0) * MTS_NSTAT * 8, size_t(nr) * MTS_NSTAT * 8);
    // device diagnostics are not part of the canonical state
    if (e == hipSuccess && v->stats)
        for (uint32_t r = 0; r < nr; ++r) v->stats[size_t(r) * MTS_NSTAT + kWheelRebuilds] = 0;
    get(v->drain, L.drain + size_t(r0) * I, size_t(nr) * I);
    get(v->hist, L.hist + size_t(r0) * kHistPerReplica * 4, size_t(nr) * kHistPerReplica * 4);
    get(v->svc, L.svc + size_t(r0) * I * 8, size_t(nr) * I * 8);
    if (h->cfg.adapt_epoch) {
        get(v->hq, L.hqr + size_t(r0) * MTS_MAX_TIERS * 4, size_t(nr) * MTS_MAX_TIERS * 4);
        get(v->hq_snap, L.hsnap + size_t(r0) * 2 * MTS_MAX_TIERS * 8, size_t(nr) * 2 * MTS_MAX_TIERS * 8);
    } else {
        // static headroom: the group's table, no counters
        for (uint32_t r = 0; r < nr && v->hq; ++r)
            std::memcpy(v->hq + size_t(r) * MTS_MAX_TIERS, &h->tables.hq[size_t(h->group_of[r0 + r]) * MTS_MAX_TIERS],
                        MTS_MAX_TIERS * 4);
        if (v->hq_snap) std::memset(v->hq_snap, 0, size_t(nr) * 2 * MTS_MAX_TIERS * 8);
    }
    return hip_rc(e);
}

int mts_import_state(mts_handle h, uint32_t r0, uint32_t nr, const mts_state_view* v)
{
    if (!h || !v || !v->meta || !v->lr || !v->seq || !v->tarr || !v->free || !v->mig || !v->next_seq || !v->stats)
        return MTS_EINVAL;
    if (r0 > h->R || nr > h->R - r0) return MTS_ERANGE;
    const size_t IS = size_t(h->I) * h->S, I = h->I;
    std::vector<uint32_t> w(size_t(nr) * IS);
    std::vector<uint32_t> rec(size_t(nr) * IS * 4);
    // structural checks keep every index the kernel derives from the state in
    // range; running requests are re-encoded relative to the handle's tick
    for (uint32_t r = 0; r < nr; ++r) {
        const uint32_t K = h->group_K[h->group_of[r0 + r]];
        for (size_t s = 0; s < IS; ++s) {
            const size_t k = size_t(r) * IS + s;
            const uint8_t m = v->meta[k];
            const uint32_t st = m & 3u, lr = v->lr[k], len = lr & 0xFFFFu, rem = lr >> 16;
            if (st == kEmpty) {
                if (m != 0) return MTS_EINVAL;
                w[k] = 0;
            } else if (st == kInbound) {
                w[k] = 3u << 30;
            } else {
                if (((m >> 2) & 15u) >= K || len == 0 || rem == 0 || rem > kMaxOutput) return MTS_EINVAL;
                if (st == kWaiting) {
                    w[k] = (1u << 30) | (rem << 16) | len;
                } else {
                    if (len + rem > 65535u) return MTS_EINVAL;
                    const uint32_t fin = uint32_t(h->tick) - 1u + rem;
                    w[k] = (2u << 30) | ((fin & 0x3FFFu) << 16) | (len + rem);
                }
            }
        }
        for (size_t i = 0; i < I; ++i) {
            const int32_t* m = v->mig + (size_t(r) * I + i) * 4;
            if (m[0] < -1 || m[0] >= int32_t(I) || m[0] == int32_t(i)) return MTS_EINVAL;
            if (m[0] >= 0 && (m[1] < 0 || m[1] >= int32_t(h->S) || m[2] < 0 || m[2] >= int32_t(h->S) || m[3] < 0))
                return MTS_EINVAL;
            const int32_t f = v->free[size_t(r) * I + i];
            if (f < -int32_t(h->cfg.kv_blocks) || f > int32_t(h->cfg.kv_blocks)) return MTS_EINVAL;
            if (v->drain && v->drain[size_t(r) * I + i] > 1) return MTS_EINVAL;
            if (v->svc && (v->svc[size_t(r) * I + i] < 0 || v->svc[size_t(r) * I + i] > (int64_t(1) << 40)))
                return MTS_EINVAL;
        }
        if (h->cfg.adapt_epoch && v->hq)
            for (uint32_t p = 0; p < MTS_MAX_TIERS; ++p) {
                const int32_t x = v->hq[size_t(r) * MTS_MAX_TIERS + p];
                if (x < 0 || uint32_t(x) > h->cfg.adapt_max || (p >= K && x != 0) ||
                    (h->cfg.zero_lowest_tier && p == K - 1 && x != 0))
                    return MTS_EINVAL;
            }
    }
    const Layout& L = h->lay;
    hipError_t e = hipStreamSynchronize(h->last);
    auto put = [&](size_t off, const void* src, size_t n) {
        if (e == hipSuccess && n) e = hipMemcpy(h->dev + off, src, n, hipMemcpyHostToDevice);
    };
    for (size_t k = 0; k < w.size(); ++k) {
        rec[4 * k] = w[k];
        rec[4 * k + 1] = v->meta[k];
        rec[4 * k + 2] = v->seq[k];
        rec[4 * k + 3] = v->tarr[k];
    }
    put(L.slot + size_t(r0) * IS * 16, rec.data(), rec.size() * 4);
    put(L.freeb + size_t(r0) * I * 4, v->free, size_t(nr) * I * 4);
    put(L.mig + size_t(r0) * I * 16, v->mig, size_t(nr) * I * 16);
    put(L.next_seq + size_t(r0) * 4, v->next_seq, size_t(nr) * 4);
    for (uint32_t r = 0; r < nr; ++r) h->seq_bound = std::max<uint64_t>(h->seq_bound, v->next_seq[r]);
    put(L.stats + size_t(r0) * MTS_NSTAT * 8, v->stats, size_t(nr) * MTS_NSTAT * 8);
    if (v->drain) {
        put(L.drain + size_t(r0) * I, v->drain, size_t(nr) * I);
    } else {
        const std::vector<uint8_t> none(size_t(nr) * I, 0);
        put(L.drain + size_t(r0) * I, none.data(), none.size());
    }
    const size_t hn = size_t(nr) * kHistPerReplica * 4;
    if (v->hist) {
        put(L.hist + size_t(r0) * kHistPerReplica * 4, v->hist, hn);
    } else if (e == hipSuccess && hn) {
        e = hipMemset(h->dev + L.hist + size_t(r0) * kHistPerReplica * 4, 0, hn);
    }
    const size_t sn = size_t(nr) * I * 8;
    if (v->svc) {
        put(L.svc + size_t(r0) * I * 8, v->svc, sn);
    } else if (e == hipSuccess && sn) {
        e = hipMemset(h->dev + L.svc + size_t(r0) * I * 8, 0, sn);
    }
    if (h->cfg.adapt_epoch) {
        // missing arrays: the group's Eq. 3 table; the imported counters as
        // the last update's
        std::vector<int32_t> hq(size_t(nr) * MTS_MAX_TIERS);
        std::vector<uint64_t> snap(size_t(nr) * 2 * MTS_MAX_TIERS);
        for (uint32_t r = 0; r < nr; ++r)
            for (uint32_t p = 0; p < MTS_MAX_TIERS; ++p) {
                const size_t k = size_t(r) * MTS_MAX_TIERS + p, k2 = size_t(r) * 2 * MTS_MAX_TIERS + p;
                hq[k] = v->hq ? v->hq[k] : h->tables.hq[size_t(h->group_of[r0 + r]) * MTS_MAX_TIERS + p];
                snap[k2] = v->hq_snap ? v->hq_snap[k2] : v->stats[size_t(r) * MTS_NSTAT + p * 8 + kAdmittedCnt];
                snap[k2 + MTS_MAX_TIERS] = v->hq_snap ? v->hq_snap[k2 + MTS_MAX_TIERS]
                                                      : v->stats[size_t(r) * MTS_NSTAT + p * 8 + kQdelay];
            }
        put(L.hqr + size_t(r0) * MTS_MAX_TIERS * 4, hq.data(), hq.size() * 4);
        put(L.hsnap + size_t(r0) * 2 * MTS_MAX_TIERS * 8, snap.data(), snap.size() * 8);
    }
    return hip_rc(e);
}

int mts_set_draining(mts_handle h, uint32_t r0, uint32_t nr, const uint8_t* flags)
{
    if (!h || (!flags && nr)) return MTS_EINVAL;
    if (r0 > h->R || nr > h->R - r0) return MTS_ERANGE;
    const size_t n = size_t(nr) * h->I;
    for (size_t k = 0; k < n; ++k)
        if (flags[k] > 1) return MTS_EINVAL;
    hipError_t e = hipStreamSynchronize(h->last);
    if (e == hipSuccess && n) e = hipMemcpy(h->dev + h->lay.drain + size_t(r0) * h->I, flags, n, hipMemcpyHostToDevice);
    return hip_rc(e);
}

int mts_get_table(mts_handle h, int which, uint32_t g, uint64_t* out, uint32_t cap, uint32_t* len, uint32_t* base)
{
    if (!h || !len || !base || (cap && !out)) return MTS_EINVAL;
    const Table* t = nullptr;
    switch (which) {
    case 0: if (g >= h->cfg.n_groups) return MTS_ERANGE; t = &h->tables.tier[g]; break;
    case 1: t = &h->tables.count; break;
    case 2: t = &h->tables.prompt; break;
    case 3: t = &h->tables.output; break;
    default: return MTS_ERANGE;
    }
    *len = uint32_t(t->q.size());
    *base = t->base;
    for (uint32_t j = 0; j < cap && j < t->q.size(); ++j) out[j] = t->q[j];
    return MTS_OK;
}

int mts_get_headroom(mts_handle h, uint32_t g, int32_t out[MTS_MAX_TIERS])
{
    if (!h || !out) return MTS_EINVAL;
    if (g >= h->cfg.n_groups) return MTS_ERANGE;
    std::memcpy(out, &h->tables.hq[size_t(g) * MTS_MAX_TIERS], MTS_MAX_TIERS * 4);
    return MTS_OK;
}

uint64_t mts_tick(mts_handle h) { return h ? h->tick : 0; }

int mts_set_tick(mts_handle h, uint64_t tick)
{
    if (!h) return MTS_EINVAL;
    if (tick > 0xFFFF0000ull) return MTS_ERANGE;
    const Params p = make_params(h);
    if (launch_shift_clock(p, uint32_t(tick - h->tick), h->last) != 0) return MTS_EDEVICE;
    if (hipStreamSynchronize(h->last) != hipSuccess) return MTS_EDEVICE;
    h->tick = tick;
    return MTS_OK;
}

int mts_set_wheel_cap(mts_handle h, uint32_t cap)
{
    if (!h || cap == 0 || cap > h->wcap_max) return MTS_EINVAL;
    // every step-kernel launch files the running requests into the wheel
    // afresh, so the capacity can change between steps
    if (hipStreamSynchronize(h->last) != hipSuccess) return MTS_EDEVICE;
    h->wcap = cap;
    return MTS_OK;
}

int mts_get_wheel(mts_handle h, uint32_t* cap, uint32_t* cap_max, uint64_t* rebuilds)
{
    if (!h) return MTS_EINVAL;
    if (cap) *cap = h->wcap;
    if (cap_max) *cap_max = h->wcap_max;
    if (rebuilds) {
        std::vector<uint64_t> st(size_t(h->R) * MTS_NSTAT);
        hipError_t e = hipStreamSynchronize(h->last);
        if (e == hipSuccess) e = hipMemcpy(st.data(), h->dev + h->lay.stats, st.size() * 8, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return MTS_EDEVICE;
        uint64_t n = 0;
        for (uint32_t r = 0; r < h->R; ++r) n += st[size_t(r) * MTS_NSTAT + kWheelRebuilds];
        *rebuilds = n;
    }
    return MTS_OK;
}

int mts_set_timing(mts_handle h, int on)
{
    if (!h || (on != 0 && on != 1)) return MTS_EINVAL;
    h->timing = on == 1;
    return MTS_OK;
}

int mts_get_timing(mts_handle h, double* step_ms, double* arrivals_ms, uint32_t* step_launches)
{
    if (!h) return MTS_EINVAL;
    double st = 0.0, ar = 0.0;
    int rc = MTS_OK;
    for (size_t k = 0; k + 2 < h->ev.size() && rc == MTS_OK; k += 3) {
        float a = 0.0f, b = 0.0f;
        if (hipEventSynchronize(h->ev[k + 2]) != hipSuccess || hipEventElapsedTime(&a, h->ev[k], h->ev[k + 1]) != hipSuccess ||
            hipEventElapsedTime(&b, h->ev[k + 1], h->ev[k + 2]) != hipSuccess)
            rc = MTS_EDEVICE;
        ar += a;
        st += b;
    }
    const uint32_t n = uint32_t(h->ev.size() / 3);
    for (hipEvent_t e : h->ev) (void)hipEventDestroy(e);
    h->ev.clear();
    if (step_ms) *step_ms = st;
    if (arrivals_ms) *arrivals_ms = ar;
    if (step_launches) *step_launches = n;
    return rc;
}

void mts_destroy(mts_handle h) { delete h; }

}  // extern "C"
