// Host-side configuration checks and table construction for libmts.
//
// Every distribution of the synthetic workload becomes a table of 32-bit
// quantised CDF values, q[j] = floor(2^32 * CDF(base + j)), the last entry
// being 2^32; a table ends at the first j whose remaining tail is below
// 2^-32 or at the distribution's upper bound.  The device samples
// base + min{j : u < q[j]} for a 32-bit uniform u.  The headroom table is
// Eq. 3 (H_p = h0 * gamma^p) in 1/256 block.
#include "mts_internal.h"

#include <cmath>
#include <cstring>

namespace mts {

namespace {

constexpr double kTwo32 = 4294967296.0;
constexpr uint64_t kOne = uint64_t(1) << 32;

double phi(double z) { return 0.5 * std::erfc(-z * 0.70710678118654752440); }

uint64_t quantise(double c)
{
    if (!(c > 0.0)) return 0;
    double x = std::floor(c * kTwo32);
    return x >= kTwo32 ? kOne : uint64_t(x);
}

bool tail_below(double c) { return (1.0 - c) * kTwo32 < 1.0; }

int tier_table(const mts_group& g, Table& t)
{
    const uint32_t K = g.K;
    t.base = 0;
    t.q.assign(K, 0);
    double w[MTS_MAX_TIERS] = {0}, total = 0.0, cum = 0.0;
    const bool weighted = g.tier_kind == MTS_TIERS_GEOMETRIC || g.tier_kind == MTS_TIERS_EXPLICIT;
    if (g.tier_kind == MTS_TIERS_GEOMETRIC) {
        w[K - 1] = 1.0;
        for (int j = int(K) - 2; j >= 0; --j) w[j] = w[j + 1] * g.p0;
    } else if (g.tier_kind == MTS_TIERS_EXPLICIT) {
        for (uint32_t j = 0; j < K; ++j) w[j] = g.probs[j];
    }
    if (weighted)
        for (uint32_t j = 0; j < K; ++j) total += w[j];
    for (uint32_t k = 0; k + 1 < K; ++k) {
        double c;
        if (g.tier_kind == MTS_TIERS_UNIFORM) c = double(k + 1) / double(K);
        else if (g.tier_kind == MTS_TIERS_GAUSS) c = phi((double(k) + 0.5 - g.p0) / g.p1);
        else { cum += w[k]; c = cum / total; }
        t.q[k] = quantise(c);
    }
    t.q[K - 1] = kOne;
    return MTS_OK;
}

int count_table(const mts_cfg& c, Table& t)
{
    t.base = 0;
    t.q.clear();
    double p, ratio = 0.0, shape = 0.0;
    if (c.arrival_kind == MTS_ARRIVAL_POISSON) {
        p = std::exp(-c.arrival_mean);
    } else {
        shape = 1.0 / (c.arrival_cv * c.arrival_cv);
        const double scale = c.arrival_mean * c.arrival_cv * c.arrival_cv;
        p = std::exp(-shape * std::log1p(scale));
        ratio = scale / (1.0 + scale);
    }
    double cum = p;
    for (uint32_t n = 0;; ++n) {
        if (n > 0) {
            if (c.arrival_kind == MTS_ARRIVAL_POISSON) p = p * c.arrival_mean / double(n);
            else p = p * ((double(n) - 1.0 + shape) / double(n)) * ratio;
            cum += p;
        }
        if (tail_below(cum)) { t.q.push_back(kOne); return MTS_OK; }
        if (n + 1 >= kMaxTable) return MTS_EINVAL;
        t.q.push_back(quantise(cum));
    }
}

int prompt_table(const mts_cfg& c, Table& t)
{
    const uint32_t lo = c.prompt_lo, hi = c.prompt_hi;
    t.base = lo;
    t.q.clear();
    for (uint32_t n = lo;; ++n) {
        double cdf = c.prompt_kind == MTS_PROMPT_UNIFORM_INT
                         ? double(n - lo + 1) / double(hi - lo + 1)
                         : phi((std::log(double(n) + 0.5) - c.prompt_mu) / c.prompt_sigma);
        if (n == hi || tail_below(cdf)) { t.q.push_back(kOne); return MTS_OK; }
        if (n - lo + 1 >= kMaxTable) return MTS_EINVAL;
        t.q.push_back(quantise(cdf));
    }
}

int output_table(const mts_cfg& c, Table& t)
{
    t.q.clear();
    if (c.output_kind == MTS_OUTPUT_GEOMETRIC) {
        const double q = 1.0 - 1.0 / c.output_param;
        double surv = 1.0;
        t.base = 1;
        for (uint32_t n = 1;; ++n) {
            surv = surv * q;
            if (surv * kTwo32 < 1.0) { t.q.push_back(kOne); return MTS_OK; }
            if (n >= kMaxTable) return MTS_EINVAL;
            t.q.push_back(quantise(1.0 - surv));
        }
    }
    const uint32_t lo = c.output_min, hi = c.output_cap;
    t.base = lo;
    for (uint32_t n = lo;; ++n) {
        const double surv = std::pow(double(lo) / (double(n) + 1.0), c.output_param);
        if (n == hi || surv * kTwo32 < 1.0) { t.q.push_back(kOne); return MTS_OK; }
        if (n - lo + 1 >= kMaxTable) return MTS_EINVAL;
        t.q.push_back(quantise(1.0 - surv));
    }
}

bool finite_pos(double v) { return std::isfinite(v) && v > 0.0; }

}  // namespace

int validate(const mts_cfg& c)
{
    if (c.abi_version != MTS_ABI_VERSION || c.reserved != 0 || c.reserved2 != 0 || c.tier_blind > 1) return MTS_EINVAL;
    if (c.dispatch_policy > MTS_POLICY_INFAAS || c.infaas_ewma_shift > 16) return MTS_EINVAL;
    if (c.infaas_alpha < 0 || c.infaas_alpha > 65536 || c.infaas_beta < 0 || c.infaas_beta > 1024 ||
        c.infaas_gamma < 0 || c.infaas_gamma > 65536)
        return MTS_EINVAL;
    if (c.infaas_pen_overloaded > (1u << 20) || c.infaas_pen_interfered > (1u << 20)) return MTS_EINVAL;
    // adaptive headroom: every H_p stays in [0, adapt_max], so the sum over
    // tiers keeps the freeness numerators below 2^30 like the static table
    if (c.adapt_margin > 256 || c.adapt_max > (1u << 29) / MTS_MAX_TIERS || c.adapt_epoch > (1u << 16)) return MTS_EINVAL;
    if (c.adapt_epoch)
        for (uint32_t p = 0; p < MTS_MAX_TIERS; ++p)
            if (c.adapt_slo[p] < 1 || c.adapt_slo[p] > (1u << 20)) return MTS_EINVAL;
    if (c.n_instances < 1 || c.n_instances > kMaxInstances) return MTS_EINVAL;
    if (c.slots_per_instance < 64 || c.slots_per_instance > kMaxSlots || c.slots_per_instance % 64) return MTS_EINVAL;
    if (c.kv_blocks < 1 || c.kv_blocks > kMaxBlocks) return MTS_EINVAL;
    if (c.block_tokens < 1 || c.block_tokens > kMaxBlockTokens || (c.block_tokens & (c.block_tokens - 1))) return MTS_EINVAL;
    if (c.zero_lowest_tier > 1) return MTS_EINVAL;
    if (!std::isfinite(c.headroom_base) || c.headroom_base < 0.0) return MTS_EINVAL;
    if (!std::isfinite(c.headroom_decay) || c.headroom_decay < 0.0 || c.headroom_decay > 1.0) return MTS_EINVAL;
    if (c.mig_interval < 1 || c.mig_stage_blocks < 1 || c.mig_max_pairs > c.n_instances / 2) return MTS_EINVAL;
    if (c.theta_num < 0 || c.theta_num >= (1 << 20) || c.theta_den < 1 || c.theta_den > 1024) return MTS_EINVAL;
    if (c.arrival_kind > MTS_ARRIVAL_GAMMA_POISSON || !finite_pos(c.arrival_mean) || c.arrival_mean > 1e5) return MTS_EINVAL;
    if (c.arrival_kind == MTS_ARRIVAL_GAMMA_POISSON && (!finite_pos(c.arrival_cv) || c.arrival_cv > 100.0)) return MTS_EINVAL;
    if (c.prompt_kind > MTS_PROMPT_LOGNORMAL || c.prompt_lo < 1 || c.prompt_hi < c.prompt_lo || c.prompt_hi > 65535) return MTS_EINVAL;
    if (c.prompt_kind == MTS_PROMPT_LOGNORMAL && (!std::isfinite(c.prompt_mu) || !finite_pos(c.prompt_sigma))) return MTS_EINVAL;
    if (c.output_kind > MTS_OUTPUT_PARETO) return MTS_EINVAL;
    if (c.output_kind == MTS_OUTPUT_GEOMETRIC && (!std::isfinite(c.output_param) || c.output_param < 1.0)) return MTS_EINVAL;
    if (c.output_kind == MTS_OUTPUT_PARETO &&
        (!finite_pos(c.output_param) || c.output_min < 1 || c.output_cap < c.output_min || c.output_cap > 65535))
        return MTS_EINVAL;
    if (c.n_groups < 1 || c.n_groups > kMaxGroups || c.groups == nullptr) return MTS_EINVAL;
    uint64_t R = 0;
    for (uint32_t g = 0; g < c.n_groups; ++g) {
        const mts_group& G = c.groups[g];
        if (G.n_replicas < 1 || G.K < 1 || G.K > MTS_MAX_TIERS || G.tier_kind > MTS_TIERS_EXPLICIT || G.reserved)
            return MTS_EINVAL;
        if (G.tier_kind == MTS_TIERS_GAUSS && (!std::isfinite(G.p0) || !finite_pos(G.p1))) return MTS_EINVAL;
        if (G.tier_kind == MTS_TIERS_GEOMETRIC && (!finite_pos(G.p0) || G.p0 > 1.0)) return MTS_EINVAL;
        if (G.tier_kind == MTS_TIERS_EXPLICIT) {
            double s = 0.0;
            for (uint32_t j = 0; j < G.K; ++j) {
                if (!std::isfinite(G.probs[j]) || G.probs[j] < 0.0) return MTS_EINVAL;
                s += G.probs[j];
            }
            if (!(s > 0.0)) return MTS_EINVAL;
        }
        R += G.n_replicas;
    }
    if (R > kMaxReplicas) return MTS_EINVAL;
    return MTS_OK;
}

void headroom(const mts_cfg& c, uint32_t K, int32_t out[MTS_MAX_TIERS])
{
    const double base = c.headroom_base * 256.0;
    double g = 1.0;
    for (uint32_t p = 0; p < MTS_MAX_TIERS; ++p) {
        out[p] = p < K ? int32_t(std::rint(base * g)) : 0;
        g = g * c.headroom_decay;
    }
    if (c.zero_lowest_tier) out[K - 1] = 0;
}

int build_tables(const mts_cfg& c, Tables& T)
{
    T.tier.resize(c.n_groups);
    T.hq.resize(size_t(c.n_groups) * MTS_MAX_TIERS);
    for (uint32_t g = 0; g < c.n_groups; ++g) {
        const double hb = c.headroom_base * 256.0;
        // keep every freeness numerator below 2^30 in magnitude
        if (hb > double(1 << 29)) return MTS_EINVAL;
        headroom(c, c.groups[g].K, &T.hq[size_t(g) * MTS_MAX_TIERS]);
        int64_t hsum = 0;
        for (uint32_t p = 0; p < MTS_MAX_TIERS; ++p) hsum += T.hq[size_t(g) * MTS_MAX_TIERS + p];
        if (hsum > (int64_t(1) << 29)) return MTS_EINVAL;
        if (c.adapt_epoch)
            for (uint32_t p = 0; p < MTS_MAX_TIERS; ++p)
                if (uint32_t(T.hq[size_t(g) * MTS_MAX_TIERS + p]) > c.adapt_max) return MTS_EINVAL;
        int rc = tier_table(c.groups[g], T.tier[g]);
        if (rc) return rc;
    }
    int rc = count_table(c, T.count);
    if (!rc) rc = prompt_table(c, T.prompt);
    if (!rc) rc = output_table(c, T.output);
    if (rc) return rc;
    // a request's length fits 16 bits and its remaining output 14 bits
    const uint64_t maxout = uint64_t(T.output.base) + T.output.q.size() - 1;
    const uint64_t maxlen = uint64_t(T.prompt.base) + T.prompt.q.size() - 1 + maxout;
    if (maxlen > 65535 || maxout > kMaxOutput) return MTS_EINVAL;
    return MTS_OK;
}

}  // namespace mts
