// Arrival sampling of libmts: every arrival of a chunk of ticks, for every
// replica, before the step kernel runs the chunk.
//
// Draws (Section 4.2 workloads; one stream per replica): Philox4x64-10 keyed
// by (seed, global replica id).  The count of tick t comes from counter
// (t, 0, 0, 0), word 0; arrival k of tick t from counter (t, k, 1, 0): tier
// from word 0, prompt length from word 1, output length from word 2 (low 32
// bits each).  A 32-bit uniform u becomes base + min{n : u < q[n]} of the
// distribution's quantised CDF table q.
//
// Output per (replica, tick): the count, and the arrivals as records
// prompt | out << 16 | tier << 32 | k << 36 sorted by tier, arrival order
// within a tier (Section 3.4: the pending queue is served tier 0 first); in
// arrival order when scheduling is tier-blind.
//
// A wave serves 64 / G ticks, G lanes each: the group's last lane draws the
// tick's count while the other G - 1 lanes draw the first G - 1 arrivals in
// the same Philox pass.  The rare tick with G or more arrivals is redrawn by
// the whole wave.
#include <hip/hip_runtime.h>

#include "mts_internal.h"
#include "mts_wave.h"

namespace mts {
namespace {

using namespace wave;

constexpr int kTiers = MTS_MAX_TIERS;

// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011) from its published
// round function and Weyl key schedule
__device__ inline void philox4x64_10(unsigned long long x[4], unsigned long long k0, unsigned long long k1)
{
    constexpr unsigned long long M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    constexpr unsigned long long W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const unsigned long long lo0 = M0 * x[0], hi0 = __umul64hi(M0, x[0]);
        const unsigned long long lo1 = M1 * x[2], hi1 = __umul64hi(M1, x[2]);
        const unsigned long long n0 = hi1 ^ x[1] ^ k0, n2 = hi0 ^ x[3] ^ k1;
        x[0] = n0; x[1] = lo1; x[2] = n2; x[3] = lo0;
        k0 += W0; k1 += W1;
    }
}

// min{n : u < q[n]} with q's last entry 2^32 implicit: the guide table g
// bounds the answer to [g[u >> shift], g[(u >> shift) + 1]] (indexed search,
// Chen and Asau 1974), a binary search finishes inside that range
__device__ __forceinline__ uint32_t sample(const uint32_t* q, const uint32_t* g, uint32_t shift, uint32_t u)
{
    const uint32_t j = u >> shift;
    uint32_t lo = g[j], hi = g[j + 1];
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (u < q[mid]) hi = mid; else lo = mid + 1;
    }
    return lo;
}

struct Draw {
    uint32_t tier;
    unsigned long long rec;
};

// tier, prompt and output length of arrival k from its Philox output x
__device__ __forceinline__ Draw arrival_of(const Params& P, const unsigned long long x[4], uint32_t k,
                                           const unsigned long long* tq, int K)
{
    const uint32_t ut = uint32_t(x[0]);
    uint32_t tier = 0;
#pragma unroll
    for (int j = 0; j < kTiers - 1; ++j) tier += (j < K - 1 && tq[j] <= ut) ? 1u : 0u;
    const uint32_t prompt = P.prompt_base + sample(P.prompt_q, P.prompt_g, P.prompt_gs, uint32_t(x[1]));
    const uint32_t outl = P.output_base + sample(P.output_q, P.output_g, P.output_gs, uint32_t(x[2]));
    Draw d;
    d.tier = tier;
    d.rec = static_cast<unsigned long long>(prompt) | (static_cast<unsigned long long>(outl) << 16) |
            (static_cast<unsigned long long>(tier) << 32) | (static_cast<unsigned long long>(k) << 36);
    return d;
}

__device__ __forceinline__ Draw draw_arrival(const Params& P, unsigned long long t, unsigned long long gid, uint32_t k,
                                             const unsigned long long* tq, int K)
{
    unsigned long long y[4] = {t, k, 1, 0};
    philox4x64_10(y, P.seed, gid);
    return arrival_of(P, y, k, tq, K);
}

// One (replica, tick) drawn by the whole wave, any number of arrivals.
__device__ void arrivals_wave(const Params& P, uint32_t r, uint32_t tl, unsigned long long t0, int lane)
{
    const unsigned long long t = t0 + tl;
    const unsigned long long gid = P.id_base + r;
    const uint32_t g = P.group_of[r];
    const int K = int(P.group_K32[g]);
    const unsigned long long* tq = P.tier_q + size_t(g) * kTiers;
    unsigned long long x[4] = {t, 0, 0, 0};
    philox4x64_10(x, P.seed, gid);
    const uint32_t n = P.count_base + sample(P.count_q, P.count_g, P.count_gs, uint32_t(x[0]));
    unsigned long long* out = P.arr_rec + (size_t(r) * P.chunk + tl) * P.arr_cap;
    if (lane == 0) P.arr_cnt[size_t(r) * P.chunk + tl] = n;
    if (n == 0) return;
    // pass 1: tier counts (tiers only)
    int cnt[kTiers];
#pragma unroll
    for (int p = 0; p < kTiers; ++p) cnt[p] = 0;
    for (uint32_t k0 = 0; k0 < n; k0 += 64) {
        const uint32_t k = k0 + lane;
        int tier = -1;
        if (k < n) {
            unsigned long long y[4] = {t, k, 1, 0};
            philox4x64_10(y, P.seed, gid);
            const uint32_t ut = uint32_t(y[0]);
            tier = 0;
#pragma unroll
            for (int j = 0; j < kTiers - 1; ++j) tier += (j < K - 1 && tq[j] <= ut) ? 1 : 0;
            if (P.blind) tier = 0;  // sorted by rank: arrival order when tier-blind
        }
#pragma unroll
        for (int p = 0; p < kTiers; ++p)
            if (p < K) cnt[p] += __popcll(ballot(tier == p));
    }
    int off[kTiers];
    int acc = 0;
#pragma unroll
    for (int p = 0; p < kTiers; ++p) { off[p] = acc; acc += cnt[p]; }
    // pass 2: draw again and scatter in tier order (a lane's draws are its own)
    for (uint32_t k0 = 0; k0 < n; k0 += 64) {
        const uint32_t k = k0 + lane;
        Draw d{~0u, 0};
        if (k < n) d = draw_arrival(P, t, gid, k, tq, K);
        int pos = 0;
        const uint32_t rk = P.blind && d.tier != ~0u ? 0u : d.tier;
#pragma unroll
        for (int p = 0; p < kTiers; ++p) {
            if (p >= K) continue;
            const unsigned long long b = ballot(rk == uint32_t(p));
            if (rk == uint32_t(p)) pos = off[p] + __popcll(b & lanemask_lt());
            off[p] += __popcll(b);
        }
        if (k < n) out[pos] = d.rec;
    }
}

template <int G>
__global__ __launch_bounds__(256) void k_arrivals(Params P, unsigned long long t0, uint32_t nt)
{
    constexpr uint32_t kTicksPerWave = 64 / G;
    const int lane = lane_id();
    const uint32_t q = uint32_t(lane) & (G - 1u), gb = uint32_t(lane) & ~(G - 1u);
    const uint32_t wv = blockIdx.x * 4 + (threadIdx.x >> 6);
    const uint32_t items = P.R * nt;
    if (wv * kTicksPerWave >= items) return;
    const uint32_t item = wv * kTicksPerWave + uint32_t(lane) / G;
    const bool live = item < items;
    const uint32_t r = live ? item / nt : 0, tl = live ? item % nt : 0;
    const unsigned long long t = t0 + tl;
    const unsigned long long gid = P.id_base + r;
    const uint32_t g = P.group_of[r];
    const int K = int(P.group_K32[g]);
    const unsigned long long* tq = P.tier_q + size_t(g) * kTiers;
    // one Philox pass: the count on the group's last lane, arrival q elsewhere
    const bool cl = q == G - 1u;
    unsigned long long x[4] = {t, cl ? 0ull : q, cl ? 0ull : 1ull, 0};
    philox4x64_10(x, P.seed, gid);
    uint32_t n = 0;
    Draw d{~0u, 0};
    if (cl) n = P.count_base + sample(P.count_q, P.count_g, P.count_gs, uint32_t(x[0]));
    else d = arrival_of(P, x, q, tq, K);
    n = uint32_t(__shfl(int(n), int(gb + G - 1u)));
    const bool fast = n < G;  // every arrival of the tick was drawn
    if (live && cl) P.arr_cnt[size_t(r) * P.chunk + tl] = n;
    const bool mine = live && fast && q < n;
    const unsigned long long gm = G == 64 ? ~0ull : ((1ull << G) - 1ull) << gb;
    int pos = 0, off = 0;
    const uint32_t rk = P.blind ? 0u : d.tier;  // sorted by rank: arrival order when tier-blind
#pragma unroll
    for (int p = 0; p < kTiers; ++p) {
        const unsigned long long b = ballot(mine && rk == uint32_t(p)) & gm;
        if (mine && rk == uint32_t(p)) pos = off + __popcll(b & lanemask_lt());
        off += __popcll(b);
    }
    if (mine) P.arr_rec[(size_t(r) * P.chunk + tl) * P.arr_cap + pos] = d.rec;
    // ticks with G or more arrivals: the whole wave draws them again
    for (unsigned long long ov = ballot(live && cl && !fast); ov; ov &= ov - 1) {
        const int l = ffs64(ov);
        arrivals_wave(P, uint32_t(rl(int(r), l)), uint32_t(rl(int(tl), l)), t0, lane);
    }
}

}  // namespace

int launch_arrivals(const Params& p, unsigned long long t0, uint32_t nt, hipStream_t stream)
{
    const uint32_t items = p.R * nt;
    const uint32_t tpw = 64 / p.arr_group;
    const uint32_t waves = (items + tpw - 1) / tpw;
    const dim3 grid((waves + 3) / 4), block(256);
    switch (p.arr_group) {
    case 16: hipLaunchKernelGGL(k_arrivals<16>, grid, block, 0, stream, p, t0, nt); break;
    case 32: hipLaunchKernelGGL(k_arrivals<32>, grid, block, 0, stream, p, t0, nt); break;
    default: hipLaunchKernelGGL(k_arrivals<64>, grid, block, 0, stream, p, t0, nt); break;
    }
    return int(hipGetLastError());
}

}  // namespace mts
