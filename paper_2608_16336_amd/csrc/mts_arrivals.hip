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

// Ticks with fewer than kDense arrivals go through the dense path; a wave
// stages at most kCap of their records in LDS at a time.
constexpr uint32_t kDense = 64;
constexpr uint32_t kCap = 512;
constexpr int kWavesPerBlock = 4;

// A wave serves 64 consecutive (replica, tick) items.  Lane l draws the count
// of item l; an inclusive wave scan lays the items' arrivals end to end, and
// the lanes then draw that flat list 64 arrivals at a time, every lane busy.
// The list is cut into segments of whole ticks that fit kCap; a segment is
// drawn into LDS, then each arrival counts the arrivals of its tick that sort
// before it (tier, then arrival order; arrival order alone when tier-blind)
// and writes its record at that rank.  Items with kDense or more arrivals are
// drawn afterwards by the whole wave, one at a time.
__global__ __launch_bounds__(64 * kWavesPerBlock) void k_arrivals(Params P, unsigned long long t0, uint32_t nt)
{
    __shared__ unsigned long long stage[kWavesPerBlock][kCap];
    __shared__ uint8_t owner[kWavesPerBlock][kCap];
    const int lane = lane_id();
    const uint32_t w = threadIdx.x >> 6;
    const uint32_t wv = blockIdx.x * kWavesPerBlock + w;
    const uint32_t items = P.R * nt;
    if (wv * 64u >= items) return;
    unsigned long long* L = stage[w];
    const uint32_t* L32 = reinterpret_cast<const uint32_t*>(L);
    uint8_t* own = owner[w];
    const uint32_t item = wv * 64u + uint32_t(lane);
    const bool live = item < items;
    const uint32_t r = live ? item / nt : 0, tl = live ? item % nt : 0;
    const uint32_t g = P.group_of[r];
    const int K = int(P.group_K32[g]);
    unsigned long long x[4] = {t0 + tl, 0, 0, 0};
    philox4x64_10(x, P.seed, P.id_base + r);
    uint32_t n = 0;
    if (live) {
        n = P.count_base + sample(P.count_q, P.count_g, P.count_gs, uint32_t(x[0]));
        P.arr_cnt[size_t(r) * P.chunk + tl] = n;
    }
    const uint32_t nd = n < kDense ? n : 0;
    uint32_t e = nd;  // inclusive scan: the item's arrivals are [e - nd, e) of the flat list
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t v = uint32_t(__shfl_up(int(e), d));
        if (lane >= d) e += v;
    }
    const uint32_t s = e - nd;
    const uint32_t total = rlu(e, 63);
    for (uint32_t base = 0; base < total;) {
        // the segment: every item whose arrivals end by base + kCap (a prefix of
        // the lanes, never empty since no dense item holds kCap arrivals)
        const unsigned long long fit = ballot(e <= base + kCap);
        const uint32_t end = rlu(e, 63 - __clzll(static_cast<long long>(fit)));
        for (uint32_t f0 = base; f0 < end; f0 += 64) {
            const uint32_t f = f0 + uint32_t(lane);
            const uint32_t fc = f < end ? f : end - 1;
            // owner: the last lane whose arrivals start at or before fc
            int i = 0;
            uint32_t si = 0;
#pragma unroll
            for (int step = 32; step; step >>= 1) {
                const uint32_t v = uint32_t(__shfl(int(s), i + step));
                if (v <= fc) { i += step; si = v; }
            }
            const uint32_t ri = uint32_t(__shfl(int(r), i)), ti = uint32_t(__shfl(int(tl), i));
            const uint32_t gi = uint32_t(__shfl(int(g), i));
            const int Ki = __shfl(K, i);
            if (f < end) {
                const Draw d = draw_arrival(P, t0 + ti, P.id_base + ri, f - si, P.tier_q + size_t(gi) * kTiers, Ki);
                L[f - base] = d.rec;
                own[f - base] = uint8_t(i);
            }
        }
        wave_sync();
        for (uint32_t f0 = base; f0 < end; f0 += 64) {
            const uint32_t f = f0 + uint32_t(lane);
            const uint32_t j = (f < end ? f : end - 1) - base;
            const int i = own[j];
            const uint32_t si = uint32_t(__shfl(int(s), i)) - base, ni = uint32_t(__shfl(int(nd), i));
            const uint32_t ri = uint32_t(__shfl(int(r), i)), ti = uint32_t(__shfl(int(tl), i));
            if (f < end) {
                // high word of a record: tier | k << 4; (tier, k) order is key order
                const uint32_t hw = L32[2 * j + 1];
                uint32_t pos = j - si;
                if (!P.blind) {
                    const uint32_t key = (hw & 15u) << 6 | (hw >> 4);
                    pos = 0;
                    for (uint32_t m = si; m < si + ni; ++m) {
                        const uint32_t hm = L32[2 * m + 1];
                        pos += ((hm & 15u) << 6 | (hm >> 4)) < key ? 1u : 0u;
                    }
                }
                P.arr_rec[(size_t(ri) * P.chunk + ti) * P.arr_cap + pos] = L[j];
            }
        }
        wave_sync();
        base = end;
    }
    for (unsigned long long ov = ballot(live && n >= kDense); ov; ov &= ov - 1) {
        const int l = ffs64(ov);
        arrivals_wave(P, rlu(r, l), rlu(tl, l), t0, lane);
    }
}

}  // namespace

int launch_arrivals(const Params& p, unsigned long long t0, uint32_t nt, hipStream_t stream)
{
    const uint32_t waves = (p.R * nt + 63) / 64;
    const dim3 grid((waves + kWavesPerBlock - 1) / kWavesPerBlock), block(64 * kWavesPerBlock);
    hipLaunchKernelGGL(k_arrivals, grid, block, 0, stream, p, t0, nt);
    return int(hipGetLastError());
}

}  // namespace mts
