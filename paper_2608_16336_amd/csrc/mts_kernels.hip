// Device code of libmts: the persistent multi-tick scheduling kernel, the
// state initialiser and the state digest.
//
// Mapping.  One block owns one replica at a time and runs all n_ticks ticks
// of it before taking the next replica (replicas never interact, so there is
// no grid-wide synchronisation).  Within a block, wave w handles instances
// w, w + nwaves, ... in the per-instance phases (A, B, C); wave 0 runs the
// replica-wide serial phases (A2, D, E).  Slot state lives in HBM in the
// canonical SoA layout (meta u8, lr u32, seq u32, tarr u32, each [R][I][S]),
// scanned 64 consecutive slots per wave instruction.  Per-instance summaries,
// the slot occupancy bitmap and the replica's counters live in LDS for the
// whole launch.
#include <hip/hip_runtime.h>

#include "mts_internal.h"

namespace mts {
namespace {

constexpr int kNstat = MTS_NSTAT;
constexpr int kTiers = MTS_MAX_TIERS;
constexpr unsigned long long kNone = ~0ull;

// ---------------------------------------------------------------------------
// LDS layout of one block (sizes depend on I and W = S / 64)
// ---------------------------------------------------------------------------
struct LdsLayout {
    uint32_t stats, occ, q, ints, tcnt, bytes, total;
};

constexpr int kIntArrays = 17;  // see Lds below
constexpr int kMisc = 16;

__host__ __device__ inline uint32_t align8(uint32_t x) { return (x + 7u) & ~7u; }

__host__ __device__ inline LdsLayout lds_layout(uint32_t I, uint32_t W)
{
    LdsLayout L;
    uint32_t o = 0;
    L.stats = o; o += kNstat * 8;
    L.occ = o;   o += I * W * 8;
    L.q = o;     o += I * 8;
    L.ints = o;  o += (I * kIntArrays + kTiers + kMisc) * 4; o = align8(o);
    L.tcnt = o;  o += I * kTiers * 2; o = align8(o);
    L.bytes = o; o += I * 2; o = align8(o);
    L.total = o;
    return L;
}

struct Lds {
    unsigned long long* stats;  // [88] this replica's counters
    unsigned long long* occ;    // [I][W] bit s%64 of word s/64: slot s not empty
    long long* q;               // [I] floor(num * 2^24 / den): exact order key of F
    int* freeb;                 // [I] free blocks
    int* B;                     // [I] running requests
    int* live;                  // [I] non-empty slots
    int* hwm;                   // [I] 1 + highest non-empty slot
    int* hol_slot;              // [I] head-of-line slot or -1
    int* hol_tier;
    unsigned* hol_seq;
    int* hol_dem;               // [I] head-of-line demand in blocks (0 if none)
    int* num;                   // [I] freeness numerator, 1/256 block
    int* den;                   // [I] max(B, 1)
    int* inb;                   // [I] blocks copied into this instance's inbound reservation
    int* mig;                   // [I][4] dst, src slot, dst slot, copied
    int* order;                 // [I] instances ranked for pairing
    int* hl;                    // [10] headroom of this replica's group
    int* misc;                  // [16] block-wide scalars
    unsigned short* tcnt;       // [I][10] running requests per tier
    unsigned char* abort_;      // [I] source migration must be released
    unsigned char* busy;        // [I] in a migration
};

__device__ inline Lds carve(char* base, uint32_t I, uint32_t W)
{
    const LdsLayout Y = lds_layout(I, W);
    Lds L;
    L.stats = reinterpret_cast<unsigned long long*>(base + Y.stats);
    L.occ = reinterpret_cast<unsigned long long*>(base + Y.occ);
    L.q = reinterpret_cast<long long*>(base + Y.q);
    int* p = reinterpret_cast<int*>(base + Y.ints);
    L.freeb = p; p += I;
    L.B = p; p += I;
    L.live = p; p += I;
    L.hwm = p; p += I;
    L.hol_slot = p; p += I;
    L.hol_tier = p; p += I;
    L.hol_seq = reinterpret_cast<unsigned*>(p); p += I;
    L.hol_dem = p; p += I;
    L.num = p; p += I;
    L.den = p; p += I;
    L.inb = p; p += I;
    L.mig = p; p += 4 * I;
    L.order = p; p += I;
    L.hl = p; p += kTiers;
    L.misc = p; p += kMisc;
    L.tcnt = reinterpret_cast<unsigned short*>(base + Y.tcnt);
    L.abort_ = reinterpret_cast<unsigned char*>(base + Y.bytes);
    L.busy = L.abort_ + I;
    return L;
}

// ---------------------------------------------------------------------------
// wave helpers (wave64)
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ unsigned long long ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ unsigned long long lanemask_lt() { return (1ull << lane_id()) - 1ull; }

__device__ __forceinline__ int wsum(int x)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

__device__ __forceinline__ unsigned long long wmax64(unsigned long long x)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        unsigned long long y = __shfl_xor(x, o);
        x = y > x ? y : x;
    }
    return x;
}

__device__ __forceinline__ unsigned long long wmin64(unsigned long long x)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        unsigned long long y = __shfl_xor(x, o);
        x = y < x ? y : x;
    }
    return x;
}

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011), written from the
// published round function and Weyl key schedule.
// ---------------------------------------------------------------------------
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

// base + min{j : u < q[j]} over a table of n entries whose last (2^32) is implicit
__device__ inline uint32_t sample(const uint32_t* q, uint32_t n, uint32_t u)
{
    uint32_t lo = 0, hi = n - 1;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (u < q[mid]) hi = mid; else lo = mid + 1;
    }
    return lo;
}

__device__ __forceinline__ int blocks_of(uint32_t len, uint32_t shift)
{
    return int((len + (1u << shift) - 1u) >> shift);
}

// Freeness of instance i (Eq. 1-4): num = 256 (free - hol) - sum of H_p over
// the tiers with a running request, den = max(B, 1); q orders F exactly.
__device__ inline void set_f(const Lds& L, int i, int K)
{
    int hs = 0;
    for (int p = 0; p < K; ++p) hs += L.tcnt[i * kTiers + p] ? L.hl[p] : 0;
    const long long num = 256ll * (L.freeb[i] - L.hol_dem[i]) - hs;
    const int den = L.B[i] > 0 ? L.B[i] : 1;
    const long long n = num * (1ll << 24);
    const long long q = n >= 0 ? n / den : -((-n + den - 1) / den);
    L.num[i] = int(num);
    L.den[i] = den;
    L.q[i] = q;
}

// dispatch key: larger F first, then smaller index; 0 is never a valid key
__device__ __forceinline__ unsigned long long dkey(long long q, int i)
{
    return (static_cast<unsigned long long>(q + (1ll << 54) + 1) << 8) | unsigned(255 - i);
}

// pairing key: smaller F first, then smaller index
__device__ __forceinline__ unsigned long long pkey(long long q, int i)
{
    return (static_cast<unsigned long long>(q + (1ll << 54) + 1) << 8) | unsigned(i);
}

// lowest empty slot of instance i (caller guarantees one exists); uniform
__device__ inline int lowest_empty(const Lds& L, int i, uint32_t W, int lane, int* word, unsigned long long* wval)
{
    const unsigned long long w = lane < int(W) ? L.occ[i * W + lane] : kNone;
    const unsigned long long fm = ballot(w != kNone);
    const int c0 = __ffsll(static_cast<long long>(fm)) - 1;
    if (c0 < 0) return -1;
    const unsigned long long w0 = __shfl(w, c0);
    const int bit = __ffsll(static_cast<long long>(~w0)) - 1;
    *word = c0;
    *wval = w0;
    return c0 * 64 + bit;
}

__device__ inline void stat_add(const Lds& L, int idx, unsigned long long v)
{
    atomicAdd(&L.stats[idx], v);
}

// ---------------------------------------------------------------------------
// The step kernel
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_step(Params P)
{
    extern __shared__ __align__(16) char lds_raw[];
    const uint32_t I = P.I, S = P.S, W = P.W;
    const Lds L = carve(lds_raw, I, W);
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int nwaves = blockDim.x >> 6;
    const uint32_t shift = P.blk_shift;
    const uint32_t bmask = (1u << shift) - 1u;

    for (uint32_t r = blockIdx.x; r < P.R; r += gridDim.x) {
        const uint32_t g = P.group_of[r];
        const int K = int(P.group_K32[g]);
        const unsigned long long gid = P.id_base + r;
        const size_t rbase = size_t(r) * I * S;

        // ---- load the replica ----
        for (int j = threadIdx.x; j < kNstat; j += blockDim.x) L.stats[j] = P.stats[size_t(r) * kNstat + j];
        for (int j = threadIdx.x; j < kTiers; j += blockDim.x) L.hl[j] = P.hq[g * kTiers + j];
        for (uint32_t i = threadIdx.x; i < I; i += blockDim.x) {
            L.freeb[i] = P.freeb[size_t(r) * I + i];
            for (int k = 0; k < 4; ++k) L.mig[4 * i + k] = P.mig[(size_t(r) * I + i) * 4 + k];
            L.abort_[i] = 0;
        }
        // high-water marks from a full scan
        for (uint32_t i = wave; i < I; i += nwaves) {
            const uint8_t* mt = P.meta + rbase + size_t(i) * S;
            int top = -1;
            for (uint32_t c = 0; c < W; ++c) {
                const unsigned long long b = ballot(mt[c * 64 + lane] != 0);
                if (b) top = int(c * 64 + 63 - __clzll(static_cast<long long>(b)));
            }
            if (lane == 0) L.hwm[i] = top + 1;
        }
        unsigned next_seq = P.next_seq[r];
        __syncthreads();

        for (unsigned long long t = P.tick0; t < P.tick0 + P.n_ticks; ++t) {
            // ================= A: decode, growth, preemption, finish =================
            for (uint32_t i = wave; i < I; i += nwaves) {
                const size_t ib = rbase + size_t(i) * S;
                uint8_t* mt = P.meta + ib;
                uint32_t* lr = P.lr + ib;
                uint32_t* sq = P.seq + ib;
                uint32_t* ta = P.tarr + ib;
                const int nch = (L.hwm[i] + 63) >> 6;
                int grow = 0;
                for (int c = 0; c < nch; ++c) {
                    const int s = c * 64 + lane;
                    bool gr = false;
                    if ((mt[s] & 3u) == kRunning) gr = (lr[s] & bmask) == 0;
                    grow += __popcll(ballot(gr));
                }
                int fr = L.freeb[i];
                while (grow > fr) {
                    // victim: the running request with the largest (tier, seq)
                    unsigned long long bk = 0;
                    int bs = 0;
                    for (int c = 0; c < nch; ++c) {
                        const int s = c * 64 + lane;
                        const unsigned m = mt[s];
                        if ((m & 3u) == kRunning) {
                            const unsigned long long k = (static_cast<unsigned long long>(((m >> 2) & 15u) + 1u) << 32) | sq[s];
                            if (k > bk) { bk = k; bs = s; }
                        }
                    }
                    const unsigned long long mx = wmax64(bk);
                    if (mx == 0) break;
                    const int wl = __ffsll(static_cast<long long>(ballot(bk == mx))) - 1;
                    const int v = __shfl(bs, wl);
                    int vb = 0, vg = 0, vt = 0, vm = 0;
                    if (lane == (v & 63)) {
                        const unsigned m = mt[v];
                        const unsigned len = lr[v] & 0xFFFFu;
                        vt = int((m >> 2) & 15u);
                        vm = (m & kMigrating) ? 1 : 0;
                        mt[v] = uint8_t((m & ~(3u | kMigrating)) | kWaiting);
                        vb = blocks_of(len, shift);
                        vg = (len & bmask) == 0;
                    }
                    vb = __shfl(vb, v & 63);
                    vg = __shfl(vg, v & 63);
                    vt = __shfl(vt, v & 63);
                    vm = __shfl(vm, v & 63);
                    fr += vb;
                    grow -= vg;
                    if (lane == 0) {
                        stat_add(L, vt * 8 + kPreempted, 1);
                        if (vm) L.abort_[i] = 1;
                    }
                }
                fr -= grow;
                int freed = 0;
                bool ab = false;
                for (int c = 0; c < nch; ++c) {
                    const int s = c * 64 + lane;
                    const unsigned m = mt[s];
                    if ((m & 3u) != kRunning) continue;
                    const unsigned v = lr[s];
                    const unsigned len = (v & 0xFFFFu) + 1u, rem = (v >> 16) - 1u;
                    if (rem == 0) {
                        freed += blocks_of(len, shift);
                        const int tier = int((m >> 2) & 15u);
                        stat_add(L, tier * 8 + kFinished, 1);
                        stat_add(L, tier * 8 + kE2e, t - ta[s]);
                        if (m & kMigrating) ab = true;
                        mt[s] = 0; lr[s] = 0; sq[s] = 0; ta[s] = 0;
                    } else {
                        lr[s] = len | (rem << 16);
                    }
                }
                fr += wsum(freed);
                const bool any_ab = ballot(ab) != 0;
                if (lane == 0) {
                    L.freeb[i] = fr;
                    if (any_ab) L.abort_[i] = 1;
                }
            }
            __syncthreads();

            // ================= A2: release aborted reservations =================
            if (wave == 0) {
                for (uint32_t i = lane; i < I; i += 64) {
                    if (!L.abort_[i]) continue;
                    L.abort_[i] = 0;
                    int* m = &L.mig[4 * i];
                    const int d = m[0];
                    if (d < 0) continue;
                    L.freeb[d] += m[3];
                    const size_t db = rbase + size_t(d) * S + m[2];
                    P.meta[db] = 0; P.lr[db] = 0; P.seq[db] = 0; P.tarr[db] = 0;
                    m[0] = -1; m[1] = 0; m[2] = 0; m[3] = 0;
                    stat_add(L, kMigAborted, 1);
                }
                for (uint32_t i = lane; i < I; i += 64) L.inb[i] = 0;
                for (uint32_t i = lane; i < I; i += 64) {
                    const int d = L.mig[4 * i];
                    if (d >= 0) L.inb[d] = L.mig[4 * i + 3];
                }
            }
            __syncthreads();

            // ================= B: admission, C: per-instance summary =================
            for (uint32_t i = wave; i < I; i += nwaves) {
                const size_t ib = rbase + size_t(i) * S;
                uint8_t* mt = P.meta + ib;
                uint32_t* lr = P.lr + ib;
                uint32_t* sq = P.seq + ib;
                uint32_t* ta = P.tarr + ib;
                const int nch = (L.hwm[i] + 63) >> 6;
                int fr = L.freeb[i];
                int hslot = -1, hdem = 0;
                unsigned long long hkey = kNone;
                for (;;) {
                    unsigned long long bk = kNone;
                    int bs = 0;
                    for (int c = 0; c < nch; ++c) {
                        const int s = c * 64 + lane;
                        const unsigned m = mt[s];
                        if ((m & 3u) == kWaiting) {
                            const unsigned long long k = (static_cast<unsigned long long>((m >> 2) & 15u) << 32) | sq[s];
                            if (k < bk) { bk = k; bs = s; }
                        }
                    }
                    const unsigned long long mn = wmin64(bk);
                    if (mn == kNone) break;
                    const int wl = __ffsll(static_cast<long long>(ballot(bk == mn))) - 1;
                    const int h = __shfl(bs, wl);
                    int need = 0;
                    if (lane == (h & 63)) need = blocks_of(lr[h] & 0xFFFFu, shift);
                    need = __shfl(need, h & 63);
                    if (need > fr) { hslot = h; hdem = need; hkey = mn; break; }
                    fr -= need;
                    if (lane == (h & 63)) {
                        const unsigned m = mt[h];
                        mt[h] = uint8_t((m & ~3u) | kRunning | kAdmitted);
                        if (!(m & kAdmitted)) {
                            const int tier = int((m >> 2) & 15u);
                            stat_add(L, tier * 8 + kAdmittedCnt, 1);
                            stat_add(L, tier * 8 + kQdelay, t - ta[h]);
                        }
                    }
                }
                // C: summary scan
                int nB = 0, nlive = 0, nwait = 0, held = 0, top = -1;
                int tc[kTiers];
#pragma unroll
                for (int p = 0; p < kTiers; ++p) tc[p] = 0;
                for (int c = 0; c < nch; ++c) {
                    const int s = c * 64 + lane;
                    const unsigned m = mt[s];
                    const unsigned st = m & 3u;
                    const bool run = st == kRunning;
                    const unsigned long long ow = ballot(st != kEmpty);
                    nB += __popcll(ballot(run));
                    nlive += __popcll(ow);
                    nwait += __popcll(ballot(st == kWaiting));
                    if (run) held += blocks_of(lr[s] & 0xFFFFu, shift);
                    const int tier = int((m >> 2) & 15u);
#pragma unroll
                    for (int p = 0; p < kTiers; ++p)
                        if (p < K) tc[p] += __popcll(ballot(run && tier == p));
                    if (ow) top = c * 64 + 63 - __clzll(static_cast<long long>(ow));
                    if (lane == 0) L.occ[i * W + c] = ow;
                }
                for (uint32_t c = nch + lane; c < W; c += 64) L.occ[i * W + c] = 0;
                held = wsum(held);
                if (lane == 0) {
                    L.freeb[i] = fr;
                    L.B[i] = nB;
                    L.live[i] = nlive;
                    L.hwm[i] = top + 1;
                    for (int p = 0; p < kTiers; ++p) L.tcnt[i * kTiers + p] = (unsigned short)(p < K ? tc[p] : 0);
                    L.hol_slot[i] = hslot;
                    L.hol_tier[i] = int(hkey >> 32);
                    L.hol_seq[i] = unsigned(hkey);
                    L.hol_dem[i] = hslot >= 0 ? hdem : 0;
                    if (fr < 0 || fr + held + L.inb[i] != int(P.M)) stat_add(L, kInvariant, 1);
                    set_f(L, int(i), K);
                    stat_add(L, kRunSlotTicks, nB);
                    stat_add(L, kWaitSlotTicks, nwait);
                }
            }
            __syncthreads();

            // ================= D: arrivals and tier-ordered dispatch =================
            if (wave == 0) {
                unsigned long long x[4] = {t, 0, 0, 0};
                philox4x64_10(x, P.seed, gid);
                const uint32_t n = P.count_base + sample(P.count_q, P.count_n, uint32_t(x[0]));
                const unsigned seq0 = next_seq;
                next_seq += n;
                unsigned long long* raw = P.scratch + size_t(blockIdx.x) * 2 * P.max_arrivals;
                unsigned long long* sorted = raw + P.max_arrivals;
                const uint32_t* tq = P.tier_q + size_t(g) * kTiers;
                int cnt[kTiers];
#pragma unroll
                for (int p = 0; p < kTiers; ++p) cnt[p] = 0;
                for (uint32_t k0 = 0; k0 < n; k0 += 64) {
                    const uint32_t k = k0 + lane;
                    const bool ok = k < n;
                    int tier = 0;
                    if (ok) {
                        unsigned long long y[4] = {t, k, 1, 0};
                        philox4x64_10(y, P.seed, gid);
                        tier = int(sample(tq, uint32_t(K), uint32_t(y[0])));
                        const uint32_t prompt = P.prompt_base + sample(P.prompt_q, P.prompt_n, uint32_t(y[1]));
                        const uint32_t out = P.output_base + sample(P.output_q, P.output_n, uint32_t(y[2]));
                        raw[k] = static_cast<unsigned long long>(prompt) | (static_cast<unsigned long long>(out) << 16) |
                                 (static_cast<unsigned long long>(tier) << 32) | (static_cast<unsigned long long>(k) << 36);
                    }
#pragma unroll
                    for (int p = 0; p < kTiers; ++p)
                        if (p < K) cnt[p] += __popcll(ballot(ok && tier == p));
                }
                int off[kTiers];
                int acc = 0;
#pragma unroll
                for (int p = 0; p < kTiers; ++p) {
                    off[p] = acc;
                    acc += p < K ? cnt[p] : 0;
                    if (lane == 0 && p < K && cnt[p]) stat_add(L, p * 8 + kArrived, cnt[p]);
                }
                // stable scatter by tier (a lane reads back only what it wrote)
                for (uint32_t k0 = 0; k0 < n; k0 += 64) {
                    const uint32_t k = k0 + lane;
                    const bool ok = k < n;
                    const unsigned long long a = ok ? raw[k] : 0;
                    const int tier = int((a >> 32) & 15u);
                    int pos = 0;
#pragma unroll
                    for (int p = 0; p < kTiers; ++p) {
                        if (p >= K) continue;
                        const unsigned long long b = ballot(ok && tier == p);
                        if (ok && tier == p) pos = off[p] + __popcll(b & lanemask_lt());
                        off[p] += __popcll(b);
                    }
                    if (ok) sorted[pos] = a;
                }
                __threadfence_block();

                int cur = -1;
                for (uint32_t j = 0; j < n; ++j) {
                    const unsigned long long a = sorted[j];
                    const int tier = int((a >> 32) & 15u);
                    if (cur < 0) {
                        unsigned long long best = 0;
                        for (uint32_t i = lane; i < I; i += 64)
                            if (L.live[i] < int(S)) {
                                const unsigned long long k = dkey(L.q[i], int(i));
                                best = k > best ? k : best;
                            }
                        best = wmax64(best);
                        if (best == 0) {
                            // no free slot anywhere: the rest of this tick's arrivals are rejected
                            for (uint32_t jj = j + lane; jj < n; jj += 64)
                                stat_add(L, int((sorted[jj] >> 32) & 15u) * 8 + kRejected, 1);
                            break;
                        }
                        cur = 255 - int(best & 255u);
                    }
                    int c0;
                    unsigned long long w0;
                    const int s = lowest_empty(L, cur, W, lane, &c0, &w0);
                    if (s < 0) {  // occupancy and live count disagree: flag and drop the arrival
                        if (lane == 0) { stat_add(L, kInvariant, 1); stat_add(L, tier * 8 + kRejected, 1); L.live[cur] = int(S); }
                        cur = -1;
                        continue;
                    }
                    const unsigned seqv = seq0 + unsigned(a >> 36);
                    const uint32_t prompt = uint32_t(a & 0xFFFFu);
                    const bool becomes = L.hol_slot[cur] < 0 || tier < L.hol_tier[cur] ||
                                         (tier == L.hol_tier[cur] && seqv < L.hol_seq[cur]);
                    if (lane == 0) {
                        const size_t sb = rbase + size_t(cur) * S + s;
                        P.meta[sb] = uint8_t(kWaiting | (unsigned(tier) << 2));
                        P.lr[sb] = uint32_t(a & 0xFFFFFFFFu);
                        P.seq[sb] = seqv;
                        P.tarr[sb] = uint32_t(t);
                        L.occ[cur * W + c0] = w0 | (1ull << (s & 63));
                        L.live[cur] += 1;
                        if (s + 1 > L.hwm[cur]) L.hwm[cur] = s + 1;
                        stat_add(L, tier * 8 + kDispatched, 1);
                        stat_add(L, kWaitSlotTicks, 1);
                        if (becomes) {
                            L.hol_slot[cur] = s;
                            L.hol_tier[cur] = tier;
                            L.hol_seq[cur] = seqv;
                            L.hol_dem[cur] = blocks_of(prompt, shift);
                            set_f(L, cur, K);
                        }
                    }
                    if (becomes || L.live[cur] >= int(S)) cur = -1;
                }
            }
            __syncthreads();

            // ================= E1: staged copies =================
            if (wave == 0) {
                for (uint32_t i = lane; i < I; i += 64) {
                    int* m = &L.mig[4 * i];
                    const int d = m[0];
                    if (d < 0) continue;
                    const size_t sb = rbase + size_t(i) * S + m[1];
                    const size_t db = rbase + size_t(d) * S + m[2];
                    const unsigned v = P.lr[sb];
                    const int b = blocks_of(v & 0xFFFFu, shift);
                    int w = b - m[3];
                    if (w > int(P.mig_stage)) w = int(P.mig_stage);
                    if (w > L.freeb[d]) {
                        L.freeb[d] += m[3];
                        P.meta[db] = 0;
                        L.occ[d * W + (m[2] >> 6)] &= ~(1ull << (m[2] & 63));
                        L.live[d] -= 1;
                        P.meta[sb] = uint8_t(P.meta[sb] & ~kMigrating);
                        m[0] = -1; m[1] = 0; m[2] = 0; m[3] = 0;
                        stat_add(L, kMigAborted, 1);
                        set_f(L, d, K);
                        continue;
                    }
                    L.freeb[d] -= w;
                    m[3] += w;
                    if (m[3] == b) {
                        const unsigned mm = P.meta[sb];
                        const int tier = int((mm >> 2) & 15u);
                        P.meta[db] = uint8_t((mm & ~(3u | kMigrating)) | kRunning);
                        P.lr[db] = v;
                        P.seq[db] = P.seq[sb];
                        P.tarr[db] = P.tarr[sb];
                        P.meta[sb] = 0; P.lr[sb] = 0; P.seq[sb] = 0; P.tarr[sb] = 0;
                        L.occ[i * W + (m[1] >> 6)] &= ~(1ull << (m[1] & 63));
                        L.live[i] -= 1;
                        L.freeb[i] += b;
                        L.B[i] -= 1;
                        L.B[d] += 1;
                        L.tcnt[i * kTiers + tier] -= 1;
                        L.tcnt[d * kTiers + tier] += 1;
                        m[0] = -1; m[1] = 0; m[2] = 0; m[3] = 0;
                        stat_add(L, kMigCommitted, 1);
                        set_f(L, int(i), K);
                    }
                    set_f(L, d, K);
                }
            }
            __syncthreads();

            // ================= E2: pairing on interval ticks =================
            if (wave == 0 && t % P.mig_interval == 0) {
                for (uint32_t i = lane; i < I; i += 64) L.busy[i] = 0;
                for (uint32_t i = lane; i < I; i += 64) {
                    const int d = L.mig[4 * i];
                    if (d >= 0) { L.busy[i] = 1; L.busy[d] = 1; }
                }
                int mine = 0;
                for (uint32_t i = lane; i < I; i += 64) {
                    if (L.busy[i]) continue;
                    ++mine;
                    const unsigned long long ki = pkey(L.q[i], int(i));
                    int rank = 0;
                    for (uint32_t j = 0; j < I; ++j)
                        if (!L.busy[j] && pkey(L.q[j], int(j)) < ki) ++rank;
                    L.order[rank] = int(i);
                }
                const int n = wsum(mine);
                for (int k = 0; k < int(P.mig_max_pairs) && k < n - 1 - k; ++k) {
                    const int src = L.order[k], dst = L.order[n - 1 - k];
                    if (L.num[src] >= 0) break;
                    const long long lhs = (long long)P.theta_den *
                        ((long long)L.num[dst] * L.den[src] - (long long)L.num[src] * L.den[dst]);
                    const long long rhs = (long long)P.theta_num * 256 * L.den[src] * L.den[dst];
                    if (lhs < rhs) break;
                    if (L.live[dst] >= int(S)) continue;
                    int c0;
                    unsigned long long w0;
                    const int ds = lowest_empty(L, dst, W, lane, &c0, &w0);
                    if (ds < 0) {
                        if (lane == 0) stat_add(L, kInvariant, 1);
                        continue;
                    }
                    const size_t dsb = rbase + size_t(dst) * S + ds;
                    const int h = L.hol_slot[src];
                    if (h >= 0) {
                        if (lane == 0) {
                            const size_t hb = rbase + size_t(src) * S + h;
                            P.meta[dsb] = P.meta[hb]; P.lr[dsb] = P.lr[hb];
                            P.seq[dsb] = P.seq[hb]; P.tarr[dsb] = P.tarr[hb];
                            P.meta[hb] = 0; P.lr[hb] = 0; P.seq[hb] = 0; P.tarr[hb] = 0;
                            L.occ[src * W + (h >> 6)] &= ~(1ull << (h & 63));
                            L.live[src] -= 1;
                            L.occ[dst * W + c0] = w0 | (1ull << (ds & 63));
                            L.live[dst] += 1;
                            if (ds + 1 > L.hwm[dst]) L.hwm[dst] = ds + 1;
                            stat_add(L, kMigQueued, 1);
                        }
                        continue;
                    }
                    // running candidate: largest tier, then fewest blocks, then newest
                    const uint8_t* mt = P.meta + rbase + size_t(src) * S;
                    const uint32_t* lr = P.lr + rbase + size_t(src) * S;
                    const uint32_t* sq = P.seq + rbase + size_t(src) * S;
                    const int nch = (L.hwm[src] + 63) >> 6;
                    unsigned long long bk = 0;
                    int bs = 0;
                    for (int c = 0; c < nch; ++c) {
                        const int s = c * 64 + lane;
                        const unsigned m = mt[s];
                        if ((m & 3u) == kRunning && !(m & kMigrating)) {
                            const unsigned long long kk =
                                (static_cast<unsigned long long>(((m >> 2) & 15u) + 1u) << 48) |
                                (static_cast<unsigned long long>(65535 - blocks_of(lr[s] & 0xFFFFu, shift)) << 32) | sq[s];
                            if (kk > bk) { bk = kk; bs = s; }
                        }
                    }
                    const unsigned long long mx = wmax64(bk);
                    if (mx == 0) continue;  // unreachable: F < 0 implies a request
                    const int cs = __shfl(bs, __ffsll(static_cast<long long>(ballot(bk == mx))) - 1);
                    if (lane == 0) {
                        P.meta[dsb] = uint8_t(kInbound);
                        L.occ[dst * W + c0] = w0 | (1ull << (ds & 63));
                        L.live[dst] += 1;
                        if (ds + 1 > L.hwm[dst]) L.hwm[dst] = ds + 1;
                        const size_t cb = rbase + size_t(src) * S + cs;
                        P.meta[cb] = uint8_t(P.meta[cb] | kMigrating);
                        int* m = &L.mig[4 * src];
                        m[0] = dst; m[1] = cs; m[2] = ds; m[3] = 0;
                        stat_add(L, kMigStarted, 1);
                    }
                }
            }
            if (threadIdx.x == 0) stat_add(L, kTicks, 1);
            __syncthreads();
        }

        // ---- store the replica ----
        for (int j = threadIdx.x; j < kNstat; j += blockDim.x) P.stats[size_t(r) * kNstat + j] = L.stats[j];
        for (uint32_t i = threadIdx.x; i < I; i += blockDim.x) {
            P.freeb[size_t(r) * I + i] = L.freeb[i];
            for (int k = 0; k < 4; ++k) P.mig[(size_t(r) * I + i) * 4 + k] = L.mig[4 * i + k];
        }
        if (threadIdx.x == 0) P.next_seq[r] = next_seq;
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// initial state: every slot empty, free = M, no migrations, zero counters
// ---------------------------------------------------------------------------
__global__ void k_init(Params P)
{
    const size_t nslots = size_t(P.R) * P.I * P.S;
    const size_t stride = size_t(gridDim.x) * blockDim.x;
    const size_t t0 = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    for (size_t s = t0; s < nslots; s += stride) { P.meta[s] = 0; P.lr[s] = 0; P.seq[s] = 0; P.tarr[s] = 0; }
    for (size_t j = t0; j < size_t(P.R) * P.I; j += stride) {
        P.freeb[j] = int32_t(P.M);
        P.mig[4 * j] = -1; P.mig[4 * j + 1] = 0; P.mig[4 * j + 2] = 0; P.mig[4 * j + 3] = 0;
    }
    for (size_t j = t0; j < size_t(P.R) * kNstat; j += stride) P.stats[j] = 0;
    for (size_t j = t0; j < P.R; j += stride) { P.next_seq[j] = 0; P.digest[j] = 0; }
}

// ---------------------------------------------------------------------------
// per-replica digest: wrapping sum of SplitMix64-finalised slot and instance
// records (Steele, Lea, Flood, OOPSLA 2014); one block per replica
// ---------------------------------------------------------------------------
__device__ inline unsigned long long mix64(unsigned long long z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__global__ __launch_bounds__(256) void k_digest(Params P, uint32_t r0)
{
    __shared__ unsigned long long part[4];
    const uint32_t r = r0 + blockIdx.x;
    const size_t IS = size_t(P.I) * P.S;
    const size_t rb = size_t(r) * IS;
    const unsigned long long gm = mix64(P.id_base + r);
    unsigned long long d = 0;
    for (size_t s = threadIdx.x; s < IS; s += blockDim.x) {
        const unsigned m = P.meta[rb + s];
        if ((m & 3u) == kEmpty) continue;
        const unsigned long long a = static_cast<unsigned long long>(P.lr[rb + s]) |
                                     (static_cast<unsigned long long>(P.seq[rb + s]) << 32);
        const unsigned long long b = static_cast<unsigned long long>(P.tarr[rb + s]) |
                                     (static_cast<unsigned long long>(m) << 32);
        const unsigned long long p = mix64(gm + 2ull * s + 1ull);
        d += mix64(p ^ a) + mix64(p ^ b);
    }
    for (uint32_t i = threadIdx.x; i < P.I; i += blockDim.x) {
        const int32_t* m = P.mig + (size_t(r) * P.I + i) * 4;
        const unsigned long long p = mix64(gm + 2ull * (IS + i) + 1ull);
        const unsigned long long c = static_cast<unsigned long long>(uint32_t(P.freeb[size_t(r) * P.I + i])) |
                                     (static_cast<unsigned long long>(uint32_t(m[0])) << 32);
        const unsigned long long e = static_cast<unsigned long long>(uint32_t(m[1])) |
                                     (static_cast<unsigned long long>(uint32_t(m[2])) << 32);
        d += mix64(p ^ c) + mix64(p ^ e) + mix64(p ^ static_cast<unsigned long long>(uint32_t(m[3])));
    }
    for (int o = 32; o > 0; o >>= 1) d += __shfl_xor(d, o);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = d;
    __syncthreads();
    if (threadIdx.x == 0) P.digest[r] = part[0] + part[1] + part[2] + part[3];
}

}  // namespace

size_t lds_bytes(uint32_t I, uint32_t S) { return lds_layout(I, S / 64).total; }

int launch_init(const Params& p, hipStream_t stream)
{
    hipLaunchKernelGGL(k_init, dim3(1024), dim3(256), 0, stream, p);
    return int(hipGetLastError());
}

int launch_step(const Params& p, uint32_t threads, uint32_t blocks, hipStream_t stream)
{
    const size_t lds = lds_bytes(p.I, p.S);
    if (lds > 64 * 1024) {
        // raise the dynamic LDS limit; the launch below reports a real failure
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_step),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
        (void)hipGetLastError();
    }
    hipLaunchKernelGGL(k_step, dim3(blocks), dim3(threads), lds, stream, p);
    return int(hipGetLastError());
}

int launch_digest(const Params& p, uint32_t r0, uint32_t nr, hipStream_t stream)
{
    if (nr == 0) return 0;
    hipLaunchKernelGGL(k_digest, dim3(nr), dim3(256), 0, stream, p, r0);
    return int(hipGetLastError());
}

}  // namespace mts
