// Device code of libmts.
//
//   k_arrivals  (mts_arrivals.hip) samples every arrival of a chunk of ticks
//               and sorts each tick's arrivals by tier.
//   k_step      the scheduling tick, one wave per replica for a whole chunk
//               of ticks: per-instance summaries live in LDS, per-instance
//               O(1) work is lane-parallel (lane i <-> instance i), slot
//               state lives in HBM and is touched only by events.
//   k_init      empty clusters; k_digest the canonical state digest.
//
// Slot record (uint4 per slot): x = slot word, y = meta, z = seq, w = arrival
// tick, so that an event reads or writes one 16-byte record.  Slot word (u32,
// bits 31..30 = status):
//   waiting   01 | rem (14 bits) | len (16 bits)
//   running   10 | fin mod 2^14  | final length (16 bits)
//   inbound   11 | 0 (with meta; seq and arrival tick keep whatever the slot
//             held last and are read as zero by the export and the digest)
//   empty     0 (the word alone marks an empty slot: meta, seq and arrival
//             tick keep whatever the slot held last; the export and the
//             digest read them as zero)
// A running request's word never changes while it runs: the tick at which it
// emits its last token (fin) and its final length determine its length at
// any tick t (final - (fin - t + 1) before the decode of t), so decoding
// writes nothing.  Its KV growth falls on ticks t with
// (final - fin - 1 + t) mod block = 0: per instance, counters indexed by that
// residue give the number of requests that need a new block at tick t in
// O(1).  A request that starts running is filed under its finish tick in a
// per-replica timing wheel, so a tick visits exactly the requests that
// finish in it.  The head of line of every instance is cached in LDS (slot,
// key, slot word, meta, arrival tick), so admission reads no HBM.
#include <hip/hip_runtime.h>

#include "mts_internal.h"
#include "mts_wave.h"

namespace mts {
namespace {

constexpr int kNstat = MTS_NSTAT;
constexpr int kTiers = MTS_MAX_TIERS;
constexpr unsigned long long kNone = ~0ull;
constexpr uint32_t kWaitW = 1u << 30, kRunW = 2u << 30, kInbW = 3u << 30;
constexpr uint32_t kFin = 0x3FFFu;
constexpr int kNoHol = -1, kHolUnknown = -2, kHolPending = -3;
constexpr int kFlagAbort = 1, kFlagBusy = 2, kFlagIntf = 4;

__device__ __forceinline__ uint32_t wst(uint32_t v) { return v >> 30; }
__device__ __forceinline__ uint32_t wlo(uint32_t v) { return v & 0xFFFFu; }
__device__ __forceinline__ uint32_t wmid(uint32_t v) { return (v >> 16) & kFin; }

// ---------------------------------------------------------------------------
// LDS of one wave (one replica)
// ---------------------------------------------------------------------------
constexpr int kInts = 20;
// placements of the previous tick's dispatch kept in LDS (at most one wave's worth)
constexpr int kLast = 64;
// requests preempted in the current tick, listed for the prefetched finish visit
constexpr int kVic = 16;
// Section 6.5 extensions: words of the device table (u32; the addresses of
// the per-replica headroom and snapshot arrays as u64 at the end)
enum { kXSlo = 0, kXAge = 10, kXPromoMin = 20, kXPromoPeriod, kXAdaptEpoch, kXAdaptUp, kXAdaptDown, kXAdaptMax,
       kXAdaptMargin, kXZeroLowest, kXHqr = 28, kXHsnap = 30, kXWords = 32 };
static_assert(kXWords == MTS_EXT_WORDS, "extension table size");

struct LdsLayout {
    uint32_t stats, occ, holk, fd, ints, res, tcnt, mig, last, vic, wc, wov, inf, qt, qn, xn, ext, blk, rsel, total;
};

// Waves per replica: the kernels for 128 or more instances run a workgroup of
// eight waves per replica (the per-instance phases are spread over the waves,
// the serial ones stay on wave 0); the others one wave.
__host__ __device__ constexpr int waves_for(uint32_t IM) { return IM >= 128 ? 8 : 1; }

__host__ __device__ inline uint32_t al8(uint32_t x) { return (x + 7u) & ~7u; }

// Per-instance arrays are sized for IM instances (a power of two >= I, at
// least 16) and come first, so that their offsets are compile-time constants
// of the kernel instantiation; the arrays whose size depends on S, the block
// size or the wheel follow.
__host__ __device__ constexpr uint32_t imax_for(uint32_t I)
{
    return I <= 16 ? 16 : I <= 32 ? 32 : I <= 64 ? 64 : I <= 128 ? 128 : 256;
}

__host__ __device__ inline LdsLayout lds_layout(uint32_t IM, uint32_t I, uint32_t W, uint32_t RB, uint32_t wsz,
                                                uint32_t policy, uint32_t qdepth, bool ext)
{
    LdsLayout L;
    uint32_t o = 0;
    L.stats = o; o += kNstat * 8;
    L.holk = o;  o += IM * 8;
    L.fd = o;    o += IM * 8;
    L.ints = o;  o += IM * kInts * 4;
    L.tcnt = o;  o += IM * kTiers / 2 * 4;
    L.mig = o;   o += IM * 16;
    L.last = o;  o += kLast * 12 + 8;
    L.vic = o;   o += kVic * 4 + 8;
    L.occ = o;   o += I * W * 8;
    L.res = o;   o += ((I * RB + 1) / 2) * 4;
    L.wc = o;    o += (wsz / 2) * 4;
    L.wov = o;   o += ((wsz + 31) / 32) * 4;
    // INFaaS only: per instance this tick's finished end-to-end sum (u64), the
    // service-time estimate (i64), the finish count and the state penalty
    o = al8(o);
    L.inf = o;   o += policy == MTS_POLICY_INFAAS ? IM * 24 : 0;
    // queue cache: per instance the qdepth waiting requests after the head of
    // line, in (tier, seq) order, 16 bytes each, and their number
    o = (o + 15u) & ~15u;
    L.qt = o;    o += IM * qdepth * 16;
    L.qn = o;    o += qdepth ? IM * 8 : 0;
    // multi-wave kernels: per instance the queue cache extension's head << 16 | count
    L.xn = o;    o += waves_for(IM) > 1 ? IM * 4 : 0;
    // adaptive headroom / promotion: the ticks left to the next promotion
    // pass and headroom update, and per instance a lower bound on the
    // arrival ticks of its waiting requests (the rest of their state stays
    // in HBM: it is touched only on pass and update ticks)
    o = al8(o);
    L.ext = o;   o += ext ? 8 + IM * 4 : 0;
    // multi-wave kernels: values the waves combine (the auto-scaling sum, an
    // abort flag, the admission work list's length and next entry)
    o = al8(o);
    L.blk = o;   o += waves_for(IM) > 1 ? 32 : 0;
    // multi-wave kernels: per wave 64 (key, slot | demand) pairs, the rescan's
    // selected requests before they are ranked (the pairing's sorted blocks
    // of 64 (key, index) pairs use the same bytes later in the tick)
    o = (o + 15u) & ~15u;
    L.rsel = o;  o += waves_for(IM) > 1 ? waves_for(IM) * 64 * 8 : 0;
    L.total = al8(o);
    return L;
}

struct Ctx {
    // LDS
    unsigned long long* stats;
    unsigned long long* occ;   // [I][W] slot not empty
    unsigned long long* holk;  // [I] head-of-line key tier << 32 | seq
    double* fd;                // [I] freeness num / den (exact order for S <= 2048)
    int *freeb, *B, *live, *nwait, *hols, *hold, *num, *den, *held, *inb, *tmask, *flags, *gtmp, *order, *pend;
    int* drn;                  // [I] draining (infinite virtual-usage sentinel)
    int* frs;                  // [I] 1: every waiting request was placed by the previous tick's dispatch
    unsigned *lw, *lsl, *lsq;  // [kLast] previous tick's placements in dispatch order: slot word,
                               // instance << 16 | tier << 12 | slot, seq
    int* lastn;                // number of those placements
    unsigned* vic;             // [kVic] instance << 16 | slot of this tick's preemption victims
    int* nvic;                 // their number (above kVic: more than the list holds)
    unsigned *hwd, *hmt, *hta; // [I] head of line: slot word, meta, arrival tick
    unsigned* res;             // [RB][I] running requests per growth residue (u16 pairs)
    unsigned* tcnt;            // [I][10] running requests per tier (u16 pairs)
    int* mig;                  // [I][4] dst, src slot, dst slot, copied
    unsigned* wc;              // [wsz / 2] entries filed per wheel bucket, two u16 per word
    unsigned* wov;             // [wsz / 32] bucket overflowed since its last visit
    // INFaaS policy only (null otherwise), per instance
    unsigned long long* fsum;  // [I] end-to-end ticks of this tick's finishes
    long long* svc;            // [I] service-time estimate, 1/256 tick
    int *fcnt, *pen;           // [I] this tick's finishes; state penalty in ticks
    // queue cache behind the head of line (td entries per instance; td = 0: none):
    // entry {seq, slot word, arrival tick, slot | tier << 12 | admitted << 16}
    uint4* qt;                 // [I][td] a ring: entry k at (qh + k) mod td
    int* qn;                   // [I] cached entries
    int* qh;                   // [I] ring position of the first entry
    // kernels for 128+ instances (null otherwise): behind the ring, up to
    // kQxDepth further waiting requests of the instance in order, in HBM
    int* xn;                   // [I] head << 16 | count
    uint4* qx;                 // [I][kQxDepth] this replica's extensions
    int td;
    uint32_t blind;            // 1: tiers order nothing (tier-blind scheduling)
    // adaptive headroom and promotion (null when both are off): the LDS
    // region read through the accessors below
    unsigned char* ext;
    // multi-wave kernels only (null otherwise): the block area, a 64-bit sum
    // and a flag the waves combine, the admission work list's length and the
    // next entry to hand out (the list itself is kept in order[])
    long long* bsum;
    int* bflag;
    int* wln;
    int* wlnext;
    int* e2go;                 // pairing runs this tick (set by wave 0)
    int* e2n2;                 // instances that can pair
    uint2* rsel;               // this wave's 64 entries of the rescan selection buffer
    // HBM: timing wheel of this replica, slot arrays, latency histograms
    uint32_t* wheel;           // [wsz][wcap] instance << 16 | slot
    uint32_t* hist;            // [2][10][MTS_HIST_BINS] queue delay, end-to-end
    uint32_t wmask, wcap;
    uint4* slot;               // [I][S] slot records of this replica
    uint32_t I, S, W, RB, shift, bmask, M, K;
    int hq[kTiers];
};

// Section 6.5 extension state in LDS, at fixed offsets from C.ext: the
// ticks left to the next promotion pass and headroom update, then per
// instance a lower bound lb on the arrival ticks of its waiting requests
// (0: unknown, the next pass reads the instance)
__device__ __forceinline__ int* xleft(const Ctx& C) { return reinterpret_cast<int*>(C.ext); }
__device__ __forceinline__ unsigned* wlb(const Ctx& C) { return reinterpret_cast<unsigned*>(C.ext + 8); }
// fields of slot record x
__device__ __forceinline__ uint32_t& s_word(const Ctx& C, size_t x) { return reinterpret_cast<uint32_t*>(C.slot + x)[0]; }
__device__ __forceinline__ uint32_t& s_meta(const Ctx& C, size_t x) { return reinterpret_cast<uint32_t*>(C.slot + x)[1]; }
__device__ __forceinline__ uint32_t& s_tarr(const Ctx& C, size_t x) { return reinterpret_cast<uint32_t*>(C.slot + x)[3]; }
// word and meta of slot record x in one 8-byte store
__device__ __forceinline__ void s_set_wm(const Ctx& C, size_t x, uint32_t w, uint32_t m)
{
    *reinterpret_cast<uint2*>(C.slot + x) = make_uint2(w, m);
}

// addresses of the per-replica headroom and snapshot arrays (null: static headroom)
__device__ __forceinline__ int32_t* ext_hqr(const Params& P)
{
    return reinterpret_cast<int32_t*>(reinterpret_cast<const unsigned long long*>(P.ext + kXHqr)[0]);
}
__device__ __forceinline__ unsigned long long* ext_hsnap(const Params& P)
{
    return reinterpret_cast<unsigned long long*>(reinterpret_cast<const unsigned long long*>(P.ext + kXHsnap)[0]);
}

template <int IM, bool INF, bool EXT>
__device__ inline Ctx carve(char* base, const Params& P)
{
    const LdsLayout Y = lds_layout(IM, P.I, P.W, P.RB, P.wsz, P.policy, P.qdepth, EXT);
    Ctx C;
    C.stats = reinterpret_cast<unsigned long long*>(base + Y.stats);
    C.occ = reinterpret_cast<unsigned long long*>(base + Y.occ);
    C.holk = reinterpret_cast<unsigned long long*>(base + Y.holk);
    C.fd = reinterpret_cast<double*>(base + Y.fd);
    int* p = reinterpret_cast<int*>(base + Y.ints);
    C.freeb = p; p += IM;
    C.B = p; p += IM;
    C.live = p; p += IM;
    C.nwait = p; p += IM;
    C.hols = p; p += IM;
    C.hold = p; p += IM;
    C.num = p; p += IM;
    C.den = p; p += IM;
    C.held = p; p += IM;
    C.inb = p; p += IM;
    C.tmask = p; p += IM;
    C.flags = p; p += IM;
    C.gtmp = p; p += IM;
    C.order = p; p += IM;
    C.pend = p; p += IM;
    C.drn = p; p += IM;
    C.frs = p; p += IM;
    C.hwd = reinterpret_cast<unsigned*>(p); p += IM;
    C.hmt = reinterpret_cast<unsigned*>(p); p += IM;
    C.hta = reinterpret_cast<unsigned*>(p); p += IM;
    C.res = reinterpret_cast<unsigned*>(base + Y.res);
    C.tcnt = reinterpret_cast<unsigned*>(base + Y.tcnt);
    C.mig = reinterpret_cast<int*>(base + Y.mig);
    C.lw = reinterpret_cast<unsigned*>(base + Y.last);
    C.lsl = C.lw + kLast;
    C.lsq = C.lsl + kLast;
    C.lastn = reinterpret_cast<int*>(C.lsq + kLast);
    C.vic = reinterpret_cast<unsigned*>(base + Y.vic);
    C.nvic = reinterpret_cast<int*>(C.vic + kVic);
    C.wc = reinterpret_cast<unsigned*>(base + Y.wc);
    C.wov = reinterpret_cast<unsigned*>(base + Y.wov);
    C.td = int(P.qdepth);
    C.blind = P.blind;
    C.qt = reinterpret_cast<uint4*>(base + Y.qt);
    C.qn = reinterpret_cast<int*>(base + Y.qn);
    C.qh = C.qn + IM;
    C.xn = waves_for(IM) > 1 ? reinterpret_cast<int*>(base + Y.xn) : nullptr;
    C.qx = nullptr;  // per replica, set with the slot records
    if (INF) {
        C.fsum = reinterpret_cast<unsigned long long*>(base + Y.inf);
        C.svc = reinterpret_cast<long long*>(base + Y.inf + IM * 8);
        C.fcnt = reinterpret_cast<int*>(base + Y.inf + IM * 16);
        C.pen = C.fcnt + IM;
    } else {
        C.fsum = nullptr; C.svc = nullptr; C.fcnt = nullptr; C.pen = nullptr;
    }
    C.ext = EXT ? reinterpret_cast<unsigned char*>(base + Y.ext) : nullptr;
    C.bsum = waves_for(IM) > 1 ? reinterpret_cast<long long*>(base + Y.blk) : nullptr;
    C.bflag = waves_for(IM) > 1 ? reinterpret_cast<int*>(base + Y.blk + 8) : nullptr;
    C.wln = waves_for(IM) > 1 ? reinterpret_cast<int*>(base + Y.blk + 12) : nullptr;
    C.wlnext = waves_for(IM) > 1 ? reinterpret_cast<int*>(base + Y.blk + 16) : nullptr;
    C.e2go = waves_for(IM) > 1 ? reinterpret_cast<int*>(base + Y.blk + 20) : nullptr;
    C.e2n2 = waves_for(IM) > 1 ? reinterpret_cast<int*>(base + Y.blk + 24) : nullptr;
    C.rsel = waves_for(IM) > 1 ? reinterpret_cast<uint2*>(base + Y.rsel) + 64 * (threadIdx.x >> 6) : nullptr;
    C.I = P.I; C.S = P.S; C.W = P.W; C.RB = P.RB;
    C.shift = P.blk_shift;
    C.bmask = (1u << P.blk_shift) - 1u;
    C.M = P.M;
    C.wmask = P.wsz - 1u;
    C.wcap = P.wcap;
    return C;
}

using namespace wave;

// Wave reductions and scans through DPP lane moves and lane reads (no LDS
// round trip): four row steps leave every lane of a 16-lane row with the
// row's reduction (quad_perm 1,0,3,2; quad_perm 2,3,0,1; row_half_mirror;
// row_mirror), the four rows are combined from lanes 0, 16, 32, 48.
template <int kCtrl>
__device__ __forceinline__ int dpp_row(int x)
{
    return __builtin_amdgcn_mov_dpp(x, kCtrl, 0xF, 0xF, false);
}
template <int kCtrl>
__device__ __forceinline__ unsigned long long dpp_row64(unsigned long long x)
{
    const unsigned lo = unsigned(dpp_row<kCtrl>(int(unsigned(x))));
    const unsigned hi = unsigned(dpp_row<kCtrl>(int(unsigned(x >> 32))));
    return (static_cast<unsigned long long>(hi) << 32) | lo;
}
__device__ __forceinline__ int wsum(int x)
{
    x += dpp_row<0xB1>(x);
    x += dpp_row<0x4E>(x);
    x += dpp_row<0x141>(x);
    x += dpp_row<0x140>(x);
    return rl(x, 0) + rl(x, 16) + rl(x, 32) + rl(x, 48);
}
__device__ __forceinline__ unsigned long long wsum64(unsigned long long x)
{
    x += dpp_row64<0xB1>(x);
    x += dpp_row64<0x4E>(x);
    x += dpp_row64<0x141>(x);
    x += dpp_row64<0x140>(x);
    return rl64(x, 0) + rl64(x, 16) + rl64(x, 32) + rl64(x, 48);
}
template <typename T>
__device__ __forceinline__ T tmax(T a, T b) { return a > b ? a : b; }
template <typename T>
__device__ __forceinline__ T tmin(T a, T b) { return a < b ? a : b; }
__device__ __forceinline__ unsigned long long wmax64(unsigned long long x)
{
    x = tmax(x, dpp_row64<0xB1>(x));
    x = tmax(x, dpp_row64<0x4E>(x));
    x = tmax(x, dpp_row64<0x141>(x));
    x = tmax(x, dpp_row64<0x140>(x));
    return tmax(tmax(rl64(x, 0), rl64(x, 16)), tmax(rl64(x, 32), rl64(x, 48)));
}
__device__ __forceinline__ unsigned long long wmin64(unsigned long long x)
{
    x = tmin(x, dpp_row64<0xB1>(x));
    x = tmin(x, dpp_row64<0x4E>(x));
    x = tmin(x, dpp_row64<0x141>(x));
    x = tmin(x, dpp_row64<0x140>(x));
    return tmin(tmin(rl64(x, 0), rl64(x, 16)), tmin(rl64(x, 32), rl64(x, 48)));
}
__device__ __forceinline__ uint32_t wmin32(uint32_t x)
{
    x = tmin(x, uint32_t(dpp_row<0xB1>(int(x))));
    x = tmin(x, uint32_t(dpp_row<0x4E>(int(x))));
    x = tmin(x, uint32_t(dpp_row<0x141>(int(x))));
    x = tmin(x, uint32_t(dpp_row<0x140>(int(x))));
    return tmin(tmin(rlu(x, 0), rlu(x, 16)), tmin(rlu(x, 32), rlu(x, 48)));
}
__device__ __forceinline__ uint32_t wmax32(uint32_t x)
{
    x = tmax(x, uint32_t(dpp_row<0xB1>(int(x))));
    x = tmax(x, uint32_t(dpp_row<0x4E>(int(x))));
    x = tmax(x, uint32_t(dpp_row<0x141>(int(x))));
    x = tmax(x, uint32_t(dpp_row<0x140>(int(x))));
    return tmax(tmax(rlu(x, 0), rlu(x, 16)), tmax(rlu(x, 32), rlu(x, 48)));
}

// wave-wide max of a double through DPP lane moves; every lane gets the result
template <int kCtrl, int kRowMask>
__device__ __forceinline__ double dpp_f64(double v)
{
    const int lo = __double2loint(v), hi = __double2hiint(v);
    const int lo2 = __builtin_amdgcn_update_dpp(lo, lo, kCtrl, kRowMask, 0xF, false);
    const int hi2 = __builtin_amdgcn_update_dpp(hi, hi, kCtrl, kRowMask, 0xF, false);
    return __hiloint2double(hi2, lo2);
}
// a lane move in which every lane reads a lane of its own row (no old value)
template <int kCtrl>
__device__ __forceinline__ double dpp_row_f64(double v)
{
    const int lo = __builtin_amdgcn_mov_dpp(__double2loint(v), kCtrl, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(v), kCtrl, 0xF, 0xF, false);
    return __hiloint2double(hi, lo);
}
// Maximum over the first NL lanes (NL = 16, 32 or 64) for every lane; the
// other lanes must not exceed it.  (The file is compiled without NaN
// support: no operand needs quieting before v_max_f64.)
template <int NL>
__device__ __forceinline__ double wave_max_f64(double v)
{
    v = fmax(v, dpp_row_f64<0xB1>(v));    // quad_perm 1,0,3,2
    v = fmax(v, dpp_row_f64<0x4E>(v));    // quad_perm 2,3,0,1
    v = fmax(v, dpp_row_f64<0x141>(v));   // row_half_mirror
    v = fmax(v, dpp_row_f64<0x140>(v));   // row_mirror: every lane of a row holds its maximum
    if (NL > 16) v = fmax(v, dpp_f64<0x142, 0xA>(v));  // row_bcast:15
    if (NL > 32) v = fmax(v, dpp_f64<0x143, 0xC>(v));  // row_bcast:31
    const int lo = __builtin_amdgcn_readlane(__double2loint(v), NL - 1);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(v), NL - 1);
    return __hiloint2double(hi, lo);
}

__device__ __forceinline__ int blocks_of(uint32_t len, uint32_t shift)
{
    return int((len + (1u << shift) - 1u) >> shift);
}

// full finish tick of a running word, given that it has not finished before t
__device__ __forceinline__ uint32_t fin_of(uint32_t v, uint32_t t) { return t + ((wmid(v) - t) & kFin); }

// Freeness of instance i (Eq. 1-4): num = 256 (free - hol demand) - sum of H_p
// over the tiers with a running request, den = max(B, 1).
__device__ inline void set_f(const Ctx& C, int i)
{
    int hs = 0;
    const int tm = C.tmask[i];
#pragma unroll
    for (int p = 0; p < kTiers; ++p) hs += (tm >> p) & 1 ? C.hq[p] : 0;
    const int num = 256 * (C.freeb[i] - C.hold[i]) - hs;
    const int den = C.B[i] > 0 ? C.B[i] : 1;
    C.num[i] = num;
    C.den[i] = den;
    C.fd[i] = double(num) / double(den);
}

// running requests of instance i whose length is r mod block_tokens: laid out
// residue-major, so that the lanes of one residue read consecutive counters
__device__ __forceinline__ uint32_t res_idx(const Ctx& C, int i, uint32_t r) { return r * C.I + uint32_t(i); }

// Counters of running requests, two u16 per LDS word (an instance holds at
// most 2048 running requests, so no half ever carries into the other).  All
// updates are atomic: lanes that work on different instances may share a word.
__device__ __forceinline__ uint32_t c16_get(const unsigned* a, uint32_t idx)
{
    return (a[idx >> 1] >> ((idx & 1u) * 16u)) & 0xFFFFu;
}
__device__ __forceinline__ uint32_t c16_inc(unsigned* a, uint32_t idx)
{
    const uint32_t sh = (idx & 1u) * 16u;
    return (atomicAdd(&a[idx >> 1], 1u << sh) >> sh) & 0xFFFFu;
}
__device__ __forceinline__ uint32_t c16_dec(unsigned* a, uint32_t idx)
{
    const uint32_t sh = (idx & 1u) * 16u;
    return (atomicSub(&a[idx >> 1], 1u << sh) >> sh) & 0xFFFFu;
}

__device__ __forceinline__ void tier_dec(const Ctx& C, int i, int tier)
{
    if (c16_dec(C.tcnt, uint32_t(i * kTiers + tier)) == 1u) atomicAnd(&C.tmask[i], ~(1 << tier));
}
__device__ __forceinline__ void tier_inc(const Ctx& C, int i, int tier)
{
    c16_inc(C.tcnt, uint32_t(i * kTiers + tier));
    atomicOr(&C.tmask[i], 1 << tier);
}

__device__ __forceinline__ void stat(const Ctx& C, int idx, unsigned long long v) { atomicAdd(&C.stats[idx], v); }

// Latency histograms in ticks: a value below 16 has its own bin; a larger
// value v with 2^e <= v < 2^(e+1) falls into one of eight sub-ranges of
// width 2^(e-3), bin 16 + 8 (e - 4) + (v >> (e - 3)) - 8.
__device__ __forceinline__ uint32_t hist_bin(uint32_t v)
{
    if (v < 16u) return v;
    const uint32_t e = 31u - uint32_t(__builtin_clz(v));
    return 8u * e - 24u + (v >> (e - 3u));
}
__device__ __forceinline__ void hist_add(const Ctx& C, int metric, int tier, uint32_t v)
{
    atomicAdd(&C.hist[(metric * kTiers + tier) * MTS_HIST_BINS + hist_bin(v)], 1u);
}

// INFaaS cost of instance i in 1/256 tick with extra queued requests:
// alpha q + beta s + gamma penalty, q = waiting + extra.  Below 2^51 by the
// configuration limits, so exact as a double.
__device__ __forceinline__ double infaas_cost(const Ctx& C, const Params& P, int i, int extra)
{
    const long long c = P.alpha256 * (C.nwait[i] + extra) + P.beta * C.svc[i] + P.gamma256 * C.pen[i];
    return double(c);
}

// number of 64-slot chunks of instance i up to its highest non-empty one; uniform
__device__ __forceinline__ int live_chunks(const Ctx& C, int i, int lane)
{
    const unsigned long long w = lane < int(C.W) ? C.occ[i * C.W + lane] : 0ull;
    const unsigned long long nz = ballot(w != 0);
    return nz ? 64 - __clzll(static_cast<long long>(nz)) : 0;
}

// position of the k-th (from 0) set bit of m; m has more than k set bits
__device__ __forceinline__ int kth_set_bit(unsigned long long m, int k)
{
    int pos = 0;
#pragma unroll
    for (int w = 32; w >= 1; w >>= 1) {
        const int c = __popcll((m >> pos) & ((1ull << w) - 1ull));
        if (k >= c) { k -= c; pos += w; }
    }
    return pos;
}

// inclusive prefix sum over the lanes of the wave, by DPP: row_shr 1, 2, 4,
// 8 (lanes reading before their row's start get 0) scan each row, then
// row_bcast:15 adds row 0's total into row 1 and row 2's into row 3, and
// row_bcast:31 adds the total of rows 0-1 into rows 2 and 3
__device__ __forceinline__ int wscan(int x, int lane)
{
    (void)lane;
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);
    return x;
}

// ---------------------------------------------------------------------------
// per-instance event handlers (uniform: the whole wave works on instance i)
// ---------------------------------------------------------------------------

__device__ __forceinline__ void qx_clear(const Ctx& C, int i)
{
    if (C.xn) C.xn[i] = 0;
}
__device__ __forceinline__ int qx_count(const Ctx& C, int i) { return C.xn ? (C.xn[i] & 0xFFFF) : 0; }

__device__ __forceinline__ void clear_hol(const Ctx& C, int i)
{
    C.hols[i] = kNoHol; C.holk[i] = kNone; C.hold[i] = 0;
    if (C.td) C.qn[i] = 0;
    qx_clear(C, i);
}

__device__ __forceinline__ void set_hol(const Ctx& C, int i, int slot, unsigned long long key, uint32_t word,
                                        uint32_t meta, uint32_t tarr)
{
    C.hols[i] = slot; C.holk[i] = key; C.hold[i] = blocks_of(wlo(word), C.shift);
    C.hwd[i] = word; C.hmt[i] = meta; C.hta[i] = tarr;
}

// Queue cache.  Invariant: the head of line, the qn[i] cached entries and
// (kernels for 128+ instances) the extension's entries are the smallest
// (tier, seq) keys among instance i's waiting requests, in order.  The functions below are per lane (lane-private
// instance i) and keep it: popping the head promotes the first cached entry
// (or leaves the head unknown, to be found by a rescan), a new waiting
// request becomes the head or enters the cache at its place when it is
// smaller than the last cached entry.
// the rank a tier gives in every ordering (queue, preemption, migration
// candidate): the tier itself, or 0 for all when scheduling is tier-blind
__device__ __forceinline__ unsigned long long rank_of(const Ctx& C, uint32_t tier)
{
    return C.blind ? 0ull : static_cast<unsigned long long>(tier);
}

__device__ __forceinline__ uint4 qc_pack(unsigned long long key, int slot, uint32_t word, uint32_t meta, uint32_t tarr)
{
    return make_uint4(uint32_t(key), word, tarr,
                      uint32_t(slot) | (((meta >> 2) & 15u) << 12) | (((meta >> 6) & 1u) << 16));
}
__device__ __forceinline__ unsigned long long qc_key(const Ctx& C, uint4 e)
{
    return (rank_of(C, (e.w >> 12) & 15u) << 32) | e.x;
}
__device__ __forceinline__ int qc_at(const Ctx& C, int i, int k)
{
    const int x = C.qh[i] + k;
    return i * C.td + (x >= C.td ? x - C.td : x);
}
// insert e at position p of instance i's cache (the last entry drops out when full)
__device__ inline void qc_insert_at(const Ctx& C, int i, int p, uint4 e)
{
    const int n = C.qn[i];
    if (n >= C.td) qx_clear(C, i);  // the last entry drops out: the extension no longer follows
    if (p == 0) {
        // in front: the ring start moves back (over the last entry when full)
        const int h = C.qh[i];
        C.qh[i] = h == 0 ? C.td - 1 : h - 1;
        C.qt[qc_at(C, i, 0)] = e;
        C.qn[i] = n < C.td ? n + 1 : C.td;
        return;
    }
    const int last = n < C.td ? n : C.td - 1;
    for (int k = last; k > p; --k) C.qt[qc_at(C, i, k)] = C.qt[qc_at(C, i, k - 1)];
    C.qt[qc_at(C, i, p)] = e;
    C.qn[i] = last + 1;
}
// the head of line of i left the queue (admitted or moved)
__device__ inline void hol_pop(const Ctx& C, int i)
{
    if (C.nwait[i] == 0) { clear_hol(C, i); return; }
    const int n = C.td ? C.qn[i] : 0;
    if (n == 0) {
        const int xv = C.xn ? C.xn[i] : 0;
        if ((xv & 0xFFFF) == 0) { C.hols[i] = kHolUnknown; return; }
        // the extension's first entry becomes the head of line
        const int xh = xv >> 16;
        const uint4 e = C.qx[size_t(i) * kQxDepth + xh];
        const uint32_t tier = (e.w >> 12) & 15u;
        set_hol(C, i, int(e.w & 0xFFFu), qc_key(C, e), e.y, kWaiting | (tier << 2) | (((e.w >> 16) & 1u) << 6), e.z);
        C.xn[i] = ((xh + 1) << 16) | ((xv & 0xFFFF) - 1);
        return;
    }
    const uint4 e = C.qt[qc_at(C, i, 0)];
    const uint32_t tier = (e.w >> 12) & 15u;
    set_hol(C, i, int(e.w & 0xFFFu), qc_key(C, e), e.y, kWaiting | (tier << 2) | (((e.w >> 16) & 1u) << 6), e.z);
    const int h = C.qh[i] + 1;
    C.qh[i] = h == C.td ? 0 : h;
    C.qn[i] = n - 1;
}
// a new waiting request of i (nwait already counts it)
__device__ inline void hol_insert(const Ctx& C, int i, unsigned long long key, int slot, uint32_t word, uint32_t meta,
                                  uint32_t tarr)
{
    const int h = C.hols[i];
    if (h == kHolUnknown) return;
    if (h == kNoHol) { set_hol(C, i, slot, key, word, meta, tarr); if (C.td) C.qn[i] = 0; qx_clear(C, i); return; }
    if (key < C.holk[i]) {
        if (C.td) qc_insert_at(C, i, 0, qc_pack(C.holk[i], h, C.hwd[i], C.hmt[i], C.hta[i]));
        set_hol(C, i, slot, key, word, meta, tarr);
        return;
    }
    if (!C.td) return;
    const int n = C.qn[i];
    int p = 0;
    while (p < n && qc_key(C, C.qt[qc_at(C, i, p)]) < key) ++p;
    if (p < n) qc_insert_at(C, i, p, qc_pack(key, slot, word, meta, tarr));
    else qx_clear(C, i);  // beyond the cached run: it may fall inside the extension
}

// file a running request under its finish tick
__device__ __forceinline__ void wheel_put(const Ctx& C, uint32_t fin, int i, int s)
{
    const uint32_t b = fin & C.wmask;
    const uint32_t sh = (b & 1u) * 16u;
    const uint32_t k = (atomicAdd(&C.wc[b >> 1], 1u << sh) >> sh) & 0xFFFFu;
    if (k < C.wcap) {
        C.wheel[size_t(b) * C.wcap + k] = (uint32_t(i) << 16) | uint32_t(s);
    } else {
        // full: keep the count at wcap and mark the bucket for an exact rebuild
        atomicSub(&C.wc[b >> 1], 1u << sh);
        atomicOr(&C.wov[b >> 5], 1u << (b & 31u));
    }
}

// A running request that leaves its slot before its finish tick (preempted,
// or moved out by a committed migration) loses its wheel entry: the entry is
// overwritten with a tombstone, so every entry of the wheel names a distinct
// running request.  A bucket that overflowed is rebuilt from the slots at its
// visit and needs nothing here.  Uniform: the whole wave calls it.
constexpr uint32_t kTomb = 0xFFFFFFFFu;
__device__ inline void wheel_erase(const Ctx& C, uint32_t fin, int i, int s, int lane)
{
    const uint32_t b = fin & C.wmask;
    if ((C.wov[b >> 5] >> (b & 31u)) & 1u) return;
    const uint32_t n = (C.wc[b >> 1] >> ((b & 1u) * 16u)) & 0xFFFFu;
    uint32_t* ent = C.wheel + size_t(b) * C.wcap;
    const uint32_t key = (uint32_t(i) << 16) | uint32_t(s);
    for (uint32_t e0 = 0; e0 < n; e0 += 64) {
        const bool hit = e0 + lane < n && ent[e0 + lane] == key;
        if (hit) ent[e0 + lane] = kTomb;
        if (ballot(hit)) break;
    }
}

// memory pressure: preempt the largest (tier, seq) running request until the
// growth of this tick fits (Section 2.2; recompute semantics)
template <int GR, int MK>
__device__ inline bool preempt(const Ctx& C, int i, uint32_t t, int lane)
{
    const size_t b = size_t(i) * C.S;
    int G = C.gtmp[i], fr = C.freeb[i];
    bool aborted = false;
    bool scan = G > fr;
    while (scan) {
        // Each lane keeps the MK largest (tier, seq) keys of its running slots,
        // descending, with the slot, its word and its meta (a running
        // request's word and meta do not change while it runs); GR chunks of
        // 64 slots are read per memory round trip.
        const int nch = live_chunks(C, i, lane);
        unsigned long long k[MK];
        uint32_t kw[MK], km[MK];
        int ks[MK];
#pragma unroll
        for (int x = 0; x < MK; ++x) { k[x] = 0; kw[x] = 0; km[x] = 0; ks[x] = 0; }
        int cnt = 0;
        for (int c0 = 0; c0 < nch; c0 += GR) {
            uint32_t v[GR], m[GR], q[GR];
#pragma unroll
            for (int g = 0; g < GR; ++g) {
                const bool in = c0 + g < nch;
                const uint4 rr = in ? C.slot[b + (c0 + g) * 64 + lane] : make_uint4(0u, 0u, 0u, 0u);
                v[g] = rr.x; m[g] = rr.y; q[g] = rr.z;
            }
#pragma unroll
            for (int g = 0; g < GR; ++g) {
                if (wst(v[g]) != 2u) continue;
                ++cnt;
                unsigned long long ck = ((rank_of(C, (m[g] >> 2) & 15u) + 1ull) << 32) | q[g];
                if (ck <= k[MK - 1]) continue;
                uint32_t cw = v[g], cm = m[g];
                int cs = (c0 + g) * 64 + lane;
#pragma unroll
                for (int x = 0; x < MK; ++x) {
                    if (ck > k[x]) {
                        const unsigned long long tk = k[x]; k[x] = ck; ck = tk;
                        const uint32_t tw = kw[x]; kw[x] = cw; cw = tw;
                        const uint32_t tm = km[x]; km[x] = cm; cm = tm;
                        const int ts = ks[x]; ks[x] = cs; cs = ts;
                    }
                }
            }
        }
        const bool more = cnt > MK;
        int taken = 0;
        scan = false;
        while (G > fr) {
            const unsigned long long mx = wmax64(k[0]);
            if (mx == 0) break;  // nothing runs
            const int wl = ffs64(ballot(k[0] == mx));
            const int vs = rl(ks[0], wl);
            const uint32_t v = rlu(kw[0], wl), m = rlu(km[0], wl);
            const bool win = lane == wl;
#pragma unroll
            for (int x = 0; x + 1 < MK; ++x) {
                k[x] = win ? k[x + 1] : k[x];
                kw[x] = win ? kw[x + 1] : kw[x];
                km[x] = win ? km[x + 1] : km[x];
                ks[x] = win ? ks[x + 1] : ks[x];
            }
            k[MK - 1] = win ? 0ull : k[MK - 1];
            taken += win ? 1 : 0;
            const bool unknown = ballot(win && more && taken >= MK) != 0;
            // the victim returns to the queue (recompute semantics: len, rem and
            // seq kept, its blocks freed)
            const uint32_t lenf = wlo(v), fin = fin_of(v, t);
            const uint32_t remb = fin - t + 1u, lenb = lenf - remb;
            const uint32_t vw = kWaitW | (remb << 16) | lenb;
            const uint32_t vmeta = (m & ~(3u | kMigrating)) | kWaiting;
            const int vb = blocks_of(lenb, C.shift);
            const int vg = (lenb & C.bmask) == 0;
            const int vt = int((m >> 2) & 15u);
            const int vr = int((lenf - fin - 1u) & C.bmask);
            const bool vm = (m & kMigrating) != 0;
            uint32_t vta = 0;
            if (lane == (vs & 63)) {
                s_set_wm(C, b + vs, vw, vmeta);
                vta = s_tarr(C, b + vs);
            }
            vta = rlu(vta, vs & 63);
            wheel_erase(C, fin, i, vs, lane);
            fr += vb;
            G -= vg;
            aborted = aborted || vm;
            if (lane == 0) {
                C.held[i] -= vb;
                C.B[i] -= 1;
                C.nwait[i] += 1;
                C.frs[i] = 0;
                C.flags[i] |= kFlagIntf;
                // (several waves may preempt at once; a count above kVic means
                // the list missed some)
                const int nv = atomicAdd(C.nvic, 1);
                if (nv < kVic) C.vic[nv] = (uint32_t(i) << 16) | uint32_t(vs);
                c16_dec(C.res, res_idx(C, i, vr));
                tier_dec(C, i, vt);
                stat(C, vt * 8 + kPreempted, 1);
                if (vm) C.flags[i] |= kFlagAbort;
                const unsigned long long key = (rank_of(C, uint32_t(vt)) << 32) | static_cast<unsigned>(mx);
                hol_insert(C, i, key, vs, vw, vmeta, vta);
                if (C.ext) wlb(C)[i] = vta < wlb(C)[i] ? vta : wlb(C)[i];
            }
            wave_sync();
            if (unknown) { scan = G > fr; break; }  // the winner's next key is unknown: read again
        }
    }
    // this tick's growth, now that it fits
    if (lane == 0) { C.freeb[i] = fr - G; C.held[i] += G; }
    wave_sync();
    return aborted;
}

// Exact finish scan of instance i, used when a wheel bucket overflowed:
// finishes the requests whose last token is at t and files again the running
// requests that share the bucket of t but finish later.
__device__ inline void finish_scan(const Ctx& C, int i, uint32_t t, int lane, bool& abort_any)
{
    const size_t b = size_t(i) * C.S;
    const int nch = live_chunks(C, i, lane);
    const uint32_t bk = t & C.wmask;
    int freed = 0, nf = 0;
    bool ab = false;
    for (int c = 0; c < nch; ++c) {
        const int s = c * 64 + lane;
        const uint4 rec = C.slot[b + s];
        const uint32_t v = rec.x;
        const bool run = wst(v) == 2u;
        const uint32_t fin = fin_of(v, t);
        const bool f = run && fin == t;
        if (f) {
            const uint32_t lenf = wlo(v);
            freed += blocks_of(lenf, C.shift);
            const uint32_t m = rec.y;
            const int tier = int((m >> 2) & 15u);
            stat(C, tier * 8 + kFinished, 1);
            const uint32_t e2e = t - rec.w;
            stat(C, tier * 8 + kE2e, e2e);
            hist_add(C, kHistE2e, tier, e2e);
            if (C.fsum) { atomicAdd(&C.fsum[i], static_cast<unsigned long long>(e2e)); atomicAdd(&C.fcnt[i], 1); }
            c16_dec(C.res, res_idx(C, i, (lenf - t - 1u) & C.bmask));
            tier_dec(C, i, tier);
            // being copied out: the source of its instance's migration record
            // (the same test as the wheel visit's)
            if (C.mig[4 * i] >= 0 && C.mig[4 * i + 1] == s) ab = true;
            s_word(C, b + s) = 0;  // the word alone marks the slot empty
        } else if (run && (fin & C.wmask) == bk) {
            wheel_put(C, fin, i, s);
        }
        const unsigned long long fb = ballot(f);
        const unsigned long long ow = ballot(v != 0 && !f);
        nf += __popcll(fb);
        if (lane == 0) C.occ[i * C.W + c] = ow;
    }
    freed = wsum(freed);
    const bool any_ab = ballot(ab) != 0;
    abort_any = abort_any || any_ab;
    if (lane == 0) {
        C.freeb[i] += freed;
        C.held[i] -= freed;
        C.B[i] -= nf;
        C.live[i] -= nf;
        if (any_ab) C.flags[i] |= kFlagAbort;
    }
    wave_sync();
}

// One batch of up to 64 entries of bucket t mod wsz (lanes with inb set),
// each with its slot's word, meta and arrival tick: entries with fin = t
// finish, those with a later fin stay in the bucket (compacted in place from
// position kept on; returns the new kept count), tombstones and entries whose
// slot changed since are dropped.
__device__ inline uint32_t finish_batch(const Ctx& C, uint32_t t, int lane, uint32_t* ent, uint32_t kept, bool inb,
                                        uint32_t e, uint32_t v, uint32_t m, uint32_t ta, bool& abort_any)
{
    const uint32_t bk = t & C.wmask;
    const int i = int(e >> 16), s = int(e & 0xFFFFu);
    const bool valid = inb && uint32_t(i) < C.I && uint32_t(s) < C.S;
    if (!valid) v = 0;
    const uint32_t fin = fin_of(v, t);
    // entries name distinct running requests (wheel_erase)
    const bool f = valid && wst(v) == 2u && fin == t;
    const bool k = valid && wst(v) == 2u && fin != t && (fin & C.wmask) == bk;
    const unsigned long long km = ballot(k);
    if (k) ent[kept + __popcll(km & lanemask_lt())] = e;
    kept += __popcll(km);
    bool ab = false;
    if (f) {
        const size_t idx = size_t(i) * C.S + s;
        const uint32_t lenf = wlo(v);
        const int bl = blocks_of(lenf, C.shift);
        const int tier = int((m >> 2) & 15u);
        stat(C, tier * 8 + kFinished, 1);
        stat(C, tier * 8 + kE2e, t - ta);
        hist_add(C, kHistE2e, tier, t - ta);
        if (C.fsum) { atomicAdd(&C.fsum[i], static_cast<unsigned long long>(t - ta)); atomicAdd(&C.fcnt[i], 1); }
        c16_dec(C.res, res_idx(C, i, (lenf - t - 1u) & C.bmask));
        tier_dec(C, i, tier);
        // being copied out: the source of its instance's migration record (the
        // slot's meta may predate the migration's start)
        ab = C.mig[4 * i] >= 0 && C.mig[4 * i + 1] == s;
        if (ab) atomicOr(&C.flags[i], kFlagAbort);
        atomicAnd(&C.occ[i * C.W + (s >> 6)], ~(1ull << (s & 63)));
        atomicAdd(&C.freeb[i], bl);
        atomicSub(&C.held[i], bl);
        atomicSub(&C.B[i], 1);
        atomicSub(&C.live[i], 1);
        s_word(C, idx) = 0;  // the word alone marks the slot empty
    }
    abort_any = abort_any || ballot(ab) != 0;
    wave_sync();
    return kept;
}

__device__ __forceinline__ void wheel_set_count(const Ctx& C, uint32_t b, uint32_t n, int lane)
{
    const uint32_t sh = (b & 1u) * 16u;
    if (lane == 0) C.wc[b >> 1] = (C.wc[b >> 1] & ~(0xFFFFu << sh)) | (n << sh);
    wave_sync();
}

// Requests that emit their last token at tick t: the bucket t mod wsz lists
// every running request with fin = t (mod wsz).
__device__ inline void finish_tick(const Ctx& C, uint32_t t, int lane, bool& abort_any)
{
    const uint32_t bk = t & C.wmask;
    const uint32_t sh = (bk & 1u) * 16u;
    const uint32_t n = (C.wc[bk >> 1] >> sh) & 0xFFFFu;
    if ((C.wov[bk >> 5] >> (bk & 31u)) & 1u) {
        // the bucket overflowed: rebuild it by scanning every instance with running requests
        if (lane == 0) {
            C.wc[bk >> 1] &= ~(0xFFFFu << sh);
            C.wov[bk >> 5] &= ~(1u << (bk & 31u));
            stat(C, kWheelRebuilds, 1);
        }
        wave_sync();
        for (uint32_t j = 0; j < (C.I + 63) / 64; ++j) {
            const uint32_t i = lane + 64 * j;
            for (unsigned long long m = ballot(i < C.I && C.B[i] > 0); m; m &= m - 1)
                finish_scan(C, int(64 * j + ffs64(m)), t, lane, abort_any);
        }
        return;
    }
    uint32_t* ent = C.wheel + size_t(bk) * C.wcap;
    uint32_t kept = 0;
    for (uint32_t e0 = 0; e0 < n; e0 += 64) {
        const bool inb = e0 + lane < n;
        const uint32_t e = inb ? ent[e0 + lane] : 0u;
        const int i = int(e >> 16), s = int(e & 0xFFFFu);
        const bool valid = inb && uint32_t(i) < C.I && uint32_t(s) < C.S;
        const size_t idx = size_t(i) * C.S + s;
        uint32_t v = 0, m = 0, ta = 0;
        if (valid) { const uint4 rec = C.slot[idx]; v = rec.x; m = rec.y; ta = rec.w; }
        kept = finish_batch(C, t, lane, ent, kept, inb, e, v, m, ta, abort_any);
    }
    wheel_set_count(C, bk, kept, lane);
}

// Adds to stats[tier * 8 + fd0], for every tier, the number of lanes of that
// tier with f0 set, and likewise for (f1, fd1) and (f2, fd2): the boundaries
// of the tiers' runs of lanes are found once.  The lanes' tiers are
// non-decreasing (arrivals are sorted by tier) unless scheduling is
// tier-blind; lanes that hold no arrival carry tier 15.
__device__ __forceinline__ void tier_stat3(const Ctx& C, int tier, bool f0, int fd0, bool f1, int fd1, bool f2, int fd2,
                                           int lane)
{
    const unsigned long long m0 = ballot(f0), m1 = ballot(f1), m2 = ballot(f2);
    if (C.blind) {
        for (int p = 0; p < int(C.K); ++p) {
            const unsigned long long tp = ballot(tier == p);
            const int c0 = __popcll(m0 & tp), c1 = __popcll(m1 & tp), c2 = __popcll(m2 & tp);
            if (lane == 0) {
                if (c0) stat(C, p * 8 + fd0, c0);
                if (c1) stat(C, p * 8 + fd1, c1);
                if (c2) stat(C, p * 8 + fd2, c2);
            }
        }
        return;
    }
    const int tn = __builtin_amdgcn_update_dpp(tier, tier, 0x130, 0xF, 0xF, false);  // wave_shl:1 (lane 63 keeps its own)
    const bool last = lane == 63 || tn != tier;
    const unsigned long long bm = ballot(last);
    if (last && tier < kTiers) {
        const unsigned long long below = bm & lanemask_lt();
        const int start = below ? 64 - __clzll(static_cast<long long>(below)) : 0;
        const unsigned long long upto = lane == 63 ? ~0ull : (1ull << (lane + 1)) - 1ull;
        const unsigned long long run = upto & ~((1ull << start) - 1ull);
        const int c0 = __popcll(m0 & run), c1 = __popcll(m1 & run), c2 = __popcll(m2 & run);
        if (c0) stat(C, tier * 8 + fd0, c0);
        if (c1) stat(C, tier * 8 + fd1, c1);
        if (c2) stat(C, tier * 8 + fd2, c2);
    }
}

// Admits the longest prefix of w ranked waiting requests of instance i (lane
// r holds the request of rank r: key, slot word, meta, arrival tick, slot)
// whose summed demand fits the free blocks, and makes the next one the head
// of line (Section 3.1: the local queue is served in priority order while
// the head fits; the result equals admitting the head of line one request at
// a time).  The list holds every waiting request of i (complete) or the w
// smallest keys of a longer queue; when all w of those fit, the head of line
// is unknown afterwards (the next rescan finds it).
// xn0 >= 0: the list is the head of line, the xn0 cached entries and the
// extension from its head xh0 on (admit_cached): the new extension is then
// a suffix of the stored one (the cache never holds more than qdepth), so
// only its head moves.
__device__ inline void admit_ranked(const Ctx& C, int i, uint32_t t, int lane, int w, unsigned long long key,
                                    uint32_t word, uint32_t meta, uint32_t ta, int slot, bool complete = true,
                                    int xn0 = -1, int xh0 = 0)
{
    const size_t b = size_t(i) * C.S;
    const int dem = lane < w ? blocks_of(wlo(word), C.shift) : 0;
    const int pre = wscan(dem, lane);
    const int fr = C.freeb[i];
    const bool adm = lane < w && pre <= fr && uint32_t(slot) < C.S;
    const int na = __popcll(ballot(adm));
    if (adm) {
        const uint32_t len = wlo(word), rem = wmid(word);
        const uint32_t fin = t + rem;
        const size_t hb = b + slot;
        s_set_wm(C, hb, kRunW | ((fin & kFin) << 16) | (len + rem), (meta & ~3u) | kRunning | kAdmitted);
        const int tier = int((meta >> 2) & 15u);
        if (!(meta & kAdmitted)) {
            stat(C, tier * 8 + kAdmittedCnt, 1);
            stat(C, tier * 8 + kQdelay, t - ta);
            hist_add(C, kHistQdelay, tier, t - ta);
        }
        c16_inc(C.res, res_idx(C, i, (len - t - 1u) & C.bmask));
        tier_inc(C, i, tier);
        wheel_put(C, fin, i, slot);
    }
    const int used = na > 0 ? rl(pre, na - 1) : 0;
    const int hs = rl(slot, na < w ? na : 0);
    const unsigned long long hk = rl64(key, na < w ? na : 0);
    const uint32_t hw = rlu(word, na < w ? na : 0), hm = rlu(meta, na < w ? na : 0),
                   ht = rlu(ta, na < w ? na : 0);
    if (lane == 0) {
        C.freeb[i] -= used;
        C.held[i] += used;
        C.B[i] += na;
        C.nwait[i] -= na;
        if (complete ? w != C.nwait[i] + na : w >= C.nwait[i] + na) stat(C, kInvariant, 1);
        if (na < w) {
            set_hol(C, i, hs, hk, hw, hm, ht);
        } else if (complete) {
            clear_hol(C, i);
        } else {
            C.hols[i] = kHolUnknown;
            if (C.td) C.qn[i] = 0;
        }
        if (C.td && na < w) { C.qn[i] = min(w - na - 1, C.td); C.qh[i] = 0; }
        if (C.xn) {
            const int xc = C.td && na < w && w - na - 1 > C.td ? w - na - 1 - C.td : 0;
            C.xn[i] = xc && xn0 >= 0 ? ((xh0 + na + C.td - xn0) << 16) | xc : xc;
        }
    }
    // the ranked list holds the smallest keys: the ones after the new head fill
    // the cache, and the ones after those its extension
    if (C.td && lane > na && lane < w && lane - na - 1 < C.td)
        C.qt[i * C.td + lane - na - 1] = qc_pack(key, slot, word, meta, ta);
    if (C.xn && C.td && xn0 < 0 && lane > na + C.td && lane < w)
        C.qx[size_t(i) * kQxDepth + (lane - na - 1 - C.td)] = qc_pack(key, slot, word, meta, ta);
    wave_sync();
}

// The ranked prefix of a rescan, taken minimum by minimum from the lanes'
// ascending lists k (MK each, with slot | demand << 12 in sd): lane r
// receives the key and sd of rank r.  The extraction stops when nothing is
// left, after 64 requests, qdepth requests after the first one whose summed
// demand exceeds the free blocks fr (the new head of line and the cache
// behind it), or when the winning lane had more waiting slots than it kept
// (more: its next key is unknown).  Returns the number taken.  KT is the key
// type: the 64-bit keys or an order-preserving 32-bit form of them, with
// all-ones as "none".
__device__ __forceinline__ uint32_t wmin_k(uint32_t x) { return wmin32(x); }
__device__ __forceinline__ unsigned long long wmin_k(unsigned long long x) { return wmin64(x); }

template <typename KT, int MK>
__device__ inline int rank_extract(KT (&k)[MK], uint32_t (&sd)[MK], bool more, int fr, int td, int lane, KT& myk,
                                   uint32_t& mysd)
{
    const KT none = static_cast<KT>(~static_cast<KT>(0));
    myk = none;
    mysd = 0;
    int got = 0, taken = 0, cum = 0, lim = 64;
    for (int r = 0; r < lim; ++r) {
        const KT mn = wmin_k(k[0]);
        if (mn == none) break;
        const int wl = ffs64(ballot(k[0] == mn));
        const uint32_t wsd = rlu(sd[0], wl);
        myk = lane == r ? mn : myk;
        mysd = lane == r ? wsd : mysd;
        got = r + 1;
        cum += int(wsd >> 12);
        if (cum > fr && lim == 64) lim = min(64, r + 1 + td);
        const bool win = lane == wl;
#pragma unroll
        for (int x = 0; x + 1 < MK; ++x) {
            k[x] = win ? k[x + 1] : k[x];
            sd[x] = win ? sd[x + 1] : sd[x];
        }
        k[MK - 1] = win ? none : k[MK - 1];
        taken += win ? 1 : 0;
        if (ballot(win && more && taken >= MK)) break;  // the winner's next key is unknown
    }
    return got;
}

// The same ranked prefix as rank_extract on 32-bit keys, found by selection
// instead of minimum by minimum: the candidates the extraction can reach are
// the keys up to the smallest last kept key of a lane with more waiting slots
// (bnd, from the caller; all keys when no lane has more).  Of those, the 64
// smallest are the keys up to a threshold found by bisection over key values
// (the keys are distinct, counted by ballots); they are gathered into this
// wave's buffer, taken out of the lists (set to none), ranked by counting and
// sent to the lane of their rank, and the prefix stops qdepth requests after
// the first one whose summed demand exceeds fr.  The latency chain is a few
// dozen scalar steps instead of one wave reduction per request.
template <int MK>
__device__ inline int rank_select(const Ctx& C, uint32_t (&k)[MK], uint32_t (&sd)[MK], uint32_t bnd, int fr, int lane,
                                  uint32_t& myk, uint32_t& mysd)
{
    constexpr uint32_t none = 0xFFFFFFFFu;
    bool vx[MK];
    int nvalid = 0;
#pragma unroll
    for (int x = 0; x < MK; ++x) {
        vx[x] = k[x] != none && k[x] <= bnd;
        nvalid += __popcll(ballot(vx[x]));
    }
    myk = none;
    mysd = 0;
    const int want = min(64, nvalid);
    if (want == 0) return 0;
    uint32_t thr = none;
    if (nvalid > 64) {
        // the smallest value with 64 candidates at or below it (a lane's
        // candidates need not start at k[0]: taken keys are none)
        uint32_t lo = none, hi = 0;
#pragma unroll
        for (int x = 0; x < MK; ++x) {
            lo = vx[x] ? tmin(lo, k[x]) : lo;
            hi = vx[x] ? tmax(hi, k[x]) : hi;
        }
        lo = wmin32(lo);
        hi = wmax32(hi);
        while (lo < hi) {
            const uint32_t mid = lo + ((hi - lo) >> 1);
            int c = 0;
#pragma unroll
            for (int x = 0; x < MK; ++x) c += __popcll(ballot(vx[x] && k[x] <= mid));
            if (c >= 64) hi = mid;
            else lo = mid + 1;
        }
        thr = lo;
    }
    // gather the want selected candidates (and take them out of the lists)
    int base = 0;
#pragma unroll
    for (int x = 0; x < MK; ++x) {
        const bool sel = vx[x] && k[x] <= thr;
        const unsigned long long m = ballot(sel);
        const int at = base + __popcll(m & lanemask_lt());  // < want <= 64
        if (sel && at < 64) C.rsel[at] = make_uint2(k[x], sd[x]);
        if (sel) k[x] = none;
        base += __popcll(m);
    }
    wave_sync();
    uint32_t ck = none, cs = 0;
    if (lane < want) { const uint2 e = C.rsel[lane]; ck = e.x; cs = e.y; }
    wave_sync();
    // (four independent counts, so that the lane reads overlap)
    int rank = 0, r1 = 0, r2 = 0, r3 = 0, j = 0;
    for (; j + 4 <= want; j += 4) {
        rank += int(rlu(ck, j) < ck);
        r1 += int(rlu(ck, j + 1) < ck);
        r2 += int(rlu(ck, j + 2) < ck);
        r3 += int(rlu(ck, j + 3) < ck);
    }
    for (; j < want; ++j) rank += int(rlu(ck, j) < ck);
    rank += r1 + r2 + r3;
    if (lane >= want) rank = lane;
    const uint32_t sk = uint32_t(__builtin_amdgcn_ds_permute(rank * 4, int(ck)));
    const uint32_t ss = uint32_t(__builtin_amdgcn_ds_permute(rank * 4, int(cs)));
    const int cum = wscan(lane < want ? int(ss >> 12) : 0, lane);
    const unsigned long long over = ballot(lane < want && cum > fr);
    // (with the extension every selected request is kept: the head of line,
    // the cache and the extension take them)
    const int got = over && !C.xn ? min(want, ffs64(over) + 1 + C.td) : want;
    if (lane < got) { myk = sk; mysd = ss; }
    return got;
}

// Head of line of instance i from its slots, with admission (Section 3.1:
// the local queue is served in (tier, seq) order while the head fits).  Each
// lane keeps the MK smallest keys of its slots, with their demand; the wave
// then takes minima round by round, lane r receiving the request of rank r,
// and stops when the winning lane had more waiting slots than it kept (its
// next key is unknown), after 64 requests, or qdepth requests after the first
// one whose cumulative demand exceeds the free blocks (the new head of line
// and the cache behind it).  A second read fetches the fields of the requests
// taken, and the longest fitting prefix is admitted at once (admit_ranked).
// The minima are taken on 32-bit keys when the candidates' seqs allow
// (rank_extract); with SEL (the kernels for 128+ instances) the same prefix
// is found by selection (rank_select), and when every request taken fits the
// candidates left up to the exhaustion bound are taken next without reading
// the slots again.  GR chunks of 64 slots are read per memory round trip.
// Returns true when every request taken was admitted and more wait (the head
// of line is still unknown).  Uniform.
template <int GR, int MK, bool SEL = false>
__device__ inline bool rescan_admit(const Ctx& C, int i, uint32_t t, int lane)
{
    const size_t b = size_t(i) * C.S;
    const int nch = live_chunks(C, i, lane);
    // per lane: its MK smallest keys, ascending, each with slot | demand << 12
    // (slot < 4096, demand < 2^16 blocks)
    unsigned long long k[MK];
    uint32_t sd[MK];
#pragma unroll
    for (int x = 0; x < MK; ++x) { k[x] = kNone; sd[x] = 0; }
    int cnt = 0;
    for (int c0 = 0; c0 < nch; c0 += GR) {
        uint32_t v[GR], m[GR], q[GR];
#pragma unroll
        for (int g = 0; g < GR; ++g) {
            const bool in = c0 + g < nch;
            const uint4 rr = in ? C.slot[b + (c0 + g) * 64 + lane] : make_uint4(0u, 0u, 0u, 0u);
            v[g] = rr.x; m[g] = rr.y; q[g] = rr.z;
        }
#pragma unroll
        for (int g = 0; g < GR; ++g) {
            if (wst(v[g]) != 1u) continue;
            ++cnt;
            unsigned long long ck = (rank_of(C, (m[g] >> 2) & 15u) << 32) | q[g];
            if (ck >= k[MK - 1]) continue;
            uint32_t cs = uint32_t((c0 + g) * 64 + lane) | (uint32_t(blocks_of(wlo(v[g]), C.shift)) << 12);
            // insertion into the lane's sorted list (the largest drops out)
#pragma unroll
            for (int x = 0; x < MK; ++x) {
                if (ck < k[x]) {
                    const unsigned long long tk = k[x]; k[x] = ck; ck = tk;
                    const uint32_t ts = sd[x]; sd[x] = cs; cs = ts;
                }
            }
        }
    }
    // rank extraction on 32-bit keys rank << 27 | (seq - lowest seq) when the
    // candidates' seqs span less than 2^27 (the order is the same; a 32-bit
    // wave minimum is a third of the 64-bit one), else on the keys themselves
    const int fr = C.freeb[i];
    const bool more = cnt > MK;
    uint32_t slo = 0xFFFFFFFFu, shi = 0;
#pragma unroll
    for (int x = 0; x < MK; ++x) {
        if (k[x] != kNone) { slo = tmin(slo, uint32_t(k[x])); shi = tmax(shi, uint32_t(k[x])); }
    }
    slo = wmin32(slo);
    shi = wmax32(shi);
    const bool c32 = shi - slo < (1u << 27) || slo > shi;
    uint32_t k32[MK];
#pragma unroll
    for (int x = 0; x < MK; ++x)
        k32[x] = k[x] == kNone ? 0xFFFFFFFFu : (uint32_t(k[x] >> 32) << 27) | (uint32_t(k[x]) - slo);
    const uint32_t bnd = SEL && c32 ? wmin32(more ? k32[MK - 1] : 0xFFFFFFFFu) : 0u;
    for (;;) {
        unsigned long long myk;
        uint32_t mysd;
        int got;
        if (c32) {
            uint32_t my32;
            if (SEL) got = rank_select<MK>(C, k32, sd, bnd, C.freeb[i], lane, my32, mysd);
            else got = rank_extract<uint32_t, MK>(k32, sd, more, fr, C.td, lane, my32, mysd);
            myk = my32 == 0xFFFFFFFFu
                      ? kNone
                      : (static_cast<unsigned long long>(my32 >> 27) << 32) | ((my32 & 0x7FFFFFFu) + slo);
        } else {
            got = rank_extract<unsigned long long, MK>(k, sd, more, fr, C.td, lane, myk, mysd);
        }
        if (got == 0) {
            if (lane == 0) clear_hol(C, i);
            wave_sync();
            return false;
        }
        const int mys = int(mysd & 0xFFFu);
        uint32_t w = 0, mt = 0, ta = 0;
        if (lane < got) { const uint4 rec = C.slot[b + mys]; w = rec.x; mt = rec.y; ta = rec.w; }
        const bool complete = got >= C.nwait[i];
        if (lane == 0) C.frs[i] = 0;
        admit_ranked(C, i, t, lane, got, myk, w, mt, ta, mys, complete);
        // (selection) every request taken was admitted and more wait: the
        // candidates left up to bnd are the next smallest keys of the queue,
        // and are taken without reading the slots again
        if (!(SEL && c32) || C.hols[i] != kHolUnknown) break;
        bool left = false;
#pragma unroll
        for (int x = 0; x < MK; ++x) left = left || (k32[x] != 0xFFFFFFFFu && k32[x] <= bnd);
        if (!ballot(left)) break;
    }
    return C.hols[i] == kHolUnknown;
}

// Admission of instance i when its head of line fits and 2..64 requests wait
// (Section 3.1: the local queue is served in priority order while the head
// fits).  The waiting requests are gathered into lanes, ranked by (tier, seq),
// and the longest prefix of the ranked list whose summed demand fits is
// admitted in one step; the next ranked request becomes the head of line.
// The result equals admitting the head of line one request at a time.  GR
// chunks of 64 slots are read per memory round trip.
template <int GR>
__device__ inline void admit_batch(const Ctx& C, int i, uint32_t t, int lane)
{
    const size_t b = size_t(i) * C.S;
    const int nch = live_chunks(C, i, lane);
    unsigned long long key = kNone;
    uint32_t word = 0, meta = 0, ta = 0;
    int slot = 0, w = 0;
    for (int c0 = 0; c0 < nch; c0 += GR) {
        uint32_t v[GR], m[GR], q[GR], a[GR];
        // all loads of the group are issued together (one memory round trip)
#pragma unroll
        for (int g = 0; g < GR; ++g) {
            const bool in = c0 + g < nch;
            const size_t sb = b + (c0 + g) * 64 + lane;
            const uint4 rr = in ? C.slot[sb] : make_uint4(0u, 0u, 0u, 0u);
            v[g] = rr.x; m[g] = rr.y; q[g] = rr.z; a[g] = rr.w;
        }
#pragma unroll
        for (int g = 0; g < GR; ++g) {
            const unsigned long long wm = ballot(wst(v[g]) == 1u);
            if (!wm) continue;
            const int cnt = __popcll(wm);
            const int k = lane - w;
            const bool take = k >= 0 && k < cnt;
            const int src = kth_set_bit(wm, take ? k : 0);
            const uint32_t pv = __shfl(v[g], src), pm = __shfl(m[g], src), pq = __shfl(q[g], src),
                           pa = __shfl(a[g], src);
            if (take) {
                word = pv; meta = pm; ta = pa;
                key = (rank_of(C, (pm >> 2) & 15u) << 32) | pq;
                slot = (c0 + g) * 64 + src;
            }
            w += cnt;
        }
    }
    if (w > 64) w = 64;  // callers guarantee at most 64 waiting requests
    // rank among the gathered keys (all distinct: seq is unique per replica)
    int rank = 0;
    for (int j = 0; j < w; ++j) rank += rl64(key, j) < key ? 1 : 0;
    if (lane >= w) rank = lane;
    // sort: lane r receives the request of rank r
    const int ad = rank * 4;
    const uint32_t k_lo = uint32_t(__builtin_amdgcn_ds_permute(ad, int(uint32_t(key))));
    const uint32_t k_hi = uint32_t(__builtin_amdgcn_ds_permute(ad, int(uint32_t(key >> 32))));
    word = uint32_t(__builtin_amdgcn_ds_permute(ad, int(word)));
    meta = uint32_t(__builtin_amdgcn_ds_permute(ad, int(meta)));
    ta = uint32_t(__builtin_amdgcn_ds_permute(ad, int(ta)));
    slot = __builtin_amdgcn_ds_permute(ad, slot);
    key = (static_cast<unsigned long long>(k_hi) << 32) | k_lo;
    admit_ranked(C, i, t, lane, w, key, word, meta, ta, slot);
}

// Admission of instance i from its head of line and the requests cached behind
// it, which are the smallest keys of its queue in order: the longest fitting
// prefix is admitted at once (admit_ranked).  When all of them fit and more
// wait, the head of line is unknown afterwards.
__device__ inline void admit_cached(const Ctx& C, int i, uint32_t t, int lane)
{
    const int n = C.qn[i];
    // (kernels for 128+ instances) the extension follows the ring: n + xc <= 63
    const int xv = C.xn ? C.xn[i] : 0, xc = xv & 0xFFFF, xh = xv >> 16;
    unsigned long long key = kNone;
    uint32_t word = 0, meta = 0, ta = 0;
    int slot = 0;
    if (lane == 0) {
        key = C.holk[i]; word = C.hwd[i]; meta = C.hmt[i]; ta = C.hta[i]; slot = C.hols[i];
    } else if (lane <= n + xc) {
        const uint4 e = lane <= n ? C.qt[qc_at(C, i, lane - 1)] : C.qx[size_t(i) * kQxDepth + xh + lane - n - 1];
        const uint32_t tier = (e.w >> 12) & 15u;
        key = qc_key(C, e);
        word = e.y;
        meta = kWaiting | (tier << 2) | (((e.w >> 16) & 1u) << 6);
        ta = e.z;
        slot = int(e.w & 0xFFFu);
    }
    const bool complete = C.nwait[i] == n + xc + 1;
    admit_ranked(C, i, t, lane, n + xc + 1, key, word, meta, ta, slot, complete, C.xn ? n : -1, xh);
}

// Admission of instance i whose waiting requests all arrived in the previous
// tick (kept in LDS by the dispatch): they are listed in dispatch order,
// which is (tier, seq) order, so no HBM read and no ranking is needed.
__device__ inline void admit_fresh(const Ctx& C, int i, uint32_t t, int lane)
{
    const int n = *C.lastn;
    const bool mine = lane < n && (C.lsl[lane] >> 16) == uint32_t(i);
    const unsigned long long mm = ballot(mine);
    const int w = __popcll(mm);
    // lane r receives the list index of the r-th request of i
    const int dest = mine ? __popcll(mm & lanemask_lt()) : w + __popcll(~mm & lanemask_lt());
    const int idx = __builtin_amdgcn_ds_permute(dest * 4, lane);
    unsigned long long key = kNone;
    uint32_t word = 0, meta = 0, ta = 0;
    int slot = 0;
    if (lane < w) {
        const uint32_t e = C.lsl[idx];
        const uint32_t tier = (e >> 12) & 15u;
        word = C.lw[idx];
        meta = kWaiting | (tier << 2);
        ta = t - 1u;
        slot = int(e & 0xFFFu);
        key = (rank_of(C, tier) << 32) | C.lsq[idx];
    }
    admit_ranked(C, i, t, lane, w, key, word, meta, ta, slot);
}

// Admission of instance i's known head of line, which fits (per lane: the
// lane-parallel rounds call it for their lanes' instances; the next head of
// line comes from the queue cache or is left unknown).
__device__ inline void admit_head(const Ctx& C, int i, uint32_t t)
{
    const int h = C.hols[i], dem = C.hold[i];
    const uint32_t w = C.hwd[i], m = C.hmt[i];
    const uint32_t len = wlo(w), rem = wmid(w);
    const uint32_t fin = t + rem;
    const size_t hb = size_t(i) * C.S + h;
    s_set_wm(C, hb, kRunW | ((fin & kFin) << 16) | (len + rem), (m & ~3u) | kRunning | kAdmitted);
    const int tier = int((m >> 2) & 15u);
    if (!(m & kAdmitted)) {
        stat(C, tier * 8 + kAdmittedCnt, 1);
        stat(C, tier * 8 + kQdelay, t - C.hta[i]);
        hist_add(C, kHistQdelay, tier, t - C.hta[i]);
    }
    C.freeb[i] -= dem;
    C.held[i] += dem;
    C.B[i] += 1;
    C.nwait[i] -= 1;
    c16_inc(C.res, res_idx(C, i, (len - t - 1u) & C.bmask));
    tier_inc(C, i, tier);
    wheel_put(C, fin, i, h);
    hol_pop(C, i);
}

// The whole admission of instance i (uniform): requests are admitted in
// (tier, seq) order while the head of line fits (Section 3.1), through the
// same steps as the lane-parallel rounds -- a rescan when the head of line
// is unknown, the previous tick's placements, a gather of a short queue, a
// cached run, or one head of line -- until the head of line does not fit or
// nothing waits.  Every step admits at least one request, or finds the head
// of line, so the loop ends.  (The kernels for 128+ instances hand instances
// to waves dynamically with it.)
template <int GR, int MK>
__device__ inline void admit_all(const Ctx& C, int i, uint32_t t, int lane)
{
    for (;;) {
        const int h = C.hols[i];
        if (h == kHolUnknown) {
            rescan_admit<GR, MK, true>(C, i, t, lane);
            continue;
        }
        if (h < 0 || C.hold[i] > C.freeb[i]) break;
        const int nw = C.nwait[i];
        const bool cached = C.td && (C.qn[i] > 0 || qx_count(C, i) > 0);
        if (nw >= 2 && nw <= 64 && C.frs[i]) {
            admit_fresh(C, i, t, lane);
        } else if (nw >= 2 && nw <= 64 && !cached) {
            admit_batch<GR>(C, i, t, lane);
        } else if (cached) {
            admit_cached(C, i, t, lane);
        } else {
            if (lane == 0) admit_head(C, i, t);
            wave_sync();
        }
    }
}

// ---------------------------------------------------------------------------
// Section 6.5 extensions, run at the start of a tick (uniform)
// ---------------------------------------------------------------------------

// Promotion pass: every waiting request of tier p >= 1 whose age t - tarr
// has reached the tier's quota (non-zero) moves to tier p - 1.  An instance
// with a promoted request loses its list of fresh placements and its queue
// cache; its head of line stays when it was not promoted and every promoted
// key is still larger, else it is found again by the admission rescan.
// lb <= the arrival tick of every waiting request of the instance, and every
// such tick is at most t (requests start to wait at the current tick or
// keep an older one): when t - lb is below the smallest quota no request can
// be old enough and the instance is not read.  lb = 0 means unknown (a
// launch starts so, as does an instance holding a request that arrived
// after t, possible only after the clock was moved back).
__device__ inline void promote_waiting(const Ctx& C, const Params& P, uint32_t t, int lane)
{
    const uint32_t qmin = P.ext[kXPromoMin];
    for (uint32_t i = 0; i < C.I; ++i) {
        if (C.nwait[i] == 0) continue;
        const uint32_t lb = wlb(C)[i];
        if (lb != 0 && t - lb < qmin) continue;
        const size_t b = size_t(i) * C.S;
        const int nch = live_chunks(C, i, lane);
        const int h = C.hols[i];
        bool any = false, late = false, head = false;
        uint32_t lo = 0xFFFFFFFFu;
        unsigned long long kmin = kNone;
        for (int c = 0; c < nch; ++c) {
            const int s = c * 64 + lane;
            const uint4 rec = C.slot[b + s];
            if (wst(rec.x) != 1u) continue;
            const uint32_t m = rec.y, tier = (m >> 2) & 15u, ta = rec.w;
            lo = ta < lo ? ta : lo;
            late = late || ta > t;
            if (tier == 0) continue;
            const uint32_t q = P.ext[kXAge + tier];
            if (q != 0 && t - ta >= q) {
                s_meta(C, b + s) = m - 4u;  // tier field at bits 2..5
                any = true;
                head = head || s == h;
                const unsigned long long k = (rank_of(C, tier - 1u) << 32) | rec.z;
                kmin = k < kmin ? k : kmin;
            }
        }
        lo = wmin32(lo);
        kmin = wmin64(kmin);
        const bool moved = ballot(any) != 0, unknown = ballot(late) != 0, hit = ballot(head) != 0;
        if (lane == 0) {
            wlb(C)[i] = unknown ? 0u : lo;
            if (moved) {
                C.frs[i] = 0;
                if (hit || h < 0 || kmin < C.holk[i]) C.hols[i] = kHolUnknown;
                else if (C.td) C.qn[i] = 0;
                qx_clear(C, i);
            }
        }
    }
    wave_sync();
}

// Adaptive headroom update of replica r: lane p < 10 handles tier p, with
// the headroom and the counter snapshots in HBM.  With a requests first
// admitted since the last update and their summed queue delay d, the
// headroom rises by a step when d > slo a, falls by a step when
// 256 d <= margin slo a, both tests in exact 128-bit arithmetic.
__device__ inline void adapt_headroom(const Ctx& C, const Params& P, uint32_t r, int lane)
{
    if (lane < kTiers) {
        const int p = lane;
        int32_t* hq = ext_hqr(P) + size_t(r) * kTiers;
        unsigned long long* snap = ext_hsnap(P) + size_t(r) * 2 * kTiers;
        const unsigned long long adm = C.stats[p * 8 + kAdmittedCnt], qd = C.stats[p * 8 + kQdelay];
        const unsigned long long a = adm - snap[p], d = qd - snap[kTiers + p];
        snap[p] = adm;
        snap[kTiers + p] = qd;
        if (p < int(C.K) && !(P.ext[kXZeroLowest] && p == int(C.K) - 1) && a != 0) {
            const unsigned long long slo = P.ext[kXSlo + p];
            const unsigned long long xl = slo * a, xh = __umul64hi(slo, a);
            const unsigned long long ms = slo * P.ext[kXAdaptMargin];  // < 2^29
            const unsigned long long yl = ms * a, yh = __umul64hi(ms, a);
            const unsigned long long dl = d << 8, dh = d >> 56;
            long long h = hq[p];
            if (xh == 0 && d > xl) {
                h += P.ext[kXAdaptUp];
                const long long mx = P.ext[kXAdaptMax];
                if (h > mx) h = mx;
            } else if (dh < yh || (dh == yh && dl <= yl)) {
                h -= P.ext[kXAdaptDown];
                if (h < 0) h = 0;
            }
            hq[p] = int32_t(h);
        }
    }
    wave_sync();
}

// ---------------------------------------------------------------------------
// k_step
// ---------------------------------------------------------------------------
// A barrier of the replica's waves (a wave-level one when a replica has one
// wave): every LDS and memory write before it is seen by every wave after it.
template <int NW>
__device__ __forceinline__ void block_sync()
{
    if (NW > 1) __syncthreads();
    else wave_sync();
}

template <int IM, bool INF, bool EXT>
__global__ __launch_bounds__(64 * waves_for(IM), IM <= 64 ? 4 : 2) void k_step(Params P, unsigned long long t0, uint32_t nt)
{
    // IPL: instances per lane when one wave covers every instance (the serial
    // phases, run by wave 0); OPL: instances per lane of the instances a wave
    // owns in the per-instance phases, instance (64 j + lane) NW + wid
    constexpr int NW = waves_for(IM);
    constexpr int IPL = (IM + 63) / 64;
    constexpr int OPL = (IM + 64 * NW - 1) / (64 * NW);
    extern __shared__ __align__(16) char lds_raw[];
    Ctx C = carve<IM, INF, EXT>(lds_raw, P);
    const int lane = lane_id();
    const int wid = NW > 1 ? int(threadIdx.x >> 6) : 0;
    const uint32_t tid = threadIdx.x;
    constexpr uint32_t NT = 64u * NW;
    const uint32_t I = P.I, S = P.S, W = P.W;
    const uint32_t wsz = P.wsz;
    constexpr bool infaas = INF;  // the global policy: INFaaS cost, else Llumnix freeness

    for (uint32_t r = blockIdx.x; r < P.R; r += gridDim.x) {
        const uint32_t g = P.group_of[r];
        C.K = P.group_K32[g];
        const int32_t* hq = P.hq + g * kTiers;
        if (EXT) {
            // (the parameters are read from memory where they are used, so that
            // none of them stays in registers through the tick loop)
            const int32_t* hqr = ext_hqr(P);
            if (hqr) hq = hqr + size_t(r) * kTiers;
            if (tid == 0) {
                const uint32_t t0u = uint32_t(t0), per = P.ext[kXPromoPeriod], ep = P.ext[kXAdaptEpoch];
                xleft(C)[0] = per ? int(t0u % per) : 0;
                xleft(C)[1] = ep ? int(t0u % ep) : 0;
            }
            for (uint32_t i = tid; i < P.I; i += NT) wlb(C)[i] = 0u;  // unknown: the first pass reads them
        }
#pragma unroll
        for (int p = 0; p < kTiers; ++p) C.hq[p] = hq[p];
        const size_t rb = size_t(r) * I * S;
        C.slot = P.slot + rb;
        if (C.xn) C.qx = P.qx + size_t(r) * I * kQxDepth;
        C.wheel = P.wheel + size_t(r) * wsz * P.wcap;
        C.hist = P.hist + size_t(r) * kHistPerReplica;

        // ---------------- prologue: derived per-instance state ----------------
        for (uint32_t j = tid; j < uint32_t(kNstat); j += NT) C.stats[j] = P.stats[size_t(r) * kNstat + j];
        for (uint32_t i = tid; i < I; i += NT) {
            C.freeb[i] = P.freeb[size_t(r) * I + i];
            C.drn[i] = P.drain[size_t(r) * I + i];
            for (int k = 0; k < 4; ++k) C.mig[4 * i + k] = P.mig[(size_t(r) * I + i) * 4 + k];
            C.inb[i] = 0;
            C.flags[i] = 0;
            C.tmask[i] = 0;
            C.frs[i] = 0;
            if (C.td) { C.qn[i] = 0; C.qh[i] = 0; }
            if (C.xn) C.xn[i] = 0;
            if (C.svc) C.svc[i] = P.svc[size_t(r) * I + i];
        }
        for (uint32_t b = tid; b < wsz / 2; b += NT) C.wc[b] = 0;
        if (tid == 0) { *C.lastn = 0; *C.nvic = 0; }
        for (uint32_t b = tid; b < (I * C.RB + 1) / 2; b += NT) C.res[b] = 0;
        for (uint32_t b = tid; b < (I * kTiers + 1) / 2; b += NT) C.tcnt[b] = 0;
        for (uint32_t b = tid; b < (wsz + 31) / 32; b += NT) C.wov[b] = 0;
        block_sync<NW>();
        for (uint32_t i = tid; i < I; i += NT) {
            const int d = C.mig[4 * i];
            if (d >= 0) C.inb[d] = C.mig[4 * i + 3];
        }
        block_sync<NW>();
        const uint32_t t0u = uint32_t(t0);
        {
            // The slots are read as one flat run of I * W chunks of 64 (chunk c
            // of instance i is flat chunk i W + c), GP chunks per memory round
            // trip; an instance is summed up after its last chunk.  The arrival
            // ticks of the heads of line are read afterwards, lane-parallel.
            // (each wave reads the chunks of the instances it owns: wid, wid + NW, ...)
            constexpr int GP = IM >= 128 ? 16 : 8;
            const uint32_t nown = NW > 1 ? (I > uint32_t(wid) ? (I - uint32_t(wid) + NW - 1) / NW : 0u) : I;
            const uint32_t nfl = nown * W;
            int nB = 0, nlive = 0, nw = 0, held = 0;
            unsigned long long bk = kNone;
            int bs = 0;
            uint32_t bv = 0, bm = 0;
            for (uint32_t f0 = 0; f0 < nfl; f0 += GP) {
                uint32_t v[GP], m[GP], q[GP];
#pragma unroll
                for (int g = 0; g < GP; ++g) {
                    const bool in = f0 + g < nfl;
                    const uint32_t fo = (f0 + g) / W;
                    const size_t fs = (size_t(fo * NW + wid) * W + (f0 + g - fo * W)) * 64 + lane;
                    const uint4 rr = in ? C.slot[fs] : make_uint4(0u, 0u, 0u, 0u);
                    v[g] = rr.x; m[g] = rr.y; q[g] = rr.z;
                }
#pragma unroll
                for (int g = 0; g < GP; ++g) {
                    const uint32_t f = f0 + g;
                    if (f >= nfl) continue;
                    const uint32_t io = f / W, c = f - io * W, i = io * NW + uint32_t(wid);
                    const int s = int(c) * 64 + lane;
                    const uint32_t st = wst(v[g]);
                    const unsigned long long ow = ballot(v[g] != 0);
                    nlive += __popcll(ow);
                    nB += __popcll(ballot(st == 2u));
                    nw += __popcll(ballot(st == 1u));
                    if (lane == 0) C.occ[i * W + c] = ow;
                    if (st == 2u) {
                        const uint32_t lenf = wlo(v[g]), fin = fin_of(v[g], t0u);
                        held += blocks_of(lenf - (fin - t0u + 1u), C.shift);
                        c16_inc(C.res, res_idx(C, i, (lenf - fin - 1u) & C.bmask));
                        c16_inc(C.tcnt, i * kTiers + int((m[g] >> 2) & 15u));
                        wheel_put(C, fin, int(i), s);
                    } else if (st == 1u) {
                        const unsigned long long k = (rank_of(C, (m[g] >> 2) & 15u) << 32) | q[g];
                        if (k < bk) { bk = k; bs = s; bv = v[g]; bm = m[g]; }
                    }
                    if (c + 1 == W) {
                        held = wsum(held);
                        const unsigned long long mn = wmin64(bk);
                        int hs = kNoHol;
                        uint32_t hw = 0, hm = 0;
                        if (mn != kNone) {
                            const int wl = ffs64(ballot(bk == mn));
                            hs = rl(bs, wl);
                            hw = rlu(bv, wl);
                            hm = rlu(bm, wl);
                        }
                        if (lane == 0) {
                            C.B[i] = nB; C.live[i] = nlive; C.nwait[i] = nw;
                            C.held[i] = held;
                            if (hs >= 0) set_hol(C, int(i), hs, mn, hw, hm, 0u);
                            else clear_hol(C, int(i));
                            int tm = 0;
                            for (int p = 0; p < kTiers; ++p) tm |= c16_get(C.tcnt, i * kTiers + p) ? (1 << p) : 0;
                            C.tmask[i] = tm;
                        }
                        wave_sync();
                        nB = 0; nlive = 0; nw = 0; held = 0;
                        bk = kNone; bs = 0; bv = 0; bm = 0;
                    }
                }
            }
            block_sync<NW>();
            for (uint32_t i = tid; i < I; i += NT) {
                const int h = C.hols[i];
                if (h >= 0) C.hta[i] = s_tarr(C, size_t(i) * S + h);
            }
        }
        unsigned next_seq = P.next_seq[r];
        uint32_t run_acc = 0, wait_acc = 0;  // per lane, at most 1024 ticks x 4 x 2048
        const unsigned long long* recs = P.arr_rec + size_t(r) * P.chunk * P.arr_cap;
        const uint32_t* cnts = P.arr_cnt + size_t(r) * P.chunk;
        block_sync<NW>();

        // the arrivals of the next tick are loaded one tick ahead; records past
        // the tick's count are never used
        const uint32_t lim = P.arr_cap < 64u ? P.arr_cap : 64u;
        // arrival counts 64 ticks at a time, lane l holding tick (tl & ~63) + l:
        // a tick's count is a lane read of a register, so no tick waits for
        // a load (and for the stores before it) to make its count uniform
        uint32_t cnt64 = uint32_t(lane) < nt ? cnts[lane] : 0u;
        // The finish visits are loaded ahead in two stages, both right after a
        // tick's own visit: the entries of the bucket two ticks ahead (pf2_n of
        // them; kNoPf: none), and the slots' word, meta and arrival tick of the
        // entries loaded a tick earlier for the next tick's bucket (pf_n, pf_e,
        // pf_v, pf_m, pf_a).  A visit uses them when its bucket still holds
        // exactly pf_n entries (appends, such as a committed migration's new
        // entry, change the count) and no preemption touched a slot in between
        // (victims' entries are dropped, more victims than the list holds drop
        // the whole set); otherwise it loads again.  A running request's word,
        // tier and arrival tick never change while it runs, and whether it is
        // being copied out is read from the migration records at the visit.
        constexpr uint32_t kNoPf = 0xFFFFFFFFu;
        uint32_t pf_n = kNoPf, pf_e = 0, pf_v = 0, pf_m = 0, pf_a = 0;
        uint32_t pf2_n = kNoPf, pf2_e = 0;
        // (wave 0) ticks to the next pairing round, and whether a migration
        // record may be active (the staged-copy phase is skipped otherwise)
        uint32_t mig_left = (P.mig_interval - t0u % P.mig_interval) % P.mig_interval;
        bool migs = false;
        for (uint32_t i = lane; i < I; i += 64) migs = migs || C.mig[4 * i] >= 0;
        migs = ballot(migs) != 0;
        unsigned long long a_nx = uint32_t(lane) < lim ? recs[lane] : 0ull;
        for (uint32_t tl = 0; tl < nt; ++tl) {
            const uint32_t t = t0u + tl;
            const uint32_t n = rlu(cnt64, int(tl & 63u));
            const unsigned long long* rec = recs + size_t(tl) * P.arr_cap;
            const unsigned long long a0 = a_nx;

            // ============ Section 6.5: promotion, adaptive headroom ============
            // (the countdowns and parameters live in LDS: nothing of this stays
            // in registers across the tick)
            if (EXT) {
                const int pl = xleft(C)[0], al = xleft(C)[1];
                const int per = int(P.ext[kXPromoPeriod]), ep = int(P.ext[kXAdaptEpoch]);
                if (wid == 0) {
                    if (per && pl == 0) promote_waiting(C, P, t, lane);
                    if (ep && al == 0) adapt_headroom(C, P, r, lane);
                }
                block_sync<NW>();
                if (ep && al == 0) {
                    const int32_t* hq = ext_hqr(P) + size_t(r) * kTiers;
#pragma unroll
                    for (int p = 0; p < kTiers; ++p) C.hq[p] = hq[p];
                }
                if (tid == 0) {
                    xleft(C)[0] = per && pl + 1 < per ? pl + 1 : 0;
                    xleft(C)[1] = ep && al + 1 < ep ? al + 1 : 0;
                }
            }

            // ===================== A: growth, preemption, finish =====================
            // an instance whose growth fits takes its blocks at once; the others
            // preempt first (and take them at the end of preempt)
            const uint32_t cres = (0u - t) & C.bmask;
            unsigned long long pre[OPL];
            bool preempting = false;
#pragma unroll
            for (int j = 0; j < OPL; ++j) {
                const uint32_t i = (uint32_t(lane) + 64u * j) * NW + uint32_t(wid);
                bool np = false;
                if (i < I) {
                    const int G = int(c16_get(C.res, res_idx(C, i, cres)));
                    const int fr = C.freeb[i];
                    np = G > fr;
                    if (np) {
                        C.gtmp[i] = G;
                    } else {
                        C.freeb[i] = fr - G;
                        C.held[i] += G;
                    }
                    if (C.flags[i] & kFlagIntf) C.flags[i] &= ~kFlagIntf;
                    if (C.fsum) { C.fsum[i] = 0; C.fcnt[i] = 0; }
                }
                pre[j] = ballot(np);
                preempting = preempting || pre[j] != 0;
            }
            // migrations to abort: set by preemption and finish, kept in a register
            // (multi-wave kernels: another wave's preemption sets the block flag)
            bool abort_any = false;
            if (preempting) {
                wave_sync();
#pragma unroll
                for (int j = 0; j < OPL; ++j)
                    for (unsigned long long m = pre[j]; m; m &= m - 1)
                        abort_any = preempt<(IM >= 128 ? 16 : 4), 2>(
                                        C, int((64u * j + ffs64(m)) * NW + uint32_t(wid)), t, lane) || abort_any;
            }
            if (NW > 1) {
                if (abort_any && lane == 0) *C.bflag = 1;
                if (tid == 0) {
                    *C.bsum = 0;  // the auto-scaling sum of this tick (phase C)
                    *C.wln = 0;   // the admission work list (phase B)
                    *C.wlnext = 0;
                }
                block_sync<NW>();
                if (wid == 0) {
                    preempting = *C.nvic != 0;
                    abort_any = *C.bflag != 0;
                }
            }
            // a preempted request is waiting now: its prefetched entries (for this
            // tick's and the next tick's visit) are dropped (its wheel entry was
            // erased); more victims than the list holds make both visits load again
            bool pf_lost = false;
            if (preempting && wid == 0) {
                const int nv = *C.nvic;
                pf_lost = nv > kVic;
                for (int v = 0; v < nv && v < kVic; ++v) {
                    if (pf_e == C.vic[v]) pf_e = kTomb;
                    if (pf2_e == C.vic[v]) pf2_e = kTomb;
                }
            }
            wave_sync();
            // the finish visit and the release of aborted migrations: wave 0
            if (wid == 0) {
            if (lane == 0) *C.nvic = 0;
            {
                const uint32_t bk = t & C.wmask;
                const uint32_t nb = (C.wc[bk >> 1] >> ((bk & 1u) * 16u)) & 0xFFFFu;
                const bool ov = (C.wov[bk >> 5] >> (bk & 31u)) & 1u;
                if (pf_n != kNoPf && !pf_lost && !ov && nb == pf_n) {
                    uint32_t* ent = C.wheel + size_t(bk) * C.wcap;
                    const uint32_t kept = finish_batch(C, t, lane, ent, 0, uint32_t(lane) < pf_n, pf_e, pf_v, pf_m, pf_a,
                                                       abort_any);
                    wheel_set_count(C, bk, kept, lane);
                } else {
                    finish_tick(C, t, lane, abort_any);
                }
                // slots of the next tick's bucket, from the entries loaded a tick ago
                pf_n = pf_lost ? kNoPf : pf2_n;
                pf_e = pf2_e;
                if (pf_n != kNoPf) {
                    const uint32_t pi = pf_e >> 16, ps = pf_e & 0xFFFFu;
                    const bool ok = uint32_t(lane) < pf_n && pi < I && ps < S;
                    const size_t idx = size_t(pi) * S + ps;
                    const uint4 rec = ok ? C.slot[idx] : make_uint4(0u, 0u, 0u, 0u);
                    pf_v = rec.x; pf_m = rec.y; pf_a = rec.w;
                }
                // entries of the bucket two ticks ahead (three distinct buckets needed)
                const uint32_t b2 = (t + 2u) & C.wmask;
                const uint32_t n2 = (C.wc[b2 >> 1] >> ((b2 & 1u) * 16u)) & 0xFFFFu;
                const bool ov2 = (C.wov[b2 >> 5] >> (b2 & 31u)) & 1u;
                pf2_n = !ov2 && n2 <= 64u && C.wmask >= 3u ? n2 : kNoPf;
                pf2_e = pf2_n != kNoPf && uint32_t(lane) < pf2_n ? C.wheel[size_t(b2) * C.wcap + lane] : 0u;
            }
            // ===================== A2: release reservations of aborted migrations =====================
            if (abort_any) {
                for (uint32_t i = lane; i < I; i += 64) {
                    if (!(C.flags[i] & kFlagAbort)) continue;
                    C.flags[i] &= ~kFlagAbort;
                    int* m = &C.mig[4 * i];
                    const int d = m[0];
                    if (d < 0) continue;
                    C.freeb[d] += m[3];
                    C.inb[d] = 0;
                    const size_t db = size_t(d) * S + m[2];
                    s_word(C, db) = 0;
                    C.occ[d * W + (m[2] >> 6)] &= ~(1ull << (m[2] & 63));
                    C.live[d] -= 1;
                    m[0] = -1; m[1] = 0; m[2] = 0; m[3] = 0;
                    stat(C, kMigAborted, 1);
                }
                wave_sync();
            }
            if (NW > 1 && lane == 0) *C.bflag = 0;
            }  // wave 0
            block_sync<NW>();

            // ===================== B: admission (lane-parallel rounds); C: freeness =====================
            // Eight-wave kernels: the instances with admission work (an unknown
            // head of line, or a known one that fits) are listed, and the waves
            // take them one at a time from the list, each admitting on its
            // instance to the end: a few long queues no longer load one wave.
            // Admissions on different instances touch only their own state and
            // shared counters, so the order does not matter.
            if (NW > 1) {
#pragma unroll
                for (int j = 0; j < OPL; ++j) {
                    const uint32_t i = (uint32_t(lane) + 64u * j) * NW + uint32_t(wid);
                    const bool need = i < I && (C.hols[i] == kHolUnknown || (C.hols[i] >= 0 && C.hold[i] <= C.freeb[i]));
                    if (need) C.order[atomicAdd(C.wln, 1)] = int(i);
                }
                block_sync<NW>();
                const int nl = *C.wln;
                for (;;) {
                    int k = 0;
                    if (lane == 0) k = atomicAdd(C.wlnext, 1);
                    k = rl(k, 0);
                    if (k >= nl) break;
                    admit_all<16, 3>(C, C.order[k], t, lane);
                }
                // phase C reads the instances each wave owns, which any wave
                // may have admitted on
                block_sync<NW>();
            } else
            for (;;) {
                // heads of line left unknown: found by a rescan, which admits at once
                bool unk = false;
#pragma unroll
                for (int j = 0; j < OPL; ++j) {
                    const uint32_t i = (uint32_t(lane) + 64u * j) * NW + uint32_t(wid);
                    for (unsigned long long m = ballot(i < I && C.hols[i] == kHolUnknown); m; m &= m - 1)
                        unk = rescan_admit<(IM >= 128 ? 16 : 4), (IM >= 128 ? 4 : 2)>(
                                  C, int((64u * j + ffs64(m)) * NW + uint32_t(wid)), t, lane) || unk;
                }
                bool any = unk;
                unsigned long long bat[OPL], frm[OPL], cch[OPL];
#pragma unroll
                for (int j = 0; j < OPL; ++j) {
                    const uint32_t i = (uint32_t(lane) + 64u * j) * NW + uint32_t(wid);
                    bool batch = false, fresh = false, cachd = false;
                    if (i < I && C.hols[i] >= 0 && C.hold[i] <= C.freeb[i]) {
                        const int nw = C.nwait[i];
                        const bool cached = C.td && C.qn[i] > 0;
                        if (nw >= 2 && nw <= 64 && C.frs[i]) {
                            fresh = true;
                        } else if (nw >= 2 && nw <= 64 && !cached) {
                            batch = true;
                        } else if (IM >= 128 && cached) {
                            // the kernels for 128+ instances admit a cached run at
                            // once (the head of line may be unknown afterwards)
                            cachd = true;
                            any = true;
                        } else {
                            // the only waiting request, a queue longer than a wave or one
                            // whose next requests are cached: admit heads of line one at a
                            // time while they fit and are known
                            do {
                                admit_head(C, int(i), t);
                            } while (C.hols[i] >= 0 && C.hold[i] <= C.freeb[i]);
                            // an unknown head of line is found by the next round's rescan
                            any = any || C.hols[i] == kHolUnknown;
                        }
                    }
                    bat[j] = ballot(batch);
                    frm[j] = ballot(fresh);
                    cch[j] = ballot(cachd);
                }
                wave_sync();
#pragma unroll
                for (int j = 0; j < OPL; ++j) {
                    for (unsigned long long m = frm[j]; m; m &= m - 1)
                        admit_fresh(C, int((64u * j + ffs64(m)) * NW + uint32_t(wid)), t, lane);
                    for (unsigned long long m = bat[j]; m; m &= m - 1)
                        admit_batch<(IM >= 128 ? 16 : 4)>(C, int((64u * j + ffs64(m)) * NW + uint32_t(wid)), t, lane);
                    for (unsigned long long m = cch[j]; m; m &= m - 1)
                        admit_cached(C, int((64u * j + ffs64(m)) * NW + uint32_t(wid)), t, lane);
                }
                if (!ballot(any)) break;
            }
            // auto-scaling signal (Section 3.6): the cluster average of the
            // normal-priority freeness F_normal = (free - head-of-line demand) /
            // max(B, 1) -- no headroom, no draining sentinel -- in fixed point,
            // floor(F_normal * 2^20) per instance, against -1/2 and 3/2
            long long fsum = 0;
#pragma unroll
            for (int j = 0; j < OPL; ++j) {
                const uint32_t i = (uint32_t(lane) + 64u * j) * NW + uint32_t(wid);
                if (i >= I) continue;
                set_f(C, int(i));
                // slot-ticks: running and waiting requests at the end of the tick.
                // Later phases move running and waiting requests between
                // instances (commits, queued moves) and add only the arrivals
                // the dispatch places, counted there
                run_acc += unsigned(C.B[i]);
                wait_acc += unsigned(C.nwait[i]);
                if (C.freeb[i] < 0 || C.freeb[i] + C.held[i] + C.inb[i] != int(C.M)) stat(C, kInvariant, 1);
                // floor(x 2^20 / den): x 2^20 is exact in a double (|x| < 2^22) and
                // the correctly rounded quotient never crosses an integer (the
                // quotient sits at least 1/den >= 2^-11 from one, more than half
                // an ulp below 2^42); the integer residual check keeps it exact
                const long long a = static_cast<long long>(C.freeb[i] - C.hold[i]) * 1048576ll;
                const long long d = C.den[i];
                long long q = static_cast<long long>(floor(double(a) / double(d)));
                const long long rr = a - q * d;
                if (rr < 0) q -= 1;
                else if (rr >= d) q += 1;
                fsum += q;
            }
            fsum = static_cast<long long>(wsum64(static_cast<unsigned long long>(fsum)));
            if (C.svc) {
                // INFaaS: service-time estimate from this tick's finishes, then
                // the state penalty (OVERLOADED before INTERFERED before ACTIVE)
#pragma unroll
                for (int j = 0; j < OPL; ++j) {
                    const uint32_t i = (uint32_t(lane) + 64u * j) * NW + uint32_t(wid);
                    if (i >= I) continue;
                    const int c = C.fcnt[i];
                    if (c > 0) {
                        // floor(256 sum / c): sum < 2^43, so 256 sum is exact in a
                        // double; the residual corrects the rounded quotient
                        const long long num = static_cast<long long>(C.fsum[i] * 256ull);
                        long long mean = static_cast<long long>(floor(double(num) / double(c)));
                        const long long rr = num - mean * c;
                        if (rr < 0) mean -= 1;
                        else if (rr >= c) mean += 1;
                        C.svc[i] += (mean - C.svc[i]) >> P.ewma_shift;  // arithmetic shift: floor
                    }
                    C.pen[i] = C.hols[i] >= 0 && C.hold[i] > C.freeb[i] ? int(P.pen_over)
                             : (C.flags[i] & kFlagIntf) ? int(P.pen_intf) : 0;
                }
            }
            if (NW > 1) {
                if (lane == 0) atomicAdd(reinterpret_cast<unsigned long long*>(C.bsum), static_cast<unsigned long long>(fsum));
                block_sync<NW>();
                fsum = *C.bsum;
            }
            if (tid == 0) {
                const long long half = static_cast<long long>(I) << 19;
                if (fsum < -half) stat(C, kScaleOut, 1);
                else if (fsum > 3 * half) stat(C, kScaleIn, 1);
            }
            wave_sync();

            // the dispatch and the migrations (phases D and E): wave 0 (pairing:
            // whether it runs this tick and how many instances can pair)
            bool e2 = false;
            int n2 = 0;
            if (wid == 0) {
            // ===================== D: tier-ordered dispatch =====================
            // an instance with an empty queue now holds, after this dispatch, only
            // this tick's arrivals; they are recorded in LDS when they fit one wave
            // (frs is written with the dispatch's write-back, from the queue length before it)
            if (lane == 0) *C.lastn = 0;
            if (n == 0)
                for (uint32_t i = lane; i < I; i += 64) C.frs[i] = C.nwait[i] == 0;
            if (n > 0) {
                const unsigned seq0 = next_seq;
                next_seq += n;
                // per-instance dispatch state in registers: lane l, register j <-> instance 64 j + l
                // key: F of the instances that can take an arrival (minus infinity
                // for a full instance and, in the first mode, for a draining one)
                // (an arrival that becomes an instance's head of line updates its
                // demand, num and F in LDS at once: only that instance's lane
                // touches them until the write-back)
                double key[IPL], fnew[IPL];
                int live_r[IPL], nadd[IPL], pend_r[IPL], num_r[IPL], hold_r[IPL];
                unsigned long long hk_r[IPL];
#pragma unroll
                for (int j = 0; j < IPL; ++j) {
                    const uint32_t i = lane + 64 * j;
                    nadd[j] = 0;
                    pend_r[j] = -1;
                    num_r[j] = 0;
                    hold_r[j] = 0;
                    fnew[j] = 0.0;
                    if (i < I) {
                        live_r[j] = C.live[i];
                        num_r[j] = C.num[i];
                        hold_r[j] = C.hold[i];
                        hk_r[j] = C.hols[i] == kNoHol ? kNone : C.holk[i];
                        key[j] = live_r[j] < int(S) && !C.drn[i] ? (infaas ? -infaas_cost(C, P, int(i), 0) : C.fd[i])
                                                                 : -__builtin_inf();
                    } else {
                        live_r[j] = int(S); hk_r[j] = 0;
                        key[j] = -__builtin_inf();
                    }
                }
                int cur = -1;
                bool full = false;
                bool drain_mode = false;  // every instance with room is draining (Section 3.4 fallback)
                int nfall = 0;
                for (uint32_t k0 = 0; k0 < n; k0 += 64) {
                    const uint32_t cn = n - k0 < 64 ? n - k0 : 64;
                    const unsigned long long a = k0 == 0 ? a0 : (lane < int(cn) ? rec[k0 + lane] : 0);
                    int tgt = -1, rank = 0;  // rank: among this batch's arrivals bound for tgt
                    uint32_t k = 0;
                    while (k < cn && !full) {
                        if (cur < 0) {
                            double lb = key[0];
#pragma unroll
                            for (int j = 1; j < IPL; ++j) lb = fmax(lb, key[j]);
                            double mv = wave_max_f64<(IM < 64 ? IM : 64)>(lb);
                            if (mv == -__builtin_inf() && !drain_mode) {
                                // no non-draining instance has a free slot: the least
                                // loaded draining one (largest F without the sentinel);
                                // slots only fill up, so the mode holds for the tick
                                drain_mode = true;
#pragma unroll
                                for (int j = 0; j < IPL; ++j) {
                                    const uint32_t i = lane + 64 * j;
                                    key[j] = i < I && live_r[j] < int(S) && C.drn[i]
                                                 ? (infaas ? -infaas_cost(C, P, int(i), nadd[j]) : C.fd[i])
                                                 : -__builtin_inf();
                                }
                                lb = key[0];
#pragma unroll
                                for (int j = 1; j < IPL; ++j) lb = fmax(lb, key[j]);
                                mv = wave_max_f64<(IM < 64 ? IM : 64)>(lb);
                            }
                            if (mv == -__builtin_inf()) { full = true; break; }
#pragma unroll
                            for (int j = IPL - 1; j >= 0; --j) {
                                const unsigned long long bm = ballot(key[j] == mv);
                                if (bm) cur = 64 * j + ffs64(bm);
                            }
                        }
                        const int jc = cur >> 6, lc = cur & 63;
                        int lv = 0, na0 = 0;
                        unsigned long long hkc = 0;
#pragma unroll
                        for (int j = 0; j < IPL; ++j)
                            if (j == jc) { lv = rl(live_r[j], lc); hkc = rl64(hk_r[j], lc); na0 = rl(nadd[j], lc); }
                        const unsigned long long ak = rl64(a, int(k));
                        const unsigned long long hk = rank_of(C, uint32_t(ak >> 32) & 15u) << 32 | (seq0 + unsigned(ak >> 36));
                        const bool becomes = hk < hkc;
                        // Arrival k goes to cur.  If it becomes cur's head of line, F of cur
                        // changes and the argmax is taken again.  Otherwise F stays, and
                        // so does the argmax for the following arrivals, none of which can
                        // become the head of line (keys increase along the arrival order):
                        // they all go to cur until its slots run out.
                        // (under INFaaS every placement raises cur's cost by alpha)
                        const bool step1 = becomes || (infaas && P.alpha256 > 0);
                        const int m = step1 ? 1 : min(int(cn - k), int(S) - lv);
                        const int nl = lv + m;
                        if (lane == lc) {
#pragma unroll
                            for (int j = 0; j < IPL; ++j) {
                                if (j != jc) continue;
                                live_r[j] = nl;
                                nadd[j] += m;
                                if (becomes) {
                                    hk_r[j] = hk;
                                    pend_r[j] = int(k0 + k);
                                    // Eq. 1-2: F moves by the change of head-of-line demand
                                    // (num and the demand stay in registers until the write-back)
                                    const int dem = blocks_of(uint32_t(ak & 0xFFFFu), C.shift);
                                    num_r[j] -= 256 * (dem - hold_r[j]);
                                    hold_r[j] = dem;
                                    fnew[j] = double(num_r[j]) / double(C.den[lc + 64 * j]);
                                    if (!infaas) key[j] = fnew[j];
                                }
                                if (infaas) key[j] -= double(P.alpha256) * double(m);
                                if (nl >= int(S)) key[j] = -__builtin_inf();
                            }
                        }
                        if (lane >= int(k) && lane < int(k) + m) { tgt = cur; rank = na0 + lane - int(k); }
                        if (step1 || nl >= int(S)) cur = -1;
                        if (drain_mode) nfall += m;
                        k += uint32_t(m);
                    }
                    // write the dispatch state back for the slot assignment and later phases
#pragma unroll
                    for (int j = 0; j < IPL; ++j) {
                        const uint32_t i = lane + 64 * j;
                        if (i >= I) continue;
                        C.live[i] = live_r[j];
                        const int nw0 = C.nwait[i];
                        if (k0 == 0) C.frs[i] = nw0 == 0 && n <= uint32_t(kLast);
                        C.nwait[i] = nw0 + nadd[j];
                        wait_acc += unsigned(nadd[j]);
                        if (pend_r[j] >= 0) {
                            C.num[i] = num_r[j];
                            C.hold[i] = hold_r[j];
                            C.fd[i] = fnew[j];
                        }
                        if (C.ext && nadd[j] > 0) wlb(C)[i] = t < wlb(C)[i] ? t : wlb(C)[i];
                        if (C.td && nadd[j] > 0) {
                            // queue cache: an arrival that became the head of line pushes
                            // the old head to the front of the cache; other arrivals may
                            // fall between cached entries, so the cache is emptied
                            if (nadd[j] > (pend_r[j] >= 0 ? 1 : 0)) {
                                C.qn[i] = 0;
                                qx_clear(C, int(i));
                            } else if (C.hols[i] >= 0) {
                                qc_insert_at(C, int(i), 0, qc_pack(C.holk[i], C.hols[i], C.hwd[i], C.hmt[i], C.hta[i]));
                            }
                        }
                        nadd[j] = 0;
                        if (pend_r[j] >= 0) {
                            C.hols[i] = kHolPending;
                            C.pend[i] = pend_r[j];
                            C.holk[i] = hk_r[j];
                            pend_r[j] = -1;
                        }
                    }
                    wave_sync();
                    // slot assignment: the arrivals bound for one instance take its
                    // lowest empty slots in arrival order
                    const int tier = int((a >> 32) & 15u);
                    int s = -1;
                    bool searched = false;
                    const unsigned long long tgm = ballot(tgt >= 0);
                    if (W > 8 && W <= uint32_t(IM) && tgm) {
                        const int ft = rl(tgt, ffs64(tgm));
                        if (!ballot(tgt >= 0 && tgt != ft)) {
                            // the whole batch goes to one instance (a burst): the
                            // inclusive prefix of its free slots per occupancy word
                            // (gtmp, free during the dispatch), and each arrival's
                            // word by binary search
                            const unsigned long long wdl = uint32_t(lane) < W ? C.occ[ft * W + lane] : kNone;
                            const int pre = wscan(64 - __popcll(wdl), lane);
                            if (uint32_t(lane) < W) C.gtmp[lane] = pre;
                            wave_sync();
                            if (tgt >= 0) {
                                int lo = 0, hi = int(W) - 1;
                                while (lo < hi) {
                                    const int mid = (lo + hi) >> 1;
                                    if (C.gtmp[mid] > rank) hi = mid;
                                    else lo = mid + 1;
                                }
                                if (C.gtmp[lo] > rank) {
                                    const int before = lo ? C.gtmp[lo - 1] : 0;
                                    s = lo * 64 + kth_set_bit(~C.occ[ft * W + lo], rank - before);
                                }
                            }
                            searched = true;
                        }
                    }
                    if (tgt >= 0 && !searched) {
                        // the rank-th empty slot, four occupancy words per step
                        int rk = rank;
                        for (uint32_t w0 = 0; w0 < W && s < 0; w0 += 4) {
                            unsigned long long wd[4];
#pragma unroll
                            for (int k = 0; k < 4; ++k) wd[k] = w0 + k < W ? C.occ[tgt * W + w0 + k] : kNone;
#pragma unroll
                            for (int k = 0; k < 4; ++k) {
                                const int z = 64 - __popcll(wd[k]);
                                if (s < 0) {
                                    if (rk < z) s = int(w0 + k) * 64 + kth_set_bit(~wd[k], rk);
                                    else rk -= z;
                                }
                            }
                        }
                    }
                    if (tgt >= 0 && s < 0) {  // occupancy and live count disagree: flag, drop the arrival
                        stat(C, kInvariant, 1);
                        stat(C, tier * 8 + kRejected, 1);
                        tgt = -2;
                    }
                    wave_sync();
                    if (n <= uint32_t(kLast)) {
                        const unsigned long long pm = ballot(tgt >= 0);
                        if (tgt >= 0) {
                            const int q = __popcll(pm & lanemask_lt());
                            C.lw[q] = kWaitW | (uint32_t((a >> 16) & 0xFFFFu) << 16) | uint32_t(a & 0xFFFFu);
                            C.lsl[q] = (uint32_t(tgt) << 16) | (uint32_t(tier) << 12) | uint32_t(s);
                            C.lsq[q] = seq0 + unsigned(a >> 36);
                        }
                        if (lane == 0) *C.lastn = __popcll(pm);
                    }
                    if (tgt >= 0) {
                        atomicOr(&C.occ[tgt * W + (s >> 6)], 1ull << (s & 63));
                        const size_t sb = size_t(tgt) * S + s;
                        const uint32_t word = kWaitW | (uint32_t((a >> 16) & 0xFFFFu) << 16) | uint32_t(a & 0xFFFFu);
                        const uint32_t meta = kWaiting | (unsigned(tier) << 2);
                        C.slot[sb] = make_uint4(word, meta, seq0 + unsigned(a >> 36), t);
                        if (C.hols[tgt] == kHolPending && C.pend[tgt] == int(k0) + lane) {
                            C.hols[tgt] = s;
                            C.hwd[tgt] = word;
                            C.hmt[tgt] = meta;
                            C.hta[tgt] = t;
                        }
                    }
                    // every arrival is dispatched (tgt >= 0) or rejected: no free slot
                    // anywhere (-1), or dropped by the occupancy check (-2, counted
                    // above)
                    const int vt = lane < int(cn) ? tier : 15;
                    tier_stat3(C, vt, lane < int(cn), kArrived, tgt >= 0, kDispatched, tgt == -1 && lane < int(cn),
                               kRejected, lane);
                    wave_sync();
                }
                if (lane == 0 && nfall) stat(C, kDrainFallback, unsigned(nfall));
            }

            if (tl + 1 < nt) {
                if (((tl + 1u) & 63u) == 0) {
                    const uint32_t* cn = uniform_ptr(cnts + tl + 1u);
                    cnt64 = tl + 1u + lane < nt ? cn[lane] : 0u;
                }
                const unsigned long long* rn = uniform_ptr(rec + P.arr_cap);
                a_nx = uint32_t(lane) < lim ? rn[lane] : 0ull;
            }

            // ===================== E1: staged copies =====================
            // a commit leaves the source slot: its wheel entry (source slot in
            // gtmp, finish tick in pend) is erased after the loop
            if (migs) {
            for (uint32_t i = lane; i < I; i += 64) C.gtmp[i] = -1;
            for (uint32_t i = lane; i < I; i += 64) {
                int* m = &C.mig[4 * i];
                const int d = m[0];
                if (d < 0) continue;
                const size_t sb = size_t(i) * S + m[1], db = size_t(d) * S + m[2];
                const uint4 srec = C.slot[sb];
                const uint32_t v = srec.x;
                const uint32_t fin = fin_of(v, t);
                const int bl = blocks_of(wlo(v) - (fin - t), C.shift);
                int w = bl - m[3];
                if (w > int(P.mig_stage)) w = int(P.mig_stage);
                if (w > C.freeb[d]) {
                    C.freeb[d] += m[3];
                    C.inb[d] = 0;
                    s_word(C, db) = 0;
                    C.occ[d * W + (m[2] >> 6)] &= ~(1ull << (m[2] & 63));
                    C.live[d] -= 1;
                    s_meta(C, sb) = srec.y & ~kMigrating;
                    m[0] = -1; m[1] = 0; m[2] = 0; m[3] = 0;
                    stat(C, kMigAborted, 1);
                    set_f(C, d);
                    continue;
                }
                C.freeb[d] -= w;
                m[3] += w;
                C.inb[d] += w;
                if (m[3] == bl) {
                    const uint32_t mm = srec.y;
                    const int tier = int((mm >> 2) & 15u);
                    const int rr = int((wlo(v) - fin - 1u) & C.bmask);
                    C.slot[db] = make_uint4(v, (mm & ~(3u | kMigrating)) | kRunning, srec.z, srec.w);
                    s_word(C, sb) = 0;
                    C.occ[i * W + (m[1] >> 6)] &= ~(1ull << (m[1] & 63));
                    C.live[i] -= 1;
                    C.freeb[i] += bl;
                    C.held[i] -= bl;
                    C.held[d] += bl;
                    C.inb[d] = 0;
                    C.B[i] -= 1;
                    C.B[d] += 1;
                    c16_dec(C.res, res_idx(C, i, rr));
                    c16_inc(C.res, res_idx(C, d, rr));
                    tier_dec(C, int(i), tier);
                    tier_inc(C, d, tier);
                    wheel_put(C, fin, d, m[2]);
                    C.gtmp[i] = m[1];
                    C.pend[i] = int(fin);
                    m[0] = -1; m[1] = 0; m[2] = 0; m[3] = 0;
                    stat(C, kMigCommitted, 1);
                    set_f(C, int(i));
                }
                set_f(C, d);
            }
            wave_sync();
#pragma unroll
            for (int j = 0; j < IPL; ++j) {
                const uint32_t i0 = lane + 64 * j;
                for (unsigned long long m = ballot(i0 < I && C.gtmp[i0] >= 0); m; m &= m - 1) {
                    const int ii = 64 * j + ffs64(m);
                    wheel_erase(C, uint32_t(C.pend[ii]), ii, C.gtmp[ii], lane);
                }
            }
            wave_sync();
            bool live = false;
            for (uint32_t i = lane; i < I; i += 64) live = live || C.mig[4 * i] >= 0;
            migs = ballot(live) != 0;
            }

            // ===================== E2: pairing on interval ticks =====================
            const bool mig_tick = mig_left == 0;
            mig_left = mig_tick ? P.mig_interval - 1u : mig_left - 1u;
            // pairing in three parts: which instances can pair and their keys
            // (wave 0), their order (wave 0 by counting ranks; in the
            // eight-wave kernels every thread counts), the pairs (wave 0)
            if (!infaas && mig_tick) {
                bool neg = false;
                for (uint32_t i = lane; i < I; i += 64) neg |= C.num[i] < 0 || C.drn[i];
                if (ballot(neg)) {
                    e2 = true;
                    for (uint32_t i = lane; i < I; i += 64) C.flags[i] &= ~kFlagBusy;
                    wave_sync();
                    for (uint32_t i = lane; i < I; i += 64) {
                        const int d = C.mig[4 * i];
                        if (d >= 0) { atomicOr(&C.flags[i], kFlagBusy); atomicOr(&C.flags[d], kFlagBusy); }
                    }
                    wave_sync();
                    // rank the instances not in a migration by (F, index): F as an
                    // order-preserving 64-bit key (a draining instance's F is minus
                    // infinity)
                    unsigned long long fk[IPL];
                    unsigned long long avm[IPL];
#pragma unroll
                    for (int j = 0; j < IPL; ++j) {
                        const uint32_t i = lane + 64 * j;
                        const bool av = i < I && !(C.flags[i] & kFlagBusy);
                        const double f = i < I && C.drn[i] ? -__builtin_inf() : (i < I ? C.fd[i] : 0.0);
                        const unsigned long long bits = static_cast<unsigned long long>(__double_as_longlong(f));
                        fk[j] = (bits >> 63) ? ~bits : bits | (1ull << 63);
                        avm[j] = ballot(av);
                        n2 += __popcll(avm[j]);
                    }
                    if (NW > 1) {
                        // the keys for the workgroup's count, in the freeness array
                        // (set again in phase C before its next use); an instance in
                        // a migration carries the largest key
#pragma unroll
                        for (int j = 0; j < IPL; ++j) {
                            const uint32_t i = lane + 64 * j;
                            if (i < I)
                                reinterpret_cast<unsigned long long*>(C.fd)[i] = (avm[j] >> lane) & 1ull ? fk[j] : kNone;
                        }
                    } else {
                        // L: every instance's rank, from every other lane's key
                        int rk[IPL];
#pragma unroll
                        for (int j = 0; j < IPL; ++j) rk[j] = 0;
#pragma unroll
                        for (int jj = 0; jj < IPL; ++jj) {
                            for (unsigned long long mm = avm[jj]; mm; mm &= mm - 1) {
                                const int l = ffs64(mm);
                                const unsigned long long kl = rl64(fk[jj], l);
                                const int il = 64 * jj + l;
#pragma unroll
                                for (int j = 0; j < IPL; ++j) {
                                    const int i = lane + 64 * j;
                                    rk[j] += (kl < fk[j] || (kl == fk[j] && il < i)) ? 1 : 0;
                                }
                            }
                        }
#pragma unroll
                        for (int j = 0; j < IPL; ++j)
                            if ((avm[j] >> lane) & 1ull) C.order[rk[j]] = lane + 64 * j;
                    }
                }
            }
            if (NW > 1 && lane == 0) { *C.e2go = e2 ? 1 : 0; *C.e2n2 = n2; }
            wave_sync();
            }  // wave 0
            block_sync<NW>();
            if (NW > 1 && *C.e2go) {
                // L in the eight-wave kernels: each instance's rank in (F, index)
                // order, in two steps: waves 0..3 each sort a block of 64
                // instances by counting (into the rescans' selection buffers,
                // free at this point of the tick), then every instance adds its
                // place in each block, found by bisection, summed in pend[]
                const unsigned long long* key = reinterpret_cast<const unsigned long long*>(C.fd);
                constexpr uint32_t kParts = NT / uint32_t(IM);
                const uint32_t nblk = (I + 63u) / 64u;
                ulonglong2* sblk = reinterpret_cast<ulonglong2*>(C.rsel - 64 * wid);
                for (uint32_t i = tid; i < I; i += NT) C.pend[i] = 0;
                if (uint32_t(wid) < nblk) {
                    // (entries past I and unavailable instances carry the largest key)
                    const uint32_t i = 64u * uint32_t(wid) + uint32_t(lane);
                    const unsigned long long kb = i < I ? key[i] : kNone;
                    int r0 = 0, r1 = 0, r2 = 0, r3 = 0;
                    for (int j = 0; j < 64; j += 4) {
                        const unsigned long long k0 = rl64(kb, j), k1 = rl64(kb, j + 1), k2 = rl64(kb, j + 2),
                                                 k3 = rl64(kb, j + 3);
                        r0 += int((k0 < kb) | ((k0 == kb) & (j < lane)));
                        r1 += int((k1 < kb) | ((k1 == kb) & (j + 1 < lane)));
                        r2 += int((k2 < kb) | ((k2 == kb) & (j + 2 < lane)));
                        r3 += int((k3 < kb) | ((k3 == kb) & (j + 3 < lane)));
                    }
                    sblk[64 * wid + r0 + r1 + r2 + r3] = make_ulonglong2(kb, i);
                }
                block_sync<NW>();
                {
                    const uint32_t i = tid % uint32_t(IM);
                    const uint32_t part = uint32_t(__builtin_amdgcn_readfirstlane(int(tid / uint32_t(IM))));
                    const unsigned long long ki = i < I ? key[i] : kNone;
                    if (ki != kNone) {
                        int rk = 0;
                        for (uint32_t bk = part; bk < nblk; bk += kParts) {
                            // entries of block bk below (ki, i)
                            int lo = 0, hi = 64;
                            while (lo < hi) {
                                const int mid = (lo + hi) >> 1;
                                const ulonglong2 e = sblk[64 * bk + mid];
                                if (e.x < ki || (e.x == ki && e.y < i)) lo = mid + 1;
                                else hi = mid;
                            }
                            rk += lo;
                        }
                        if (rk) atomicAdd(&C.pend[i], rk);
                    }
                }
                block_sync<NW>();
                for (uint32_t i = tid; i < I; i += NT)
                    if (key[i] != kNone) C.order[C.pend[i]] = int(i);
                block_sync<NW>();
            }
            if (wid == 0) {
                if (NW > 1) { e2 = *C.e2go != 0; n2 = *C.e2n2; }
                if (e2) {
                    const int npairs = min(int(P.mig_max_pairs), n2 / 2);
                    // Pairs (L[k], L[n2 - 1 - k]) use disjoint instances and one
                    // snapshot of F, so the stopping pair is found for all pairs at
                    // once (lane k tests pair k), the queued moves of the pairs
                    // before it run in parallel, and only the staged copies, which
                    // scan a source's slots with the whole wave, go one at a time.
                    for (int k0 = 0; k0 < npairs; k0 += 64) {
                        const int k = k0 + lane;
                        const bool in = k < npairs;
                        const int src = in ? C.order[k] : 0, dst = in ? C.order[n2 - 1 - k] : 0;
                        bool stop = false;
                        if (in) {
                            if (C.drn[dst]) {
                                // a draining destination: every instance left is draining
                                stop = true;
                            } else if (!C.drn[src]) {
                                // (a draining source is overloaded and any destination is
                                // more than theta freer)
                                const long long lhs = (long long)P.theta_den *
                                    ((long long)C.num[dst] * C.den[src] - (long long)C.num[src] * C.den[dst]);
                                const long long rhs = (long long)P.theta_num * 256 * C.den[src] * C.den[dst];
                                stop = C.num[src] >= 0 || lhs < rhs;
                            }
                        }
                        const unsigned long long sm = ballot(stop);
                        const int kstop = sm ? ffs64(sm) : 64;
                        // the destination's lowest empty slot; a full one skips its pair
                        int ds = -1;
                        if (in && lane < kstop && C.live[dst] < int(S)) {
                            for (uint32_t w = 0; w < W; ++w) {
                                const unsigned long long word = C.occ[dst * W + w];
                                if (word != kNone) { ds = int(w) * 64 + ffs64(~word); break; }
                            }
                        }
                        const bool act = ds >= 0;
                        const int h = act ? C.hols[src] : kNoHol;
                        if (act && h >= 0) {
                            // queued move of the source's head of line (fields cached in LDS)
                            const size_t dsb = size_t(dst) * S + ds, hb = size_t(src) * S + h;
                            const uint32_t hw = C.hwd[src], hm = C.hmt[src], ht = C.hta[src];
                            const unsigned long long key = C.holk[src];
                            C.slot[dsb] = make_uint4(hw, hm, uint32_t(key), ht);
                            s_word(C, hb) = 0;
                            C.occ[src * W + (h >> 6)] &= ~(1ull << (h & 63));
                            C.occ[dst * W + (ds >> 6)] |= 1ull << (ds & 63);
                            C.live[src] -= 1; C.nwait[src] -= 1;
                            C.live[dst] += 1; C.nwait[dst] += 1;
                            C.frs[src] = 0; C.frs[dst] = 0;
                            hol_insert(C, dst, key, ds, hw, hm, ht);
                            hol_pop(C, src);
                            stat(C, kMigQueued, 1);
                            if (C.ext) wlb(C)[dst] = ht < wlb(C)[dst] ? ht : wlb(C)[dst];
                        }
                        wave_sync();
                        // staged copies: running candidate of largest tier, then fewest
                        // blocks, then newest
                        for (unsigned long long pm = ballot(act && h < 0); pm; pm &= pm - 1) {
                            const int l = ffs64(pm);
                            const int psrc = rl(src, l), pdst = rl(dst, l), pds = rl(ds, l);
                            const size_t sbase = size_t(psrc) * S;
                            const int nch = live_chunks(C, psrc, lane);
                            unsigned long long bk = 0;
                            int bs = 0;
                            // GC chunks of 64 slots per memory round trip
                            constexpr int GC = IM >= 128 ? 16 : 4;
                            for (int c0 = 0; c0 < nch; c0 += GC) {
                                uint32_t v[GC], m[GC], q[GC];
#pragma unroll
                                for (int g = 0; g < GC; ++g) {
                                    const bool in = c0 + g < nch;
                                    const size_t sb = sbase + (c0 + g) * 64 + lane;
                                    const uint4 rr = in ? C.slot[sb] : make_uint4(0u, 0u, 0u, 0u);
                                    v[g] = rr.x; m[g] = rr.y; q[g] = rr.z;
                                }
#pragma unroll
                                for (int g = 0; g < GC; ++g) {
                                    if (wst(v[g]) == 2u && !(m[g] & kMigrating)) {
                                        const uint32_t fin = fin_of(v[g], t);
                                        const unsigned long long kk =
                                            ((rank_of(C, (m[g] >> 2) & 15u) + 1ull) << 48) |
                                            (static_cast<unsigned long long>(65535 - blocks_of(wlo(v[g]) - (fin - t), C.shift)) << 32) |
                                            q[g];
                                        if (kk > bk) { bk = kk; bs = (c0 + g) * 64 + lane; }
                                    }
                                }
                            }
                            const unsigned long long mx = wmax64(bk);
                            if (mx == 0) continue;  // nothing to move (an empty draining source)
                            const int cs = rl(bs, ffs64(ballot(bk == mx)));
                            if (lane == 0) {
                                const size_t dsb = size_t(pdst) * S + pds;
                                s_set_wm(C, dsb, kInbW, kInbound);
                                C.occ[pdst * W + (pds >> 6)] |= 1ull << (pds & 63);
                                C.live[pdst] += 1;
                                s_meta(C, sbase + cs) |= kMigrating;
                                int* m = &C.mig[4 * psrc];
                                m[0] = pdst; m[1] = cs; m[2] = pds; m[3] = 0;
                                stat(C, kMigStarted, 1);
                            }
                            migs = true;
                            wave_sync();
                        }
                        if (sm) break;
                    }
                }
                wave_sync();
            }
            block_sync<NW>();
        }

        // ---------------- epilogue ----------------
        const unsigned long long run_sum = wsum64(run_acc), wait_sum = wsum64(wait_acc);
        if (lane == 0) {
            stat(C, kRunSlotTicks, run_sum);
            stat(C, kWaitSlotTicks, wait_sum);
            if (wid == 0) stat(C, kTicks, nt);
        }
        block_sync<NW>();
        for (uint32_t j = tid; j < uint32_t(kNstat); j += NT) P.stats[size_t(r) * kNstat + j] = C.stats[j];
        for (uint32_t i = tid; i < I; i += NT) {
            P.freeb[size_t(r) * I + i] = C.freeb[i];
            if (C.svc) P.svc[size_t(r) * I + i] = C.svc[i];
            for (int k = 0; k < 4; ++k) P.mig[(size_t(r) * I + i) * 4 + k] = C.mig[4 * i + k];
        }
        if (tid == 0) P.next_seq[r] = next_seq;
        block_sync<NW>();
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
    for (size_t s = t0; s < nslots; s += stride) P.slot[s] = make_uint4(0u, 0u, 0u, 0u);
    for (size_t j = t0; j < size_t(P.R) * P.I; j += stride) {
        P.freeb[j] = int32_t(P.M);
        P.mig[4 * j] = -1; P.mig[4 * j + 1] = 0; P.mig[4 * j + 2] = 0; P.mig[4 * j + 3] = 0;
        P.drain[j] = 0;
    }
    for (size_t j = t0; j < size_t(P.R) * kHistPerReplica; j += stride) P.hist[j] = 0;
    for (size_t j = t0; j < size_t(P.R) * P.I; j += stride) P.svc[j] = 0;
    for (size_t j = t0; j < size_t(P.R) * kNstat; j += stride) P.stats[j] = 0;
    for (size_t j = t0; j < P.R; j += stride) { P.next_seq[j] = 0; P.digest[j] = 0; }
    if (P.hsnap)
        for (size_t j = t0; j < size_t(P.R) * 2 * kTiers; j += stride) P.hsnap[j] = 0;
}

// ---------------------------------------------------------------------------
// moving the clock by delta ticks keeps every running request's remaining
// output: its finish tick moves by the same delta
// ---------------------------------------------------------------------------
__global__ void k_shift_clock(Params P, uint32_t delta)
{
    const size_t nslots = size_t(P.R) * P.I * P.S;
    const size_t stride = size_t(gridDim.x) * blockDim.x;
    for (size_t s = size_t(blockIdx.x) * blockDim.x + threadIdx.x; s < nslots; s += stride) {
        uint32_t* w = reinterpret_cast<uint32_t*>(P.slot + s);
        const uint32_t v = *w;
        if (wst(v) == 2u) *w = (v & ~(kFin << 16)) | (((wmid(v) + delta) & kFin) << 16);
    }
}

// ---------------------------------------------------------------------------
// per-replica digest of the canonical state at tick `tick` (the next tick to
// run): wrapping sum of SplitMix64-finalised slot and instance records
// (Steele, Lea, Flood, OOPSLA 2014); one block per replica
// ---------------------------------------------------------------------------
__device__ inline unsigned long long mix64(unsigned long long z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// canonical len | rem << 16 of a slot word at tick `tick`
__device__ inline uint32_t canonical_lr(uint32_t v, uint32_t tick)
{
    if (wst(v) == 1u) return wlo(v) | (wmid(v) << 16);
    if (wst(v) == 2u) {
        const uint32_t rem = (wmid(v) - tick + 1u) & kFin;
        return (wlo(v) - rem) | (rem << 16);
    }
    return 0;
}

__global__ __launch_bounds__(256) void k_digest(Params P, uint32_t r0, uint32_t tick)
{
    __shared__ unsigned long long part[4];
    const uint32_t r = r0 + blockIdx.x;
    const size_t IS = size_t(P.I) * P.S;
    const size_t rb = size_t(r) * IS;
    const unsigned long long gm = mix64(P.id_base + r);
    unsigned long long d = 0;
    for (size_t s = threadIdx.x; s < IS; s += blockDim.x) {
        // an empty slot has a zero word; an inbound reservation's seq and
        // arrival tick are zero in the canonical state (the device leaves them)
        const uint4 rec = P.slot[rb + s];
        const uint32_t hw = rec.x;
        if (hw == 0u) continue;
        const bool inb = wst(hw) == kInbound;
        const unsigned m = rec.y;
        const unsigned long long a = static_cast<unsigned long long>(canonical_lr(hw, tick)) |
                                     (static_cast<unsigned long long>(inb ? 0u : rec.z) << 32);
        const unsigned long long b = static_cast<unsigned long long>(inb ? 0u : rec.w) |
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
        const unsigned long long f = static_cast<unsigned long long>(uint32_t(m[3])) |
                                     (static_cast<unsigned long long>(P.drain[size_t(r) * P.I + i]) << 32);
        d += mix64(p ^ c) + mix64(p ^ e) + mix64(p ^ f);
    }
    for (int o = 32; o > 0; o >>= 1) d += __shfl_xor(d, o);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = d;
    __syncthreads();
    if (threadIdx.x == 0) P.digest[r] = part[0] + part[1] + part[2] + part[3];
}

}  // namespace

size_t lds_bytes(uint32_t I, uint32_t S, uint32_t RB, uint32_t wsz, uint32_t policy, uint32_t qdepth, bool ext)
{
    return lds_layout(imax_for(I), I, S / 64, RB, wsz, policy, qdepth, ext).total;
}

int launch_init(const Params& p, hipStream_t stream)
{
    hipLaunchKernelGGL(k_init, dim3(1024), dim3(256), 0, stream, p);
    return int(hipGetLastError());
}


namespace {

template <bool INF, bool EXT>
const void* step_fn_t(uint32_t I)
{
    switch (imax_for(I)) {
    case 16: return reinterpret_cast<const void*>(&k_step<16, INF, EXT>);
    case 32: return reinterpret_cast<const void*>(&k_step<32, INF, EXT>);
    case 64: return reinterpret_cast<const void*>(&k_step<64, INF, EXT>);
    case 128: return reinterpret_cast<const void*>(&k_step<128, INF, EXT>);
    default: return reinterpret_cast<const void*>(&k_step<256, INF, EXT>);
    }
}

// the kernels with the adaptive-headroom / promotion code are separate
// instantiations, so that the others carry none of its registers
bool ext_on(const Params& p) { return p.adapt_epoch != 0 || p.promo_period != 0; }

const void* step_fn(const Params& p)
{
    if (p.policy == MTS_POLICY_INFAAS) return ext_on(p) ? step_fn_t<true, true>(p.I) : step_fn_t<true, false>(p.I);
    return ext_on(p) ? step_fn_t<false, true>(p.I) : step_fn_t<false, false>(p.I);
}

template <bool INF, bool EXT>
void launch_step_t(const Params& p, unsigned long long t0, uint32_t nt, uint32_t blocks, size_t lds, hipStream_t stream)
{
    switch (imax_for(p.I)) {
    case 16: hipLaunchKernelGGL((k_step<16, INF, EXT>), dim3(blocks), dim3(64 * waves_for(16)), lds, stream, p, t0, nt); break;
    case 32: hipLaunchKernelGGL((k_step<32, INF, EXT>), dim3(blocks), dim3(64 * waves_for(32)), lds, stream, p, t0, nt); break;
    case 64: hipLaunchKernelGGL((k_step<64, INF, EXT>), dim3(blocks), dim3(64 * waves_for(64)), lds, stream, p, t0, nt); break;
    case 128: hipLaunchKernelGGL((k_step<128, INF, EXT>), dim3(blocks), dim3(64 * waves_for(128)), lds, stream, p, t0, nt); break;
    default: hipLaunchKernelGGL((k_step<256, INF, EXT>), dim3(blocks), dim3(64 * waves_for(256)), lds, stream, p, t0, nt); break;
    }
}

size_t step_lds(const Params& p)
{
    const size_t lds = lds_bytes(p.I, p.S, p.RB, p.wsz, p.policy, p.qdepth, ext_on(p));
    if (lds > 64 * 1024) {
        // raise the dynamic LDS limit; a real failure shows up at the launch
        (void)hipFuncSetAttribute(step_fn(p), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
        (void)hipGetLastError();
    }
    return lds;
}

}  // namespace

int step_threads(const Params& p) { return 64 * waves_for(imax_for(p.I)); }

int step_blocks_per_cu(const Params& p)
{
    const size_t lds = step_lds(p);
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, step_fn(p), step_threads(p), lds) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    return nb;
}

int launch_step(const Params& p, unsigned long long t0, uint32_t nt, uint32_t blocks, hipStream_t stream)
{
    const size_t lds = step_lds(p);
    if (p.policy == MTS_POLICY_INFAAS) {
        if (ext_on(p)) launch_step_t<true, true>(p, t0, nt, blocks, lds, stream);
        else launch_step_t<true, false>(p, t0, nt, blocks, lds, stream);
    } else {
        if (ext_on(p)) launch_step_t<false, true>(p, t0, nt, blocks, lds, stream);
        else launch_step_t<false, false>(p, t0, nt, blocks, lds, stream);
    }
    return int(hipGetLastError());
}

int launch_shift_clock(const Params& p, uint32_t delta, hipStream_t stream)
{
    hipLaunchKernelGGL(k_shift_clock, dim3(1024), dim3(256), 0, stream, p, delta);
    return int(hipGetLastError());
}

int launch_digest(const Params& p, uint32_t r0, uint32_t nr, uint32_t tick, hipStream_t stream)
{
    if (nr == 0) return 0;
    hipLaunchKernelGGL(k_digest, dim3(nr), dim3(256), 0, stream, p, r0, tick);
    return int(hipGetLastError());
}

}  // namespace mts
