// Wave-level helpers shared by the device sources of libmts (one wave of 64
// lanes; gfx950).
#pragma once

#include <hip/hip_runtime.h>

namespace mts {
namespace wave {

__device__ __forceinline__ int lane_id() { return __lane_id(); }
__device__ __forceinline__ unsigned long long ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ unsigned long long lanemask_lt() { return (1ull << lane_id()) - 1ull; }
__device__ __forceinline__ int ffs64(unsigned long long m) { return __ffsll(static_cast<long long>(m)) - 1; }

__device__ __forceinline__ int rl(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ unsigned rlu(unsigned v, int l) { return unsigned(__builtin_amdgcn_readlane(int(v), l)); }
__device__ __forceinline__ unsigned long long rl64(unsigned long long v, int l)
{
    const unsigned lo = rlu(unsigned(v), l), hi = rlu(unsigned(v >> 32), l);
    return (static_cast<unsigned long long>(hi) << 32) | lo;
}

// A wave-uniform pointer made opaque to the optimiser (its two halves go
// through readfirstlane): addresses built on it stay a scalar base plus a
// lane offset instead of becoming 64-bit per-lane induction variables
template <typename T>
__device__ __forceinline__ T* uniform_ptr(T* p)
{
    const unsigned long long v = reinterpret_cast<unsigned long long>(p);
    const unsigned lo = unsigned(__builtin_amdgcn_readfirstlane(int(unsigned(v))));
    const unsigned hi = unsigned(__builtin_amdgcn_readfirstlane(int(unsigned(v >> 32))));
    return reinterpret_cast<T*>((static_cast<unsigned long long>(hi) << 32) | lo);
}

// Lanes of the wave exchange values through LDS and HBM: every write by a
// subset of lanes that other lanes read later is followed by this point, so
// that no later load is moved above it and every later load sees the write.
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    __builtin_amdgcn_wave_barrier();
}

}  // namespace wave
}  // namespace mts
