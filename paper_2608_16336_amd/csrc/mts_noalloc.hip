// Static device scratch of mts_step_noalloc: the arrival staging (per-tick
// counts and tier-sorted records of a chunk of ticks) lives in a file-scope
// device array instead of the caller's buffer, so that stepping allocates
// nothing.  Each GPU holds its own copy of the array, whose device address
// is looked up once per device by scratch_setup (called from mts_create with
// that device current) and kept here; host code never passes the array's
// name to a kernel or a copy, only that address.
#include <hip/hip_runtime.h>

#include <mutex>

#include "mts_internal.h"

namespace mts {
namespace {

constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

std::mutex g_mu;
char* g_ptr[kMaxDevices];  // device address of `scratch` on each device (null: not looked up)

}  // namespace

int scratch_setup(int device)
{
    if (device < 0 || device >= kMaxDevices) return MTS_EDEVICE;
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_ptr[device]) return MTS_OK;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
        (void)hipGetLastError();
        return MTS_EDEVICE;
    }
    g_ptr[device] = static_cast<char*>(p);
    return MTS_OK;
}

char* scratch_ptr(int device)
{
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_mu);
    return g_ptr[device];
}

}  // namespace mts
