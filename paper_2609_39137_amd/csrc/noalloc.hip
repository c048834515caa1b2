// Fixed device scratch for idb_router_step_noalloc: the router step's
// workspace (slice candidates and the merge's ticket) in a file-scope device
// array instead of caller memory, for callers that cannot allocate.
//
// Each device that loads the library holds its own copy of the array, at its
// own address, until the process ends.  Host code never passes the array's
// name to a kernel (in host code it is only a stand-in for the symbol): the
// device address comes from hipGetSymbolAddress, taken once per device with
// that device current, and is kept per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "idb.h"
#include "internal.h"

namespace idb {

namespace {

constexpr size_t kScratchBytes = IDB_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "whole 256-byte units");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

size_t noalloc_scratch_bytes() { return kScratchBytes; }

hipError_t noalloc_scratch(int device, void** out) {
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[device]) {
        // the caller made `device` current
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_ptr[device] = p;
    }
    *out = g_ptr[device];
    return hipSuccess;
}

}  // namespace idb
