// The static plan table of cpdp_plan_build_static: a file-scope device array,
// one copy per GPU, and the per-device lookup of its address.  No kernel
// lives here; the plan kernels get the address as their table argument, the
// same way they get a table the caller allocated.
#include <hip/hip_runtime.h>

#include <mutex>

#include "plan_scratch.h"

namespace cpdp {
namespace {

constexpr int kMaxDevices = 64;

// In host code this name is a host-side stand-in for the symbol, not device
// memory: host code uses only the address plan_scratch() resolves for the
// current device.
static __device__ __align__(256) int64_t scratch[kPlanScratchWords];

std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

}  // namespace

int plan_scratch(void** ptr) {
    int d = 0;
    hipError_t e = hipGetDevice(&d);
    if (e != hipSuccess) return (int)e;
    if (d < 0 || d >= kMaxDevices) return -1;
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_addr[d] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return (int)e;
        if (p == nullptr) return -1;
        g_addr[d] = p;
    }
    *ptr = g_addr[d];
    return 0;
}

int plan_scratch_device(const void* table) {
    if (table == nullptr) return -1;
    std::lock_guard<std::mutex> lock(g_mu);
    for (int d = 0; d < kMaxDevices; ++d)
        if (g_addr[d] == table) return d;
    return -1;
}

}  // namespace cpdp
