// Device memory the library itself owns: one fixed plan table per GPU, for
// cpdp_plan_build_static (plans built by callers that cannot allocate).
// Plain C++ declarations, so the host validation layer builds with any host
// compiler; the array and the code that resolves its address live in
// plan_scratch.hip.
#pragma once
#include <stdint.h>

namespace cpdp {

// 64-bit words of the static plan table (256 KiB per GPU, kept until the
// process ends).
constexpr int64_t kPlanScratchWords = 32768;

// Device address of the current device's static table in *ptr (resolved
// with hipGetSymbolAddress the first time a device asks, then cached per
// device).  Returns 0, or the HIP error of hipGetDevice / hipGetSymbolAddress
// (-1 for a device ordinal beyond the cache).
int plan_scratch(void** ptr);

// Ordinal of the device whose static table sits at `table`, or -1 when
// `table` is no device's static table (or that device's address was never
// resolved).
int plan_scratch_device(const void* table);

}  // namespace cpdp
