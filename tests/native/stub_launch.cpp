// Host-only stand-ins for the gfx950 launchers, so the C-ABI validation layer
// (cpdp_api.cpp) can be built with g++ under AddressSanitizer/UBSan on a
// machine without a GPU.  Every launcher records that it was reached.
#include "cpdp_launch.h"
#include "plan_scratch.h"

int g_launches = 0;

namespace cpdp {
int launch_state_init(Param, Mom, const void*, void*, void*, float*, float*, float*, int, int64_t,
                      int64_t, void*) {
    return ++g_launches, 0;
}
int launch_local_step(Opt, const OptParams&, Param, Grad, Mom, void*, void*, float*, const void*, int,
                      int64_t, int64_t, void*) {
    return ++g_launches, 0;
}
int launch_sync(Sync, Opt, const OptParams&, Param, Grad, Mom, void*, void*, float*, const void*,
                float*, float*, int, int64_t, int64_t, float, float, unsigned, void*) {
    return ++g_launches, 0;
}
int launch_state_init_plan(Param, const int64_t*, int, int, int64_t, void*) {
    return ++g_launches, 0;
}
int launch_local_step_plan(Opt, const OptParams&, Param, const int64_t*, int, int, int64_t,
                           void*) {
    return ++g_launches, 0;
}
int launch_sync_plan(Sync, Opt, const OptParams&, Param, const int64_t*, int, int, int64_t, float,
                     float, unsigned, void*) {
    return ++g_launches, 0;
}
int launch_local_step_table(Opt, Param, const int64_t*, void*, float*, float*, const float*, int,
                            int64_t, int64_t, void*) {
    return ++g_launches, 0;
}
int launch_sync_table(Sync, Opt, Param, const int64_t*, void*, float*, float*, const float*,
                      float*, float*, int, int64_t, int64_t, unsigned, void*) {
    return ++g_launches, 0;
}
int launch_local_step_plan_table(Opt, Param, const int64_t*, int, int, int64_t, const int64_t*,
                                 void*) {
    return ++g_launches, 0;
}
int launch_sync_plan_table(Sync, Opt, Param, const int64_t*, int, int, int64_t, const int64_t*,
                           unsigned, void*) {
    return ++g_launches, 0;
}
int launch_step_table_set(int64_t*, int64_t, void*) { return ++g_launches, 0; }
int launch_step_table_advance(int64_t*, void*) { return ++g_launches, 0; }
int read_step_table_position(const int64_t*, int64_t* position) { return *position = 0, 0; }
int64_t g_uploaded_bytes = 0;
int upload_bytes(void*, const void*, int64_t bytes) { return g_uploaded_bytes = bytes, 0; }
int launch_count_unsynced(Param, const void*, const float*, int, int64_t, int64_t, uint64_t*,
                          void*) {
    return ++g_launches, 0;
}
int64_t coords_per_block() { return 1024; }
int g_uploaded_words = 0;
int upload_plan(void*, const int64_t*, int64_t words) { return g_uploaded_words = (int)words, 0; }
bool grid_fits(int rows, int64_t P) { return rows >= 1 && (P + 1023) / 1024 <= kMaxBlocks / rows; }
const char* hip_error_string(int) { return "stub"; }
// a host array stands in for the device's static plan table
alignas(256) int64_t g_plan_scratch[kPlanScratchWords];
int plan_scratch(void** ptr) { return *ptr = g_plan_scratch, 0; }
int plan_scratch_device(const void* table) { return table == g_plan_scratch ? 0 : -1; }
}  // namespace cpdp
