// Multi-tensor plans with the scalars of each step read from a device step
// table (graph replay of schedules over a model held as separate tensors).
#include "cpdp_plan_impl.h"

namespace cpdp {

int launch_local_step_plan_table(Opt opt, Param pt, const int64_t* plan, int W, int n,
                                 int64_t total_chunks, const int64_t* table, void* stream) {
    return local_plan_any(opt, pt, TableScalars{table}, plan, W, n, total_chunks, stream);
}

int launch_sync_plan_table(Sync mode, Opt opt, Param pt, const int64_t* plan, int W, int n,
                           int64_t total_chunks, const int64_t* table, unsigned flags,
                           void* stream) {
    return sync_plan_any(mode, opt, pt, TableScalars{table}, plan, W, n, total_chunks, flags,
                         stream);
}

}  // namespace cpdp
