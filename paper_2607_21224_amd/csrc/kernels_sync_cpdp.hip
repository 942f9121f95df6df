// Flat-layout synchronisation kernels of one strategy (CPDP).
#include "cpdp_sync_impl.h"

namespace cpdp {

template int launch_sync_mode<Sync::CPDP>(Opt, const OptParams&, Param, void*, float*,
                                              float*, const float*, float*, float*, int,
                                              int64_t, int64_t, float, float, unsigned,
                                              void*);

}  // namespace cpdp
