// Flat-layout synchronisation kernels of one strategy (CPDP).
#include "cpdp_sync_impl.h"

namespace cpdp {

template int launch_sync_mode<Sync::CPDP>(Opt, const OptParams&, Param, Grad, Mom, void*,
                                              void*, float*, const void*, float*, float*, int,
                                              int64_t, int64_t, float, float, unsigned,
                                              void*);

}  // namespace cpdp
