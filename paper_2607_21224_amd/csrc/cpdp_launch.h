// Internal interface between the C ABI (cpdp_api.cpp: validation, dispatch)
// and the gfx950 kernels (cpdp_kernels.hip).  Plain C++ types only, so the
// validation layer builds with any host compiler.  Every launcher assumes its
// arguments were validated (P > 0, aligned, non-overlapping) and returns 0 on
// success or the HIP error code of a failed launch.
#pragma once
#include <stdint.h>

namespace cpdp {

enum class Param { F32, BF16 };

int launch_state_init(Param pt, const void* theta0, void* params, float* mom,
                      float* slow, float* anchor, int W, int64_t P, int64_t ld,
                      void* stream);

int launch_local_step(Param pt, void* params, float* mom, const float* grads,
                      int W, int64_t P, int64_t ld, float lr, float mu,
                      void* stream);

// Synchronisation step of one of the three strategies (CPDP reconcile,
// LocalSGD averaging, DDP gradient step).  slow/anchor are read and written
// by CPDP; LocalSGD writes anchor only when it is not NULL; DDP uses neither.
enum class Sync { CPDP, LocalSGD, DDP };

int launch_sync(Sync mode, Param pt, void* params, float* mom,
                const float* grads, float* slow, float* anchor, int W,
                int64_t P, int64_t ld, float lr, float mu, float beta,
                float alpha, void* stream);

// True when a launch over P coordinates (rows = W for the row-parallel local
// step, 1 otherwise) fits in one grid.
bool grid_fits(int rows, int64_t P);

const char* hip_error_string(int err);

}  // namespace cpdp
