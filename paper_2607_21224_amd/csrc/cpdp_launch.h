// Internal interface between the C ABI (cpdp_api.cpp: validation, dispatch)
// and the gfx950 kernels (kernels_*.hip).  Plain C++ types only, so the
// validation layer builds with any host compiler.  Every launcher assumes its
// arguments were validated (P > 0, aligned, non-overlapping) and returns 0 on
// success or the HIP error code of a failed launch.
#pragma once
#include <stdint.h>

namespace cpdp {

enum class Param { F32, BF16 };

// Gradient and momentum storage of the flat local and synchronisation steps:
// fp32, or bf16 (momentum SGD without variants only; the general optimizers,
// plans and step tables take fp32).
enum class Grad { F32, BF16 };
enum class Mom { F32, BF16 };

// The per-replica optimizer update: momentum SGD, SGD with coupled weight
// decay, or AdamW.
enum class Opt { SGD, SGD_WD, ADAMW };

// Scalars of one optimizer update, in the fp32 form the kernels use.  The
// AdamW entries that depend on the step count t are folded on the host.
struct OptParams {
    float lr;            // learning rate
    float mu;            // SGD momentum, or AdamW beta1
    float wd;            // SGD coupled weight decay
    float omb1;          // AdamW: 1 - beta1
    float beta2;         // AdamW
    float omb2;          // AdamW: 1 - beta2
    float eps;           // AdamW
    float step_size;     // AdamW: lr / (1 - beta1^t)
    float sqrt_bc2;      // AdamW: sqrt(1 - beta2^t)
    float decay;         // AdamW: 1 - lr * weight_decay
};

// Synchronisation step of one of the three strategies (CPDP reconcile,
// LocalSGD averaging, DDP gradient step).  slow/anchor are read and written
// by CPDP; LocalSGD writes anchor only when it is not NULL; DDP uses neither.
// mom2 (AdamW second moments) is used by Opt::ADAMW only.
enum class Sync { CPDP, LocalSGD, DDP };

// Optional variants of a synchronisation step (bit flags): write the gradient
// mean back into every gradient row; average the optimizer state over the
// replicas after the step.
constexpr unsigned kSyncWriteGbar = 1u;
constexpr unsigned kSyncAverageState = 2u;

int launch_state_init(Param pt, Mom mt, const void* theta0, void* params, void* mom,
                      float* mom2, float* slow, float* anchor, int W, int64_t P,
                      int64_t ld, void* stream);

int launch_local_step(Opt opt, const OptParams& o, Param pt, Grad gt, Mom mt, void* params,
                      void* mom, float* mom2, const void* grads, int W,
                      int64_t P, int64_t ld, void* stream);

int launch_sync(Sync mode, Opt opt, const OptParams& o, Param pt, Grad gt, Mom mt,
                void* params, void* mom, float* mom2, const void* grads, float* slow,
                float* anchor, int W, int64_t P, int64_t ld, float beta,
                float alpha, unsigned flags, void* stream);

// launch_sync for one strategy; each is instantiated in its own translation
// unit (kernels_sync_<strategy>.hip).
template <Sync M>
int launch_sync_mode(Opt opt, const OptParams& o, Param pt, Grad gt, Mom mt, void* params,
                     void* mom, float* mom2, const void* grads, float* slow, float* anchor,
                     int W, int64_t P, int64_t ld, float beta, float alpha, unsigned flags,
                     void* stream);

// Multi-tensor plan table in device memory, as 64-bit words:
//   [0] W  [1] n  [2] total chunks  [3] reserved
//   chunk_start[n + 1]   first chunk of every tensor (chunk = coords_per_block())
//   numel[n]
//   params[W*n], mom[W*n], mom2[W*n], grads[W*n]   device addresses, [i*n + t]
//   slow[n], anchor[n]                              device addresses (0 = none)
constexpr int64_t kPlanHeaderWords = 4;
inline int64_t plan_words(int W, int n) {
    return kPlanHeaderWords + (int64_t)(n + 1) + n + 4 * (int64_t)W * n + 2 * (int64_t)n;
}

int launch_state_init_plan(Param pt, const int64_t* plan, int W, int n,
                           int64_t total_chunks, void* stream);

int launch_local_step_plan(Opt opt, const OptParams& o, Param pt, const int64_t* plan,
                           int W, int n, int64_t total_chunks, void* stream);

int launch_sync_plan(Sync mode, Opt opt, const OptParams& o, Param pt,
                     const int64_t* plan, int W, int n, int64_t total_chunks,
                     float beta, float alpha, unsigned flags, void* stream);

// Step table in device memory: per-step scalars the table kernels read at
// run time, so a captured graph can replay steps whose scalars differ (AdamW
// bias correction, a learning-rate schedule).
//   words [0] position (index of the entry the next step uses)  [1] n_steps
//   then n_steps StepEntry records
// A table kernel whose position is outside [0, n_steps) returns without
// touching anything; the advance kernel stops at n_steps.
struct StepEntry {
    OptParams o;         // the update's scalars, folded as for a direct call
    float beta;          // SlowMo beta (CPDP steps)
    float alpha_lr;      // alpha * lr, the SlowMo step length
    float reserved[4];
};
static_assert(sizeof(StepEntry) == 64, "step table entries are 64 bytes");
constexpr int64_t kStepTableHeaderWords = 2;
inline int64_t step_table_bytes(int n_steps) {
    return kStepTableHeaderWords * (int64_t)sizeof(int64_t) +
           (int64_t)n_steps * (int64_t)sizeof(StepEntry);
}

int launch_local_step_table(Opt opt, Param pt, const int64_t* table, void* params, float* mom,
                            float* mom2, const float* grads, int W, int64_t P, int64_t ld,
                            void* stream);

int launch_sync_table(Sync mode, Opt opt, Param pt, const int64_t* table, void* params,
                      float* mom, float* mom2, const float* grads, float* slow, float* anchor,
                      int W, int64_t P, int64_t ld, unsigned flags, void* stream);

// Plan steps with the scalars of a step table's current entry.
int launch_local_step_plan_table(Opt opt, Param pt, const int64_t* plan, int W, int n,
                                 int64_t total_chunks, const int64_t* table, void* stream);
int launch_sync_plan_table(Sync mode, Opt opt, Param pt, const int64_t* plan, int W, int n,
                           int64_t total_chunks, const int64_t* table, unsigned flags,
                           void* stream);

// One-thread kernels on the table's position word (graph-capturable: no
// memset, no copy).
int launch_step_table_set(int64_t* table, int64_t position, void* stream);
int launch_step_table_advance(int64_t* table, void* stream);

// Synchronous device-to-host read of a table's position word.
int read_step_table_position(const int64_t* table, int64_t* position);

// Synchronous host-to-device copy of a filled step table.
int upload_bytes(void* dev, const void* host, int64_t bytes);

// Zero *count, then add the number of coordinates p < P at which some
// replica's stored parameter differs bitwise from the anchor rounded to the
// parameter storage type.
int launch_count_unsynced(Param pt, const void* params, const float* anchor, int W, int64_t P,
                          int64_t ld, uint64_t* count, void* stream);

// Coordinates one block of the flat and plan kernels covers.
int64_t coords_per_block();

// Synchronous host-to-device copy of a plan table; returns the HIP status.
int upload_plan(void* dev, const int64_t* host, int64_t words);

// Most blocks a launch may cover (a grid holds at most 2^31 - 1).
constexpr int64_t kMaxBlocks = 0x7FFFFFFF - 8;

// True when a launch over P coordinates (rows = W for the row-parallel local
// step, 1 otherwise) fits in one grid.
bool grid_fits(int rows, int64_t P);

const char* hip_error_string(int err);

}  // namespace cpdp
