// Multi-tensor plans: the same steps over a model held as separate tensors,
// described by a device table (layout in cpdp_launch.h), with the scalars
// passed by value; plan initialisation.
#include "cpdp_plan_impl.h"

namespace cpdp {
namespace {

// ---- plan initialisation: every replica <- the reference model ----------------

template <class PS, bool FULL>
__device__ __forceinline__ void init_plan_chunk(const float* anchor, typename PS::T* params,
                                                float* mom, float* mom2, float* slow, int n) {
    float a[kVec];
    const float zero[kVec] = {0.0f, 0.0f, 0.0f, 0.0f};
    load_f32<FULL, false>(anchor, n, a);
    PS::template store<FULL, kNTS>(params, n, a);
    store_f32<FULL, kNTS>(mom, n, zero);
    if (mom2 != nullptr) store_f32<FULL, kNTS>(mom2, n, zero);
    if (slow != nullptr) store_f32<FULL, kNTS>(slow, n, zero);
}

template <class PS>
__global__ __launch_bounds__(kBlock) void state_init_plan_kernel(const int64_t* __restrict__ plan,
                                                                 int W, int n,
                                                                 int64_t total_chunks) {
    const PlanView v = plan_view(plan, W, n);
    const int64_t row = blockIdx.x / total_chunks;
    const int64_t b = blockIdx.x - row * total_chunks;
    const int64_t t = plan_tensor(v, n, b);
    const int64_t P = v.numel[t];
    const int64_t p0 = ((b - v.chunk_start[t]) * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    const int64_t k = row * n + t;
    auto at = [&](int64_t addr) { return reinterpret_cast<float*>(addr) + p0; };
    const float* anchor = at(v.anchor[t]);
    auto* params = reinterpret_cast<typename PS::T*>(v.params[k]) + p0;
    float* mom2 = v.mom2[k] != 0 ? at(v.mom2[k]) : nullptr;
    float* slow = row == 0 && v.slow[t] != 0 ? at(v.slow[t]) : nullptr;
    if (p0 + kVec <= P)
        init_plan_chunk<PS, true>(anchor, params, at(v.mom[k]), mom2, slow, kVec);
    else
        init_plan_chunk<PS, false>(anchor, params, at(v.mom[k]), mom2, slow, (int)(P - p0));
}

}  // namespace

int launch_state_init_plan(Param pt, const int64_t* plan, int W, int n, int64_t total_chunks,
                           void* stream) {
    const int64_t blocks = total_chunks * W;
    return pt == Param::BF16
               ? launch(state_init_plan_kernel<ParamBF16>, blocks, stream, plan, W, n, total_chunks)
               : launch(state_init_plan_kernel<ParamF32>, blocks, stream, plan, W, n, total_chunks);
}

int launch_local_step_plan(Opt opt, const OptParams& o, Param pt, const int64_t* plan, int W,
                           int n, int64_t total_chunks, void* stream) {
    return local_plan_any(opt, pt, DirectScalars{o, 0.0f, 0.0f}, plan, W, n, total_chunks,
                          stream);
}

int launch_sync_plan(Sync mode, Opt opt, const OptParams& o, Param pt, const int64_t* plan, int W,
                     int n, int64_t total_chunks, float beta, float alpha, unsigned flags,
                     void* stream) {
    return sync_plan_any(mode, opt, pt, DirectScalars{o, beta, alpha * o.lr}, plan, W, n,
                         total_chunks, flags, stream);
}

int64_t coords_per_block() { return (int64_t)kBlock * kVec; }

int upload_plan(void* dev, const int64_t* host, int64_t words) {
    return (int)hipMemcpy(dev, host, (size_t)words * sizeof(int64_t), hipMemcpyHostToDevice);
}

}  // namespace cpdp
