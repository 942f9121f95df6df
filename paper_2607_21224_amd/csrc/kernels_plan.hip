// Multi-tensor plans: the same steps over a model held as separate tensors,
// described by a device table (layout in cpdp_launch.h).
#include "cpdp_device.h"

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

// multi-tensor plan: block (row, chunk b) -> replica row, tensor t, its chunk
template <Opt O, class PS>
__global__ __launch_bounds__(kBlock) void local_step_plan_kernel(OptParams o,
                                                                 const int64_t* __restrict__ plan,
                                                                 int W, int n,
                                                                 int64_t total_chunks) {
    const PlanView v = plan_view(plan, W, n);
    const int64_t row = blockIdx.x / total_chunks;
    const int64_t b = blockIdx.x - row * total_chunks;
    const int64_t t = plan_tensor(v, n, b);
    const int64_t P = v.numel[t];
    const int64_t p0 = ((b - v.chunk_start[t]) * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    const Table<PS> r{v.params, v.mom, v.mom2, v.grads, n, t};
    const int i = (int)row;
    local_dispatch<O, PS>(o, r.prm(i), r.m(i), O == Opt::ADAMW ? r.v(i) : nullptr, r.g(i), p0, P);
}

// multi-tensor plan: block b -> tensor t and its chunk; run-time W
template <Sync M, Opt O, class PS, bool EXTRA>
__global__ __launch_bounds__(kBlock) void sync_plan_kernel(OptParams o,
                                                           const int64_t* __restrict__ plan, int W,
                                                           int n, float beta, float alpha_lr,
                                                           float inv_w, unsigned flags) {
    const PlanView v = plan_view(plan, W, n);
    const int64_t b = blockIdx.x;
    const int64_t t = plan_tensor(v, n, b);
    const int64_t P = v.numel[t];
    const int64_t p0 = ((b - v.chunk_start[t]) * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    const Table<PS> r{v.params, v.mom, v.mom2, v.grads, n, t};
    float* slow = reinterpret_cast<float*>(v.slow[t]);
    float* anchor = reinterpret_cast<float*>(v.anchor[t]);
    if (p0 + kVec <= P)
        sync_chunk<M, O, 0, PS, true, EXTRA>(o, r, slow, anchor, W, p0, kVec, beta, alpha_lr,
                                             inv_w, flags);
    else
        sync_chunk<M, O, 0, PS, false, EXTRA>(o, r, slow, anchor, W, p0, (int)(P - p0), beta,
                                              alpha_lr, inv_w, flags);
}

template <Opt O>
int local_plan_o(Param pt, const OptParams& o, const int64_t* plan, int W, int n,
                 int64_t total_chunks, void* stream) {
    const int64_t blocks = total_chunks * W;
    return pt == Param::BF16 ? launch(local_step_plan_kernel<O, ParamBF16>, blocks, stream, o, plan,
                                      W, n, total_chunks)
                             : launch(local_step_plan_kernel<O, ParamF32>, blocks, stream, o, plan,
                                      W, n, total_chunks);
}

template <Sync M, Opt O, class PS>
int sync_plan_t(const OptParams& o, const int64_t* plan, int W, int n, int64_t total_chunks,
                float beta, float alpha, unsigned flags, void* stream) {
    const float alpha_lr = alpha * o.lr;
    const float inv_w = 1.0f / (float)W;
    if (flags != 0)
        return launch(sync_plan_kernel<M, O, PS, true>, total_chunks, stream, o, plan, W, n, beta,
                      alpha_lr, inv_w, flags);
    return launch(sync_plan_kernel<M, O, PS, false>, total_chunks, stream, o, plan, W, n, beta,
                  alpha_lr, inv_w, flags);
}

template <Sync M, Opt O>
int sync_plan_p(Param pt, const OptParams& o, const int64_t* plan, int W, int n,
                int64_t total_chunks, float beta, float alpha, unsigned flags, void* stream) {
    return pt == Param::BF16
               ? sync_plan_t<M, O, ParamBF16>(o, plan, W, n, total_chunks, beta, alpha, flags,
                                              stream)
               : sync_plan_t<M, O, ParamF32>(o, plan, W, n, total_chunks, beta, alpha, flags,
                                             stream);
}

template <Sync M>
int sync_plan_o(Opt opt, Param pt, const OptParams& o, const int64_t* plan, int W, int n,
                int64_t total_chunks, float beta, float alpha, unsigned flags, void* stream) {
    switch (opt) {
        case Opt::SGD_WD:
            return sync_plan_p<M, Opt::SGD_WD>(pt, o, plan, W, n, total_chunks, beta, alpha,
                                               flags, stream);
        case Opt::ADAMW:
            return sync_plan_p<M, Opt::ADAMW>(pt, o, plan, W, n, total_chunks, beta, alpha, flags,
                                              stream);
        default:
            return sync_plan_p<M, Opt::SGD>(pt, o, plan, W, n, total_chunks, beta, alpha, flags,
                                            stream);
    }
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
    switch (opt) {
        case Opt::SGD_WD: return local_plan_o<Opt::SGD_WD>(pt, o, plan, W, n, total_chunks, stream);
        case Opt::ADAMW: return local_plan_o<Opt::ADAMW>(pt, o, plan, W, n, total_chunks, stream);
        default: return local_plan_o<Opt::SGD>(pt, o, plan, W, n, total_chunks, stream);
    }
}

int launch_sync_plan(Sync mode, Opt opt, const OptParams& o, Param pt, const int64_t* plan, int W,
                     int n, int64_t total_chunks, float beta, float alpha, unsigned flags,
                     void* stream) {
    switch (mode) {
        case Sync::LocalSGD:
            return sync_plan_o<Sync::LocalSGD>(opt, pt, o, plan, W, n, total_chunks, beta, alpha,
                                               flags, stream);
        case Sync::DDP:
            return sync_plan_o<Sync::DDP>(opt, pt, o, plan, W, n, total_chunks, beta, alpha, flags,
                                          stream);
        default:
            return sync_plan_o<Sync::CPDP>(opt, pt, o, plan, W, n, total_chunks, beta, alpha,
                                           flags, stream);
    }
}

int64_t coords_per_block() { return (int64_t)kBlock * kVec; }

int upload_plan(void* dev, const int64_t* host, int64_t words) {
    return (int)hipMemcpy(dev, host, (size_t)words * sizeof(int64_t), hipMemcpyHostToDevice);
}

}  // namespace cpdp
