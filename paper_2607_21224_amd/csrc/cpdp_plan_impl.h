// Multi-tensor plan kernels of the local and synchronisation steps and their
// dispatch, generic over where a step's scalars come from (DirectScalars:
// launch arguments; TableScalars: a device step table).  kernels_plan.hip
// and kernels_plan_table.hip instantiate one source each.
#pragma once

#include "cpdp_device.h"

namespace cpdp {
namespace {

// cell (row, chunk b), in the local step's block order -> replica row, tensor t,
// its chunk
template <Opt O, class PS, class Src>
__global__ __launch_bounds__(kBlock) void local_step_plan_kernel(Src src,
                                                                 const int64_t* __restrict__ plan,
                                                                 int W, int n,
                                                                 int64_t total_chunks) {
    const int64_t cell = local_cell(total_chunks * W);
    if (cell < 0) return;
    const PlanView v = plan_view(plan, W, n);
    const int64_t row = cell / total_chunks;
    const int64_t b = cell - row * total_chunks;
    const int64_t t = plan_tensor(v, n, b);
    const int64_t P = v.numel[t];
    const int64_t p0 = ((b - v.chunk_start[t]) * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    StepEntry e;
    if (!src.get(e)) return;
    const Table<PS> r{v.params, v.mom, v.mom2, v.grads, n, t};
    const int i = (int)row;
    local_dispatch<O, PS>(e.o, r.prm(i), r.m(i), O == Opt::ADAMW ? r.v(i) : nullptr, r.g(i), p0,
                          P);
}

// block b -> tensor t and its chunk; run-time W
template <Sync M, Opt O, class PS, bool EXTRA, class Src>
__global__ __launch_bounds__(kBlock) void sync_plan_kernel(Src src,
                                                           const int64_t* __restrict__ plan, int W,
                                                           int n, float inv_w, unsigned flags) {
    const PlanView v = plan_view(plan, W, n);
    const int64_t b = blockIdx.x;
    const int64_t t = plan_tensor(v, n, b);
    const int64_t P = v.numel[t];
    const int64_t p0 = ((b - v.chunk_start[t]) * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    StepEntry e;
    if (!src.get(e)) return;
    const Table<PS> r{v.params, v.mom, v.mom2, v.grads, n, t};
    float* slow = reinterpret_cast<float*>(v.slow[t]);
    float* anchor = reinterpret_cast<float*>(v.anchor[t]);
    if (p0 + kVec <= P)
        sync_chunk<M, O, 0, PS, true, EXTRA>(e.o, r, slow, anchor, W, p0, kVec, e.beta,
                                             e.alpha_lr, inv_w, flags);
    else
        sync_chunk<M, O, 0, PS, false, EXTRA>(e.o, r, slow, anchor, W, p0, (int)(P - p0),
                                              e.beta, e.alpha_lr, inv_w, flags);
}

template <Opt O, class Src>
int local_plan_o(Param pt, Src src, const int64_t* plan, int W, int n, int64_t total_chunks,
                 void* stream) {
    const int64_t blocks = local_grid(total_chunks * W);
    return pt == Param::BF16 ? launch(local_step_plan_kernel<O, ParamBF16, Src>, blocks, stream,
                                      src, plan, W, n, total_chunks)
                             : launch(local_step_plan_kernel<O, ParamF32, Src>, blocks, stream,
                                      src, plan, W, n, total_chunks);
}

template <class Src>
int local_plan_any(Opt opt, Param pt, Src src, const int64_t* plan, int W, int n,
                   int64_t total_chunks, void* stream) {
    switch (opt) {
        case Opt::SGD_WD: return local_plan_o<Opt::SGD_WD>(pt, src, plan, W, n, total_chunks, stream);
        case Opt::ADAMW: return local_plan_o<Opt::ADAMW>(pt, src, plan, W, n, total_chunks, stream);
        default: return local_plan_o<Opt::SGD>(pt, src, plan, W, n, total_chunks, stream);
    }
}

template <Sync M, Opt O, class PS, class Src>
int sync_plan_t(Src src, const int64_t* plan, int W, int n, int64_t total_chunks,
                unsigned flags, void* stream) {
    const float inv_w = 1.0f / (float)W;
    if (flags != 0)
        return launch(sync_plan_kernel<M, O, PS, true, Src>, total_chunks, stream, src, plan, W,
                      n, inv_w, flags);
    return launch(sync_plan_kernel<M, O, PS, false, Src>, total_chunks, stream, src, plan, W, n,
                  inv_w, flags);
}

template <Sync M, Opt O, class Src>
int sync_plan_p(Param pt, Src src, const int64_t* plan, int W, int n, int64_t total_chunks,
                unsigned flags, void* stream) {
    return pt == Param::BF16
               ? sync_plan_t<M, O, ParamBF16>(src, plan, W, n, total_chunks, flags, stream)
               : sync_plan_t<M, O, ParamF32>(src, plan, W, n, total_chunks, flags, stream);
}

template <Sync M, class Src>
int sync_plan_o(Opt opt, Param pt, Src src, const int64_t* plan, int W, int n,
                int64_t total_chunks, unsigned flags, void* stream) {
    switch (opt) {
        case Opt::SGD_WD:
            return sync_plan_p<M, Opt::SGD_WD>(pt, src, plan, W, n, total_chunks, flags, stream);
        case Opt::ADAMW:
            return sync_plan_p<M, Opt::ADAMW>(pt, src, plan, W, n, total_chunks, flags, stream);
        default:
            return sync_plan_p<M, Opt::SGD>(pt, src, plan, W, n, total_chunks, flags, stream);
    }
}

template <class Src>
int sync_plan_any(Sync mode, Opt opt, Param pt, Src src, const int64_t* plan, int W, int n,
                  int64_t total_chunks, unsigned flags, void* stream) {
    switch (mode) {
        case Sync::LocalSGD:
            return sync_plan_o<Sync::LocalSGD>(opt, pt, src, plan, W, n, total_chunks, flags,
                                               stream);
        case Sync::DDP:
            return sync_plan_o<Sync::DDP>(opt, pt, src, plan, W, n, total_chunks, flags, stream);
        default:
            return sync_plan_o<Sync::CPDP>(opt, pt, src, plan, W, n, total_chunks, flags, stream);
    }
}

}  // namespace
}  // namespace cpdp
