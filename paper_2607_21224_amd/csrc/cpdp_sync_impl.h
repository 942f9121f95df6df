// The flat-layout synchronisation kernels (CPDP reconcile, LocalSGD averaging,
// DDP gradient step) and their dispatch over update rule, parameter,
// gradient and momentum storage types, and W.  Each strategy is instantiated in a translation unit of its own
// (kernels_sync_<strategy>.hip) so the three compile in parallel.
#pragma once

#include "cpdp_device.h"

namespace cpdp {
namespace {

template <Sync M, Opt O, int WT, class PS, bool EXTRA, class GS, class MS>
__global__ __launch_bounds__(kBlock) void sync_kernel(
    OptParams o, typename PS::T* __restrict__ params, typename MS::T* __restrict__ mom,
    float* __restrict__ mom2, GradPtr<EXTRA, GS> __restrict__ grads, float* __restrict__ slow,
    float* __restrict__ anchor, int W, int64_t ld, int64_t P, float beta, float alpha_lr,
    float inv_w, unsigned flags) {
    const int64_t p0 = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    // Strided holds mutable row pointers; without EXTRA no store to the
    // gradient rows is instantiated
    const Strided<PS, GS, MS> r{params, mom, mom2, const_cast<typename GS::T*>(grads), ld};
    if (p0 + kVec <= P)
        sync_chunk<M, O, WT, PS, true, EXTRA>(o, r, slow, anchor, W, p0, kVec, beta, alpha_lr,
                                              inv_w, flags);
    else
        sync_chunk<M, O, WT, PS, false, EXTRA>(o, r, slow, anchor, W, p0, (int)(P - p0), beta,
                                               alpha_lr, inv_w, flags);
}

template <Sync M, Opt O, int WT, class PS, bool EXTRA = false, class GS = ParamF32,
          class MS = ParamF32>
int sync_w(const OptParams& o, const SyncArgs& a) {
    using T = typename PS::T;
    const float alpha_lr = a.alpha * o.lr;
    const float inv_w = 1.0f / (float)a.W;
    // the variants run only from the entry points whose gradient argument is
    // mutable (flags != 0), so dropping const here restores the caller's type
    const GradPtr<EXTRA, GS> grads =
        const_cast<typename GS::T*>(static_cast<const typename GS::T*>(a.grads));
    return launch(sync_kernel<M, O, WT, PS, EXTRA, GS, MS>, blocks_for(a.P), a.stream, o,
                  static_cast<T*>(a.params), static_cast<typename MS::T*>(a.mom), a.mom2, grads,
                  a.slow, a.anchor, a.W, a.ld, a.P, a.beta, alpha_lr, inv_w, a.flags);
}

template <Sync M, Opt O, class PS, class GS = ParamF32, class MS = ParamF32>
int sync_t(const OptParams& o, const SyncArgs& a) {
    if constexpr (std::is_same<GS, ParamF32>::value && std::is_same<MS, ParamF32>::value) {
        if (a.flags != 0) return sync_w<M, O, 0, PS, true>(o, a);
    }
    switch (a.W) {
        case 1: return sync_w<M, O, 1, PS, false, GS, MS>(o, a);
        case 2: return sync_w<M, O, 2, PS, false, GS, MS>(o, a);
        case 4: return sync_w<M, O, 4, PS, false, GS, MS>(o, a);
        case 8: return sync_w<M, O, 8, PS, false, GS, MS>(o, a);
        case 16: return sync_w<M, O, 16, PS, false, GS, MS>(o, a);
        case 32: return sync_w<M, O, 32, PS, false, GS, MS>(o, a);
        default: return sync_w<M, O, 0, PS, false, GS, MS>(o, a);
    }
}

// bf16 gradients or momentum: momentum SGD without variants only (the
// validation layer enforces it)
template <Sync M, class PS>
int sync_narrow(Grad gt, Mom mt, const OptParams& o, const SyncArgs& a) {
    if (a.flags != 0) return (int)hipErrorInvalidValue;
    if (gt == Grad::BF16)
        return mt == Mom::BF16 ? sync_t<M, Opt::SGD, PS, ParamBF16, ParamBF16>(o, a)
                               : sync_t<M, Opt::SGD, PS, ParamBF16, ParamF32>(o, a);
    return sync_t<M, Opt::SGD, PS, ParamF32, ParamBF16>(o, a);
}

template <Sync M, Opt O>
int sync_p(Param pt, Grad gt, Mom mt, const OptParams& o, const SyncArgs& a) {
    if (gt == Grad::BF16 || mt == Mom::BF16) {
        if constexpr (O == Opt::SGD)
            return pt == Param::BF16 ? sync_narrow<M, ParamBF16>(gt, mt, o, a)
                                     : sync_narrow<M, ParamF32>(gt, mt, o, a);
        return (int)hipErrorInvalidValue;
    }
    return pt == Param::BF16 ? sync_t<M, O, ParamBF16>(o, a) : sync_t<M, O, ParamF32>(o, a);
}

template <Sync M>
int sync_o(Opt opt, Param pt, Grad gt, Mom mt, const OptParams& o, const SyncArgs& a) {
    switch (opt) {
        case Opt::SGD_WD: return sync_p<M, Opt::SGD_WD>(pt, gt, mt, o, a);
        case Opt::ADAMW: return sync_p<M, Opt::ADAMW>(pt, gt, mt, o, a);
        default: return sync_p<M, Opt::SGD>(pt, gt, mt, o, a);
    }
}

}  // namespace

template <Sync M>
int launch_sync_mode(Opt opt, const OptParams& o, Param pt, Grad gt, Mom mt, void* params,
                     void* mom, float* mom2, const void* grads, float* slow, float* anchor,
                     int W, int64_t P, int64_t ld, float beta, float alpha, unsigned flags,
                     void* stream) {
    const SyncArgs a{params, mom, mom2, grads, slow, anchor, W, P, ld, beta, alpha, flags, stream};
    return sync_o<M>(opt, pt, gt, mt, o, a);
}

}  // namespace cpdp
