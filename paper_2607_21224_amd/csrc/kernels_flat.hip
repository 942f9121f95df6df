// Flat layout (one (W, ld) row block per family): state initialisation, the
// local optimizer step, and the dispatch of the synchronisation steps to
// their per-strategy translation units.
#include "cpdp_device.h"

namespace cpdp {
namespace {

// ---- state initialisation ---------------------------------------------------

template <class PS, class MS, bool FULL>
__device__ __forceinline__ void init_chunk(const typename PS::T* theta0, typename PS::T* params,
                                           typename MS::T* mom, float* mom2, float* slow,
                                           float* anchor, int W, int64_t ld, int64_t p0, int n) {
    float th[kVec];
    const float zero[kVec] = {0.0f, 0.0f, 0.0f, 0.0f};
    PS::template load<FULL, false>(theta0 + p0, n, th);
    for (int i = 0; i < W; ++i) {
        const int64_t off = (int64_t)i * ld + p0;
        PS::template store<FULL, kNTS>(params + off, n, th);
        MS::template store<FULL, kNTS>(mom + off, n, zero);
        if (mom2 != nullptr) store_f32<FULL, kNTS>(mom2 + off, n, zero);
    }
    store_f32<FULL, kNTS>(slow + p0, n, zero);
    store_f32<FULL, kNTS>(anchor + p0, n, th);
}

template <class PS, class MS>
__global__ __launch_bounds__(kBlock) void state_init_kernel(
    const typename PS::T* __restrict__ theta0, typename PS::T* __restrict__ params,
    typename MS::T* __restrict__ mom, float* __restrict__ mom2, float* __restrict__ slow,
    float* __restrict__ anchor, int W, int64_t ld, int64_t P) {
    const int64_t p0 = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    if (p0 + kVec <= P)
        init_chunk<PS, MS, true>(theta0, params, mom, mom2, slow, anchor, W, ld, p0, kVec);
    else
        init_chunk<PS, MS, false>(theta0, params, mom, mom2, slow, anchor, W, ld, p0,
                                  (int)(P - p0));
}

template <Opt O, class PS, class GS, class MS>
__global__ __launch_bounds__(kBlock) void local_step_kernel(
    OptParams o, typename PS::T* __restrict__ params, typename MS::T* __restrict__ mom,
    float* __restrict__ mom2, const typename GS::T* __restrict__ grads, int64_t ld, int64_t P,
    int64_t blocks_per_row, int64_t cells) {
    const int64_t cell = local_cell(cells);
    if (cell < 0) return;
    const int64_t row = cell / blocks_per_row;
    const int64_t col = cell - row * blocks_per_row;
    const int64_t p0 = (col * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    const int64_t off = row * ld;
    local_dispatch<O, PS, GS, MS>(o, params + off, mom + off, mom2 + off, grads + off, p0, P);
}

template <class PS, class MS>
int state_init_t(const void* theta0, void* params, void* mom, float* mom2, float* slow,
                 float* anchor, int W, int64_t P, int64_t ld, void* stream) {
    using T = typename PS::T;
    return launch(state_init_kernel<PS, MS>, blocks_for(P), stream,
                  static_cast<const T*>(theta0), static_cast<T*>(params),
                  static_cast<typename MS::T*>(mom), mom2, slow, anchor, W, ld, P);
}

template <Opt O, class PS, class GS, class MS>
int local_step_t(const OptParams& o, void* params, void* mom, float* mom2, const void* grads,
                 int W, int64_t P, int64_t ld, void* stream) {
    using T = typename PS::T;
    const int64_t bpr = blocks_for(P);
    return launch(local_step_kernel<O, PS, GS, MS>, local_grid(bpr * W), stream, o,
                  static_cast<T*>(params), static_cast<typename MS::T*>(mom), mom2,
                  static_cast<const typename GS::T*>(grads), ld, P, bpr, bpr * W);
}

template <Opt O, class PS>
int local_step_gm(const OptParams& o, Grad gt, Mom mt, void* params, void* mom, float* mom2,
                  const void* grads, int W, int64_t P, int64_t ld, void* stream) {
    if constexpr (O != Opt::SGD) {
        // the general optimizers take fp32 gradients and momentum (the
        // validation layer enforces it)
        if (gt != Grad::F32 || mt != Mom::F32) return (int)hipErrorInvalidValue;
        return local_step_t<O, PS, ParamF32, ParamF32>(o, params, mom, mom2, grads, W, P, ld,
                                                       stream);
    } else {
        if (gt == Grad::BF16)
            return mt == Mom::BF16
                       ? local_step_t<O, PS, ParamBF16, ParamBF16>(o, params, mom, mom2, grads, W,
                                                                   P, ld, stream)
                       : local_step_t<O, PS, ParamBF16, ParamF32>(o, params, mom, mom2, grads, W,
                                                                  P, ld, stream);
        return mt == Mom::BF16
                   ? local_step_t<O, PS, ParamF32, ParamBF16>(o, params, mom, mom2, grads, W, P,
                                                              ld, stream)
                   : local_step_t<O, PS, ParamF32, ParamF32>(o, params, mom, mom2, grads, W, P,
                                                             ld, stream);
    }
}

template <Opt O>
int local_step_p(const OptParams& o, Param pt, Grad gt, Mom mt, void* params, void* mom,
                 float* mom2, const void* grads, int W, int64_t P, int64_t ld, void* stream) {
    return pt == Param::BF16
               ? local_step_gm<O, ParamBF16>(o, gt, mt, params, mom, mom2, grads, W, P, ld,
                                             stream)
               : local_step_gm<O, ParamF32>(o, gt, mt, params, mom, mom2, grads, W, P, ld,
                                            stream);
}

}  // namespace

int launch_state_init(Param pt, Mom mt, const void* theta0, void* params, void* mom,
                      float* mom2, float* slow, float* anchor, int W, int64_t P, int64_t ld,
                      void* stream) {
    if (pt == Param::BF16)
        return mt == Mom::BF16
                   ? state_init_t<ParamBF16, ParamBF16>(theta0, params, mom, mom2, slow, anchor,
                                                        W, P, ld, stream)
                   : state_init_t<ParamBF16, ParamF32>(theta0, params, mom, mom2, slow, anchor,
                                                       W, P, ld, stream);
    return mt == Mom::BF16
               ? state_init_t<ParamF32, ParamBF16>(theta0, params, mom, mom2, slow, anchor, W, P,
                                                   ld, stream)
               : state_init_t<ParamF32, ParamF32>(theta0, params, mom, mom2, slow, anchor, W, P,
                                                  ld, stream);
}

int launch_local_step(Opt opt, const OptParams& o, Param pt, Grad gt, Mom mt, void* params,
                      void* mom, float* mom2, const void* grads, int W, int64_t P, int64_t ld,
                      void* stream) {
    switch (opt) {
        case Opt::SGD_WD:
            return local_step_p<Opt::SGD_WD>(o, pt, gt, mt, params, mom, mom2, grads, W, P, ld,
                                             stream);
        case Opt::ADAMW:
            return local_step_p<Opt::ADAMW>(o, pt, gt, mt, params, mom, mom2, grads, W, P, ld,
                                            stream);
        default:
            return local_step_p<Opt::SGD>(o, pt, gt, mt, params, mom, mom2, grads, W, P, ld,
                                          stream);
    }
}

int launch_sync(Sync mode, Opt opt, const OptParams& o, Param pt, Grad gt, Mom mt, void* params,
                void* mom, float* mom2, const void* grads, float* slow, float* anchor, int W,
                int64_t P, int64_t ld, float beta, float alpha, unsigned flags, void* stream) {
    switch (mode) {
        case Sync::LocalSGD:
            return launch_sync_mode<Sync::LocalSGD>(opt, o, pt, gt, mt, params, mom, mom2, grads,
                                                    slow, anchor, W, P, ld, beta, alpha, flags,
                                                    stream);
        case Sync::DDP:
            return launch_sync_mode<Sync::DDP>(opt, o, pt, gt, mt, params, mom, mom2, grads, slow,
                                               anchor, W, P, ld, beta, alpha, flags, stream);
        default:
            return launch_sync_mode<Sync::CPDP>(opt, o, pt, gt, mt, params, mom, mom2, grads,
                                                slow, anchor, W, P, ld, beta, alpha, flags,
                                                stream);
    }
}

}  // namespace cpdp
