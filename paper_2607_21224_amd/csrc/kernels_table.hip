// Step tables: the local and synchronisation steps with their scalars read
// from a device table, and the kernels that move the table's position.
#include "cpdp_device.h"

namespace cpdp {
namespace {

template <Opt O, class PS>
__global__ __launch_bounds__(kBlock) void local_step_table_kernel(
    const int64_t* __restrict__ table, typename PS::T* __restrict__ params,
    float* __restrict__ mom, float* __restrict__ mom2, const float* __restrict__ grads,
    int64_t ld, int64_t P, int64_t blocks_per_row, int64_t cells) {
    const int64_t cell = local_cell(cells);
    if (cell < 0) return;
    const int64_t row = cell / blocks_per_row;
    const int64_t col = cell - row * blocks_per_row;
    const int64_t p0 = (col * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    StepEntry e;
    if (!step_entry(table, e)) return;
    const int64_t off = row * ld;
    local_dispatch<O, PS>(e.o, params + off, mom + off, mom2 + off, grads + off, p0, P);
}

// run-time W (replica batches of kChunk): one instantiation per strategy,
// update and parameter type, whatever W is
template <Sync M, Opt O, class PS, bool EXTRA>
__global__ __launch_bounds__(kBlock) void sync_table_kernel(
    const int64_t* __restrict__ table, typename PS::T* __restrict__ params,
    float* __restrict__ mom, float* __restrict__ mom2, GradPtr<EXTRA> __restrict__ grads,
    float* __restrict__ slow, float* __restrict__ anchor, int W, int64_t ld, int64_t P,
    float inv_w, unsigned flags) {
    const int64_t p0 = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    StepEntry e;
    if (!step_entry(table, e)) return;
    const Strided<PS> r{params, mom, mom2, const_cast<float*>(grads), ld};
    if (p0 + kVec <= P)
        sync_chunk<M, O, 0, PS, true, EXTRA>(e.o, r, slow, anchor, W, p0, kVec, e.beta,
                                             e.alpha_lr, inv_w, flags);
    else
        sync_chunk<M, O, 0, PS, false, EXTRA>(e.o, r, slow, anchor, W, p0, (int)(P - p0),
                                              e.beta, e.alpha_lr, inv_w, flags);
}

// position word updates: one lane of one block, an ordinary (vector) store
__global__ __launch_bounds__(64) void step_table_set_kernel(int64_t* table, int64_t position) {
    if (blockIdx.x == 0 && threadIdx.x == 0) table[0] = position;
}

__global__ __launch_bounds__(64) void step_table_advance_kernel(int64_t* table) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        const int64_t pos = table[0];
        if (pos < table[1]) table[0] = pos + 1;
    }
}

template <Opt O>
int local_table_o(Param pt, const int64_t* table, void* params, float* mom, float* mom2,
                  const float* grads, int W, int64_t P, int64_t ld, void* stream) {
    const int64_t bpr = blocks_for(P);
    if (pt == Param::BF16)
        return launch(local_step_table_kernel<O, ParamBF16>, local_grid(bpr * W), stream,
                      table, static_cast<uint16_t*>(params), mom, mom2, grads, ld, P, bpr,
                      bpr * W);
    return launch(local_step_table_kernel<O, ParamF32>, local_grid(bpr * W), stream, table,
                  static_cast<float*>(params), mom, mom2, grads, ld, P, bpr, bpr * W);
}

template <Sync M, Opt O, class PS>
int sync_table_t(const int64_t* table, const SyncArgs& a) {
    using T = typename PS::T;
    const float inv_w = 1.0f / (float)a.W;
    // step tables take fp32 gradients
    const float* grads = static_cast<const float*>(a.grads);
    if (a.flags != 0)
        return launch(sync_table_kernel<M, O, PS, true>, blocks_for(a.P), a.stream, table,
                      static_cast<T*>(a.params), static_cast<float*>(a.mom), a.mom2,
                      const_cast<float*>(grads),
                      a.slow, a.anchor, a.W, a.ld, a.P, inv_w, a.flags);
    return launch(sync_table_kernel<M, O, PS, false>, blocks_for(a.P), a.stream, table,
                  static_cast<T*>(a.params), static_cast<float*>(a.mom), a.mom2, grads, a.slow,
                  a.anchor, a.W,
                  a.ld, a.P, inv_w, a.flags);
}

template <Sync M, Opt O>
int sync_table_p(Param pt, const int64_t* table, const SyncArgs& a) {
    return pt == Param::BF16 ? sync_table_t<M, O, ParamBF16>(table, a)
                             : sync_table_t<M, O, ParamF32>(table, a);
}

template <Sync M>
int sync_table_o(Opt opt, Param pt, const int64_t* table, const SyncArgs& a) {
    switch (opt) {
        case Opt::SGD_WD: return sync_table_p<M, Opt::SGD_WD>(pt, table, a);
        case Opt::ADAMW: return sync_table_p<M, Opt::ADAMW>(pt, table, a);
        default: return sync_table_p<M, Opt::SGD>(pt, table, a);
    }
}

}  // namespace

int launch_local_step_table(Opt opt, Param pt, const int64_t* table, void* params, float* mom,
                            float* mom2, const float* grads, int W, int64_t P, int64_t ld,
                            void* stream) {
    switch (opt) {
        case Opt::SGD_WD:
            return local_table_o<Opt::SGD_WD>(pt, table, params, mom, mom2, grads, W, P, ld, stream);
        case Opt::ADAMW:
            return local_table_o<Opt::ADAMW>(pt, table, params, mom, mom2, grads, W, P, ld, stream);
        default:
            return local_table_o<Opt::SGD>(pt, table, params, mom, mom2, grads, W, P, ld, stream);
    }
}

int launch_sync_table(Sync mode, Opt opt, Param pt, const int64_t* table, void* params,
                      float* mom, float* mom2, const float* grads, float* slow, float* anchor,
                      int W, int64_t P, int64_t ld, unsigned flags, void* stream) {
    const SyncArgs a{params, mom, mom2, grads, slow, anchor, W, P, ld, 0.0f, 1.0f, flags, stream};
    switch (mode) {
        case Sync::LocalSGD: return sync_table_o<Sync::LocalSGD>(opt, pt, table, a);
        case Sync::DDP: return sync_table_o<Sync::DDP>(opt, pt, table, a);
        default: return sync_table_o<Sync::CPDP>(opt, pt, table, a);
    }
}

int launch_step_table_set(int64_t* table, int64_t position, void* stream) {
    void* argv[] = {static_cast<void*>(&table), static_cast<void*>(&position)};
    return (int)hipLaunchKernel(reinterpret_cast<const void*>(step_table_set_kernel), dim3(1),
                                dim3(64), argv, 0, static_cast<hipStream_t>(stream));
}

int launch_step_table_advance(int64_t* table, void* stream) {
    void* argv[] = {static_cast<void*>(&table)};
    return (int)hipLaunchKernel(reinterpret_cast<const void*>(step_table_advance_kernel), dim3(1),
                                dim3(64), argv, 0, static_cast<hipStream_t>(stream));
}

int read_step_table_position(const int64_t* table, int64_t* position) {
    return (int)hipMemcpy(position, table, sizeof(int64_t), hipMemcpyDeviceToHost);
}

int upload_bytes(void* dev, const void* host, int64_t bytes) {
    return (int)hipMemcpy(dev, host, (size_t)bytes, hipMemcpyHostToDevice);
}

}  // namespace cpdp
