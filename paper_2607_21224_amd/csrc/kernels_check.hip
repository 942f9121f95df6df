// Failure detection (replicas that do not hold the reference model) and
// launch-shape helpers shared with the validation layer.
#include "cpdp_device.h"

namespace cpdp {
namespace {

// ---- failure detection: replicas that do not hold the reference model ------------
//
// Right after a synchronisation every replica stores R(anchor) (the broadcast
// of Algorithm 1).  Each thread checks its 4 coordinates over all W replicas,
// bit for bit (a NaN matches a NaN), the counts are summed across the
// wavefront with shuffles, and one lane per wavefront adds a nonzero sum to
// the result with a vector atomic.

__device__ __forceinline__ bool same_stored(float a, float b) {
    if (a != a && b != b) return true;  // NaN stored as NaN
    return __float_as_uint(a) == __float_as_uint(b);
}

template <class PS, bool FULL>
__device__ __forceinline__ unsigned long long count_chunk(const typename PS::T* params,
                                                          const float* anchor, int W, int64_t ld,
                                                          int64_t p0, int n) {
    float a[kVec], x[kVec];
    bool differs[kVec] = {false, false, false, false};
    load_f32<FULL, false>(anchor + p0, n, a);
#pragma unroll
    for (int k = 0; k < kVec; ++k) a[k] = PS::round(a[k]);
    for (int i = 0; i < W; ++i) {
        PS::template load<FULL, false>(params + (int64_t)i * ld + p0, n, x);
#pragma unroll
        for (int k = 0; k < kVec; ++k) differs[k] = differs[k] || !same_stored(x[k], a[k]);
    }
    unsigned long long bad = 0;
#pragma unroll
    for (int k = 0; k < kVec; ++k) bad += (k < n && differs[k]) ? 1u : 0u;
    return bad;
}

template <class PS>
__global__ __launch_bounds__(kBlock) void count_unsynced_kernel(
    const typename PS::T* __restrict__ params, const float* __restrict__ anchor, int W,
    int64_t ld, int64_t P, unsigned long long* __restrict__ count) {
    const int64_t p0 = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * kVec;
    unsigned long long bad = 0;
    if (p0 + kVec <= P)
        bad = count_chunk<PS, true>(params, anchor, W, ld, p0, kVec);
    else if (p0 < P)
        bad = count_chunk<PS, false>(params, anchor, W, ld, p0, (int)(P - p0));
    // every lane takes part in the shuffles, including those past P
    for (int off = warpSize / 2; off > 0; off >>= 1) bad += __shfl_xor(bad, off);
    if ((threadIdx.x % warpSize) == 0 && bad != 0) atomicAdd(count, bad);
}

__global__ __launch_bounds__(64) void zero_count_kernel(unsigned long long* count) {
    if (blockIdx.x == 0 && threadIdx.x == 0) *count = 0;
}

}  // namespace

int launch_count_unsynced(Param pt, const void* params, const float* anchor, int W, int64_t P,
                          int64_t ld, uint64_t* count, void* stream) {
    auto* c = reinterpret_cast<unsigned long long*>(count);
    void* zargv[] = {static_cast<void*>(&c)};
    hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(zero_count_kernel), dim3(1),
                                   dim3(64), zargv, 0, static_cast<hipStream_t>(stream));
    if (e != hipSuccess || P == 0) return (int)e;
    if (pt == Param::BF16)
        return launch(count_unsynced_kernel<ParamBF16>, blocks_for(P), stream,
                      static_cast<const uint16_t*>(params), anchor, W, ld, P, c);
    return launch(count_unsynced_kernel<ParamF32>, blocks_for(P), stream,
                  static_cast<const float*>(params), anchor, W, ld, P, c);
}

bool grid_fits(int rows, int64_t P) {
    return rows >= 1 && blocks_for(P) <= kMaxBlocks / rows;
}

const char* hip_error_string(int err) { return hipGetErrorString((hipError_t)err); }

}  // namespace cpdp
