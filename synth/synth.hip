// Device side of the seeded input generator (definition in synth/gen.py),
// plus a plain copy kernel used to calibrate bandwidth and HBM counters.
//
// Holds none of the CPDP arithmetic.  The generator draws the numbers that
// stand in for the initial model and for backward-pass gradients; a GPU test
// checks it bit for bit against the numpy implementation.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kBlock = 256;
constexpr int kVec = 4;
constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kC1 = 0xD1B54A32D192ED03ull;
constexpr uint64_t kC2 = 0xABC98388FB8FAC03ull;
constexpr uint64_t kC3 = 0x8CB92BA72F3D8DD7ull;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z ^= z >> 30;
    z *= 0xBF58476D1CE4E5B9ull;
    z ^= z >> 27;
    z *= 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ float draw(uint64_t key, uint64_t p, float sigma, uint32_t thr,
                                      float scale) {
    const uint64_t base = key + 4ull * p * kGamma;
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        const uint64_t h = mix64(base + (uint64_t)(j + 1) * kGamma);
#pragma unroll
        for (int f = 0; f < 4; ++f) s += (int64_t)((h >> (16 * f)) & 0xFFFFull);
    }
    const float z = (float)(s - 393210) * 0x1p-16f;
    float v = z * sigma;
    if (thr != 0u) {
        const uint64_t h3 = mix64(base + 4ull * kGamma);
        if ((uint32_t)(h3 & 0xFFFFFFFFull) < thr) v = v * scale;
    }
    return v;
}

__global__ __launch_bounds__(kBlock) void fill_normal_kernel(float* __restrict__ out,
                                                             int64_t ld, int64_t P,
                                                             int64_t blocks_per_row,
                                                             uint64_t seed, uint64_t kind,
                                                             uint64_t t, float sigma,
                                                             uint32_t thr, float scale) {
    const int64_t row = blockIdx.x / blocks_per_row;
    const int64_t col = blockIdx.x - row * blocks_per_row;
    const int64_t p0 = (col * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    uint64_t key = mix64(seed ^ (kind * kC1));
    key = mix64(key ^ (t * kC2));
    key = mix64(key ^ ((uint64_t)row * kC3));
    float* dst = out + row * ld;
#pragma unroll
    for (int k = 0; k < kVec; ++k)
        if (p0 + k < P) dst[p0 + k] = draw(key, (uint64_t)(p0 + k), sigma, thr, scale);
}

// The reference copy for the bandwidth ceiling: 128-bit nontemporal loads and
// stores, and the blocks dealt to the 8 XCDs (workgroup b runs on XCD b % 8) in
// contiguous eighths of the buffer, the fastest full-size copy measured on
// MI355X.  blocks = 8 * ceil(chunks / 8); the padding blocks exit.
__global__ __launch_bounds__(kBlock) void copy_kernel(float* __restrict__ dst,
                                                      const float* __restrict__ src,
                                                      int64_t n, int64_t chunks) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const int64_t per = (chunks + 7) / 8;
    const int64_t c = (int64_t)(blockIdx.x % 8) * per + (int64_t)(blockIdx.x / 8);
    if (c >= chunks) return;
    const int64_t p0 = (c * kBlock + threadIdx.x) * kVec;
    if (p0 + kVec <= n) {
        const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src + p0));
        __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(dst + p0));
    } else {
        for (int64_t p = p0; p < n; ++p) dst[p] = src[p];
    }
}

int64_t blocks_for(int64_t n) { return (n + kBlock * kVec - 1) / (kBlock * kVec); }

template <class T>
struct same_type {
    using type = T;
};

// Returns the status of this launch itself (not a stale error left by an
// earlier runtime call in the thread, which hipGetLastError would report).
template <class... Args>
int launch(void (*kernel)(Args...), int64_t blocks, void* stream,
           typename same_type<Args>::type... args) {
    void* argv[] = {static_cast<void*>(&args)...};
    return (int)hipLaunchKernel(reinterpret_cast<const void*>(kernel), dim3((unsigned)blocks),
                                dim3(kBlock), argv, 0, static_cast<hipStream_t>(stream));
}

}  // namespace

extern "C" {

// Fill rows [0, rows) of a (rows x ld) fp32 buffer, coordinates [0, P) of each
// row, with stream key(seed, kind, t, row).  thr = 0 disables outliers.
// Returns 0 or a HIP error code; -1 for invalid sizes.
int synth_fill_normal(float* out, int rows, int64_t P, int64_t ld, uint64_t seed, int kind,
                      int64_t t, float sigma, uint32_t outlier_thr, float outlier_scale,
                      void* stream) {
    if (rows < 1 || P < 0 || ld < P || out == nullptr) return -1;
    if (P == 0) return 0;
    const int64_t bpr = blocks_for(P);
    if (bpr > 0x7FFFFFFF / rows) return -1;
    return launch(fill_normal_kernel, bpr * rows, stream, out, ld, P, bpr, seed, (uint64_t)kind,
                  (uint64_t)t, sigma, outlier_thr, outlier_scale);
}

// dst[0:n] = src[0:n] (fp32, 16-byte aligned), a plain streaming copy.
int synth_copy_f32(float* dst, const float* src, int64_t n, void* stream) {
    if (n < 0 || dst == nullptr || src == nullptr) return -1;
    if (n == 0) return 0;
    const int64_t chunks = blocks_for(n);
    if (chunks > 0x7FFFFFFF - 8) return -1;
    return launch(copy_kernel, (chunks + 7) / 8 * 8, stream, dst, src, n, chunks);
}

}  // extern "C"
