// Device side of the seeded input generator (definition in synth/gen.py),
// plus two measurement kernels: a plain copy that calibrates bandwidth and the
// HBM counters, and a traffic-shape kernel that streams any set of rows with
// no arithmetic to speak of, the bandwidth ceiling of a traffic shape.
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


// ---- traffic-shape kernel ------------------------------------------------------
//
// Moves the bytes of a streaming pass with a given set of rows and nothing
// else: every thread loads 4 consecutive coordinates of every read row
// (128-bit loads of fp32 rows, 64-bit of bf16 rows, nontemporal), folds the
// loaded bits into an XOR, and stores each read row that is also written
// back to its write address unchanged (in place, the state keeps its exact
// bits), then the XOR into every extra write-only row.  Read rows are taken
// in batches of B, all loads of a batch before its stores, as the reconcile
// takes its replica batches.  A block of T threads covers 4T coordinates
// (the library's kernels use T = 64, 256 coordinates); blocks go round robin
// to the XCDs, or (xcd = 1) in contiguous eighths like the copy kernel.
//
// Row table in device memory, 64-bit words: for each read row r
// [3r] address, [3r+1] write address (0 = read only), [3r+2] 1 for bf16
// (2-byte) rows; then one address per write-only row (fp32, 4 bytes).
// Coordinate p of a row with address a sits at
//   a + (p / tile) * tile_stride + (p % tile) * esize
// so tile = the row length with tile_stride = 0 gives plain rows, and
// tile = T with tile_stride = rows * T * esize a tile-major layout whose
// tiles of T coordinates hold one segment of every row back to back.
// The XOR is written to `sink` only when it equals `sentinel`, which keeps
// every load live; sink is a 1 KiB scratch buffer.
constexpr int kShapeMaxRead = 256;
constexpr int kShapeMaxWriteOnly = 64;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kShapeMaxThreads = 1024;

template <int B>
__global__ __launch_bounds__(kShapeMaxThreads) void shape_kernel(const int64_t* __restrict__ rows, int n_rd,
                                                       int n_wo, int64_t P, int64_t chunks,
                                                       int64_t tile, int64_t tile_stride,
                                                       int xcd, uint32_t sentinel,
                                                       uint32_t* __restrict__ sink) {
    int64_t c = blockIdx.x;
    if (xcd) {
        const int64_t per = (chunks + 7) / 8;
        c = (int64_t)(blockIdx.x % 8) * per + (int64_t)(blockIdx.x / 8);
    }
    if (c >= chunks) return;
    const int64_t p0 = (c * (int64_t)blockDim.x + threadIdx.x) * kVec;
    if (p0 + kVec > P) return;  // P is a multiple of kVec (checked on the host)
    const int64_t tile_off = (p0 / tile) * tile_stride;
    const int64_t in_tile = p0 % tile;
    uint32_t acc = 0;
    for (int r0 = 0; r0 < n_rd; r0 += B) {
        u32x4 x[B];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            x[b] = u32x4{0u, 0u, 0u, 0u};
            const int r = r0 + b;
            if (r < n_rd) {
                const char* a = reinterpret_cast<const char*>(rows[3 * r]) + tile_off;
                if (rows[3 * r + 2]) {
                    const u32x2 v = __builtin_nontemporal_load(
                        reinterpret_cast<const u32x2*>(a + in_tile * 2));
                    x[b].x = v.x;
                    x[b].y = v.y;
                } else {
                    x[b] = __builtin_nontemporal_load(
                        reinterpret_cast<const u32x4*>(a + in_tile * 4));
                }
            }
        }
#pragma unroll
        for (int b = 0; b < B; ++b) acc ^= x[b].x ^ x[b].y ^ x[b].z ^ x[b].w;
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int r = r0 + b;
            if (r < n_rd && rows[3 * r + 1] != 0) {
                char* a = reinterpret_cast<char*>(rows[3 * r + 1]) + tile_off;
                if (rows[3 * r + 2])
                    __builtin_nontemporal_store(u32x2{x[b].x, x[b].y},
                                                reinterpret_cast<u32x2*>(a + in_tile * 2));
                else
                    __builtin_nontemporal_store(x[b], reinterpret_cast<u32x4*>(a + in_tile * 4));
            }
        }
    }
    const int64_t* wo = rows + 3 * (int64_t)n_rd;
    for (int j = 0; j < n_wo; ++j) {
        char* a = reinterpret_cast<char*>(wo[j]) + tile_off;
        __builtin_nontemporal_store(u32x4{acc, acc, acc, acc},
                                    reinterpret_cast<u32x4*>(a + in_tile * 4));
    }
    if (acc == sentinel) sink[threadIdx.x % 256] = acc;
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


// One pass of the traffic-shape kernel (see shape_kernel) over coordinates
// [0, P) of the rows described by the device table `rows` (n_read read rows,
// n_write_only write-only rows).  tile = 0 means plain rows; otherwise tile
// is a multiple of 1024 coordinates and tile_stride the bytes between tiles.
// batch is 8 or 16; xcd = 1 deals blocks to the XCDs in contiguous eighths.
// The caller guarantees that every address the table names covers the
// coordinates the pass touches (the Python binding checks it against the
// tensors it takes them from).  Returns 0, a HIP error code, or -1 for
// invalid arguments.
int synth_shape_stream(const int64_t* rows, int n_read, int n_write_only, int64_t P,
                       int64_t tile, int64_t tile_stride, int xcd, int batch, int threads,
                       uint32_t sentinel, uint32_t* sink, void* stream) {
    if (rows == nullptr || sink == nullptr || n_read < 0 || n_read > kShapeMaxRead ||
        n_write_only < 0 || n_write_only > kShapeMaxWriteOnly || n_read + n_write_only < 1 ||
        P < 0 || P % kVec != 0 || tile < 0 || tile_stride < 0 || (xcd != 0 && xcd != 1) ||
        threads < 64 || threads > kShapeMaxThreads || (threads & (threads - 1)) != 0)
        return -1;
    const int64_t per_block = (int64_t)threads * kVec;
    if (tile != 0 && tile % per_block != 0) return -1;
    if (P == 0) return 0;
    const int64_t chunks = (P + per_block - 1) / per_block;
    if (chunks > 0x7FFFFFFF - 8) return -1;
    const int64_t t = tile == 0 ? P : tile;
    const int64_t blocks = xcd ? (chunks + 7) / 8 * 8 : chunks;
    const int64_t ts = tile == 0 ? (int64_t)0 : tile_stride;
    void* argv[] = {&rows, &n_read, &n_write_only, &P, const_cast<int64_t*>(&chunks),
                    const_cast<int64_t*>(&t), const_cast<int64_t*>(&ts), &xcd, &sentinel, &sink};
    const void* k = batch == 8    ? reinterpret_cast<const void*>(shape_kernel<8>)
                    : batch == 16 ? reinterpret_cast<const void*>(shape_kernel<16>)
                                  : nullptr;
    if (k == nullptr) return -1;
    return (int)hipLaunchKernel(k, dim3((unsigned)blocks), dim3((unsigned)threads), argv, 0,
                                static_cast<hipStream_t>(stream));
}

}  // extern "C"
