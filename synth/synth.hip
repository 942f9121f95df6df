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

#include <type_traits>

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

// The reference copy for the bandwidth ceiling: one wavefront per block (256
// coordinates), 128-bit nontemporal loads and stores, blocks in plain order,
// the fastest full-size copy measured on MI355X (1-2 % ahead of 256-thread
// blocks and of blocks dealt to the XCDs in contiguous eighths).
constexpr int kCopyBlock = 64;

__global__ __launch_bounds__(kCopyBlock) void copy_kernel(float* __restrict__ dst,
                                                          const float* __restrict__ src,
                                                          int64_t n) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const int64_t p0 = ((int64_t)blockIdx.x * kCopyBlock + threadIdx.x) * kVec;
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
// to the XCDs, or (xcd = 1) in contiguous eighths of the coordinates.
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

// The row addresses are integers from a table; these casts put the accesses in
// the global address space, so that they compile to global loads and stores
// like the library's (a generic pointer gives flat accesses, which also count
// against the LDS counter).
#define SHAPE_GLOBAL __attribute__((address_space(1)))
template <class V>
__device__ __forceinline__ V gload(const char* p) {
    return __builtin_nontemporal_load((const SHAPE_GLOBAL V*)p);
}
template <class V>
__device__ __forceinline__ void gstore(V v, char* p) {
    __builtin_nontemporal_store(v, (SHAPE_GLOBAL V*)p);
}

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
                    const u32x2 v = gload<u32x2>(a + in_tile * 2);
                    x[b].x = v.x;
                    x[b].y = v.y;
                } else {
                    x[b] = gload<u32x4>(a + in_tile * 4);
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
                    gstore(u32x2{x[b].x, x[b].y}, a + in_tile * 2);
                else
                    gstore(x[b], a + in_tile * 4);
            }
        }
    }
    const int64_t* wo = rows + 3 * (int64_t)n_rd;
    for (int j = 0; j < n_wo; ++j) {
        char* a = reinterpret_cast<char*>(wo[j]) + tile_off;
        gstore(u32x4{acc, acc, acc, acc}, a + in_tile * 4);
    }
    if (acc == sentinel) sink[threadIdx.x % 256] = acc;
}

// ---- traffic shape in the synchronisation steps' own order -------------------
//
// The same rows as the shape kernel above, loaded and stored in the order the
// library's synchronisation kernels issue them, with no arithmetic: one
// 64-thread block per 256 coordinates, replica batches of 4, and
//   S = 0, the reconcile: the W gradient rows in batches of 4; the anchor and
//          the SlowMo row; per batch the momentum (and second-moment) rows
//          and the parameter rows of 4 replicas, then their momentum stores;
//          the SlowMo and anchor stores; the W parameter stores last (they
//          carry the broadcast, which exists only after the parameter mean);
//   S = 1, the LocalSGD sync: per batch each replica's gradient, momentum
//          (second-moment) and parameter rows, then the momentum stores;
//          the write-only anchor; the W parameter stores last;
//   S = 2, the DDP step: the W gradient rows in batches of 4; per batch the
//          momentum (second-moment) and parameter rows, then per replica its
//          momentum, (second-moment) and parameter stores.
// Every store writes back the bits its row held (the parameter rows are
// kept in registers until the end), the write-only anchor gets the XOR.
// The table is the shape kernel's, in a fixed order (n = W gradient rows,
// R = 2, or 3 with second moments):
//   S = 0  g_0..g_{W-1}, then (m_i, [v_i], theta_i) for i < W, then u, anchor
//   S = 1  (g_i, m_i, [v_i], theta_i) for i < W; write-only: the anchor
//   S = 2  g_0..g_{W-1}, then (m_i, [v_i], theta_i) for i < W
// NP: the parameter rows are bf16 (held as 2 words).

// Row access of the order kernel: a scalar base (from the table) plus a 32-bit
// byte offset, the form the library's loads take; N = bf16 row.
template <bool N>
__device__ __forceinline__ u32x4 shape_ld(const int64_t* __restrict__ rows, int r, uint32_t p0) {
    const char* a = reinterpret_cast<const char*>(rows[3 * r]);
    if constexpr (N) {
        const u32x2 v = gload<u32x2>(a + p0 * 2u);
        return u32x4{v.x, v.y, 0u, 0u};
    } else {
        return gload<u32x4>(a + p0 * 4u);
    }
}

template <bool N>
__device__ __forceinline__ void shape_st(const int64_t* __restrict__ rows, int r, uint32_t p0,
                                         u32x4 x) {
    char* a = reinterpret_cast<char*>(rows[3 * r + 1]);
    if constexpr (N)
        gstore(u32x2{x.x, x.y}, a + p0 * 2u);
    else
        gstore(x, a + p0 * 4u);
}

__device__ __forceinline__ uint32_t fold(u32x4 x) { return x.x ^ x.y ^ x.z ^ x.w; }

// NP, NG, NM: parameter, gradient, momentum rows are bf16 (the second-moment,
// SlowMo and anchor rows are fp32)
template <int S, bool ADAM, int W, bool NP, bool NG, bool NM>
__global__ __launch_bounds__(64) void shape_sync_kernel(const int64_t* __restrict__ rows,
                                                        int64_t P, uint32_t sentinel,
                                                        uint32_t* __restrict__ sink) {
    constexpr int C = W < 4 ? W : 4;
    constexpr int R = ADAM ? 3 : 2;
    constexpr int G = S == 1 ? 1 : 0;  // LocalSGD: gradient row inside the replica's rows
    // P * 4 < 2^32 (checked on the host), so coordinates and byte offsets fit 32 bits
    const uint32_t p0 = (blockIdx.x * 64u + threadIdx.x) * kVec;
    if ((int64_t)p0 + kVec > P) return;  // P is a multiple of kVec (checked on the host)
    auto row_g = [](int i) { return S == 1 ? i * (R + 1) : i; };
    auto row_m = [](int i) { return S == 1 ? i * (R + 1) + 1 : W + i * R; };
    auto row_t = [](int i) { return S == 1 ? i * (R + 1) + R : W + i * R + R - 1; };
    uint32_t acc = 0;
    if constexpr (S != 1) {
#pragma unroll
        for (int i0 = 0; i0 < W; i0 += C) {
            u32x4 g[C];
#pragma unroll
            for (int c = 0; c < C; ++c) g[c] = shape_ld<NG>(rows, row_g(i0 + c), p0);
#pragma unroll
            for (int c = 0; c < C; ++c) acc ^= fold(g[c]);
        }
    }
    u32x4 a{0u, 0u, 0u, 0u}, u{0u, 0u, 0u, 0u};
    if constexpr (S == 0) {
        a = shape_ld<false>(rows, W + W * R + 1, p0);
        u = shape_ld<false>(rows, W + W * R, p0);
        acc ^= fold(a) ^ fold(u);
    }
    using PT = typename std::conditional<NP, u32x2, u32x4>::type;
    PT late[S == 2 ? 1 : W];
#pragma unroll
    for (int i0 = 0; i0 < W; i0 += C) {
        u32x4 g[C], m[C], v[C], th[C];
#pragma unroll
        for (int c = 0; c < C; ++c) {
            if constexpr (G) g[c] = shape_ld<NG>(rows, row_g(i0 + c), p0);
            m[c] = shape_ld<NM>(rows, row_m(i0 + c), p0);
            if constexpr (ADAM) v[c] = shape_ld<false>(rows, row_m(i0 + c) + 1, p0);
            th[c] = shape_ld<NP>(rows, row_t(i0 + c), p0);
        }
#pragma unroll
        for (int c = 0; c < C; ++c) {
            if constexpr (G) acc ^= fold(g[c]);
            acc ^= fold(m[c]) ^ fold(th[c]);
            if constexpr (ADAM) acc ^= fold(v[c]);
        }
#pragma unroll
        for (int c = 0; c < C; ++c) {
            shape_st<NM>(rows, row_m(i0 + c), p0, m[c]);
            if constexpr (ADAM) shape_st<false>(rows, row_m(i0 + c) + 1, p0, v[c]);
            if constexpr (S == 2) {
                shape_st<NP>(rows, row_t(i0 + c), p0, th[c]);
            } else if constexpr (NP) {
                late[i0 + c] = u32x2{th[c].x, th[c].y};
            } else {
                late[i0 + c] = th[c];
            }
        }
    }
    if constexpr (S == 0) {
        shape_st<false>(rows, W + W * R, p0, u);
        shape_st<false>(rows, W + W * R + 1, p0, a);
    }
    if constexpr (S == 1) {
        char* an = reinterpret_cast<char*>(rows[3 * W * (R + 1)]);
        gstore(u32x4{acc, acc, acc, acc}, an + p0 * 4u);
    }
    if constexpr (S != 2) {
#pragma unroll
        for (int i = 0; i < W; ++i) {
            if constexpr (NP)
                shape_st<true>(rows, row_t(i), p0, u32x4{late[i].x, late[i].y, 0u, 0u});
            else
                shape_st<false>(rows, row_t(i), p0, late[i]);
        }
    }
    if (acc == sentinel) sink[threadIdx.x] = acc;
}

template <int S, bool ADAM, bool NP, bool NG, bool NM>
const void* shape_sync_for_w(int W) {
    switch (W) {
        case 4: return reinterpret_cast<const void*>(shape_sync_kernel<S, ADAM, 4, NP, NG, NM>);
        case 8: return reinterpret_cast<const void*>(shape_sync_kernel<S, ADAM, 8, NP, NG, NM>);
        case 16: return reinterpret_cast<const void*>(shape_sync_kernel<S, ADAM, 16, NP, NG, NM>);
        case 32: return reinterpret_cast<const void*>(shape_sync_kernel<S, ADAM, 32, NP, NG, NM>);
        default: return nullptr;
    }
}

// bf16 gradient and momentum rows exist on the momentum-SGD reconcile only,
// as in the library
template <int S>
const void* shape_sync_for(bool adam, bool np, bool ng, bool nm, int W) {
    if (adam && (ng || nm)) return nullptr;
    if (adam) return np ? shape_sync_for_w<S, true, true, false, false>(W)
                        : shape_sync_for_w<S, true, false, false, false>(W);
    if constexpr (S != 0) {
        if (ng || nm) return nullptr;
        return np ? shape_sync_for_w<S, false, true, false, false>(W)
                  : shape_sync_for_w<S, false, false, false, false>(W);
    } else {
        const int k = (np ? 4 : 0) | (ng ? 2 : 0) | (nm ? 1 : 0);
        switch (k) {
            case 0: return shape_sync_for_w<S, false, false, false, false>(W);
            case 1: return shape_sync_for_w<S, false, false, false, true>(W);
            case 2: return shape_sync_for_w<S, false, false, true, false>(W);
            case 3: return shape_sync_for_w<S, false, false, true, true>(W);
            case 4: return shape_sync_for_w<S, false, true, false, false>(W);
            case 5: return shape_sync_for_w<S, false, true, false, true>(W);
            case 6: return shape_sync_for_w<S, false, true, true, false>(W);
            default: return shape_sync_for_w<S, false, true, true, true>(W);
        }
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
    const int64_t blocks = (n + kCopyBlock * kVec - 1) / (kCopyBlock * kVec);
    if (blocks > 0x7FFFFFFF) return -1;
    void* argv[] = {&dst, &src, &n};
    return (int)hipLaunchKernel(reinterpret_cast<const void*>(copy_kernel),
                                dim3((unsigned)blocks), dim3(kCopyBlock), argv, 0,
                                static_cast<hipStream_t>(stream));
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

// One pass of the traffic shape of a synchronisation step in the library's
// own load and store order (see shape_sync_kernel): sync 0 = the reconcile,
// 1 = the LocalSGD sync, 2 = the DDP step; adam = second-moment rows present;
// W in {4, 8, 16, 32}; param_bf16, grad_bf16, mom_bf16 = those rows are bf16
// (gradient and momentum rows only on the reconcile without second moments).
// The table `rows` follows the layout stated at shape_sync_kernel, its bf16
// flags unread; the caller guarantees that every address covers coordinates
// [0, P).  Returns 0, a HIP error code, or -1 for invalid arguments.
int synth_shape_sync(const int64_t* rows, int sync, int adam, int W, int param_bf16,
                     int grad_bf16, int mom_bf16, int64_t P, uint32_t sentinel, uint32_t* sink,
                     void* stream) {
    if (rows == nullptr || sink == nullptr || sync < 0 || sync > 2 || (adam != 0 && adam != 1) ||
        (param_bf16 != 0 && param_bf16 != 1) || (grad_bf16 != 0 && grad_bf16 != 1) ||
        (mom_bf16 != 0 && mom_bf16 != 1) || P < 0 || P % kVec != 0 ||
        P > (int64_t)0x3FFFFFFF)
        return -1;
    const bool a = adam, np = param_bf16, ng = grad_bf16, nm = mom_bf16;
    const void* k = sync == 0   ? shape_sync_for<0>(a, np, ng, nm, W)
                    : sync == 1 ? shape_sync_for<1>(a, np, ng, nm, W)
                                : shape_sync_for<2>(a, np, ng, nm, W);
    if (k == nullptr) return -1;
    if (P == 0) return 0;
    const int64_t blocks = (P + 64 * kVec - 1) / (64 * kVec);
    void* argv[] = {&rows, &P, &sentinel, &sink};
    return (int)hipLaunchKernel(k, dim3((unsigned)blocks), dim3(64), argv, 0,
                                static_cast<hipStream_t>(stream));
}

}  // extern "C"
