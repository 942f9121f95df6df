// gfx950 kernels of the CPDP reconcile hot path: state initialisation, the
// local optimizer step, and the fused synchronisation step of the three
// strategies (CPDP reconcile, LocalSGD averaging, DDP gradient step), each for
// momentum SGD, SGD with weight decay, or AdamW.
//
// All of them are HBM-streaming kernels: nothing here is a dense contraction, so
// there is no MFMA and no LDS.  Every thread owns VEC = 4 consecutive
// coordinates and moves them with 128-bit (fp32) or 64-bit (bf16) vector
// accesses; a wavefront therefore touches 1 KiB (fp32) of each array row per
// access, fully coalesced.  Every output element is written by exactly one
// thread, there are no atomics and no inter-block dependencies, and the
// cross-replica sums run in a fixed order (replica 0, 1, ..., W-1) inside one
// thread, so results are bitwise independent of the launch shape.
//
// Arithmetic is fp32 with explicit fmaf in the optimizer updates and the
// SlowMo step (the library is built with -ffp-contract=off so nothing else is
// fused).  bf16 parameters are widened on load and rounded to nearest-even on
// every store, including the x_i fed to the parameter mean, where the
// framework implementation writes the optimizer's result to the parameter
// tensor before averaging it (Sec. 4.2).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "cpdp_launch.h"

namespace cpdp {
namespace {

#ifndef CPDP_BLOCK
#define CPDP_BLOCK 256
#endif
constexpr int kBlock = CPDP_BLOCK;
constexpr int kVec = 4;

// State tensors are streamed exactly once per call; nontemporal accesses keep
// them from displacing anything useful in L2 / MALL.
#ifndef CPDP_NT_LOAD
#define CPDP_NT_LOAD 1
#endif
#ifndef CPDP_NT_STORE
#define CPDP_NT_STORE 1
#endif
constexpr bool kNTL = CPDP_NT_LOAD != 0;
constexpr bool kNTS = CPDP_NT_STORE != 0;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <bool NT, class V>
__device__ __forceinline__ V vload(const V* p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    else return *p;
}

template <bool NT, class V>
__device__ __forceinline__ void vstore(V* p, V v) {
    if constexpr (NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}

// ---- fp32 lanes: FULL = all 4 coordinates valid, else the first n --------

template <bool FULL, bool NT>
__device__ __forceinline__ void load_f32(const float* p, int n, float (&x)[kVec]) {
    if constexpr (FULL) {
        f32x4 v = vload<NT>(reinterpret_cast<const f32x4*>(p));
        x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
    } else {
#pragma unroll
        for (int k = 0; k < kVec; ++k) x[k] = k < n ? p[k] : 0.0f;
    }
}

template <bool FULL, bool NT>
__device__ __forceinline__ void store_f32(float* p, int n, const float (&x)[kVec]) {
    if constexpr (FULL) {
        f32x4 v = {x[0], x[1], x[2], x[3]};
        vstore<NT>(reinterpret_cast<f32x4*>(p), v);
    } else {
#pragma unroll
        for (int k = 0; k < kVec; ++k)
            if (k < n) p[k] = x[k];
    }
}

// ---- parameter storage ----------------------------------------------------

struct ParamF32 {
    using T = float;
    __device__ static __forceinline__ float round(float x) { return x; }
    template <bool FULL, bool NT>
    __device__ static __forceinline__ void load(const T* p, int n, float (&x)[kVec]) {
        load_f32<FULL, NT>(p, n, x);
    }
    template <bool FULL, bool NT>
    __device__ static __forceinline__ void store(T* p, int n, const float (&x)[kVec]) {
        store_f32<FULL, NT>(p, n, x);
    }
};

__device__ __forceinline__ uint32_t bf16_bits(float f) {
    uint32_t b = __float_as_uint(f);
    if ((b & 0x7FFFFFFFu) > 0x7F800000u) return (b >> 16) | 0x40u;  // keep NaN quiet
    b += 0x7FFFu + ((b >> 16) & 1u);                                  // nearest, ties even
    return b >> 16;
}

__device__ __forceinline__ float bf16_value(uint32_t h) { return __uint_as_float(h << 16); }

struct ParamBF16 {
    using T = uint16_t;
    __device__ static __forceinline__ float round(float x) { return bf16_value(bf16_bits(x)); }
    template <bool FULL, bool NT>
    __device__ static __forceinline__ void load(const T* p, int n, float (&x)[kVec]) {
        if constexpr (FULL) {
            u32x2 v = vload<NT>(reinterpret_cast<const u32x2*>(p));
            x[0] = __uint_as_float(v.x << 16);
            x[1] = __uint_as_float(v.x & 0xFFFF0000u);
            x[2] = __uint_as_float(v.y << 16);
            x[3] = __uint_as_float(v.y & 0xFFFF0000u);
        } else {
#pragma unroll
            for (int k = 0; k < kVec; ++k) x[k] = k < n ? bf16_value(p[k]) : 0.0f;
        }
    }
    template <bool FULL, bool NT>
    __device__ static __forceinline__ void store(T* p, int n, const float (&x)[kVec]) {
        if constexpr (FULL) {
            u32x2 v = {bf16_bits(x[0]) | (bf16_bits(x[1]) << 16),
                       bf16_bits(x[2]) | (bf16_bits(x[3]) << 16)};
            vstore<NT>(reinterpret_cast<u32x2*>(p), v);
        } else {
#pragma unroll
            for (int k = 0; k < kVec; ++k)
                if (k < n) p[k] = (uint16_t)bf16_bits(x[k]);
        }
    }
};

// ---- state initialisation ---------------------------------------------------

template <class PS, bool FULL>
__device__ __forceinline__ void init_chunk(const typename PS::T* theta0, typename PS::T* params,
                                           float* mom, float* mom2, float* slow, float* anchor,
                                           int W, int64_t ld, int64_t p0, int n) {
    float th[kVec];
    const float zero[kVec] = {0.0f, 0.0f, 0.0f, 0.0f};
    PS::template load<FULL, false>(theta0 + p0, n, th);
    for (int i = 0; i < W; ++i) {
        const int64_t off = (int64_t)i * ld + p0;
        PS::template store<FULL, kNTS>(params + off, n, th);
        store_f32<FULL, kNTS>(mom + off, n, zero);
        if (mom2 != nullptr) store_f32<FULL, kNTS>(mom2 + off, n, zero);
    }
    store_f32<FULL, kNTS>(slow + p0, n, zero);
    store_f32<FULL, kNTS>(anchor + p0, n, th);
}

template <class PS>
__global__ __launch_bounds__(kBlock) void state_init_kernel(
    const typename PS::T* __restrict__ theta0, typename PS::T* __restrict__ params,
    float* __restrict__ mom, float* __restrict__ mom2, float* __restrict__ slow,
    float* __restrict__ anchor, int W, int64_t ld, int64_t P) {
    const int64_t p0 = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    if (p0 + kVec <= P)
        init_chunk<PS, true>(theta0, params, mom, mom2, slow, anchor, W, ld, p0, kVec);
    else
        init_chunk<PS, false>(theta0, params, mom, mom2, slow, anchor, W, ld, p0,
                              (int)(P - p0));
}

// ---- the per-replica optimizer update -------------------------------------------
//
// One coordinate of one replica: th is the stored parameter (widened), m / v
// the optimizer state, g the gradient the update uses.  Returns the new
// parameter, rounded to the parameter storage type (the value the optimizer
// writes to the parameter tensor).
//   SGD     m <- mu m + g;              th <- th - lr m
//   SGD_WD  d = g + wd th;  m <- mu m + d;  th <- th - lr m      (coupled L2)
//   ADAMW   th <- round(th (1 - lr wd));  m <- b1 m + (1-b1) g;
//           v <- b2 v + (1-b2) g^2;
//           th <- th - (lr / (1-b1^t)) m / (sqrt(v) / sqrt(1-b2^t) + eps)
// The AdamW bias-correction factors and the decay factor are folded into
// OptParams on the host (they depend on the step count only) and enter the
// arithmetic as fp32 values, as they do in the framework's fp32 tensor ops.

template <Opt O, class PS>
__device__ __forceinline__ float opt_update(const OptParams& o, float th, float& m, float& v,
                                            float g) {
    if constexpr (O == Opt::SGD) {
        m = fmaf(o.mu, m, g);
        return PS::round(fmaf(-o.lr, m, th));
    } else if constexpr (O == Opt::SGD_WD) {
        const float d = fmaf(o.wd, th, g);
        m = fmaf(o.mu, m, d);
        return PS::round(fmaf(-o.lr, m, th));
    } else {
        const float t = PS::round(th * o.decay);
        m = fmaf(o.omb1, g, o.mu * m);
        v = fmaf(o.omb2, g * g, o.beta2 * v);
        const float denom = sqrtf(v) / o.sqrt_bc2 + o.eps;
        return PS::round(fmaf(-o.step_size, m / denom, t));
    }
}

// ---- replica addressing ------------------------------------------------------------
//
// Where replica i's row of each family starts.  Strided is the flat layout of
// the C ABI (base + i*ld); Table is a multi-tensor plan (one device pointer
// per replica and tensor, replica-major).  Both expose the same accessors, so
// the step code below is written once.

template <class PS>
struct Strided {
    typename PS::T* params;
    float* mom;
    float* mom2;
    float* grads;
    int64_t ld;
    __device__ __forceinline__ typename PS::T* prm(int i) const { return params + (int64_t)i * ld; }
    __device__ __forceinline__ float* m(int i) const { return mom + (int64_t)i * ld; }
    __device__ __forceinline__ float* v(int i) const { return mom2 + (int64_t)i * ld; }
    __device__ __forceinline__ float* g(int i) const { return grads + (int64_t)i * ld; }
};

template <class PS>
struct Table {
    const int64_t* params;  // 64-bit device addresses, entry i*n + t
    const int64_t* mom;
    const int64_t* mom2;
    const int64_t* grads;
    int64_t n, t;
    __device__ __forceinline__ typename PS::T* prm(int i) const {
        return reinterpret_cast<typename PS::T*>(params[i * n + t]);
    }
    __device__ __forceinline__ float* m(int i) const { return reinterpret_cast<float*>(mom[i * n + t]); }
    __device__ __forceinline__ float* v(int i) const { return reinterpret_cast<float*>(mom2[i * n + t]); }
    __device__ __forceinline__ float* g(int i) const { return reinterpret_cast<float*>(grads[i * n + t]); }
};

// The sections of a plan table (layout documented in cpdp_launch.h).
struct PlanView {
    const int64_t* chunk_start;
    const int64_t* numel;
    const int64_t* params;
    const int64_t* mom;
    const int64_t* mom2;
    const int64_t* grads;
    const int64_t* slow;
    const int64_t* anchor;
};

__device__ __forceinline__ PlanView plan_view(const int64_t* plan, int64_t W, int64_t n) {
    PlanView v;
    v.chunk_start = plan + kPlanHeaderWords;
    v.numel = v.chunk_start + (n + 1);
    v.params = v.numel + n;
    v.mom = v.params + W * n;
    v.mom2 = v.mom + W * n;
    v.grads = v.mom2 + W * n;
    v.slow = v.grads + W * n;
    v.anchor = v.slow + n;
    return v;
}

// tensor holding chunk b: the largest t < n with chunk_start[t] <= b (an
// empty tensor never qualifies as the last such t, since b < chunk_start[n])
__device__ __forceinline__ int64_t plan_tensor(const PlanView& v, int64_t n, int64_t b) {
    int64_t lo = 0, hi = n;
    while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (v.chunk_start[mid] <= b) lo = mid;
        else hi = mid;
    }
    return lo;
}

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

// ---- local step: one replica row per block, 4 coordinates per thread -------

template <Opt O, class PS, bool FULL>
__device__ __forceinline__ void local_chunk(const OptParams& o, typename PS::T* params,
                                            float* mom, float* mom2, const float* grads,
                                            int n) {
    float g[kVec], m[kVec], v[kVec] = {0.0f, 0.0f, 0.0f, 0.0f}, th[kVec];
    load_f32<FULL, kNTL>(grads, n, g);
    load_f32<FULL, kNTL>(mom, n, m);
    if constexpr (O == Opt::ADAMW) load_f32<FULL, kNTL>(mom2, n, v);
    PS::template load<FULL, kNTL>(params, n, th);
#pragma unroll
    for (int k = 0; k < kVec; ++k) th[k] = opt_update<O, PS>(o, th[k], m[k], v[k], g[k]);
    store_f32<FULL, kNTS>(mom, n, m);
    if constexpr (O == Opt::ADAMW) store_f32<FULL, kNTS>(mom2, n, v);
    PS::template store<FULL, kNTS>(params, n, th);
}

template <Opt O, class PS>
__device__ __forceinline__ void local_dispatch(const OptParams& o, typename PS::T* params,
                                               float* mom, float* mom2, const float* grads,
                                               int64_t p0, int64_t P) {
    if (p0 + kVec <= P)
        local_chunk<O, PS, true>(o, params + p0, mom + p0, mom2 + p0, grads + p0, kVec);
    else
        local_chunk<O, PS, false>(o, params + p0, mom + p0, mom2 + p0, grads + p0,
                                  (int)(P - p0));
}

template <Opt O, class PS>
__global__ __launch_bounds__(kBlock) void local_step_kernel(
    OptParams o, typename PS::T* __restrict__ params, float* __restrict__ mom,
    float* __restrict__ mom2, const float* __restrict__ grads, int64_t ld, int64_t P,
    int64_t blocks_per_row) {
    const int64_t row = blockIdx.x / blocks_per_row;
    const int64_t col = blockIdx.x - row * blocks_per_row;
    const int64_t p0 = (col * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    const int64_t off = row * ld;
    local_dispatch<O, PS>(o, params + off, mom + off, mom2 + off, grads + off, p0, P);
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

// ---- fused synchronisation steps ----------------------------------------------
//
// One thread owns 4 coordinates across all W replicas.  WT > 0 fixes W at
// compile time (fully unrolled); WT == 0 takes W at run time (batches of
// kChunk, then single replicas).  Within a batch all loads are issued before
// any store.  The batching matters because the compiler cannot prove that two
// replica rows never alias (ld is a run-time value, plan pointers are data),
// so a store for replica i would otherwise hold back the loads of replica
// i+1 and the thread would wait one round trip to HBM per replica.
//
// Sync::CPDP      gradient mean, synchronized optimizer step, parameter mean,
//                 SlowMo, copy-back (the reconcile).
// Sync::LocalSGD  each replica steps on its own gradient, then the parameter
//                 mean is copied back (no gradient mean, no SlowMo).
// Sync::DDP       gradient mean and the same optimizer step on every replica,
//                 no parameter mean.
//
// EXTRA = true enables the optional variants selected by `flags` (run-time W
// only): kSyncWriteGbar stores the gradient mean into every gradient row;
// kSyncAverageState replaces every replica's optimizer state by the replica
// mean after the step.

#ifndef CPDP_RECON_CHUNK
#define CPDP_RECON_CHUNK 8
#endif
constexpr int kChunk = CPDP_RECON_CHUNK;

// per-thread values carried across replica batches
struct SyncAcc {
    float gbar[kVec];  // gradient mean
    float a[kVec];     // anchor (CPDP) / averaged model (LocalSGD)
    float u[kVec];     // SlowMo state
    float s[kVec];     // sum of x_i - reference
    float x0[kVec];    // LocalSGD reference: replica 0's x
    float msum[kVec];  // optimizer-state sums (state reconciliation)
    float vsum[kVec];
};

template <int C, bool FULL, class Rows>
__device__ __forceinline__ void grad_batch(const Rows& r, int i0, int64_t p0, int n,
                                           float (&acc)[kVec]) {
    float g[C][kVec];
#pragma unroll
    for (int c = 0; c < C; ++c) load_f32<FULL, kNTL>(r.g(i0 + c) + p0, n, g[c]);
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
        for (int k = 0; k < kVec; ++k) acc[k] += g[c][k];
}

template <Sync M, Opt O, int C, class PS, bool FULL, class Rows>
__device__ __forceinline__ void step_batch(const OptParams& o, const Rows& r, int i0, int64_t p0,
                                           int n, SyncAcc& z, bool avg_state) {
    constexpr bool kAdam = O == Opt::ADAMW;
    float m[C][kVec], v[C][kVec], th[C][kVec], g[C][kVec];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        if constexpr (M == Sync::LocalSGD) load_f32<FULL, kNTL>(r.g(i0 + c) + p0, n, g[c]);
        load_f32<FULL, kNTL>(r.m(i0 + c) + p0, n, m[c]);
        if constexpr (kAdam) load_f32<FULL, kNTL>(r.v(i0 + c) + p0, n, v[c]);
        PS::template load<FULL, kNTL>(r.prm(i0 + c) + p0, n, th[c]);
    }
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
        for (int k = 0; k < kVec; ++k) {
            const float gk = M == Sync::LocalSGD ? g[c][k] : z.gbar[k];
            const float x = opt_update<O, PS>(o, th[c][k], m[c][k], v[c][k], gk);
            if constexpr (M == Sync::CPDP) {
                z.s[k] += x - z.a[k];
            } else if constexpr (M == Sync::LocalSGD) {
                if (i0 + c == 0) z.x0[k] = x;
                z.s[k] += x - z.x0[k];
            } else {
                th[c][k] = x;
            }
        }
#pragma unroll
    for (int c = 0; c < C; ++c) {
        if (avg_state) {
#pragma unroll
            for (int k = 0; k < kVec; ++k) {
                z.msum[k] += m[c][k];
                if constexpr (kAdam) z.vsum[k] += v[c][k];
            }
        } else {
            store_f32<FULL, kNTS>(r.m(i0 + c) + p0, n, m[c]);
            if constexpr (kAdam) store_f32<FULL, kNTS>(r.v(i0 + c) + p0, n, v[c]);
        }
        if constexpr (M == Sync::DDP) PS::template store<FULL, kNTS>(r.prm(i0 + c) + p0, n, th[c]);
    }
}

template <Sync M, Opt O, int WT, class PS, bool FULL, bool EXTRA, class Rows>
__device__ __forceinline__ void sync_chunk(const OptParams& o, const Rows& r, float* slow,
                                           float* anchor, int W, int64_t p0, int n, float beta,
                                           float alpha_lr, float inv_w, unsigned flags) {
    static_assert(!EXTRA || WT == 0, "variants run on the run-time-W kernel");
    constexpr int C = WT > 0 ? (WT < kChunk ? WT : kChunk) : kChunk;
    static_assert(WT <= 0 || WT % C == 0, "replica batches must tile W");
    constexpr bool kAdam = O == Opt::ADAMW;
    const int nw = WT > 0 ? WT : W;
    const bool avg_state = EXTRA && (flags & kSyncAverageState);
    SyncAcc z;
#pragma unroll
    for (int k = 0; k < kVec; ++k)
        z.gbar[k] = z.a[k] = z.u[k] = z.s[k] = z.x0[k] = z.msum[k] = z.vsum[k] = 0.0f;

    // gradient mean (the gradient AllReduce of a synchronisation step),
    // summed in the fixed order i = 0, 1, ..., W-1
    if constexpr (M != Sync::LocalSGD) {
        float acc[kVec] = {0.0f, 0.0f, 0.0f, 0.0f};
        if constexpr (WT > 0) {
#pragma unroll
            for (int i0 = 0; i0 < WT; i0 += C) grad_batch<C, FULL>(r, i0, p0, n, acc);
        } else {
            int i0 = 0;
            for (; i0 + C <= nw; i0 += C) grad_batch<C, FULL>(r, i0, p0, n, acc);
            for (; i0 < nw; ++i0) grad_batch<1, FULL>(r, i0, p0, n, acc);
        }
#pragma unroll
        for (int k = 0; k < kVec; ++k) z.gbar[k] = acc[k] * inv_w;
        if (EXTRA && (flags & kSyncWriteGbar))
            for (int i = 0; i < nw; ++i) store_f32<FULL, kNTS>(r.g(i) + p0, n, z.gbar);
    }

    if constexpr (M == Sync::CPDP) {
        load_f32<FULL, kNTL>(anchor + p0, n, z.a);
        load_f32<FULL, kNTL>(slow + p0, n, z.u);
    }

    // optimizer step of every replica.  The parameter mean is accumulated as
    // a sum of differences to a reference that is close to every x_i (the
    // anchor for CPDP, replica 0's x for LocalSGD), so the small deviations
    // keep their precision.
    if constexpr (WT > 0) {
#pragma unroll
        for (int i0 = 0; i0 < WT; i0 += C) step_batch<M, O, C, PS, FULL>(o, r, i0, p0, n, z, avg_state);
    } else {
        int i0 = 0;
        for (; i0 + C <= nw; i0 += C) step_batch<M, O, C, PS, FULL>(o, r, i0, p0, n, z, avg_state);
        for (; i0 < nw; ++i0) step_batch<M, O, 1, PS, FULL>(o, r, i0, p0, n, z, avg_state);
    }
    if (avg_state) {
#pragma unroll
        for (int k = 0; k < kVec; ++k) {
            z.msum[k] *= inv_w;
            z.vsum[k] *= inv_w;
        }
        for (int i = 0; i < nw; ++i) {
            store_f32<FULL, kNTS>(r.m(i) + p0, n, z.msum);
            if constexpr (kAdam) store_f32<FULL, kNTS>(r.v(i) + p0, n, z.vsum);
        }
    }
    if constexpr (M == Sync::DDP) return;

    if constexpr (M == Sync::CPDP) {
        // SlowMo outer step: u <- beta u + (a - avg)/lr ; new = a - alpha lr u
#pragma unroll
        for (int k = 0; k < kVec; ++k) {
            const float drift = z.s[k] * inv_w;  // avg - a
            z.u[k] = fmaf(beta, z.u[k], -drift / o.lr);
            z.a[k] = fmaf(-alpha_lr, z.u[k], z.a[k]);
        }
        store_f32<FULL, kNTS>(slow + p0, n, z.u);
        store_f32<FULL, kNTS>(anchor + p0, n, z.a);
    } else {
#pragma unroll
        for (int k = 0; k < kVec; ++k) z.a[k] = fmaf(z.s[k], inv_w, z.x0[k]);
        if (anchor != nullptr) store_f32<FULL, kNTS>(anchor + p0, n, z.a);
    }

    // copy the reconciled model back into every replica
#pragma unroll
    for (int i = 0; i < nw; ++i) PS::template store<FULL, kNTS>(r.prm(i) + p0, n, z.a);
}

// The gradient rows are written only by the variants (the gradient-mean
// write-back), so only those instantiations take them as mutable.
template <bool EXTRA>
using GradPtr = typename std::conditional<EXTRA, float*, const float*>::type;

template <Sync M, Opt O, int WT, class PS, bool EXTRA>
__global__ __launch_bounds__(kBlock) void sync_kernel(
    OptParams o, typename PS::T* __restrict__ params, float* __restrict__ mom,
    float* __restrict__ mom2, GradPtr<EXTRA> __restrict__ grads, float* __restrict__ slow,
    float* __restrict__ anchor, int W, int64_t ld, int64_t P, float beta, float alpha_lr,
    float inv_w, unsigned flags) {
    const int64_t p0 = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * kVec;
    if (p0 >= P) return;
    // Strided holds mutable row pointers; without EXTRA no store to the
    // gradient rows is instantiated
    const Strided<PS> r{params, mom, mom2, const_cast<float*>(grads), ld};
    if (p0 + kVec <= P)
        sync_chunk<M, O, WT, PS, true, EXTRA>(o, r, slow, anchor, W, p0, kVec, beta, alpha_lr,
                                              inv_w, flags);
    else
        sync_chunk<M, O, WT, PS, false, EXTRA>(o, r, slow, anchor, W, p0, (int)(P - p0), beta,
                                               alpha_lr, inv_w, flags);
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

// ---- step tables: the scalars of the current step read from device memory -----
//
// Every thread reads the position word and that entry (the same addresses for
// the whole grid, so they are served from cache).  A position outside the
// table means the table is used up: the kernel returns without touching the
// state, so replaying a captured graph past its table cannot run a step with
// undefined scalars.

__device__ __forceinline__ bool step_entry(const int64_t* table, StepEntry& e) {
    const int64_t pos = table[0];
    if (pos < 0 || pos >= table[1]) return false;
    e = reinterpret_cast<const StepEntry*>(table + kStepTableHeaderWords)[pos];
    return true;
}

template <Opt O, class PS>
__global__ __launch_bounds__(kBlock) void local_step_table_kernel(
    const int64_t* __restrict__ table, typename PS::T* __restrict__ params,
    float* __restrict__ mom, float* __restrict__ mom2, const float* __restrict__ grads,
    int64_t ld, int64_t P, int64_t blocks_per_row) {
    const int64_t row = blockIdx.x / blocks_per_row;
    const int64_t col = blockIdx.x - row * blocks_per_row;
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

// ---- launch helpers -------------------------------------------------------------

inline int64_t blocks_for(int64_t P) { return (P + (int64_t)kBlock * kVec - 1) / ((int64_t)kBlock * kVec); }

template <class T>
struct same_type {
    using type = T;
};

// Argument types come from the kernel's signature only (the trailing
// parameters are a non-deduced context), so every argument is converted to
// exactly what the kernel takes before its address goes into argv.
template <class... Args>
int launch(void (*kernel)(Args...), int64_t blocks, void* stream,
           typename same_type<Args>::type... args) {
    void* argv[] = {static_cast<void*>(&args)...};
    hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kernel),
                                   dim3((unsigned)blocks), dim3(kBlock), argv, 0,
                                   static_cast<hipStream_t>(stream));
    return (int)e;
}

template <class PS>
int state_init_t(const void* theta0, void* params, float* mom, float* mom2, float* slow,
                 float* anchor, int W, int64_t P, int64_t ld, void* stream) {
    using T = typename PS::T;
    return launch(state_init_kernel<PS>, blocks_for(P), stream, static_cast<const T*>(theta0),
                  static_cast<T*>(params), mom, mom2, slow, anchor, W, ld, P);
}

template <Opt O, class PS>
int local_step_t(const OptParams& o, void* params, float* mom, float* mom2, const float* grads,
                 int W, int64_t P, int64_t ld, void* stream) {
    using T = typename PS::T;
    const int64_t bpr = blocks_for(P);
    return launch(local_step_kernel<O, PS>, bpr * W, stream, o, static_cast<T*>(params), mom,
                  mom2, grads, ld, P, bpr);
}

template <Opt O>
int local_step_p(const OptParams& o, Param pt, void* params, float* mom, float* mom2,
                 const float* grads, int W, int64_t P, int64_t ld, void* stream) {
    return pt == Param::BF16
               ? local_step_t<O, ParamBF16>(o, params, mom, mom2, grads, W, P, ld, stream)
               : local_step_t<O, ParamF32>(o, params, mom, mom2, grads, W, P, ld, stream);
}

struct SyncArgs {
    void* params;
    float* mom;
    float* mom2;
    const float* grads;
    float* slow;
    float* anchor;
    int W;
    int64_t P, ld;
    float beta, alpha;
    unsigned flags;
    void* stream;
};

template <Sync M, Opt O, int WT, class PS, bool EXTRA = false>
int sync_w(const OptParams& o, const SyncArgs& a) {
    using T = typename PS::T;
    const float alpha_lr = a.alpha * o.lr;
    const float inv_w = 1.0f / (float)a.W;
    // the variants run only from the entry points whose gradient argument is
    // mutable (flags != 0), so dropping const here restores the caller's type
    const GradPtr<EXTRA> grads = const_cast<float*>(a.grads);
    return launch(sync_kernel<M, O, WT, PS, EXTRA>, blocks_for(a.P), a.stream, o,
                  static_cast<T*>(a.params), a.mom, a.mom2, grads, a.slow, a.anchor, a.W,
                  a.ld, a.P, a.beta, alpha_lr, inv_w, a.flags);
}

template <Sync M, Opt O, class PS>
int sync_t(const OptParams& o, const SyncArgs& a) {
    if (a.flags != 0) return sync_w<M, O, 0, PS, true>(o, a);
    switch (a.W) {
        case 1: return sync_w<M, O, 1, PS>(o, a);
        case 2: return sync_w<M, O, 2, PS>(o, a);
        case 4: return sync_w<M, O, 4, PS>(o, a);
        case 8: return sync_w<M, O, 8, PS>(o, a);
        case 16: return sync_w<M, O, 16, PS>(o, a);
        case 32: return sync_w<M, O, 32, PS>(o, a);
        default: return sync_w<M, O, 0, PS>(o, a);
    }
}

template <Sync M, Opt O>
int sync_p(Param pt, const OptParams& o, const SyncArgs& a) {
    return pt == Param::BF16 ? sync_t<M, O, ParamBF16>(o, a) : sync_t<M, O, ParamF32>(o, a);
}

template <Sync M>
int sync_o(Opt opt, Param pt, const OptParams& o, const SyncArgs& a) {
    switch (opt) {
        case Opt::SGD_WD: return sync_p<M, Opt::SGD_WD>(pt, o, a);
        case Opt::ADAMW: return sync_p<M, Opt::ADAMW>(pt, o, a);
        default: return sync_p<M, Opt::SGD>(pt, o, a);
    }
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

template <Opt O>
int local_table_o(Param pt, const int64_t* table, void* params, float* mom, float* mom2,
                  const float* grads, int W, int64_t P, int64_t ld, void* stream) {
    const int64_t bpr = blocks_for(P);
    if (pt == Param::BF16)
        return launch(local_step_table_kernel<O, ParamBF16>, bpr * W, stream, table,
                      static_cast<uint16_t*>(params), mom, mom2, grads, ld, P, bpr);
    return launch(local_step_table_kernel<O, ParamF32>, bpr * W, stream, table,
                  static_cast<float*>(params), mom, mom2, grads, ld, P, bpr);
}

template <Sync M, Opt O, class PS>
int sync_table_t(const int64_t* table, const SyncArgs& a) {
    using T = typename PS::T;
    const float inv_w = 1.0f / (float)a.W;
    if (a.flags != 0)
        return launch(sync_table_kernel<M, O, PS, true>, blocks_for(a.P), a.stream, table,
                      static_cast<T*>(a.params), a.mom, a.mom2, const_cast<float*>(a.grads),
                      a.slow, a.anchor, a.W, a.ld, a.P, inv_w, a.flags);
    return launch(sync_table_kernel<M, O, PS, false>, blocks_for(a.P), a.stream, table,
                  static_cast<T*>(a.params), a.mom, a.mom2, a.grads, a.slow, a.anchor, a.W,
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

int launch_state_init(Param pt, const void* theta0, void* params, float* mom, float* mom2,
                      float* slow, float* anchor, int W, int64_t P, int64_t ld, void* stream) {
    return pt == Param::BF16
               ? state_init_t<ParamBF16>(theta0, params, mom, mom2, slow, anchor, W, P, ld,
                                         stream)
               : state_init_t<ParamF32>(theta0, params, mom, mom2, slow, anchor, W, P, ld,
                                        stream);
}

int launch_local_step(Opt opt, const OptParams& o, Param pt, void* params, float* mom,
                      float* mom2, const float* grads, int W, int64_t P, int64_t ld,
                      void* stream) {
    switch (opt) {
        case Opt::SGD_WD:
            return local_step_p<Opt::SGD_WD>(o, pt, params, mom, mom2, grads, W, P, ld, stream);
        case Opt::ADAMW:
            return local_step_p<Opt::ADAMW>(o, pt, params, mom, mom2, grads, W, P, ld, stream);
        default:
            return local_step_p<Opt::SGD>(o, pt, params, mom, mom2, grads, W, P, ld, stream);
    }
}

int launch_sync(Sync mode, Opt opt, const OptParams& o, Param pt, void* params, float* mom,
                float* mom2, const float* grads, float* slow, float* anchor, int W, int64_t P,
                int64_t ld, float beta, float alpha, unsigned flags, void* stream) {
    const SyncArgs a{params, mom, mom2, grads, slow, anchor, W, P, ld, beta, alpha, flags, stream};
    switch (mode) {
        case Sync::LocalSGD: return sync_o<Sync::LocalSGD>(opt, pt, o, a);
        case Sync::DDP: return sync_o<Sync::DDP>(opt, pt, o, a);
        default: return sync_o<Sync::CPDP>(opt, pt, o, a);
    }
}

bool grid_fits(int rows, int64_t P) {
    return rows >= 1 && blocks_for(P) <= (int64_t)0x7FFFFFFF / rows;
}

const char* hip_error_string(int err) { return hipGetErrorString((hipError_t)err); }

}  // namespace cpdp
