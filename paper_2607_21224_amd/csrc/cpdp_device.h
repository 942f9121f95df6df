// Device building blocks of the gfx950 kernels of the CPDP reconcile hot path
// (state initialisation, the local optimizer step, and the fused
// synchronisation step of the three strategies -- CPDP reconcile, LocalSGD
// averaging, DDP gradient step -- each for momentum SGD, SGD with weight
// decay, or AdamW).  The kernels and their launchers live in the kernels_*.hip
// translation units, which are compiled in parallel; everything here is
// templates and inline functions in an anonymous namespace, so each unit
// instantiates only what it launches.
//
// All of them are HBM-streaming kernels: nothing here is a dense contraction, so
// there is no MFMA and no LDS.  Every thread owns VEC = 4 consecutive
// coordinates and moves them with 128-bit (fp32) or 64-bit (bf16) vector
// accesses (parameters, and on the plain momentum-SGD entry points also the
// gradients and the momentum, may be stored as bf16); a wavefront therefore touches 1 KiB (fp32) of each array row per
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
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "cpdp_launch.h"

namespace cpdp {
namespace {

// One wavefront per block.  On MI355X 64-thread blocks ran the reconcile
// 2.6-3.1 % and the local step 1-3.7 % faster than 256-thread blocks on the
// fp32 ResNet-50 / ViT-S sized states (level on the 32-replica bf16 state);
// a kernel streaming the reconcile's rows with no arithmetic gains as much,
// so the difference is in how the memory system sees the blocks, not in the
// code.  Results do not depend on it (every thread owns its 4 coordinates).
#ifndef CPDP_BLOCK
#define CPDP_BLOCK 64
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

template <Opt O, class PS, class MS = ParamF32>
__device__ __forceinline__ float opt_update(const OptParams& o, float th, float& m, float& v,
                                            float g) {
    // the momentum buffer is stored (rounded to its storage type MS) before
    // the parameter update reads it, as the framework's in-place buffer does
    if constexpr (O == Opt::SGD) {
        m = MS::round(fmaf(o.mu, m, g));
        return PS::round(fmaf(-o.lr, m, th));
    } else if constexpr (O == Opt::SGD_WD) {
        const float d = fmaf(o.wd, th, g);
        m = MS::round(fmaf(o.mu, m, d));
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

template <class PS, class GS_ = ParamF32, class MS_ = ParamF32>
struct Strided {
    using GS = GS_;  // gradient storage type
    using MS = MS_;  // momentum storage type
    typename PS::T* params;
    typename MS::T* mom;
    float* mom2;
    typename GS::T* grads;
    int64_t ld;
    __device__ __forceinline__ typename PS::T* prm(int i) const { return params + (int64_t)i * ld; }
    __device__ __forceinline__ typename MS::T* m(int i) const { return mom + (int64_t)i * ld; }
    __device__ __forceinline__ float* v(int i) const { return mom2 + (int64_t)i * ld; }
    __device__ __forceinline__ typename GS::T* g(int i) const { return grads + (int64_t)i * ld; }
};

template <class PS>
struct Table {
    using GS = ParamF32;    // plans hold fp32 gradients
    using MS = ParamF32;    // and fp32 momentum
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

// ---- block order of the local step ---------------------------------------------
//
// The local step's blocks are the cells (replica row, column of kBlock * kVec
// coordinates) of a W x columns grid, taken in plain replica-major order: the
// hardware hands workgroup b of a launch to XCD b % 8, so each XCD streams
// every eighth column.  Dealing the blocks to the XCDs in contiguous eighths
// of the state instead was 4-5 % faster for the momentum-SGD update with
// 256-thread blocks, but 0.6-2.9 % slower with the 64-thread blocks used
// here (and level for AdamW), so the plain order stays.

// blocks of a local-step launch over `cells` cells
inline int64_t local_grid(int64_t cells) { return cells; }

// the cell of this block, or -1 for a block past the last cell
__device__ __forceinline__ int64_t local_cell(int64_t cells) {
    return (int64_t)blockIdx.x < cells ? (int64_t)blockIdx.x : -1;
}

// ---- local step: one replica row per block, 4 coordinates per thread -------

template <Opt O, class PS, class GS, class MS, bool FULL>
__device__ __forceinline__ void local_chunk(const OptParams& o, typename PS::T* params,
                                            typename MS::T* mom, float* mom2,
                                            const typename GS::T* grads, int n) {
    float g[kVec], m[kVec], v[kVec] = {0.0f, 0.0f, 0.0f, 0.0f}, th[kVec];
    GS::template load<FULL, kNTL>(grads, n, g);
    MS::template load<FULL, kNTL>(mom, n, m);
    if constexpr (O == Opt::ADAMW) load_f32<FULL, kNTL>(mom2, n, v);
    PS::template load<FULL, kNTL>(params, n, th);
#pragma unroll
    for (int k = 0; k < kVec; ++k) th[k] = opt_update<O, PS, MS>(o, th[k], m[k], v[k], g[k]);
    MS::template store<FULL, kNTS>(mom, n, m);
    if constexpr (O == Opt::ADAMW) store_f32<FULL, kNTS>(mom2, n, v);
    PS::template store<FULL, kNTS>(params, n, th);
}

template <Opt O, class PS, class GS = ParamF32, class MS = ParamF32>
__device__ __forceinline__ void local_dispatch(const OptParams& o, typename PS::T* params,
                                               typename MS::T* mom, float* mom2,
                                               const typename GS::T* grads, int64_t p0,
                                               int64_t P) {
    if (p0 + kVec <= P)
        local_chunk<O, PS, GS, MS, true>(o, params + p0, mom + p0, mom2 + p0, grads + p0,
                                         kVec);
    else
        local_chunk<O, PS, GS, MS, false>(o, params + p0, mom + p0, mom2 + p0, grads + p0,
                                          (int)(P - p0));
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

// Replica batch of the synchronisation steps.  With 64-thread blocks,
// batches of 4 were level with or up to 1.5 % faster than batches of 8 (and
// batches of 2 slower) on the reconcile of the four full-size states; the
// batching does not change the arithmetic or its order.
#ifndef CPDP_RECON_CHUNK
#define CPDP_RECON_CHUNK 4
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
    for (int c = 0; c < C; ++c)
        Rows::GS::template load<FULL, kNTL>(r.g(i0 + c) + p0, n, g[c]);
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
        if constexpr (M == Sync::LocalSGD)
            Rows::GS::template load<FULL, kNTL>(r.g(i0 + c) + p0, n, g[c]);
        Rows::MS::template load<FULL, kNTL>(r.m(i0 + c) + p0, n, m[c]);
        if constexpr (kAdam) load_f32<FULL, kNTL>(r.v(i0 + c) + p0, n, v[c]);
        PS::template load<FULL, kNTL>(r.prm(i0 + c) + p0, n, th[c]);
    }
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
        for (int k = 0; k < kVec; ++k) {
            const float gk = M == Sync::LocalSGD ? g[c][k] : z.gbar[k];
            const float x = opt_update<O, PS, typename Rows::MS>(o, th[c][k], m[c][k], v[c][k],
                                                                 gk);
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
            Rows::MS::template store<FULL, kNTS>(r.m(i0 + c) + p0, n, m[c]);
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
            for (int i = 0; i < nw; ++i)
                Rows::GS::template store<FULL, kNTS>(r.g(i) + p0, n, z.gbar);
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
            Rows::MS::template store<FULL, kNTS>(r.m(i) + p0, n, z.msum);
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
template <bool EXTRA, class GS = ParamF32>
using GradPtr = typename std::conditional<EXTRA, typename GS::T*, const typename GS::T*>::type;

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

// Where a step's scalars come from: the launch arguments, or the entry at the
// position of a device step table (no entry when the table is used up).
struct DirectScalars {
    OptParams o;
    float beta;
    float alpha_lr;
    __device__ __forceinline__ bool get(StepEntry& e) const {
        e.o = o;
        e.beta = beta;
        e.alpha_lr = alpha_lr;
        return true;
    }
};

struct TableScalars {
    const int64_t* table;
    __device__ __forceinline__ bool get(StepEntry& e) const { return step_entry(table, e); }
};

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

struct SyncArgs {
    void* params;
    void* mom;          // fp32 or bf16 rows (Mom)
    float* mom2;
    const void* grads;  // fp32 or bf16 rows (Grad)
    float* slow;
    float* anchor;
    int W;
    int64_t P, ld;
    float beta, alpha;
    unsigned flags;
    void* stream;
};

}  // namespace
}  // namespace cpdp
