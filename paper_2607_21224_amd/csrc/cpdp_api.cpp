// C ABI of the CPDP hot path: argument validation on the host, storage-type
// dispatch, and the kernel launches on the caller's stream.  No HIP call is
// made before every argument has been checked, so an invalid call never
// touches the GPU.  The contract of every entry point is documented in
// include/cpdp.h.
#include "cpdp.h"

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <mutex>
#include <utility>
#include <vector>

#include "cpdp_launch.h"
#include "plan_scratch.h"

namespace {

struct Range {
    uintptr_t lo, hi;  // [lo, hi) in bytes; empty when lo == hi
};

bool overlap(const Range& a, const Range& b) {
    return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool is_dtype(int dt) { return dt == CPDP_F32 || dt == CPDP_BF16; }

size_t esize(int dt) { return dt == CPDP_BF16 ? 2 : 4; }

// Largest element count whose byte size stays far from any address-space
// overflow (2^60 bytes); real buffers are many orders of magnitude smaller.
constexpr int64_t kMaxElems = (int64_t)1 << 57;

int check_shape(int W, int64_t P, int64_t ld, int K) {
    if (W < 1 || P < 0 || ld < P || K < 1) return CPDP_ERR_INVALID_ARG;
    if (ld > kMaxElems || (int64_t)(W - 1) > kMaxElems / (ld > 0 ? ld : 1))
        return CPDP_ERR_INVALID_ARG;
    return CPDP_OK;
}

// Byte range of a W-row family with row stride ld (only [0, P) of each row
// belongs to it, but the span from the first to the last used element is
// what may not be shared with another argument).
Range rows(const void* base, int W, int64_t P, int64_t ld, size_t es) {
    uintptr_t lo = reinterpret_cast<uintptr_t>(base);
    return {lo, lo + (uintptr_t)(((int64_t)(W - 1) * ld + P) * (int64_t)es)};
}

Range vec(const void* base, int64_t P, size_t es) {
    uintptr_t lo = reinterpret_cast<uintptr_t>(base);
    return {lo, lo + (uintptr_t)(P * (int64_t)es)};
}

int check_pointers(const void* const* ptrs, const Range* ranges, const size_t* es, int n,
                   int64_t ld) {
    for (int k = 0; k < n; ++k)
        if (ptrs[k] == nullptr) return CPDP_ERR_NULL;
    // a range that wraps past the end of the address space cannot be a buffer
    // (and would slip through the overlap test as an empty range)
    for (int k = 0; k < n; ++k)
        if (ranges[k].hi < ranges[k].lo) return CPDP_ERR_INVALID_ARG;
    for (int k = 0; k < n; ++k) {
        if (!aligned16(ptrs[k])) return CPDP_ERR_MISALIGNED;
        if (es[k] != 0 && ((int64_t)(ld * (int64_t)es[k]) & 15) != 0) return CPDP_ERR_MISALIGNED;
    }
    for (int a = 0; a < n; ++a)
        for (int b = a + 1; b < n; ++b)
            if (overlap(ranges[a], ranges[b])) return CPDP_ERR_OVERLAP;
    return CPDP_OK;
}

bool finite(float x) { return std::isfinite(x); }

int check_lr_mu(float lr, float mu) {
    if (!(finite(lr) && lr > 0.0f)) return CPDP_ERR_INVALID_ARG;
    if (!(mu >= 0.0f && mu < 1.0f)) return CPDP_ERR_INVALID_ARG;
    return CPDP_OK;
}

int hip_status(int err) { return err == 0 ? CPDP_OK : CPDP_ERR_HIP; }

cpdp::Param param_kind(int dt) { return dt == CPDP_BF16 ? cpdp::Param::BF16 : cpdp::Param::F32; }

cpdp::Grad grad_kind(int dt) { return dt == CPDP_BF16 ? cpdp::Grad::BF16 : cpdp::Grad::F32; }

cpdp::Mom mom_kind(int dt) { return dt == CPDP_BF16 ? cpdp::Mom::BF16 : cpdp::Mom::F32; }

cpdp::OptParams plain_sgd(float lr, float mu) {
    cpdp::OptParams o{};
    o.lr = lr;
    o.mu = mu;
    return o;
}

// Validates an optimizer descriptor and folds it into kernel scalars.
int make_opt(const cpdp_optimizer* opt, cpdp::Opt* kind, cpdp::OptParams* o) {
    if (opt == nullptr) return CPDP_ERR_NULL;
    *o = cpdp::OptParams{};
    const float lr = opt->lr, wd = opt->weight_decay;
    if (!(finite(lr) && lr > 0.0f)) return CPDP_ERR_INVALID_ARG;
    if (!(opt->momentum >= 0.0f && opt->momentum < 1.0f)) return CPDP_ERR_INVALID_ARG;
    if (!(finite(wd) && wd >= 0.0f)) return CPDP_ERR_INVALID_ARG;
    o->lr = lr;
    o->mu = opt->momentum;
    if (opt->kind == CPDP_OPT_SGD) {
        *kind = wd != 0.0f ? cpdp::Opt::SGD_WD : cpdp::Opt::SGD;
        o->wd = wd;
        return CPDP_OK;
    }
    if (opt->kind != CPDP_OPT_ADAMW) return CPDP_ERR_INVALID_ARG;
    const float b2 = opt->beta2, eps = opt->eps;
    if (!(b2 >= 0.0f && b2 < 1.0f)) return CPDP_ERR_INVALID_ARG;
    if (!(finite(eps) && eps > 0.0f)) return CPDP_ERR_INVALID_ARG;
    if (opt->step < 1) return CPDP_ERR_INVALID_ARG;
    if (!((double)lr * wd < 1.0)) return CPDP_ERR_INVALID_ARG;
    *kind = cpdp::Opt::ADAMW;
    const double t = (double)opt->step;
    const double bc1 = 1.0 - std::pow((double)opt->momentum, t);
    const double bc2 = 1.0 - std::pow((double)b2, t);
    if (!(bc1 > 0.0 && bc2 > 0.0)) return CPDP_ERR_INVALID_ARG;
    o->omb1 = 1.0f - opt->momentum;
    o->beta2 = b2;
    o->omb2 = 1.0f - b2;
    o->eps = eps;
    o->step_size = (float)((double)lr / bc1);
    o->sqrt_bc2 = (float)std::sqrt(bc2);
    o->decay = (float)(1.0 - (double)lr * wd);
    return CPDP_OK;
}

// Hash of every field of a plan handle except the seal itself (splitmix64
// finaliser steps over the fields in declaration order).
uint64_t plan_seal(const cpdp_plan* p) {
    uint64_t h = 0x243F6A8885A308D3ull;
    auto mix = [&h](uint64_t x) {
        h ^= x;
        h ^= h >> 30;
        h *= 0xBF58476D1CE4E5B9ull;
        h ^= h >> 27;
        h *= 0x94D049BB133111EBull;
        h ^= h >> 31;
    };
    mix(reinterpret_cast<uintptr_t>(p->table));
    mix((uint64_t)(uint32_t)p->W);
    mix((uint64_t)(uint32_t)p->n_tensors);
    mix((uint64_t)(uint32_t)p->param_dt);
    mix((uint64_t)(uint32_t)p->has_mom2);
    mix((uint64_t)(uint32_t)p->has_slow_mom);
    mix((uint64_t)(uint32_t)p->has_anchor);
    mix((uint64_t)p->total_chunks);
    mix((uint64_t)p->total_numel);
    return h;
}

// Pointer checks of a local step with a general optimizer (mom2 only for AdamW).
int check_local_ptrs(void* params, void* mom, void* mom2, const void* grads, int W, int64_t P,
                     int64_t ld, size_t sp, bool adam) {
    const void* ptrs[] = {params, mom, grads, mom2};
    const Range ranges[] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, 4),
                            rows(grads, W, P, ld, 4), rows(mom2, W, P, ld, 4)};
    const size_t row_es[] = {sp, 4, 4, 4};
    return check_pointers(ptrs, ranges, row_es, adam ? 4 : 3, ld);
}

// The buffers a synchronisation step of `strategy` reads or writes, checked;
// on success *slow, *anc and *m2 are the ones the kernels get (NULL when the
// strategy or update does not use them).
int check_sync_ptrs(int strategy, bool adam, void* params, void* mom, void* mom2, void* grads,
                    float* slow_mom, float* anchor, int W, int64_t P, int64_t ld, size_t sp,
                    float** slow, float** anc, void** m2) {
    const bool cpdp_sync = strategy == CPDP_SYNC_CPDP;
    *slow = cpdp_sync ? slow_mom : nullptr;
    *anc = strategy == CPDP_SYNC_DDP ? nullptr : anchor;
    *m2 = adam ? mom2 : nullptr;
    if (cpdp_sync && (slow_mom == nullptr || anchor == nullptr)) return CPDP_ERR_NULL;
    if (adam && mom2 == nullptr) return CPDP_ERR_NULL;
    const void* ptrs[6] = {params, mom, grads};
    Range ranges[6] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, 4),
                       rows(grads, W, P, ld, 4)};
    size_t row_es[6] = {sp, 4, 4};
    int n = 3;
    if (*m2) { ptrs[n] = *m2; ranges[n] = rows(*m2, W, P, ld, 4); row_es[n++] = 4; }
    if (*slow) { ptrs[n] = *slow; ranges[n] = vec(*slow, P, 4); row_es[n++] = 0; }
    if (*anc) { ptrs[n] = *anc; ranges[n] = vec(*anc, P, 4); row_es[n++] = 0; }
    return check_pointers(ptrs, ranges, row_es, n, ld);
}

bool valid_strategy(int strategy) {
    return strategy == CPDP_SYNC_CPDP || strategy == CPDP_SYNC_LOCALSGD ||
           strategy == CPDP_SYNC_DDP;
}

cpdp::Sync sync_mode(int strategy) {
    return strategy == CPDP_SYNC_CPDP       ? cpdp::Sync::CPDP
           : strategy == CPDP_SYNC_LOCALSGD ? cpdp::Sync::LocalSGD
                                            : cpdp::Sync::DDP;
}

constexpr unsigned kKnownFlags = CPDP_SYNC_WRITE_GRAD_MEAN | CPDP_SYNC_AVERAGE_OPT_STATE;

// Hash of a step-table handle's fields except the seal (same construction as
// the plan seal).
uint64_t step_table_seal(const cpdp_step_table* t) {
    uint64_t h = 0x13198A2E03707344ull;
    auto mix = [&h](uint64_t x) {
        h ^= x;
        h ^= h >> 30;
        h *= 0xBF58476D1CE4E5B9ull;
        h ^= h >> 27;
        h *= 0x94D049BB133111EBull;
        h ^= h >> 31;
    };
    mix(reinterpret_cast<uintptr_t>(t->table));
    mix((uint64_t)(uint32_t)t->n_steps);
    mix((uint64_t)(uint32_t)t->update);
    return h;
}

// A usable step-table handle: filled by cpdp_step_table_fill and unchanged.
int check_step_table(const cpdp_step_table* t, cpdp::Opt* kind) {
    if (t == nullptr || t->table == nullptr) return CPDP_ERR_NULL;
    if (t->n_steps < 1 || t->update < 0 || t->update > 2) return CPDP_ERR_INVALID_ARG;
    if (t->seal != step_table_seal(t)) return CPDP_ERR_INVALID_ARG;
    *kind = t->update == 2 ? cpdp::Opt::ADAMW : t->update == 1 ? cpdp::Opt::SGD_WD : cpdp::Opt::SGD;
    return CPDP_OK;
}

}  // namespace

extern "C" {

int cpdp_state_init(const void* theta0, void* params, void* mom, float* slow_mom,
                    float* anchor, int W, int64_t P, int64_t ld, int K, int param_dt,
                    int mom_dt, void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (!is_dtype(param_dt) || !is_dtype(mom_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt), sm = esize(mom_dt);
    const void* ptrs[] = {theta0, params, mom, slow_mom, anchor};
    const Range ranges[] = {vec(theta0, P, sp), rows(params, W, P, ld, sp),
                            rows(mom, W, P, ld, sm), vec(slow_mom, P, 4), vec(anchor, P, 4)};
    const size_t row_es[] = {0, sp, sm, 0, 0};
    if (int s = check_pointers(ptrs, ranges, row_es, 5, ld)) return s;
    return hip_status(cpdp::launch_state_init(param_kind(param_dt), mom_kind(mom_dt), theta0,
                                              params, mom, nullptr, slow_mom, anchor, W, P, ld,
                                              stream));
}

int cpdp_local_step(void* params, void* mom, const void* grads, int W, int64_t P, int64_t ld,
                    int K, float lr, float mu, int param_dt, int grad_dt, int mom_dt,
                    void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (int s = check_lr_mu(lr, mu)) return s;
    if (!is_dtype(param_dt) || !is_dtype(grad_dt) || !is_dtype(mom_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(W, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt), sg = esize(grad_dt), sm = esize(mom_dt);
    const void* ptrs[] = {params, mom, grads};
    const Range ranges[] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, sm),
                            rows(grads, W, P, ld, sg)};
    const size_t row_es[] = {sp, sm, sg};
    if (int s = check_pointers(ptrs, ranges, row_es, 3, ld)) return s;
    return hip_status(cpdp::launch_local_step(cpdp::Opt::SGD, plain_sgd(lr, mu),
                                              param_kind(param_dt), grad_kind(grad_dt),
                                              mom_kind(mom_dt), params, mom, nullptr, grads, W,
                                              P, ld, stream));
}

int cpdp_reconcile(void* params, void* mom, const void* grads, float* slow_mom, float* anchor,
                   int W, int64_t P, int64_t ld, int K, float lr, float mu, float beta,
                   float alpha, int param_dt, int grad_dt, int mom_dt, void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (int s = check_lr_mu(lr, mu)) return s;
    if (!(beta >= 0.0f && beta < 1.0f)) return CPDP_ERR_INVALID_ARG;
    if (!(finite(alpha) && alpha > 0.0f)) return CPDP_ERR_INVALID_ARG;
    if (!is_dtype(param_dt) || !is_dtype(grad_dt) || !is_dtype(mom_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt), sg = esize(grad_dt), sm = esize(mom_dt);
    const void* ptrs[] = {params, mom, grads, slow_mom, anchor};
    const Range ranges[] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, sm),
                            rows(grads, W, P, ld, sg), vec(slow_mom, P, 4), vec(anchor, P, 4)};
    const size_t row_es[] = {sp, sm, sg, 0, 0};
    if (int s = check_pointers(ptrs, ranges, row_es, 5, ld)) return s;
    return hip_status(cpdp::launch_sync(cpdp::Sync::CPDP, cpdp::Opt::SGD, plain_sgd(lr, mu),
                                        param_kind(param_dt), grad_kind(grad_dt),
                                        mom_kind(mom_dt), params, mom, nullptr, grads, slow_mom,
                                        anchor, W, P, ld, beta, alpha, 0u, stream));
}

int cpdp_localsgd_sync(void* params, void* mom, const void* grads, float* anchor, int W,
                       int64_t P, int64_t ld, int K, float lr, float mu, int param_dt,
                       int grad_dt, int mom_dt, void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (int s = check_lr_mu(lr, mu)) return s;
    if (!is_dtype(param_dt) || !is_dtype(grad_dt) || !is_dtype(mom_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt), sg = esize(grad_dt), sm = esize(mom_dt);
    // anchor is optional: validate it only when given
    const int n = anchor != nullptr ? 4 : 3;
    const void* ptrs[] = {params, mom, grads, anchor};
    const Range ranges[] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, sm),
                            rows(grads, W, P, ld, sg), vec(anchor, P, 4)};
    const size_t row_es[] = {sp, sm, sg, 0};
    if (int s = check_pointers(ptrs, ranges, row_es, n, ld)) return s;
    return hip_status(cpdp::launch_sync(cpdp::Sync::LocalSGD, cpdp::Opt::SGD, plain_sgd(lr, mu),
                                        param_kind(param_dt), grad_kind(grad_dt),
                                        mom_kind(mom_dt), params, mom, nullptr, grads, nullptr,
                                        anchor, W, P, ld, 0.0f, 1.0f, 0u, stream));
}

int cpdp_ddp_step(void* params, void* mom, const void* grads, int W, int64_t P, int64_t ld,
                  float lr, float mu, int param_dt, int grad_dt, int mom_dt, void* stream) {
    if (int s = check_shape(W, P, ld, 1)) return s;
    if (int s = check_lr_mu(lr, mu)) return s;
    if (!is_dtype(param_dt) || !is_dtype(grad_dt) || !is_dtype(mom_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt), sg = esize(grad_dt), sm = esize(mom_dt);
    const void* ptrs[] = {params, mom, grads};
    const Range ranges[] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, sm),
                            rows(grads, W, P, ld, sg)};
    const size_t row_es[] = {sp, sm, sg};
    if (int s = check_pointers(ptrs, ranges, row_es, 3, ld)) return s;
    return hip_status(cpdp::launch_sync(cpdp::Sync::DDP, cpdp::Opt::SGD, plain_sgd(lr, mu),
                                        param_kind(param_dt), grad_kind(grad_dt),
                                        mom_kind(mom_dt), params, mom, nullptr, grads, nullptr,
                                        nullptr, W, P, ld, 0.0f, 1.0f, 0u, stream));
}

int cpdp_state_init_opt(const void* theta0, void* params, void* mom, void* mom2,
                        float* slow_mom, float* anchor, int W, int64_t P, int64_t ld, int K,
                        int param_dt, void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (!is_dtype(param_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt);
    const int n = mom2 != nullptr ? 6 : 5;
    const void* ptrs[] = {theta0, params, mom, slow_mom, anchor, mom2};
    const Range ranges[] = {vec(theta0, P, sp),    rows(params, W, P, ld, sp),
                            rows(mom, W, P, ld, 4), vec(slow_mom, P, 4),
                            vec(anchor, P, 4),      rows(mom2, W, P, ld, 4)};
    const size_t row_es[] = {0, sp, 4, 0, 0, 4};
    if (int s = check_pointers(ptrs, ranges, row_es, n, ld)) return s;
    return hip_status(cpdp::launch_state_init(param_kind(param_dt), cpdp::Mom::F32, theta0,
                                              params, mom, static_cast<float*>(mom2), slow_mom,
                                              anchor, W, P, ld, stream));
}

int cpdp_local_step_opt(void* params, void* mom, void* mom2, const void* grads, int W,
                        int64_t P, int64_t ld, int K, const cpdp_optimizer* opt, int param_dt,
                        void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    cpdp::Opt kind;
    cpdp::OptParams o;
    if (int s = make_opt(opt, &kind, &o)) return s;
    if (!is_dtype(param_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(W, P)) return CPDP_ERR_INVALID_ARG;
    const bool adam = kind == cpdp::Opt::ADAMW;
    const size_t sp = esize(param_dt);
    if (int s = check_local_ptrs(params, mom, mom2, grads, W, P, ld, sp, adam)) return s;
    return hip_status(cpdp::launch_local_step(kind, o, param_kind(param_dt), cpdp::Grad::F32,
                                              cpdp::Mom::F32, params, mom,
                                              adam ? static_cast<float*>(mom2) : nullptr, grads,
                                              W, P, ld, stream));
}

int cpdp_sync_step_opt(int strategy, void* params, void* mom, void* mom2, void* grads,
                       float* slow_mom, float* anchor, int W, int64_t P, int64_t ld, int K,
                       const cpdp_optimizer* opt, float beta, float alpha, unsigned flags,
                       int param_dt, void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (flags & ~kKnownFlags) return CPDP_ERR_INVALID_ARG;
    if (!valid_strategy(strategy)) return CPDP_ERR_INVALID_ARG;
    cpdp::Opt kind;
    cpdp::OptParams o;
    if (int s = make_opt(opt, &kind, &o)) return s;
    if (strategy == CPDP_SYNC_CPDP) {
        if (!(beta >= 0.0f && beta < 1.0f)) return CPDP_ERR_INVALID_ARG;
        if (!(finite(alpha) && alpha > 0.0f)) return CPDP_ERR_INVALID_ARG;
    }
    if (!is_dtype(param_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    float* slow;
    float* anc;
    void* m2;
    if (int s = check_sync_ptrs(strategy, kind == cpdp::Opt::ADAMW, params, mom, mom2, grads,
                                slow_mom, anchor, W, P, ld, esize(param_dt), &slow, &anc, &m2))
        return s;
    const cpdp::Sync mode = sync_mode(strategy);
    return hip_status(cpdp::launch_sync(mode, kind, o, param_kind(param_dt), cpdp::Grad::F32,
                                        cpdp::Mom::F32, params, mom,
                                        static_cast<float*>(m2), grads, slow, anc, W, P, ld,
                                        beta, alpha, flags, stream));
}

int64_t cpdp_plan_bytes(int W, int n_tensors) {
    if (W < 1 || n_tensors < 1) return 0;
    return cpdp::plan_words(W, n_tensors) * (int64_t)sizeof(int64_t);
}

namespace {

using Span = std::pair<uintptr_t, uintptr_t>;

// Fill the words of a plan table (layout in cpdp_launch.h) and validate every
// described range: non-NULL, 16-byte aligned, no overlaps.  `ranges` has room
// for at least 4*W*n + 2*n entries (sorted in place).  On success *chunks and
// *total hold the plan's chunk and element counts.
int fill_plan(int64_t* tab, int64_t words, Span* ranges, int W, int n, const int64_t* numel,
              void* const* params, void* const* mom, void* const* mom2, void* const* grads,
              float* const* slow_mom, float* const* anchor, int param_dt, int64_t* chunks_out,
              int64_t* total_out) {
    const int64_t per_block = cpdp::coords_per_block();
    const size_t sp = esize(param_dt);
    std::fill(tab, tab + words, (int64_t)0);
    int64_t* start = tab + cpdp::kPlanHeaderWords;
    int64_t* cnt = start + (n + 1);
    int64_t* tp = cnt + n;
    int64_t* tm = tp + (int64_t)W * n;
    int64_t* tv = tm + (int64_t)W * n;
    int64_t* tg = tv + (int64_t)W * n;
    int64_t* ts = tg + (int64_t)W * n;
    int64_t* ta = ts + n;
    size_t nr = 0;
    auto add = [&](const void* p, int64_t elems, size_t es) -> int {
        if (p == nullptr) return CPDP_ERR_NULL;
        if (!aligned16(p)) return CPDP_ERR_MISALIGNED;
        const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
        const uintptr_t hi = lo + (uintptr_t)(elems * (int64_t)es);
        if (hi < lo) return CPDP_ERR_INVALID_ARG;
        ranges[nr++] = Span(lo, hi);
        return CPDP_OK;
    };
    int64_t chunks = 0, total = 0;
    for (int t = 0; t < n; ++t) {
        const int64_t P = numel[t];
        if (P < 0 || P > kMaxElems) return CPDP_ERR_INVALID_ARG;
        start[t] = chunks;
        cnt[t] = P;
        chunks += (P + per_block - 1) / per_block;
        total += P;
        // W * chunks blocks must fit one launch; checked as the sum grows so
        // that it cannot overflow
        if (chunks > cpdp::kMaxBlocks / W) return CPDP_ERR_INVALID_ARG;
        for (int i = 0; i < W; ++i) {
            const int64_t k = (int64_t)i * n + t;
            tp[k] = (int64_t)reinterpret_cast<uintptr_t>(params[k]);
            tm[k] = (int64_t)reinterpret_cast<uintptr_t>(mom[k]);
            tg[k] = (int64_t)reinterpret_cast<uintptr_t>(grads[k]);
            if (mom2 != nullptr) tv[k] = (int64_t)reinterpret_cast<uintptr_t>(mom2[k]);
            if (P == 0) continue;
            if (int s = add(params[k], P, sp)) return s;
            if (int s = add(mom[k], P, 4)) return s;
            if (int s = add(grads[k], P, 4)) return s;
            if (mom2 != nullptr)
                if (int s = add(mom2[k], P, 4)) return s;
        }
        if (slow_mom != nullptr) ts[t] = (int64_t)reinterpret_cast<uintptr_t>(slow_mom[t]);
        if (anchor != nullptr) ta[t] = (int64_t)reinterpret_cast<uintptr_t>(anchor[t]);
        if (P == 0) continue;
        if (slow_mom != nullptr)
            if (int s = add(slow_mom[t], P, 4)) return s;
        if (anchor != nullptr)
            if (int s = add(anchor[t], P, 4)) return s;
    }
    start[n] = chunks;
    std::sort(ranges, ranges + nr);
    for (size_t k = 1; k < nr; ++k)
        if (ranges[k].first < ranges[k - 1].second) return CPDP_ERR_OVERLAP;
    tab[0] = W;
    tab[1] = n;
    tab[2] = chunks;
    *chunks_out = chunks;
    *total_out = total;
    return CPDP_OK;
}

void set_plan_fields(cpdp_plan* plan, int W, int n, int param_dt, bool has_mom2, bool has_slow,
                     bool has_anchor, int64_t chunks, int64_t total) {
    plan->W = W;
    plan->n_tensors = n;
    plan->param_dt = param_dt;
    plan->has_mom2 = has_mom2;
    plan->has_slow_mom = has_slow;
    plan->has_anchor = has_anchor;
    plan->total_chunks = chunks;
    plan->total_numel = total;
}

int check_plan_args(const cpdp_plan* plan, int W, int n, const int64_t* numel,
                    void* const* params, void* const* mom, void* const* grads, int param_dt) {
    if (plan == nullptr || numel == nullptr || params == nullptr || mom == nullptr ||
        grads == nullptr)
        return CPDP_ERR_NULL;
    if (W < 1 || n < 1 || W > 4096 || n > (1 << 24)) return CPDP_ERR_INVALID_ARG;
    if (!is_dtype(param_dt)) return CPDP_ERR_DTYPE;
    return CPDP_OK;
}

// The static plan tables (cpdp_plan_build_static): host buffers the build
// fills before its copy, and per device the seal of the plan its table
// currently holds.  One lock serialises static builds and seal lookups.
constexpr int kStaticDevices = 64;
std::mutex g_static_mu;
int64_t g_static_words[cpdp::kPlanScratchWords];
Span g_static_ranges[cpdp::kPlanScratchWords];
uint64_t g_static_seal[kStaticDevices];    // seal handed out by the last build (0: none)
uint64_t g_static_fields[kStaticDevices];  // plan_seal() of that build's handle fields
uint64_t g_static_builds = 0;

}  // namespace

int cpdp_plan_build(cpdp_plan* plan, int64_t plan_bytes, int W, int n, const int64_t* numel,
                    void* const* params, void* const* mom, void* const* mom2,
                    void* const* grads, float* const* slow_mom, float* const* anchor,
                    int param_dt) {
    if (int s = check_plan_args(plan, W, n, numel, params, mom, grads, param_dt)) return s;
    if (plan->table == nullptr) return CPDP_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(plan->table) & 7u) != 0) return CPDP_ERR_MISALIGNED;
    // a table the library owns is filled by cpdp_plan_build_static only
    if (cpdp::plan_scratch_device(plan->table) >= 0) return CPDP_ERR_INVALID_ARG;
    const int64_t words = cpdp::plan_words(W, n);
    if (plan_bytes < words * (int64_t)sizeof(int64_t)) return CPDP_ERR_INVALID_ARG;

    std::vector<int64_t> tab((size_t)words, 0);
    std::vector<Span> ranges((size_t)(4 * (int64_t)W * n + 2 * (int64_t)n));
    int64_t chunks = 0, total = 0;
    if (int s = fill_plan(tab.data(), words, ranges.data(), W, n, numel, params, mom, mom2,
                          grads, slow_mom, anchor, param_dt, &chunks, &total))
        return s;
    if (cpdp::upload_plan(plan->table, tab.data(), words) != 0) return CPDP_ERR_HIP;
    set_plan_fields(plan, W, n, param_dt, mom2 != nullptr, slow_mom != nullptr,
                    anchor != nullptr, chunks, total);
    plan->seal = plan_seal(plan);
    return CPDP_OK;
}

int cpdp_plan_build_static(cpdp_plan* plan, int W, int n, const int64_t* numel,
                           void* const* params, void* const* mom, void* const* mom2,
                           void* const* grads, float* const* slow_mom, float* const* anchor,
                           int param_dt) {
    if (int s = check_plan_args(plan, W, n, numel, params, mom, grads, param_dt)) return s;
    const int64_t words = cpdp::plan_words(W, n);
    if (words > cpdp::kPlanScratchWords) return CPDP_ERR_TOO_LARGE;

    std::lock_guard<std::mutex> lock(g_static_mu);
    int64_t chunks = 0, total = 0;
    if (int s = fill_plan(g_static_words, words, g_static_ranges, W, n, numel, params, mom, mom2,
                          grads, slow_mom, anchor, param_dt, &chunks, &total))
        return s;
    void* table = nullptr;
    if (cpdp::plan_scratch(&table) != 0) return CPDP_ERR_HIP;
    const int dev = cpdp::plan_scratch_device(table);
    if (dev < 0 || dev >= kStaticDevices) return CPDP_ERR_HIP;
    // plans built on this device before now stop working from here on, even
    // if the copy below fails: their table is about to change
    g_static_seal[dev] = 0;
    if (cpdp::upload_plan(table, g_static_words, words) != 0) return CPDP_ERR_HIP;
    plan->table = table;
    set_plan_fields(plan, W, n, param_dt, mom2 != nullptr, slow_mom != nullptr,
                    anchor != nullptr, chunks, total);
    // the seal also carries the build count, so a handle from an earlier static
    // build on this device no longer matches
    const uint64_t build = ++g_static_builds;
    const uint64_t fields = plan_seal(plan);
    uint64_t seal = fields ^ (build * 0x9E3779B97F4A7C15ull);
    if (seal == 0) seal = 1;  // 0 marks a device without a valid static plan
    plan->seal = seal;
    g_static_fields[dev] = fields;
    g_static_seal[dev] = seal;
    return CPDP_OK;
}

static int check_plan(const cpdp_plan* plan) {
    if (plan == nullptr || plan->table == nullptr) return CPDP_ERR_NULL;
    if (plan->W < 1 || plan->n_tensors < 1 || plan->total_chunks < 0) return CPDP_ERR_INVALID_ARG;
    if (!is_dtype(plan->param_dt)) return CPDP_ERR_DTYPE;
    return CPDP_OK;
}

// The launch shape and the table layout the kernels assume come from the
// handle, so a step call runs only on the exact fields cpdp_plan_build wrote.
// A plan on a device's static table must carry the seal of that table's last
// static build, with the fields that build wrote.
static int check_seal(const cpdp_plan* plan) {
    const int dev = cpdp::plan_scratch_device(plan->table);
    if (dev >= 0) {
        const uint64_t fields = plan_seal(plan);
        std::lock_guard<std::mutex> lock(g_static_mu);
        return dev < kStaticDevices && g_static_seal[dev] != 0 &&
                       plan->seal == g_static_seal[dev] && fields == g_static_fields[dev]
                   ? CPDP_OK
                   : CPDP_ERR_INVALID_ARG;
    }
    return plan->seal == plan_seal(plan) ? CPDP_OK : CPDP_ERR_INVALID_ARG;
}

int cpdp_state_init_plan(const cpdp_plan* plan, void* stream) {
    if (int s = check_plan(plan)) return s;
    if (!plan->has_anchor) return CPDP_ERR_NULL;
    if (int s = check_seal(plan)) return s;
    if (plan->total_chunks == 0) return CPDP_OK;
    return hip_status(cpdp::launch_state_init_plan(param_kind(plan->param_dt),
                                                   static_cast<const int64_t*>(plan->table),
                                                   plan->W, plan->n_tensors, plan->total_chunks,
                                                   stream));
}

int cpdp_local_step_plan(const cpdp_plan* plan, int K, const cpdp_optimizer* opt, void* stream) {
    if (int s = check_plan(plan)) return s;
    if (K < 1) return CPDP_ERR_INVALID_ARG;
    cpdp::Opt kind;
    cpdp::OptParams o;
    if (int s = make_opt(opt, &kind, &o)) return s;
    if (kind == cpdp::Opt::ADAMW && !plan->has_mom2) return CPDP_ERR_NULL;
    if (int s = check_seal(plan)) return s;
    if (plan->total_chunks == 0) return CPDP_OK;
    return hip_status(cpdp::launch_local_step_plan(kind, o, param_kind(plan->param_dt),
                                                   static_cast<const int64_t*>(plan->table),
                                                   plan->W, plan->n_tensors, plan->total_chunks,
                                                   stream));
}

int cpdp_sync_step_plan(int strategy, const cpdp_plan* plan, int K, const cpdp_optimizer* opt,
                        float beta, float alpha, unsigned flags, void* stream) {
    if (int s = check_plan(plan)) return s;
    if (K < 1) return CPDP_ERR_INVALID_ARG;
    if (!valid_strategy(strategy)) return CPDP_ERR_INVALID_ARG;
    if (flags & ~kKnownFlags) return CPDP_ERR_INVALID_ARG;
    cpdp::Opt kind;
    cpdp::OptParams o;
    if (int s = make_opt(opt, &kind, &o)) return s;
    if (strategy == CPDP_SYNC_CPDP) {
        if (!(beta >= 0.0f && beta < 1.0f)) return CPDP_ERR_INVALID_ARG;
        if (!(finite(alpha) && alpha > 0.0f)) return CPDP_ERR_INVALID_ARG;
        if (!plan->has_slow_mom || !plan->has_anchor) return CPDP_ERR_NULL;
    }
    if (kind == cpdp::Opt::ADAMW && !plan->has_mom2) return CPDP_ERR_NULL;
    if (int s = check_seal(plan)) return s;
    if (plan->total_chunks == 0) return CPDP_OK;
    return hip_status(cpdp::launch_sync_plan(sync_mode(strategy), kind, o, param_kind(plan->param_dt),
                                             static_cast<const int64_t*>(plan->table), plan->W,
                                             plan->n_tensors, plan->total_chunks, beta, alpha,
                                             flags, stream));
}

int64_t cpdp_step_table_bytes(int n_steps) {
    if (n_steps < 1) return 0;
    return cpdp::step_table_bytes(n_steps);
}

int cpdp_step_table_fill(cpdp_step_table* t, int64_t table_bytes, int n_steps,
                         const cpdp_optimizer* opt, const float* beta, const float* alpha) {
    if (t == nullptr || t->table == nullptr || opt == nullptr) return CPDP_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(t->table) & 15u) != 0) return CPDP_ERR_MISALIGNED;
    if (n_steps < 1 || n_steps > (1 << 24)) return CPDP_ERR_INVALID_ARG;
    const int64_t bytes = cpdp::step_table_bytes(n_steps);
    if (table_bytes < bytes) return CPDP_ERR_INVALID_ARG;
    std::vector<unsigned char> host((size_t)bytes, 0);
    int64_t* header = reinterpret_cast<int64_t*>(host.data());
    header[0] = 0;
    header[1] = n_steps;
    auto* entries = reinterpret_cast<cpdp::StepEntry*>(header + cpdp::kStepTableHeaderWords);
    cpdp::Opt first = cpdp::Opt::SGD;
    for (int s = 0; s < n_steps; ++s) {
        cpdp::Opt kind;
        cpdp::OptParams o;
        if (int st = make_opt(&opt[s], &kind, &o)) return st;
        if (s == 0) first = kind;
        else if (kind != first) return CPDP_ERR_INVALID_ARG;
        const float b = beta != nullptr ? beta[s] : 0.0f;
        const float a = alpha != nullptr ? alpha[s] : 1.0f;
        if (!(b >= 0.0f && b < 1.0f)) return CPDP_ERR_INVALID_ARG;
        if (!(finite(a) && a > 0.0f)) return CPDP_ERR_INVALID_ARG;
        entries[s].o = o;
        entries[s].beta = b;
        entries[s].alpha_lr = a * o.lr;  // as the direct launch computes it
    }
    if (cpdp::upload_bytes(t->table, host.data(), bytes) != 0) return CPDP_ERR_HIP;
    t->n_steps = n_steps;
    t->update = first == cpdp::Opt::ADAMW ? 2 : first == cpdp::Opt::SGD_WD ? 1 : 0;
    t->seal = step_table_seal(t);
    return CPDP_OK;
}

int cpdp_step_table_set_position(const cpdp_step_table* t, int64_t position, void* stream) {
    cpdp::Opt kind;
    if (int s = check_step_table(t, &kind)) return s;
    if (position < 0 || position > t->n_steps) return CPDP_ERR_INVALID_ARG;
    return hip_status(
        cpdp::launch_step_table_set(static_cast<int64_t*>(t->table), position, stream));
}

int cpdp_step_table_advance(const cpdp_step_table* t, void* stream) {
    cpdp::Opt kind;
    if (int s = check_step_table(t, &kind)) return s;
    return hip_status(cpdp::launch_step_table_advance(static_cast<int64_t*>(t->table), stream));
}

int cpdp_step_table_position(const cpdp_step_table* t, int64_t* position) {
    cpdp::Opt kind;
    if (int s = check_step_table(t, &kind)) return s;
    if (position == nullptr) return CPDP_ERR_NULL;
    return hip_status(
        cpdp::read_step_table_position(static_cast<const int64_t*>(t->table), position));
}

int cpdp_local_step_table(void* params, void* mom, void* mom2, const void* grads, int W,
                          int64_t P, int64_t ld, int K, const cpdp_step_table* t, int param_dt,
                          void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    cpdp::Opt kind;
    if (int s = check_step_table(t, &kind)) return s;
    if (!is_dtype(param_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(W, P)) return CPDP_ERR_INVALID_ARG;
    const bool adam = kind == cpdp::Opt::ADAMW;
    if (int s = check_local_ptrs(params, mom, mom2, grads, W, P, ld, esize(param_dt), adam))
        return s;
    return hip_status(cpdp::launch_local_step_table(
        kind, param_kind(param_dt), static_cast<const int64_t*>(t->table), params,
        static_cast<float*>(mom), adam ? static_cast<float*>(mom2) : nullptr,
        static_cast<const float*>(grads), W, P, ld, stream));
}

int cpdp_sync_step_table(int strategy, void* params, void* mom, void* mom2, void* grads,
                         float* slow_mom, float* anchor, int W, int64_t P, int64_t ld, int K,
                         const cpdp_step_table* t, unsigned flags, int param_dt, void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (flags & ~kKnownFlags) return CPDP_ERR_INVALID_ARG;
    if (!valid_strategy(strategy)) return CPDP_ERR_INVALID_ARG;
    cpdp::Opt kind;
    if (int s = check_step_table(t, &kind)) return s;
    if (!is_dtype(param_dt)) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    float* slow;
    float* anc;
    void* m2;
    if (int s = check_sync_ptrs(strategy, kind == cpdp::Opt::ADAMW, params, mom, mom2, grads,
                                slow_mom, anchor, W, P, ld, esize(param_dt), &slow, &anc, &m2))
        return s;
    return hip_status(cpdp::launch_sync_table(
        sync_mode(strategy), kind, param_kind(param_dt), static_cast<const int64_t*>(t->table),
        params, static_cast<float*>(mom), static_cast<float*>(m2),
        static_cast<const float*>(grads), slow, anc, W, P, ld, flags, stream));
}

int cpdp_local_step_plan_table(const cpdp_plan* plan, int K, const cpdp_step_table* t,
                               void* stream) {
    if (int s = check_plan(plan)) return s;
    if (K < 1) return CPDP_ERR_INVALID_ARG;
    cpdp::Opt kind;
    if (int s = check_step_table(t, &kind)) return s;
    if (kind == cpdp::Opt::ADAMW && !plan->has_mom2) return CPDP_ERR_NULL;
    if (int s = check_seal(plan)) return s;
    if (plan->total_chunks == 0) return CPDP_OK;
    return hip_status(cpdp::launch_local_step_plan_table(
        kind, param_kind(plan->param_dt), static_cast<const int64_t*>(plan->table), plan->W,
        plan->n_tensors, plan->total_chunks, static_cast<const int64_t*>(t->table), stream));
}

int cpdp_sync_step_plan_table(int strategy, const cpdp_plan* plan, int K,
                              const cpdp_step_table* t, unsigned flags, void* stream) {
    if (int s = check_plan(plan)) return s;
    if (K < 1) return CPDP_ERR_INVALID_ARG;
    if (!valid_strategy(strategy)) return CPDP_ERR_INVALID_ARG;
    if (flags & ~kKnownFlags) return CPDP_ERR_INVALID_ARG;
    cpdp::Opt kind;
    if (int s = check_step_table(t, &kind)) return s;
    if (strategy == CPDP_SYNC_CPDP && (!plan->has_slow_mom || !plan->has_anchor))
        return CPDP_ERR_NULL;
    if (kind == cpdp::Opt::ADAMW && !plan->has_mom2) return CPDP_ERR_NULL;
    if (int s = check_seal(plan)) return s;
    if (plan->total_chunks == 0) return CPDP_OK;
    return hip_status(cpdp::launch_sync_plan_table(
        sync_mode(strategy), kind, param_kind(plan->param_dt),
        static_cast<const int64_t*>(plan->table), plan->W, plan->n_tensors, plan->total_chunks,
        static_cast<const int64_t*>(t->table), flags, stream));
}

int cpdp_count_unsynced(const void* params, const float* anchor, int W, int64_t P, int64_t ld,
                        int param_dt, uint64_t* count, void* stream) {
    if (int s = check_shape(W, P, ld, 1)) return s;
    if (!is_dtype(param_dt)) return CPDP_ERR_DTYPE;
    if (count == nullptr) return CPDP_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(count) & 7u) != 0) return CPDP_ERR_MISALIGNED;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    if (P > 0) {
        const size_t sp = esize(param_dt);
        const void* ptrs[] = {params, anchor, count};
        const Range ranges[] = {rows(params, W, P, ld, sp), vec(anchor, P, 4), vec(count, 1, 8)};
        const size_t row_es[] = {sp, 0, 0};
        if (int s = check_pointers(ptrs, ranges, row_es, 2, ld)) return s;
        // the count may not lie inside either input
        if (overlap(ranges[2], ranges[0]) || overlap(ranges[2], ranges[1])) return CPDP_ERR_OVERLAP;
    }
    return hip_status(cpdp::launch_count_unsynced(param_kind(param_dt), params, anchor, W, P, ld,
                                                  count, stream));
}

int cpdp_is_sync_step(int64_t t, int K, int64_t T) {
    if (t < 1 || K < 1 || T < 0 || (T > 0 && t > T)) return -CPDP_ERR_INVALID_ARG;
    return (t % K == 0 || (T > 0 && t == T)) ? 1 : 0;
}

int cpdp_period_for_epoch(int64_t epoch, int64_t warmup_epochs, int K) {
    if (epoch < 0 || warmup_epochs < 0 || K < 1) return -CPDP_ERR_INVALID_ARG;
    return epoch < warmup_epochs ? 1 : K;
}

float cpdp_lr_at(int64_t step, int64_t total_steps, int64_t warmup_steps, float base_lr,
                 float min_lr) {
    const float nan = std::numeric_limits<float>::quiet_NaN();
    if (step < 0 || step >= total_steps || warmup_steps < 0 || warmup_steps > total_steps)
        return nan;
    if (!(finite(base_lr) && base_lr > 0.0f && finite(min_lr) && min_lr >= 0.0f &&
          min_lr <= base_lr))
        return nan;
    if (step < warmup_steps) return (float)((double)base_lr * (double)(step + 1) / (double)warmup_steps);
    const double span = (double)std::max<int64_t>(1, total_steps - warmup_steps);
    const double frac = (double)(step - warmup_steps) / span;
    const double pi = 3.14159265358979323846;
    return (float)((double)min_lr + ((double)base_lr - (double)min_lr) * 0.5 * (1.0 + std::cos(pi * frac)));
}

float cpdp_linear_scaled_lr(float base_lr, int64_t base_batch, int64_t global_batch) {
    if (!(finite(base_lr) && base_lr > 0.0f) || base_batch < 1 || global_batch < 1)
        return std::numeric_limits<float>::quiet_NaN();
    return (float)((double)base_lr * (double)global_batch / (double)base_batch);
}

const char* cpdp_status_str(int status) {
    switch (status) {
        case CPDP_OK: return "CPDP_OK";
        case CPDP_ERR_INVALID_ARG: return "CPDP_ERR_INVALID_ARG: W, P, ld, K or a hyperparameter out of range";
        case CPDP_ERR_NULL: return "CPDP_ERR_NULL: a required pointer is NULL";
        case CPDP_ERR_MISALIGNED: return "CPDP_ERR_MISALIGNED: pointer or row stride not 16-byte aligned";
        case CPDP_ERR_OVERLAP: return "CPDP_ERR_OVERLAP: argument ranges overlap";
        case CPDP_ERR_DTYPE: return "CPDP_ERR_DTYPE: unsupported storage-type combination";
        case CPDP_ERR_HIP: return "CPDP_ERR_HIP: the HIP runtime rejected the launch";
        case CPDP_ERR_TOO_LARGE:
            return "CPDP_ERR_TOO_LARGE: the plan table exceeds the library's fixed "
                   "CPDP_PLAN_STATIC_BYTES buffer";
        default: return "CPDP: unknown status";
    }
}

}  // extern "C"
