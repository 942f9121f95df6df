// C ABI of the CPDP hot path: argument validation on the host, storage-type
// dispatch, and the kernel launches on the caller's stream.  No HIP call is
// made before every argument has been checked, so an invalid call never
// touches the GPU.  The contract of every entry point is documented in
// include/cpdp.h.
#include "cpdp.h"

#include <cmath>
#include <cstdint>

#include "cpdp_launch.h"

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

}  // namespace

extern "C" {

int cpdp_state_init(const void* theta0, void* params, void* mom, float* slow_mom,
                    float* anchor, int W, int64_t P, int64_t ld, int K, int param_dt,
                    int mom_dt, void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (!is_dtype(param_dt) || mom_dt != CPDP_F32) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt);
    const void* ptrs[] = {theta0, params, mom, slow_mom, anchor};
    const Range ranges[] = {vec(theta0, P, sp), rows(params, W, P, ld, sp),
                            rows(mom, W, P, ld, 4), vec(slow_mom, P, 4), vec(anchor, P, 4)};
    const size_t row_es[] = {0, sp, 4, 0, 0};
    if (int s = check_pointers(ptrs, ranges, row_es, 5, ld)) return s;
    return hip_status(cpdp::launch_state_init(param_kind(param_dt), theta0, params,
                                              static_cast<float*>(mom), slow_mom, anchor, W, P,
                                              ld, stream));
}

int cpdp_local_step(void* params, void* mom, const void* grads, int W, int64_t P, int64_t ld,
                    int K, float lr, float mu, int param_dt, int grad_dt, int mom_dt,
                    void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (int s = check_lr_mu(lr, mu)) return s;
    if (!is_dtype(param_dt) || grad_dt != CPDP_F32 || mom_dt != CPDP_F32) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(W, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt);
    const void* ptrs[] = {params, mom, grads};
    const Range ranges[] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, 4),
                            rows(grads, W, P, ld, 4)};
    const size_t row_es[] = {sp, 4, 4};
    if (int s = check_pointers(ptrs, ranges, row_es, 3, ld)) return s;
    return hip_status(cpdp::launch_local_step(param_kind(param_dt), params,
                                              static_cast<float*>(mom),
                                              static_cast<const float*>(grads), W, P, ld, lr, mu,
                                              stream));
}

int cpdp_reconcile(void* params, void* mom, const void* grads, float* slow_mom, float* anchor,
                   int W, int64_t P, int64_t ld, int K, float lr, float mu, float beta,
                   float alpha, int param_dt, int grad_dt, int mom_dt, void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (int s = check_lr_mu(lr, mu)) return s;
    if (!(beta >= 0.0f && beta < 1.0f)) return CPDP_ERR_INVALID_ARG;
    if (!(finite(alpha) && alpha > 0.0f)) return CPDP_ERR_INVALID_ARG;
    if (!is_dtype(param_dt) || grad_dt != CPDP_F32 || mom_dt != CPDP_F32) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt);
    const void* ptrs[] = {params, mom, grads, slow_mom, anchor};
    const Range ranges[] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, 4),
                            rows(grads, W, P, ld, 4), vec(slow_mom, P, 4), vec(anchor, P, 4)};
    const size_t row_es[] = {sp, 4, 4, 0, 0};
    if (int s = check_pointers(ptrs, ranges, row_es, 5, ld)) return s;
    return hip_status(cpdp::launch_sync(cpdp::Sync::CPDP, param_kind(param_dt), params,
                                        static_cast<float*>(mom), static_cast<const float*>(grads),
                                        slow_mom, anchor, W, P, ld, lr, mu, beta, alpha, stream));
}

int cpdp_localsgd_sync(void* params, void* mom, const void* grads, float* anchor, int W,
                       int64_t P, int64_t ld, int K, float lr, float mu, int param_dt,
                       int grad_dt, int mom_dt, void* stream) {
    if (int s = check_shape(W, P, ld, K)) return s;
    if (int s = check_lr_mu(lr, mu)) return s;
    if (!is_dtype(param_dt) || grad_dt != CPDP_F32 || mom_dt != CPDP_F32) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt);
    // anchor is optional: validate it only when given
    const int n = anchor != nullptr ? 4 : 3;
    const void* ptrs[] = {params, mom, grads, anchor};
    const Range ranges[] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, 4),
                            rows(grads, W, P, ld, 4), vec(anchor, P, 4)};
    const size_t row_es[] = {sp, 4, 4, 0};
    if (int s = check_pointers(ptrs, ranges, row_es, n, ld)) return s;
    return hip_status(cpdp::launch_sync(cpdp::Sync::LocalSGD, param_kind(param_dt), params,
                                        static_cast<float*>(mom), static_cast<const float*>(grads),
                                        nullptr, anchor, W, P, ld, lr, mu, 0.0f, 1.0f, stream));
}

int cpdp_ddp_step(void* params, void* mom, const void* grads, int W, int64_t P, int64_t ld,
                  float lr, float mu, int param_dt, int grad_dt, int mom_dt, void* stream) {
    if (int s = check_shape(W, P, ld, 1)) return s;
    if (int s = check_lr_mu(lr, mu)) return s;
    if (!is_dtype(param_dt) || grad_dt != CPDP_F32 || mom_dt != CPDP_F32) return CPDP_ERR_DTYPE;
    if (P == 0) return CPDP_OK;
    if (!cpdp::grid_fits(1, P)) return CPDP_ERR_INVALID_ARG;
    const size_t sp = esize(param_dt);
    const void* ptrs[] = {params, mom, grads};
    const Range ranges[] = {rows(params, W, P, ld, sp), rows(mom, W, P, ld, 4),
                            rows(grads, W, P, ld, 4)};
    const size_t row_es[] = {sp, 4, 4};
    if (int s = check_pointers(ptrs, ranges, row_es, 3, ld)) return s;
    return hip_status(cpdp::launch_sync(cpdp::Sync::DDP, param_kind(param_dt), params,
                                        static_cast<float*>(mom), static_cast<const float*>(grads),
                                        nullptr, nullptr, W, P, ld, lr, mu, 0.0f, 1.0f, stream));
}

int cpdp_is_sync_step(int64_t t, int K, int64_t T) {
    if (t < 1 || K < 1 || T < 0 || (T > 0 && t > T)) return -CPDP_ERR_INVALID_ARG;
    return (t % K == 0 || (T > 0 && t == T)) ? 1 : 0;
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
        default: return "CPDP: unknown status";
    }
}

}  // extern "C"
