// Drives every C-ABI entry point through valid and invalid arguments on the
// host (fake, never dereferenced device addresses) and checks the returned
// status and whether a launch was reached.  Built with sanitizers by
// tests/test_native_sanitizers.py; exits non-zero on the first mismatch.
#include <cmath>
#include <cstdint>
#include <cstdio>

#include "cpdp.h"

extern int g_launches;

static int failures = 0;
#define EXPECT(call, want_status, want_launch)                                            \
    do {                                                                                  \
        int before = g_launches;                                                          \
        int got = (call);                                                                 \
        bool launched = g_launches != before;                                             \
        if (got != (want_status) || launched != (want_launch)) {                          \
            std::printf("FAIL line %d: status %d (want %d) launched %d (want %d)\n",      \
                        __LINE__, got, (int)(want_status), (int)launched, (int)(want_launch)); \
            ++failures;                                                                   \
        }                                                                                 \
    } while (0)

int main() {
    auto at = [](int k) { return reinterpret_cast<void*>((uintptr_t)(1ull << 40) + ((uintptr_t)k << 36)); };
    void *pa = at(0), *mo = at(1), *gr = at(2), *m2 = at(6), *th = at(5);
    float *u = static_cast<float*>(at(3)), *an = static_cast<float*>(at(4));
    const int W = 8;
    const int64_t P = 1000, ld = 1024;

    EXPECT(cpdp_reconcile(pa, mo, gr, u, an, W, P, ld, 4, 0.1f, 0.9f, 0.5f, 1.0f, 0, 0, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_reconcile(pa, mo, gr, u, an, W, P, ld, 4, 0.1f, 0.9f, 1.0f, 1.0f, 0, 0, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
    EXPECT(cpdp_reconcile(pa, mo, gr, u, an, W, P, ld, 4, NAN, 0.9f, 0.5f, 1.0f, 0, 0, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
    EXPECT(cpdp_reconcile(pa, pa, gr, u, an, W, P, ld, 4, 0.1f, 0.9f, 0.5f, 1.0f, 0, 0, 0, nullptr), CPDP_ERR_OVERLAP, false);
    EXPECT(cpdp_reconcile(nullptr, mo, gr, u, an, W, P, ld, 4, 0.1f, 0.9f, 0.5f, 1.0f, 0, 0, 0, nullptr), CPDP_ERR_NULL, false);
    EXPECT(cpdp_reconcile(pa, mo, gr, u, an, W, 0, ld, 4, 0.1f, 0.9f, 0.5f, 1.0f, 0, 0, 0, nullptr), CPDP_OK, false);
    EXPECT(cpdp_reconcile(pa, mo, gr, u, an, W, P, ld, 4, 0.1f, 0.9f, 0.5f, 1.0f, 1, 0, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_reconcile(pa, mo, gr, u, an, W, P, 1004, 4, 0.1f, 0.9f, 0.5f, 1.0f, 1, 0, 0, nullptr), CPDP_ERR_MISALIGNED, false);
    EXPECT(cpdp_reconcile(pa, mo, gr, u, an, W, (int64_t)1 << 42, (int64_t)1 << 42, 4, 0.1f, 0.9f, 0.5f, 1.0f, 0, 0, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
    EXPECT(cpdp_reconcile(pa, mo, gr, u, an, 1 << 30, P, (int64_t)1 << 40, 4, 0.1f, 0.9f, 0.5f, 1.0f, 0, 0, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
    EXPECT(cpdp_local_step(pa, mo, gr, W, P, ld, 4, 0.1f, 0.9f, 0, 0, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_local_step(pa, mo, gr, W, P, ld, 4, 0.1f, 1.0f, 0, 0, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
    EXPECT(cpdp_state_init(th, pa, mo, u, an, W, P, ld, 4, 0, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_state_init(th, pa, mo, u, an, W, P, ld, 4, 0, 1, nullptr), CPDP_OK, true);  // bf16 momentum
    EXPECT(cpdp_state_init(th, pa, mo, u, an, W, P, ld, 4, 0, 2, nullptr), CPDP_ERR_DTYPE, false);
    EXPECT(cpdp_localsgd_sync(pa, mo, gr, nullptr, W, P, ld, 4, 0.1f, 0.9f, 0, 0, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_ddp_step(pa, mo, gr, W, P, ld, 0.1f, 0.9f, 0, 0, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_ddp_step(pa, mo, gr, W, P, ld, 0.1f, 0.9f, 0, 1, 0, nullptr), CPDP_OK, true);  // bf16 grads
    EXPECT(cpdp_ddp_step(pa, mo, gr, W, P, ld, 0.1f, 0.9f, 0, 2, 0, nullptr), CPDP_ERR_DTYPE, false);

    cpdp_optimizer adam = {CPDP_OPT_ADAMW, 5e-4f, 0.9f, 0.999f, 1e-8f, 0.05f, 1};
    cpdp_optimizer sgd = {CPDP_OPT_SGD, 0.1f, 0.9f, 0.0f, 0.0f, 5e-4f, 0};
    EXPECT(cpdp_state_init_opt(th, pa, mo, m2, u, an, W, P, ld, 4, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_local_step_opt(pa, mo, m2, gr, W, P, ld, 4, &adam, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_local_step_opt(pa, mo, nullptr, gr, W, P, ld, 4, &adam, 0, nullptr), CPDP_ERR_NULL, false);
    EXPECT(cpdp_local_step_opt(pa, mo, nullptr, gr, W, P, ld, 4, &sgd, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_local_step_opt(pa, mo, m2, gr, W, P, ld, 4, nullptr, 0, nullptr), CPDP_ERR_NULL, false);
    for (int s = 0; s < 3; ++s)
        for (unsigned f = 0; f < 4; ++f)
            EXPECT(cpdp_sync_step_opt(s, pa, mo, m2, gr, u, an, W, P, ld, 4, &adam, 0.5f, 1.0f, f, 0, nullptr), CPDP_OK, true);
    EXPECT(cpdp_sync_step_opt(0, pa, mo, m2, gr, u, an, W, P, ld, 4, &adam, 0.5f, 1.0f, 8u, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
    EXPECT(cpdp_sync_step_opt(3, pa, mo, m2, gr, u, an, W, P, ld, 4, &adam, 0.5f, 1.0f, 0u, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
    EXPECT(cpdp_sync_step_opt(2, pa, mo, nullptr, gr, nullptr, nullptr, W, P, ld, 4, &sgd, 0.5f, 1.0f, 0u, 0, nullptr), CPDP_OK, true);
    adam.step = 0;
    EXPECT(cpdp_local_step_opt(pa, mo, m2, gr, W, P, ld, 4, &adam, 0, nullptr), CPDP_ERR_INVALID_ARG, false);

    {
        // a 3-tensor plan over fake, far-apart addresses (never dereferenced)
        const int n = 3;
        const int64_t numel[n] = {100, 0, 1027};
        void* tp[W * n];
        void* tm[W * n];
        void* tv[W * n];
        void* tg[W * n];
        float* ts[n];
        float* ta[n];
        int k = 0;
        auto far = [&](void) { return reinterpret_cast<void*>((uintptr_t)(1ull << 44) + ((uintptr_t)(k++) << 24)); };
        for (int j = 0; j < W * n; ++j) { tp[j] = far(); tm[j] = far(); tv[j] = far(); tg[j] = far(); }
        for (int t = 0; t < n; ++t) { ts[t] = static_cast<float*>(far()); ta[t] = static_cast<float*>(far()); }
        cpdp_plan plan = {};
        plan.table = at(7);
        const int64_t bytes = cpdp_plan_bytes(W, n);
        EXPECT(cpdp_plan_build(&plan, bytes, W, n, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_OK, false);
        if (plan.total_chunks != 3 || plan.total_numel != 1127) { std::printf("FAIL plan totals\n"); ++failures; }
        EXPECT(cpdp_plan_build(&plan, bytes - 8, W, n, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_ERR_INVALID_ARG, false);
        void* keep = tg[0];
        tg[0] = tm[0];  // tensor 0 is non-empty: its grads would alias its momentum
        EXPECT(cpdp_plan_build(&plan, bytes, W, n, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_ERR_OVERLAP, false);
        tg[0] = keep;
        tg[1] = tm[0];  // tensor 1 is empty: its pointers are not ranges
        EXPECT(cpdp_plan_build(&plan, bytes, W, n, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_OK, false);
        tg[1] = far();
        EXPECT(cpdp_plan_build(&plan, bytes, W, n, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_OK, false);
        EXPECT(cpdp_state_init_plan(&plan, nullptr), CPDP_OK, true);
        EXPECT(cpdp_local_step_plan(&plan, 4, &sgd, nullptr), CPDP_OK, true);
        EXPECT(cpdp_sync_step_plan(0, &plan, 4, &sgd, 0.5f, 1.0f, 3u, nullptr), CPDP_OK, true);
        EXPECT(cpdp_sync_step_plan(0, &plan, 4, &sgd, 1.5f, 1.0f, 0u, nullptr), CPDP_ERR_INVALID_ARG, false);
        // an edited handle no longer matches its seal and never reaches a launch
        plan.W += 1;
        EXPECT(cpdp_local_step_plan(&plan, 4, &sgd, nullptr), CPDP_ERR_INVALID_ARG, false);
        plan.W -= 1;
        plan.total_chunks += 1;
        EXPECT(cpdp_sync_step_plan(0, &plan, 4, &sgd, 0.5f, 1.0f, 0u, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_state_init_plan(&plan, nullptr), CPDP_ERR_INVALID_ARG, false);
        plan.total_chunks -= 1;
        plan.table = at(8);
        EXPECT(cpdp_local_step_plan(&plan, 4, &sgd, nullptr), CPDP_ERR_INVALID_ARG, false);
        plan.table = at(7);
        EXPECT(cpdp_local_step_plan(&plan, 4, &sgd, nullptr), CPDP_OK, true);
        EXPECT(cpdp_plan_build(&plan, bytes, W, n, numel, tp, tm, nullptr, tg, nullptr, nullptr, 0), CPDP_OK, false);
        EXPECT(cpdp_sync_step_plan(0, &plan, 4, &sgd, 0.5f, 1.0f, 0u, nullptr), CPDP_ERR_NULL, false);
        EXPECT(cpdp_sync_step_plan(2, &plan, 4, &sgd, 0.5f, 1.0f, 0u, nullptr), CPDP_OK, true);
        adam.step = 1;
        EXPECT(cpdp_local_step_plan(&plan, 4, &adam, nullptr), CPDP_ERR_NULL, false);

        // the allocation-free build: the library's own table, stale handles
        // rejected, oversized plans refused before any runtime call
        cpdp_plan sp = {};
        EXPECT(cpdp_plan_build_static(&sp, W, n, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_OK, false);
        if (sp.table == nullptr || sp.total_chunks != 3) { std::printf("FAIL static plan\n"); ++failures; }
        EXPECT(cpdp_local_step_plan(&sp, 4, &sgd, nullptr), CPDP_OK, true);
        cpdp_plan sp2 = {};
        EXPECT(cpdp_plan_build_static(&sp2, W, n - 1, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_OK, false);
        EXPECT(cpdp_local_step_plan(&sp, 4, &sgd, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_local_step_plan(&sp2, 4, &sgd, nullptr), CPDP_OK, true);
        cpdp_plan into = sp2;  // cpdp_plan_build never writes the library's table
        EXPECT(cpdp_plan_build(&into, bytes, W, n, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_local_step_plan(&sp2, 4, &sgd, nullptr), CPDP_OK, true);
        sp2.W += 1;  // an edited static handle fails its seal too
        EXPECT(cpdp_local_step_plan(&sp2, 4, &sgd, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_plan_build_static(&sp, 4096, 1024, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_ERR_TOO_LARGE, false);
        EXPECT(cpdp_plan_build_static(nullptr, W, n, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_ERR_NULL, false);
        EXPECT(cpdp_plan_build_static(&sp, W, n, numel, tp, tm, tv, tg, ts, ta, 9), CPDP_ERR_DTYPE, false);
    }

    {
        // step tables over a fake aligned table address (never dereferenced)
        const int n = 4;
        cpdp_optimizer steps[n];
        for (int s = 0; s < n; ++s) {
            steps[s] = adam;
            steps[s].step = s + 1;
            steps[s].lr = 1e-3f * (float)(s + 1);
        }
        const float betas[n] = {0.5f, 0.5f, 0.5f, 0.5f};
        cpdp_step_table tab = {};
        const int64_t tb = cpdp_step_table_bytes(n);
        if (tb != 16 + 64 * n) { std::printf("FAIL step table bytes\n"); ++failures; }
        EXPECT(cpdp_step_table_fill(&tab, tb, n, steps, betas, nullptr), CPDP_ERR_NULL, false);
        tab.table = at(9);
        EXPECT(cpdp_step_table_fill(&tab, tb - 1, n, steps, betas, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_step_table_fill(&tab, tb, 0, steps, betas, nullptr), CPDP_ERR_INVALID_ARG, false);
        steps[2].kind = CPDP_OPT_SGD;  // mixed update rules
        EXPECT(cpdp_step_table_fill(&tab, tb, n, steps, betas, nullptr), CPDP_ERR_INVALID_ARG, false);
        steps[2].kind = CPDP_OPT_ADAMW;
        steps[3].step = 0;  // an entry that a direct call would reject
        EXPECT(cpdp_step_table_fill(&tab, tb, n, steps, betas, nullptr), CPDP_ERR_INVALID_ARG, false);
        steps[3].step = 4;
        const float bad_beta[n] = {0.5f, 1.0f, 0.5f, 0.5f};
        EXPECT(cpdp_step_table_fill(&tab, tb, n, steps, bad_beta, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_step_table_fill(&tab, tb, n, steps, betas, nullptr), CPDP_OK, false);
        if (tab.n_steps != n || tab.update != 2) { std::printf("FAIL step table handle\n"); ++failures; }
        EXPECT(cpdp_local_step_table(pa, mo, m2, gr, W, P, ld, 4, &tab, 0, nullptr), CPDP_OK, true);
        EXPECT(cpdp_local_step_table(pa, mo, nullptr, gr, W, P, ld, 4, &tab, 0, nullptr), CPDP_ERR_NULL, false);
        EXPECT(cpdp_sync_step_table(0, pa, mo, m2, gr, u, an, W, P, ld, 4, &tab, 3u, 0, nullptr), CPDP_OK, true);
        EXPECT(cpdp_sync_step_table(0, pa, mo, m2, gr, nullptr, an, W, P, ld, 4, &tab, 0u, 0, nullptr), CPDP_ERR_NULL, false);
        EXPECT(cpdp_sync_step_table(1, pa, mo, m2, gr, nullptr, nullptr, W, P, ld, 4, &tab, 0u, 0, nullptr), CPDP_OK, true);
        EXPECT(cpdp_sync_step_table(5, pa, mo, m2, gr, u, an, W, P, ld, 4, &tab, 0u, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_sync_step_table(0, pa, mo, m2, gr, u, an, W, P, ld, 4, &tab, 16u, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_step_table_advance(&tab, nullptr), CPDP_OK, true);
        EXPECT(cpdp_step_table_set_position(&tab, 0, nullptr), CPDP_OK, true);
        EXPECT(cpdp_step_table_set_position(&tab, n, nullptr), CPDP_OK, true);
        EXPECT(cpdp_step_table_set_position(&tab, n + 1, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_step_table_set_position(&tab, -1, nullptr), CPDP_ERR_INVALID_ARG, false);
        int64_t pos = -1;
        EXPECT(cpdp_step_table_position(&tab, &pos), CPDP_OK, false);
        EXPECT(cpdp_step_table_position(&tab, nullptr), CPDP_ERR_NULL, false);
        tab.n_steps += 1;  // an edited handle is rejected everywhere
        EXPECT(cpdp_local_step_table(pa, mo, m2, gr, W, P, ld, 4, &tab, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_step_table_advance(&tab, nullptr), CPDP_ERR_INVALID_ARG, false);
        tab.n_steps -= 1;
        tab.update = 0;
        EXPECT(cpdp_sync_step_table(0, pa, mo, m2, gr, u, an, W, P, ld, 4, &tab, 0u, 0, nullptr), CPDP_ERR_INVALID_ARG, false);
        tab.update = 2;
        EXPECT(cpdp_local_step_table(pa, mo, m2, gr, W, P, ld, 4, &tab, 0, nullptr), CPDP_OK, true);

        // plans driven by the step table
        const int nt = 2;
        const int64_t numel[nt] = {100, 7};
        void* tp[W * nt];
        void* tm[W * nt];
        void* tv[W * nt];
        void* tg[W * nt];
        float* ts[nt];
        float* ta[nt];
        int k = 64;
        auto far = [&](void) { return reinterpret_cast<void*>((uintptr_t)(1ull << 44) + ((uintptr_t)(k++) << 24)); };
        for (int j = 0; j < W * nt; ++j) { tp[j] = far(); tm[j] = far(); tv[j] = far(); tg[j] = far(); }
        for (int j = 0; j < nt; ++j) { ts[j] = static_cast<float*>(far()); ta[j] = static_cast<float*>(far()); }
        cpdp_plan plan = {};
        plan.table = at(11);
        EXPECT(cpdp_plan_build(&plan, cpdp_plan_bytes(W, nt), W, nt, numel, tp, tm, tv, tg, ts, ta, 0), CPDP_OK, false);
        EXPECT(cpdp_local_step_plan_table(&plan, 4, &tab, nullptr), CPDP_OK, true);
        EXPECT(cpdp_sync_step_plan_table(0, &plan, 4, &tab, 3u, nullptr), CPDP_OK, true);
        EXPECT(cpdp_sync_step_plan_table(2, &plan, 4, &tab, 0u, nullptr), CPDP_OK, true);
        EXPECT(cpdp_sync_step_plan_table(4, &plan, 4, &tab, 0u, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_sync_step_plan_table(0, &plan, 4, &tab, 64u, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_local_step_plan_table(&plan, 0, &tab, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_local_step_plan_table(&plan, 4, nullptr, nullptr), CPDP_ERR_NULL, false);
        tab.n_steps += 1;
        EXPECT(cpdp_local_step_plan_table(&plan, 4, &tab, nullptr), CPDP_ERR_INVALID_ARG, false);
        tab.n_steps -= 1;
        plan.W += 1;
        EXPECT(cpdp_sync_step_plan_table(1, &plan, 4, &tab, 0u, nullptr), CPDP_ERR_INVALID_ARG, false);
        plan.W -= 1;
        // an AdamW table needs the plan's second moments; CPDP needs u and anchor
        EXPECT(cpdp_plan_build(&plan, cpdp_plan_bytes(W, nt), W, nt, numel, tp, tm, nullptr, tg, nullptr, nullptr, 0), CPDP_OK, false);
        EXPECT(cpdp_local_step_plan_table(&plan, 4, &tab, nullptr), CPDP_ERR_NULL, false);
        EXPECT(cpdp_sync_step_plan_table(0, &plan, 4, &tab, 0u, nullptr), CPDP_ERR_NULL, false);
    }

    {
        uint64_t* cnt = static_cast<uint64_t*>(at(10));
        EXPECT(cpdp_count_unsynced(pa, an, W, P, ld, 0, cnt, nullptr), CPDP_OK, true);
        EXPECT(cpdp_count_unsynced(pa, an, W, 0, ld, 0, cnt, nullptr), CPDP_OK, true);  // zeroes the count
        EXPECT(cpdp_count_unsynced(pa, an, W, P, ld, 0, nullptr, nullptr), CPDP_ERR_NULL, false);
        EXPECT(cpdp_count_unsynced(pa, nullptr, W, P, ld, 0, cnt, nullptr), CPDP_ERR_NULL, false);
        EXPECT(cpdp_count_unsynced(pa, an, W, P, ld, 0, reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(cnt) + 4), nullptr), CPDP_ERR_MISALIGNED, false);
        EXPECT(cpdp_count_unsynced(pa, an, W, P, ld, 0, reinterpret_cast<uint64_t*>(an), nullptr), CPDP_ERR_OVERLAP, false);
        EXPECT(cpdp_count_unsynced(pa, an, W, P, P - 1, 0, cnt, nullptr), CPDP_ERR_INVALID_ARG, false);
        EXPECT(cpdp_count_unsynced(pa, an, W, P, ld, 3, cnt, nullptr), CPDP_ERR_DTYPE, false);
    }

    EXPECT(cpdp_is_sync_step(4, 4, 0), 1, false);
    EXPECT(cpdp_is_sync_step(3, 4, 0), 0, false);
    EXPECT(cpdp_is_sync_step(0, 4, 0), -CPDP_ERR_INVALID_ARG, false);
    EXPECT(cpdp_period_for_epoch(0, 2, 4), 1, false);
    EXPECT(cpdp_period_for_epoch(2, 2, 4), 4, false);
    if (!std::isnan(cpdp_lr_at(10, 10, 0, 0.1f, 0.0f))) { std::printf("FAIL lr_at range\n"); ++failures; }
    for (int s = -3; s < 12; ++s) (void)cpdp_status_str(s);
    std::printf("%s (%d launches)\n", failures ? "FAILED" : "OK", g_launches);
    return failures ? 1 : 0;
}
