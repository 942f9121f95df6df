/* Exercises every oracle function on tiny arrays, for sanitizer builds of
 * the oracle (tests/test_native_sanitizers.py).  Prints one checksum. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct { int kind; double lr, mu, beta2, eps, wd; int64_t step; } opt_t;
void oracle_state_init(int, int64_t, int, int, const double*, double*, double*, double*, double*);
void oracle_local_step(int, int64_t, int, int, double*, double*, const double*, double, double);
void oracle_reconcile(int, int64_t, int, int, int, double*, double*, const double*, double*, double*, double, double, double, double);
void oracle_reconcile_vform(int, int64_t, int, int, int, double*, double*, const double*, double*, double*, double, double, double);
void oracle_localsgd_sync(int, int64_t, int, int, int, double*, double*, const double*, double*, double, double);
void oracle_ddp_step(int, int64_t, int, int, int, double*, double*, const double*, double, double);
void oracle_local_step_opt(int, int64_t, int, int, int, double*, double*, double*, const double*, const opt_t*);
void oracle_sync_opt(int, int, int64_t, int, int, int, double*, double*, double*, double*, double*, double*, const opt_t*, double, double, unsigned);
double oracle_round(int, double);

int main(void) {
    enum { W = 5, P = 7 };
    double th0[P], params[W * P], mom[W * P], mom2[W * P], g[W * P], slow[P], anchor[P];
    for (int p = 0; p < P; ++p) th0[p] = 0.01 * (p - 3);
    for (int k = 0; k < W * P; ++k) { g[k] = 0.001 * ((k * 7) % 11 - 5); mom2[k] = 0.0; }
    double sum = 0.0;
    for (int dt = 0; dt < 3; ++dt) {
        oracle_state_init(W, P, dt, 0, th0, params, mom, slow, anchor);
        oracle_local_step(W, P, dt, 0, params, mom, g, 0.1, 0.9);
        oracle_reconcile(W, P, dt, 0, 0, params, mom, g, slow, anchor, 0.1, 0.9, 0.5, 1.0);
        oracle_reconcile_vform(W, P, dt, 0, 0, params, mom, g, slow, anchor, 0.1, 0.9, 0.5);
        oracle_localsgd_sync(W, P, dt, 0, 0, params, mom, g, anchor, 0.1, 0.9);
        oracle_localsgd_sync(W, P, dt, 0, 0, params, mom, g, NULL, 0.1, 0.9);
        oracle_ddp_step(W, P, dt, 0, 0, params, mom, g, 0.1, 0.9);
        opt_t sgd = {0, 0.1, 0.9, 0.0, 0.0, 5e-4, 0}, adam = {1, 5e-4, 0.9, 0.999, 1e-8, 0.05, 1};
        oracle_local_step_opt(W, P, dt, 0, 0, params, mom, NULL, g, &sgd);
        oracle_local_step_opt(W, P, dt, 0, 0, params, mom, mom2, g, &adam);
        for (int s = 0; s < 3; ++s)
            for (unsigned f = 0; f < 4; ++f) {
                adam.step++;
                oracle_sync_opt(s, W, P, dt, 0, 0, params, mom, mom2, g, slow, anchor, &adam, 0.5, 1.0, f);
            }
        for (int k = 0; k < W * P; ++k) sum += params[k] + mom[k] + mom2[k];
        sum += oracle_round(1, 1.00390625) + oracle_round(0, 0.1);
    }
    printf("oracle checksum %.17g\n", sum);
    return 0;
}
