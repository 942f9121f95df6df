/*
 * CPDP oracle: plain, slow CPU reference for the reconcile hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no code, header or constant with the HIP
 * library: it is a second, independent statement of the method.
 *
 * What it computes (Controlled Periodic Data Parallelism with SlowMo):
 *   - initialisation            Algorithm 1 (CPDP with SlowMo), the two
 *                               "Initialize" statements: every worker starts
 *                               from the same parameters, velocity 0,
 *                               reference model = initial parameters.
 *   - local update phase        Sec. 3.2, Eq. (local_update), executed as the
 *                               framework optimizer does it (Sec. 4.2): SGD
 *                               with a per-worker momentum buffer
 *                               (buf <- mu*buf + g; theta <- theta - lr*buf).
 *                               mu = 0 gives Eq. (local_update) exactly.
 *   - synchronization phase     Sec. 3.2 stages 1-2, Sec. 3.3 Eqs. (Delta, v,
 *                               theta_new, broadcast, reference update),
 *                               in the execution order fixed by Sec. 4.2:
 *                               gradient mean -> optimizer step with the mean
 *                               gradient (momentum buffers stay local) ->
 *                               parameter mean -> SlowMo -> copy back.
 *   - baselines of Sec. 5.3     oracle_localsgd_sync (local step, then
 *                               parameter averaging; no gradient AllReduce,
 *                               no SlowMo) and oracle_ddp_step (gradient
 *                               mean and the same step on every worker, no
 *                               averaging), run with the same cadence.
 *   - SlowMo, u-form            u <- beta*u + (ref - avg)/lr,
 *                               new = ref - alpha*lr*u.  With v = -lr*u,
 *                               alpha = 1 and a constant lr this is exactly
 *                               the paper's v <- beta*v + (avg - ref),
 *                               new = ref + v (Sec. 3.3); the v-form is also
 *                               provided (oracle_reconcile_vform).
 *
 * Arithmetic: every value is held in a double.  Stored tensors are rounded to
 * their storage type exactly where the framework implementation writes a
 * tensor (parameters after the optimizer step, momentum buffers, the fp32
 * mean gradient, SlowMo state, reference model).  Rounding is
 * round-to-nearest-even; bf16 rounds the fp32 value (two-step), the way a
 * device holding fp32 intermediates stores bf16.  A storage type of "f64"
 * disables rounding for that family, which turns the oracle into an exact-
 * arithmetic statement of the algorithm (used against rational brute force).
 *
 * Layout: replica i of a per-replica family occupies [i*P, (i+1)*P).  Every
 * coordinate is independent of every other, so any subset of coordinates can
 * be run on its own.
 *
 * Pins (tests check this file against): a hand-derived worked example of
 * Algorithm 1, exact rational brute force, closed forms for constant
 * gradients, reductions to PyTorch's SGD (K = 1 and W = 1), replica-permutation
 * invariance, fixed points, Table 2's synchronisation counts, and a mutation
 * test that plants mistakes in a copy of this file.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* storage types understood by the oracle (its own numbering) */
#define ORACLE_F32 0
#define ORACLE_BF16 1
#define ORACLE_F64 2

static double round_to_f32(double x) { return (double)(float)x; }

/* bf16 = upper half of an fp32 bit pattern, rounded to nearest, ties to even */
static double round_to_bf16(double x) {
    float f = (float)x;
    if (isnan(f)) return (double)f;
    uint32_t b;
    memcpy(&b, &f, sizeof b);
    uint32_t lsb = (b >> 16) & 1u;
    b = (b + 0x7FFFu + lsb) & 0xFFFF0000u;
    memcpy(&f, &b, sizeof f);
    return (double)f;
}

static double store_as(int dt, double x) {
    if (dt == ORACLE_F32) return round_to_f32(x);
    if (dt == ORACLE_BF16) return round_to_bf16(x);
    return x;
}

/* exported so the tests can check the rounding against library conversions */
double oracle_round(int dt, double x) { return store_as(dt, x); }

/*
 * Algorithm 1, initialisation: theta_i <- theta for every worker, SlowMo
 * state <- 0, reference model <- theta.  theta0 is taken as the parameter
 * storage type holds it; the reference model keeps that representable value.
 */
void oracle_state_init(int W, int64_t P, int param_dt, int aux_dt,
                       const double* theta0, double* params, double* mom,
                       double* slow, double* anchor) {
    for (int64_t p = 0; p < P; ++p) {
        double th = store_as(param_dt, theta0[p]);
        for (int i = 0; i < W; ++i) {
            params[(int64_t)i * P + p] = th;
            mom[(int64_t)i * P + p] = 0.0;
        }
        slow[p] = 0.0;
        anchor[p] = store_as(aux_dt, th);
    }
}

/*
 * Local update phase (s_t = 0): each worker steps on its own gradient with
 * its own momentum buffer; no communication.
 */
void oracle_local_step(int W, int64_t P, int param_dt, int mom_dt,
                       double* params, double* mom, const double* grads,
                       double lr, double mu) {
    for (int i = 0; i < W; ++i) {
        for (int64_t p = 0; p < P; ++p) {
            int64_t k = (int64_t)i * P + p;
            double buf = store_as(mom_dt, mu * mom[k] + grads[k]);
            mom[k] = buf;
            params[k] = store_as(param_dt, params[k] - lr * buf);
        }
    }
}

/*
 * Synchronization phase (s_t = 1), u-form SlowMo.
 *   1. gbar = (1/W) sum_i g_i                     (stored in fp32 like .grad)
 *   2. buf_i <- mu*buf_i + gbar; x_i = theta_i - lr*buf_i   (optimizer step)
 *   3. avg = (1/W) sum_i x_i                      (parameter average)
 *   4. u <- beta*u + (ref - avg)/lr
 *   5. new = ref - alpha*lr*u
 *   6. theta_i <- new for all i; ref <- new       (momentum buffers untouched)
 */
void oracle_reconcile(int W, int64_t P, int param_dt, int mom_dt, int aux_dt,
                      double* params, double* mom, const double* grads,
                      double* slow, double* anchor,
                      double lr, double mu, double beta, double alpha) {
    for (int64_t p = 0; p < P; ++p) {
        double gsum = 0.0;
        for (int i = 0; i < W; ++i) gsum += grads[(int64_t)i * P + p];
        double gbar = store_as(aux_dt, gsum / (double)W);

        double xsum = 0.0;
        for (int i = 0; i < W; ++i) {
            int64_t k = (int64_t)i * P + p;
            double buf = store_as(mom_dt, mu * mom[k] + gbar);
            mom[k] = buf;
            double x = store_as(param_dt, params[k] - lr * buf);
            xsum += x;
        }
        double avg = xsum / (double)W;

        double ref = anchor[p];
        double u = store_as(aux_dt, beta * slow[p] + (ref - avg) / lr);
        double fresh = store_as(aux_dt, ref - alpha * lr * u);

        slow[p] = u;
        anchor[p] = fresh;
        for (int i = 0; i < W; ++i)
            params[(int64_t)i * P + p] = store_as(param_dt, fresh);
    }
}

/*
 * Synchronization phase in the paper's own variables (Sec. 3.3):
 *   Delta = avg - ref;  v <- beta*v + Delta;  new = ref + v;
 *   theta_i <- new;  ref <- new.
 * Stages 1-3 are the same as in oracle_reconcile.
 */
void oracle_reconcile_vform(int W, int64_t P, int param_dt, int mom_dt,
                            int aux_dt, double* params, double* mom,
                            const double* grads, double* velocity,
                            double* anchor, double lr, double mu,
                            double beta) {
    for (int64_t p = 0; p < P; ++p) {
        double gsum = 0.0;
        for (int i = 0; i < W; ++i) gsum += grads[(int64_t)i * P + p];
        double gbar = store_as(aux_dt, gsum / (double)W);

        double xsum = 0.0;
        for (int i = 0; i < W; ++i) {
            int64_t k = (int64_t)i * P + p;
            double buf = store_as(mom_dt, mu * mom[k] + gbar);
            mom[k] = buf;
            xsum += store_as(param_dt, params[k] - lr * buf);
        }
        double avg = xsum / (double)W;

        double ref = anchor[p];
        double delta = avg - ref;
        double v = store_as(aux_dt, beta * velocity[p] + delta);
        double fresh = store_as(aux_dt, ref + v);

        velocity[p] = v;
        anchor[p] = fresh;
        for (int i = 0; i < W; ++i)
            params[(int64_t)i * P + p] = store_as(param_dt, fresh);
    }
}

/*
 * LocalSGD synchronisation step (Sec. 5.3, second baseline; Table 2 row
 * "LocalSGD"): no gradient AllReduce and no SlowMo.  Every worker takes its
 * own optimizer step with its local gradient, then the parameters are
 * averaged and the average is copied back into every worker.  The averaged
 * model is also stored in `anchor` (if not NULL) as the reference model.
 * Momentum buffers stay local.
 */
void oracle_localsgd_sync(int W, int64_t P, int param_dt, int mom_dt,
                          int aux_dt, double* params, double* mom,
                          const double* grads, double* anchor, double lr,
                          double mu) {
    for (int64_t p = 0; p < P; ++p) {
        double xsum = 0.0;
        for (int i = 0; i < W; ++i) {
            int64_t k = (int64_t)i * P + p;
            double buf = store_as(mom_dt, mu * mom[k] + grads[k]);
            mom[k] = buf;
            xsum += store_as(param_dt, params[k] - lr * buf);
        }
        double avg = store_as(aux_dt, xsum / (double)W);
        if (anchor) anchor[p] = avg;
        for (int i = 0; i < W; ++i)
            params[(int64_t)i * P + p] = store_as(param_dt, avg);
    }
}

/*
 * Synchronous DDP step (Sec. 3.1 Eqs. for gbar and the update; Sec. 5.3,
 * first baseline): the gradient is averaged over the workers at every step
 * and every worker applies the same optimizer step with it; there is no
 * parameter averaging.  Momentum buffers are per worker (they stay equal when
 * the workers start equal).
 */
void oracle_ddp_step(int W, int64_t P, int param_dt, int mom_dt, int aux_dt,
                     double* params, double* mom, const double* grads,
                     double lr, double mu) {
    for (int64_t p = 0; p < P; ++p) {
        double gsum = 0.0;
        for (int i = 0; i < W; ++i) gsum += grads[(int64_t)i * P + p];
        double gbar = store_as(aux_dt, gsum / (double)W);
        for (int i = 0; i < W; ++i) {
            int64_t k = (int64_t)i * P + p;
            double buf = store_as(mom_dt, mu * mom[k] + gbar);
            mom[k] = buf;
            params[k] = store_as(param_dt, params[k] - lr * buf);
        }
    }
}

/* ------------------------------------------------------------------------
 * General optimizers (Sec. 5.2 / Table 3: SGD with momentum and weight decay
 * for ResNet-50, AdamW for ViT-S), with the optimizer state kept per worker
 * (Sec. 3.2 last paragraph, Sec. 4.2).  Semantics and storage points follow
 * the PyTorch optimizers the paper's implementation calls:
 *   SGD    d = g + wd*theta (stored); buf <- mu*buf + d; theta <- theta - lr*buf
 *   AdamW  theta <- theta*(1 - lr*wd)                  (stored)
 *          m <- b1*m + (1-b1)*g;  v <- b2*v + (1-b2)*g^2
 *          theta <- theta - (lr/(1-b1^t)) * m / (sqrt(v)/sqrt(1-b2^t) + eps)
 * with t the 1-based step count of this update.  The derived scalars
 * 1 - lr*wd, lr/(1-b1^t) and sqrt(1-b2^t) are computed in double and then
 * stored in the gradient storage type (fp32): that is the value an fp32
 * tensor operation of the framework multiplies or divides by.
 * ------------------------------------------------------------------------ */
typedef struct {
    int kind;      /* 0 = SGD, 1 = AdamW */
    double lr;
    double mu;     /* SGD momentum, or AdamW beta1 */
    double beta2;  /* AdamW */
    double eps;    /* AdamW */
    double wd;     /* weight decay: coupled for SGD, decoupled for AdamW */
    int64_t step;  /* AdamW bias-correction step count (1-based) */
} oracle_opt;

static void optimizer_update(const oracle_opt* o, int param_dt, int mom_dt,
                             int grad_dt, double* theta, double* m, double* v,
                             double g) {
    if (o->kind == 0) {
        double d = o->wd != 0.0 ? store_as(grad_dt, g + o->wd * *theta) : g;
        *m = store_as(mom_dt, o->mu * *m + d);
        *theta = store_as(param_dt, *theta - o->lr * *m);
    } else {
        double decay = store_as(grad_dt, 1.0 - o->lr * o->wd);
        double th = o->wd != 0.0 ? store_as(param_dt, *theta * decay) : *theta;
        *m = store_as(mom_dt, o->mu * *m + (1.0 - o->mu) * g);
        *v = store_as(mom_dt, o->beta2 * *v + (1.0 - o->beta2) * g * g);
        double bc1 = 1.0 - pow(o->mu, (double)o->step);
        double bc2 = 1.0 - pow(o->beta2, (double)o->step);
        double step_size = store_as(grad_dt, o->lr / bc1);
        double sqrt_bc2 = store_as(grad_dt, sqrt(bc2));
        double denom = sqrt(*v) / sqrt_bc2 + o->eps;
        *theta = store_as(param_dt, th - step_size * *m / denom);
    }
}

/* local step with a general optimizer; mom2 holds AdamW's second moments;
 * aux_dt is the storage type of gradient-sized temporaries (fp32 like .grad) */
void oracle_local_step_opt(int W, int64_t P, int param_dt, int mom_dt,
                           int aux_dt, double* params, double* mom,
                           double* mom2, const double* grads,
                           const oracle_opt* o) {
    for (int i = 0; i < W; ++i)
        for (int64_t p = 0; p < P; ++p) {
            int64_t k = (int64_t)i * P + p;
            optimizer_update(o, param_dt, mom_dt, aux_dt, &params[k], &mom[k],
                             mom2 ? &mom2[k] : NULL, grads[k]);
        }
}

/*
 * Synchronisation step of a strategy with a general optimizer.
 *   strategy 0 (CPDP): gradient mean, optimizer step with it, parameter mean,
 *                      SlowMo (u-form, beta, alpha), copy-back.
 *   strategy 1 (LocalSGD): optimizer step with the local gradient, parameter
 *                      mean, copy-back (anchor <- mean if anchor != NULL).
 *   strategy 2 (DDP): gradient mean, optimizer step with it; no averaging.
 * The SlowMo step length is the optimizer's lr, as in the SGD reconcile.
 * flags (variants the paper names but does not use):
 *   1  write the gradient mean back into every replica's gradient row, as a
 *      DDP AllReduce leaves it in .grad (CPDP and DDP; LocalSGD has none).
 *   2  optimizer-state reconciliation (Sec. 4.2 "Implication for Optimizer
 *      State", Sec. 7 future work): after the optimizer step every replica's
 *      momentum (and AdamW second moment) is replaced by the replica mean.
 */
void oracle_sync_opt(int strategy, int W, int64_t P, int param_dt, int mom_dt,
                     int aux_dt, double* params, double* mom, double* mom2,
                     double* grads, double* slow, double* anchor,
                     const oracle_opt* o, double beta, double alpha,
                     unsigned flags) {
    for (int64_t p = 0; p < P; ++p) {
        double gbar = 0.0;
        if (strategy != 1) {
            double gsum = 0.0;
            for (int i = 0; i < W; ++i) gsum += grads[(int64_t)i * P + p];
            gbar = store_as(aux_dt, gsum / (double)W);
        }
        double xsum = 0.0;
        for (int i = 0; i < W; ++i) {
            int64_t k = (int64_t)i * P + p;
            optimizer_update(o, param_dt, mom_dt, aux_dt, &params[k], &mom[k],
                             mom2 ? &mom2[k] : NULL,
                             strategy == 1 ? grads[k] : gbar);
            xsum += params[k];
        }
        if ((flags & 1u) && strategy != 1)
            for (int i = 0; i < W; ++i) grads[(int64_t)i * P + p] = gbar;
        if (flags & 2u) {
            double msum = 0.0, vsum = 0.0;
            for (int i = 0; i < W; ++i) {
                msum += mom[(int64_t)i * P + p];
                if (mom2) vsum += mom2[(int64_t)i * P + p];
            }
            for (int i = 0; i < W; ++i) {
                mom[(int64_t)i * P + p] = store_as(mom_dt, msum / (double)W);
                if (mom2) mom2[(int64_t)i * P + p] = store_as(mom_dt, vsum / (double)W);
            }
        }
        if (strategy == 2) continue;
        double avg = xsum / (double)W;
        double fresh;
        if (strategy == 0) {
            double ref = anchor[p];
            double u = store_as(aux_dt, beta * slow[p] + (ref - avg) / o->lr);
            fresh = store_as(aux_dt, ref - alpha * o->lr * u);
            slow[p] = u;
            anchor[p] = fresh;
        } else {
            fresh = store_as(aux_dt, avg);
            if (anchor) anchor[p] = fresh;
        }
        for (int i = 0; i < W; ++i)
            params[(int64_t)i * P + p] = store_as(param_dt, fresh);
    }
}
