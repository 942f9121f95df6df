/*
 * cpdp.h -- C ABI of the Controlled Periodic Data Parallelism (CPDP) reconcile
 * hot path on one AMD Instinct MI355X (gfx950).
 *
 * The method (paper: "Controlled Periodic Synchronization for Efficient
 * Data-Parallel Training"): W worker replicas take independent momentum-SGD
 * steps; every K steps they are reconciled by a gradient mean, a synchronized
 * optimizer step with that mean, a parameter mean, and a SlowMo outer update
 * whose result is copied back to every replica.  On one GPU all W replicas
 * live in HBM and the cross-worker means (the AllReduce of the paper's DDP
 * deployment) are computed inside one kernel.
 *
 * Layout (all entry points)
 *   A per-replica family (params, mom, grads) is W rows of P coordinates with
 *   a row stride of ld elements: replica i, coordinate p is at base[i*ld + p].
 *   Elements p in [P, ld) of every row are never read or written.
 *   slow_mom (u) and anchor (the reference model theta_ref) are P fp32 values.
 *   All pointers are device pointers owned by the caller; the library never
 *   allocates, frees or keeps them.  Each family must start on a 16-byte
 *   boundary and ld * sizeof(element) must be a multiple of 16.  The ranges
 *   of different arguments must not overlap (CPDP_ERR_OVERLAP), and a range
 *   that would run past the end of the address space is CPDP_ERR_INVALID_ARG.
 *
 * Storage types (param_dt, grad_dt, mom_dt): each CPDP_F32 or CPDP_BF16 on
 *   the entry points that take them (cpdp_state_init: params, momentum;
 *   cpdp_local_step, cpdp_reconcile, cpdp_localsgd_sync, cpdp_ddp_step: all
 *   three).  The general-optimizer, plan and step-table entry points take a
 *   param_dt only and use fp32 gradients and optimizer state.  All arithmetic
 *   is fp32: bf16 values are widened exactly on load, and every bf16 value is
 *   rounded to nearest-even when it is written.  The momentum buffer is
 *   rounded to its storage type before the parameter update reads it (the
 *   framework's in-place buffer).  Any other code returns CPDP_ERR_DTYPE.
 *
 * Hyperparameters are fp32: lr > 0 and finite (Sec. 3.1), 0 <= mu < 1,
 *   0 <= beta < 1 (Sec. 3.1), alpha > 0 and finite, K >= 1 (Sec. 3.1).
 *   K is validated but does not enter the arithmetic: the caller decides
 *   which step synchronises (cpdp_is_sync_step).
 *
 * Streams and errors
 *   `stream` is a hipStream_t passed as void* (NULL = the null stream).  Every
 *   device entry point validates all arguments on the host first and returns
 *   a cpdp_status without touching the GPU when one is invalid; otherwise it
 *   enqueues its kernel(s) on `stream` and returns CPDP_OK, or CPDP_ERR_HIP if
 *   the launch failed.  Results are ready when the stream is synchronised.
 *   P = 0 is a valid no-op.  NaN and Inf propagate without being checked.
 *   Calls are reentrant; two calls that touch the same buffers on different
 *   streams without ordering race.
 */
#ifndef CPDP_H
#define CPDP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { CPDP_F32 = 0, CPDP_BF16 = 1 } cpdp_dtype;

typedef enum {
    CPDP_OK = 0,
    CPDP_ERR_INVALID_ARG = 1, /* W, P, ld, K or a hyperparameter out of range */
    CPDP_ERR_NULL = 2,        /* a required pointer is NULL (P > 0)          */
    CPDP_ERR_MISALIGNED = 3,  /* pointer or row stride not 16-byte aligned   */
    CPDP_ERR_OVERLAP = 4,     /* two argument ranges overlap                 */
    CPDP_ERR_DTYPE = 5,       /* unsupported storage-type combination        */
    CPDP_ERR_HIP = 6,         /* the HIP runtime rejected the launch         */
    CPDP_ERR_TOO_LARGE = 7    /* beyond a fixed library buffer
                                 (cpdp_plan_build_static)                    */
} cpdp_status;

/*
 * Initialisation of Algorithm 1 (CPDP with SlowMo): every replica starts from
 * theta0, the SlowMo state starts at 0 and the reference model at theta0.
 *   theta0   [P] in param_dt (read)
 *   params   [W x ld] param_dt  <- theta0 in every row
 *   mom      [W x ld] mom_dt    <- 0
 *   slow_mom [P] fp32           <- 0
 *   anchor   [P] fp32           <- theta0 (widened)
 */
int cpdp_state_init(const void* theta0, void* params, void* mom,
                    float* slow_mom, float* anchor, int W, int64_t P,
                    int64_t ld, int K, int param_dt, int mom_dt, void* stream);

/*
 * Local update phase (Sec. 3.2, Eq. local_update, run as the framework's SGD
 * optimizer with a per-replica momentum buffer, Sec. 4.2), for every replica
 * i and coordinate p < P, with no communication:
 *   mom_i   <- mu * mom_i + grad_i
 *   param_i <- param_i - lr * mom_i
 * grads [W x ld] are read only; params and mom are updated in place.
 */
int cpdp_local_step(void* params, void* mom, const void* grads, int W,
                    int64_t P, int64_t ld, int K, float lr, float mu,
                    int param_dt, int grad_dt, int mom_dt, void* stream);

/*
 * Synchronization phase (Sec. 3.2 stages one and two, Sec. 3.3 SlowMo, in
 * the execution order of Sec. 4.2), in one pass over HBM.  Per coordinate p:
 *   gbar    = (1/W) * sum_i grad_i          (fixed order i = 0..W-1)
 *   mom_i  <- mu * mom_i + gbar             (stored; buffers stay per replica)
 *   x_i     = param_i - lr * mom_i          (rounded to param_dt)
 *   avg     = (1/W) * sum_i x_i             (accumulated as x_i - anchor)
 *   u      <- beta * u + (anchor - avg) / lr
 *   new     = anchor - alpha * lr * u
 *   param_i <- new for every i;  anchor <- new
 * With v = -lr*u and alpha = 1 this is the paper's v <- beta v + (avg - ref),
 * new = ref + v.  grads are read only (the mean is not written back).
 */
int cpdp_reconcile(void* params, void* mom, const void* grads,
                   float* slow_mom, float* anchor, int W, int64_t P,
                   int64_t ld, int K, float lr, float mu, float beta,
                   float alpha, int param_dt, int grad_dt, int mom_dt,
                   void* stream);

/*
 * LocalSGD synchronisation step, the second baseline of Sec. 5.3 (Table 2,
 * one parameter AllReduce per period): no gradient mean and no SlowMo.  Per
 * coordinate p < P:
 *   mom_i   <- mu * mom_i + grad_i          (each replica's own gradient)
 *   x_i      = param_i - lr * mom_i         (rounded to param_dt)
 *   avg      = (1/W) * sum_i x_i
 *   param_i <- avg for every i;  anchor <- avg if anchor != NULL
 * Arguments and layout as cpdp_reconcile; anchor is optional ([P] fp32).
 */
int cpdp_localsgd_sync(void* params, void* mom, const void* grads,
                       float* anchor, int W, int64_t P, int64_t ld, int K,
                       float lr, float mu, int param_dt, int grad_dt,
                       int mom_dt, void* stream);

/*
 * Synchronous DDP step, the first baseline of Sec. 5.3 (Sec. 3.1: gradient
 * AllReduce and identical updates at every step, no parameter averaging).
 * Called at every step (the K = 1 schedule).  Per coordinate p < P:
 *   gbar     = (1/W) * sum_i grad_i         (fixed order i = 0..W-1)
 *   mom_i   <- mu * mom_i + gbar
 *   param_i <- param_i - lr * mom_i
 * Arguments and layout as cpdp_local_step.
 */
int cpdp_ddp_step(void* params, void* mom, const void* grads, int W,
                  int64_t P, int64_t ld, float lr, float mu, int param_dt,
                  int grad_dt, int mom_dt, void* stream);

/* ------------------------------------------------------------------------
 * General optimizers.  The paper trains ResNet-50 with SGD (momentum 0.9,
 * weight decay 5e-4) and ViT-S with AdamW (lr 5e-4, weight decay 0.05)
 * (Sec. 5.2, Table 3); optimizer state always stays per replica and is never
 * averaged (Sec. 3.2 last paragraph, Sec. 4.2).  Update of one replica with
 * the gradient g it uses (its own on local and LocalSGD steps, the replica
 * mean on CPDP and DDP steps), PyTorch semantics:
 *   CPDP_OPT_SGD    d = g + weight_decay * theta
 *                   mom <- momentum * mom + d;   theta <- theta - lr * mom
 *   CPDP_OPT_ADAMW  theta <- theta * (1 - lr * weight_decay)     (stored)
 *                   mom  <- b1 mom + (1 - b1) g;  mom2 <- b2 mom2 + (1 - b2) g^2
 *                   theta <- theta - lr / (1 - b1^step) * mom
 *                                    / (sqrt(mom2) / sqrt(1 - b2^step) + eps)
 *                   with b1 = momentum, b2 = beta2, step = 1-based count of
 *                   this update (it advances on local and sync steps alike).
 * The SlowMo step of a CPDP reconcile uses the optimizer's lr.  Validation:
 * lr > 0 finite, 0 <= momentum < 1, weight_decay >= 0 finite; AdamW also
 * 0 <= beta2 < 1, eps > 0 finite, step >= 1, lr * weight_decay < 1.
 * ------------------------------------------------------------------------ */
typedef enum { CPDP_OPT_SGD = 0, CPDP_OPT_ADAMW = 1 } cpdp_optimizer_kind;

typedef struct cpdp_optimizer {
    int kind;           /* cpdp_optimizer_kind */
    float lr;
    float momentum;     /* SGD momentum, or AdamW beta1 */
    float beta2;        /* AdamW only */
    float eps;          /* AdamW only */
    float weight_decay; /* SGD: added to the gradient; AdamW: decoupled */
    int64_t step;       /* AdamW only: 1-based step count of this update */
} cpdp_optimizer;

typedef enum {
    CPDP_SYNC_CPDP = 0,     /* cpdp_reconcile's computation */
    CPDP_SYNC_LOCALSGD = 1, /* cpdp_localsgd_sync's computation */
    CPDP_SYNC_DDP = 2       /* cpdp_ddp_step's computation */
} cpdp_sync_kind;

/*
 * cpdp_state_init, also zeroing mom2 ([W x ld] fp32, AdamW second moments)
 * when it is not NULL.  Momentum families are fp32.
 */
int cpdp_state_init_opt(const void* theta0, void* params, void* mom,
                        void* mom2, float* slow_mom, float* anchor, int W,
                        int64_t P, int64_t ld, int K, int param_dt,
                        void* stream);

/*
 * Local update phase with a general optimizer.  mom2 ([W x ld] fp32) is
 * required for AdamW and ignored for SGD; grads and mom are fp32.
 * Returns CPDP_ERR_NULL when opt is NULL or AdamW lacks mom2.
 */
int cpdp_local_step_opt(void* params, void* mom, void* mom2,
                        const void* grads, int W, int64_t P, int64_t ld,
                        int K, const cpdp_optimizer* opt, int param_dt,
                        void* stream);

/* Optional variants of a synchronisation step (bit flags). */
enum {
    /* Write the replica-mean gradient into every replica's gradient row, as a
     * DDP AllReduce leaves it in .grad (CPDP and DDP steps; LocalSGD has no
     * gradient mean and ignores the flag).  Costs 4*W bytes per coordinate. */
    CPDP_SYNC_WRITE_GRAD_MEAN = 1,
    /* Optimizer-state reconciliation, the variant Sec. 4.2 names and Sec. 7
     * leaves to future work: after the step every replica's momentum (and
     * AdamW second moment) is replaced by the replica mean.  No extra bytes. */
    CPDP_SYNC_AVERAGE_OPT_STATE = 2
};

/*
 * Synchronisation step of a strategy (cpdp_sync_kind) with a general
 * optimizer, in one pass over HBM.  slow_mom and anchor are required for
 * CPDP_SYNC_CPDP (with beta, alpha as in cpdp_reconcile), anchor is optional
 * for CPDP_SYNC_LOCALSGD, and neither is used by CPDP_SYNC_DDP (beta, alpha
 * are then ignored).  mom2 as in cpdp_local_step_opt.  grads are read only
 * unless flags has CPDP_SYNC_WRITE_GRAD_MEAN.  Unknown flag bits return
 * CPDP_ERR_INVALID_ARG.
 */
int cpdp_sync_step_opt(int strategy, void* params, void* mom, void* mom2,
                       void* grads, float* slow_mom, float* anchor, int W,
                       int64_t P, int64_t ld, int K,
                       const cpdp_optimizer* opt, float beta, float alpha,
                       unsigned flags, int param_dt, void* stream);

/* ------------------------------------------------------------------------
 * Multi-tensor plans.  A framework holds a model as separate parameter
 * tensors (ResNet-50: 161, ViT-S blocks + head: 146), and the paper's
 * implementation updates them tensor by tensor (Sec. 4.2).  A plan describes
 * n_tensors tensors per replica, each family's tensors anywhere in device
 * memory, so one launch per step covers all of them with the same arithmetic
 * as the flat entry points (coordinates are independent, so the result of a
 * tensor equals that of the same values in a flat buffer).
 *
 * The table lives in device memory the caller allocates (cpdp_plan_bytes
 * bytes, 8-byte aligned) and keeps alive while the plan is used;
 * cpdp_plan_build fills it once with a synchronous copy.  The cpdp_plan
 * struct is the host handle the step calls take; its fields are read-only
 * for the caller (they are sealed, see cpdp_plan.seal).
 * ------------------------------------------------------------------------ */
typedef struct cpdp_plan {
    void* table;          /* device memory, >= cpdp_plan_bytes(W, n_tensors)  */
    int W;                /* replicas                                           */
    int n_tensors;
    int param_dt;         /* storage type of every parameter tensor             */
    int has_mom2;         /* second-moment tensors given (AdamW)                */
    int has_slow_mom;     /* SlowMo state tensors given (CPDP)                  */
    int has_anchor;       /* reference-model tensors given (CPDP, LocalSGD)     */
    int64_t total_chunks; /* filled by cpdp_plan_build                          */
    int64_t total_numel;  /* filled by cpdp_plan_build: sum of numel            */
    uint64_t seal;        /* filled by cpdp_plan_build: a hash of every field
                             above; a step call on a handle whose fields no
                             longer match it returns CPDP_ERR_INVALID_ARG, so
                             an edited handle can never make a kernel read the
                             table with the wrong layout                        */
} cpdp_plan;

/* Device bytes of a plan table for W replicas of n_tensors tensors. */
int64_t cpdp_plan_bytes(int W, int n_tensors);

/*
 * Fill plan->table (and plan's total_* fields) from host arrays:
 *   numel[n]                     elements of tensor t (>= 0)
 *   params, mom, grads [W*n]     device pointer of replica i, tensor t at
 *                                [i*n + t]; params in param_dt, the rest fp32
 *   mom2 [W*n] or NULL           AdamW second moments (fp32)
 *   slow_mom, anchor [n] or NULL SlowMo state and reference model (fp32)
 * Every pointer of a non-empty tensor must be non-NULL and 16-byte aligned,
 * and no two of the described ranges may overlap (CPDP_ERR_NULL,
 * CPDP_ERR_MISALIGNED, CPDP_ERR_OVERLAP).  W, n_tensors >= 1 and plan_bytes
 * >= cpdp_plan_bytes, else CPDP_ERR_INVALID_ARG.  The copy is synchronous.
 */
int cpdp_plan_build(cpdp_plan* plan, int64_t plan_bytes, int W, int n_tensors,
                    const int64_t* numel, void* const* params,
                    void* const* mom, void* const* mom2, void* const* grads,
                    float* const* slow_mom, float* const* anchor,
                    int param_dt);

/* Bytes of the library's own plan table on each GPU (cpdp_plan_build_static). */
#define CPDP_PLAN_STATIC_BYTES 262144

/*
 * cpdp_plan_build for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments and checks as cpdp_plan_build, but the table is a fixed
 * array of CPDP_PLAN_STATIC_BYTES that the library keeps on every GPU it runs
 * on until the process ends; plan->table is set to that array's address on
 * the current device (its input value is ignored).  The call allocates
 * nothing, on the device or on the host; it copies the table synchronously,
 * like cpdp_plan_build.
 *   - CPDP_ERR_TOO_LARGE when cpdp_plan_bytes(W, n_tensors) exceeds
 *     CPDP_PLAN_STATIC_BYTES (no HIP call is made); CPDP_ERR_HIP when the
 *     array's address cannot be resolved or the copy fails.
 *   - One table per GPU: a static build replaces the table of the previous
 *     static build on that GPU.  Step calls on a plan from an earlier static
 *     build then return CPDP_ERR_INVALID_ARG instead of reading the new
 *     table; cpdp_plan_build never writes into this array.
 *   - A static build while kernels of an earlier static plan on that GPU may
 *     still be running races with them: synchronize the GPU first.  Static
 *     builds themselves are serialised by the library.
 */
int cpdp_plan_build_static(cpdp_plan* plan, int W, int n_tensors,
                           const int64_t* numel, void* const* params,
                           void* const* mom, void* const* mom2, void* const* grads,
                           float* const* slow_mom, float* const* anchor,
                           int param_dt);

/*
 * Initialisation of Algorithm 1 over a plan: the reference model (the plan's
 * anchor tensors, fp32, filled by the caller with the initial parameters) is
 * copied into every replica (rounded to param_dt), the momentum, second-
 * moment (if any) and SlowMo (if any) tensors are zeroed.  Needs anchor.
 */
int cpdp_state_init_plan(const cpdp_plan* plan, void* stream);

/* cpdp_local_step_opt over every tensor of a plan (one launch). */
int cpdp_local_step_plan(const cpdp_plan* plan, int K,
                         const cpdp_optimizer* opt, void* stream);

/*
 * cpdp_sync_step_opt over every tensor of a plan (one launch).  CPDP needs
 * a plan with slow_mom and anchor; AdamW needs mom2 (else CPDP_ERR_NULL).
 */
int cpdp_sync_step_plan(int strategy, const cpdp_plan* plan, int K,
                        const cpdp_optimizer* opt, float beta, float alpha,
                        unsigned flags, void* stream);

/* ------------------------------------------------------------------------
 * Step tables.  A training loop changes scalars every step: AdamW's bias
 * correction uses the step count, and the learning rate follows a schedule
 * (Sec. 4.3).  The entry points above take those scalars by value, so a HIP
 * graph captured over them replays the captured values.  A step table holds
 * the scalars of n_steps consecutive steps in device memory together with a
 * position word; the *_table entry points read the entry at the position, and
 * cpdp_step_table_advance moves it on.  A graph that captures a period's
 * steps and advances therefore runs the next period's scalars on every replay.
 *
 * The table's memory is the caller's (cpdp_step_table_bytes bytes, 16-byte
 * aligned), kept alive while the table is used; cpdp_step_table_fill writes it
 * once with a synchronous copy and sets the position to 0.  A step whose
 * position is outside [0, n_steps) (the table is used up) changes nothing;
 * cpdp_step_table_advance stops at n_steps, where cpdp_step_table_position
 * reports it.  All steps of a table use one update rule (momentum SGD, SGD
 * with weight decay, or AdamW), fixed when it is filled.
 * ------------------------------------------------------------------------ */
typedef struct cpdp_step_table {
    void* table;     /* device memory, >= cpdp_step_table_bytes(n_steps)      */
    int n_steps;     /* filled by cpdp_step_table_fill                        */
    int update;      /* filled: 0 momentum SGD, 1 SGD with weight decay,
                        2 AdamW                                               */
    uint64_t seal;   /* filled: a hash of the fields above; calls on a handle
                        whose fields changed since return CPDP_ERR_INVALID_ARG */
} cpdp_step_table;

/* Device bytes of a step table of n_steps entries (0 if n_steps < 1). */
int64_t cpdp_step_table_bytes(int n_steps);

/*
 * Fill a step table from host arrays of n_steps entries: opt[s] is the
 * optimizer of step s (its step field is AdamW's 1-based count for that
 * step), beta[s] and alpha[s] the SlowMo coefficients of a CPDP sync at that
 * step (NULL: 0 and 1).  Every entry is validated as cpdp_sync_step_opt
 * validates its arguments, and all entries must select the same update rule
 * (CPDP_ERR_INVALID_ARG otherwise).  Scalars are folded exactly as a direct
 * call folds them, so a table step is bitwise the corresponding direct call.
 * NULL handle, table or opt: CPDP_ERR_NULL; table not 16-byte aligned:
 * CPDP_ERR_MISALIGNED; n_steps < 1 or table_bytes too small:
 * CPDP_ERR_INVALID_ARG.  The copy is synchronous.
 */
int cpdp_step_table_fill(cpdp_step_table* t, int64_t table_bytes, int n_steps,
                         const cpdp_optimizer* opt, const float* beta,
                         const float* alpha);

/* Set the position (0 <= position <= n_steps) with a one-thread kernel on
 * `stream` (no memset or copy, so it may be captured in a graph). */
int cpdp_step_table_set_position(const cpdp_step_table* t, int64_t position,
                                 void* stream);

/* Advance the position by one (not past n_steps), one-thread kernel. */
int cpdp_step_table_advance(const cpdp_step_table* t, void* stream);

/* Synchronous read of the position (waits for the device copy; not for use
 * under graph capture). */
int cpdp_step_table_position(const cpdp_step_table* t, int64_t* position);

/* cpdp_local_step_opt with the scalars of the table's current entry.  mom2 is
 * required for an AdamW table.  Does not advance the position. */
int cpdp_local_step_table(void* params, void* mom, void* mom2, const void* grads,
                          int W, int64_t P, int64_t ld, int K,
                          const cpdp_step_table* t, int param_dt, void* stream);

/* cpdp_sync_step_opt with the scalars (and beta, alpha) of the table's
 * current entry.  Does not advance the position. */
int cpdp_sync_step_table(int strategy, void* params, void* mom, void* mom2,
                         void* grads, float* slow_mom, float* anchor, int W,
                         int64_t P, int64_t ld, int K, const cpdp_step_table* t,
                         unsigned flags, int param_dt, void* stream);

/* cpdp_local_step_plan / cpdp_sync_step_plan with the scalars (and beta,
 * alpha) of a step table's current entry; the update rule is the table's.
 * An AdamW table needs a plan with mom2.  Do not advance the position. */
int cpdp_local_step_plan_table(const cpdp_plan* plan, int K,
                               const cpdp_step_table* t, void* stream);
int cpdp_sync_step_plan_table(int strategy, const cpdp_plan* plan, int K,
                              const cpdp_step_table* t, unsigned flags,
                              void* stream);

/*
 * Failure detection.  Right after a CPDP reconcile or a LocalSGD sync every
 * replica holds the reference model in the parameter storage type (the
 * broadcast of Algorithm 1, Sec. 3.3), and the paper relies on exactly that
 * consistency at every synchronisation and at the epoch end (Sec. 3.1).  This
 * call counts the coordinates p < P at which at least one replica's stored
 * parameter differs bitwise from R(anchor) (a NaN matches a NaN); a nonzero
 * count after a synchronisation means a missed or partial one.
 *   params [W x ld] param_dt, anchor [P] fp32: read only
 *   count  device pointer to one uint64, 8-byte aligned: overwritten (a
 *          one-thread kernel zeroes it first, so the call may be captured in
 *          a graph); read it after synchronising the stream.
 * Validation as cpdp_reconcile for the arguments it shares.
 */
int cpdp_count_unsynced(const void* params, const float* anchor, int W,
                        int64_t P, int64_t ld, int param_dt, uint64_t* count,
                        void* stream);

/*
 * Synchronisation indicator (Sec. 3.2) with the forced synchronisation at the
 * end of an epoch (Sec. 3.1, Sec. 4.2).  Host only, no GPU work.
 *   t: 1-based step counter inside the epoch; K: period (>= 1);
 *   T: steps per epoch, or 0 when there is no epoch boundary.
 * Returns 1 if step t synchronises (t mod K == 0, or t == T), 0 if it is a
 * local step, or -CPDP_ERR_INVALID_ARG if t < 1, K < 1, T < 0 or t > T > 0.
 */
int cpdp_is_sync_step(int64_t t, int K, int64_t T);

/*
 * Synchronisation period in force during 0-based epoch `epoch`: 1 for the
 * first warmup_epochs epochs (CPDP and LocalSGD run fully synchronously during
 * warmup, Sec. 3.4, Sec. 4.3, Sec. 5.3), K afterwards.  Host only.
 * Returns -CPDP_ERR_INVALID_ARG if epoch < 0, warmup_epochs < 0 or K < 1.
 */
int cpdp_period_for_epoch(int64_t epoch, int64_t warmup_epochs, int K);

/*
 * Learning rate of 0-based step `step` of a run of total_steps steps: linear
 * warmup, lr = base_lr * (step + 1) / warmup_steps for step < warmup_steps,
 * then cosine annealing from base_lr to min_lr over the remaining steps,
 * lr = min_lr + (base_lr - min_lr) * (1 + cos(pi * s / S)) / 2 with
 * s = step - warmup_steps, S = max(1, total_steps - warmup_steps)
 * (Sec. 4.3 names cosine annealing with linear warmup; the exact curve is
 * a reading of that passage).  Host only.  Returns NaN if step < 0,
 * step >= total_steps, warmup_steps < 0, warmup_steps > total_steps,
 * base_lr <= 0, min_lr < 0 or min_lr > base_lr.
 */
float cpdp_lr_at(int64_t step, int64_t total_steps, int64_t warmup_steps,
                 float base_lr, float min_lr);

/*
 * Linear learning-rate scaling with the global batch (Sec. 4.3, Sec. 5.3 and
 * Table 4): lr = base_lr * global_batch / base_batch, computed in double and
 * rounded to fp32 (Table 4: base 0.1 at a global batch of 256 gives 0.15,
 * 0.20, 0.30, 0.40 at 384, 512, 768, 1024).  The result is the base_lr a
 * schedule (cpdp_lr_at) starts from.  Host only.  Returns NaN if base_lr is
 * not finite and > 0, or either batch is < 1.
 */
float cpdp_linear_scaled_lr(float base_lr, int64_t base_batch, int64_t global_batch);

/* Static, human-readable name of a status code (never NULL). */
const char* cpdp_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* CPDP_H */
