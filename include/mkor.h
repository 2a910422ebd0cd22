/*
 * mkor.h - C ABI of the MI355X (gfx950) implementation of MKOR's per-step
 * hot path (arXiv 2306.01685, "MKOR: Momentum-Enabled Kronecker-Factor-Based
 * Optimizer Using Rank-1 Updates").
 *
 * For every layer of a grouped list the library runs, on the caller's HIP
 * stream, the second-order branch of Algorithm 1 with the rank-1 means handed
 * in as inputs:
 *
 *   1. norm-based stabiliser of each inverse factor   (Algorithm 1, the two
 *      stabilisation lines; Eq. 9-11; "Exploding Gradients Problem")
 *   2. momentum rank-1 Sherman-Morrison update of each inverse factor
 *      (Algorithm 1, SM-based factor inversion; Eq. 4-7)
 *   3. preconditioning dW_hat = Linv * G * Rinv with the updated factors
 *      (Algorithm 1, precondition line; Eq. 2)
 *   4. rescaling dW = (||G||_F / ||dW_hat||_F) * dW_hat
 *      (Algorithm 1, rescale line; "Rescaling Gradients")
 *   5. first-order layers: dW = G (Algorithm 1, else-branch)
 *
 * Orientation.  The gradient G of a layer is stored d_in x d_out, row-major.
 * Linv is d_in x d_in and is driven by the mean activation a (length d_in);
 * Rinv is d_out x d_out and is driven by the mean output gradient g (length
 * d_out).  The paper writes the transposed gradient; since both factors are
 * symmetric the two forms are the same update.
 *
 * Update of one factor P with vector x (both sides use the same rule):
 *   nu    = ||P||              (induced infinity norm = max abs row sum, or
 *                               max |entry|, see mkor_params.norm_kind)
 *   P_hat = zeta P + (1 - zeta) I   if nu > eps (strict),  else P
 *   u     = P_hat x,  s = x^T u
 *   MKOR_SM_EXACT:     P <- (1/gamma) (P_hat - k u u^T),
 *                      k = (1 - gamma) / (gamma + (1 - gamma) s)
 *                      (the Sherman-Morrison inverse of the momentum
 *                      accumulation M_t = gamma M_hat_{t-1} + (1 - gamma) x x^T
 *                      of Eq. 4/5; the default)
 *   MKOR_SM_PAPER_EQ6: P <- gamma P_hat
 *                            + (1 - gamma) / (gamma^2 (1 + gamma (1 - gamma) s)) u u^T
 *                      (Eq. 6/7 exactly as printed, which is not the inverse
 *                      of Eq. 4/5; kept as an option)
 *
 * Factor state.  The library carries each inverse factor as its caller
 * buffer S plus one pending rank-1 term kept in the workspace:
 *     current factor  P = c1 S + c2 I + sgn w w^T.
 * A step streams every factor once: it first writes the previous step's
 * pending term into S, computes the norm and the matrix-vector product of the
 * stabiliser and SM update on those values, and leaves this step's update as
 * the new pending term; the preconditioning applies that term while it loads
 * the factor, so it multiplies with the updated factor.  Results are the same
 * values a write-back after every update would give (element for element the
 * same roundings).  The factor of a split-path layer's first GEMM (Rinv, or
 * Linv when G is bf16 and d_in > d_out) is written only every other step: the
 * step in between leaves it in S with two pending terms, evaluated one after
 * the other with the same roundings, so the factor values are unchanged; the
 * preconditioning applies both algebraically, so dW matches a write-back
 * after every step to rounding, and bit for bit after mkor_sync_factors.
 * Consequently, after mkor_step or mkor_update_factors the buffers Linv and
 * Rinv hold the factors as of the previous update or the one before;
 * mkor_sync_factors writes the current factors into them.  Call it before
 * reading, saving or modifying Linv / Rinv, and before mkor_plan_destroy if
 * the factors are to be kept.  A new plan starts with no pending term.
 * With bf16 factors (factor_dtype) S is the bf16-rounded factor: writing a
 * pending term into S rounds it to bf16, and the next update's norm and
 * matrix-vector product use the rounded values, while the preconditioning
 * multiplies with the updated factor before that rounding (c1 S + c2 I +
 * sgn w w^T, evaluated in fp32).  So with bf16 factors a mkor_sync_factors
 * between an update and a preconditioning changes the preconditioning: it
 * then uses the rounded factor.
 *
 * Memory and ownership.
 *   - Every buffer named in mkor_layer, and the workspace, is device memory
 *     owned by the caller.  The library never allocates or frees device
 *     memory; its only allocation is the host-side mkor_plan object.
 *   - Matrices are dense, row-major, contiguous (leading dimension = row
 *     length).  Every pointer must be 16-byte aligned; the workspace must be
 *     256-byte aligned.
 *   - Pointers are captured by mkor_plan_create.  Before each step the
 *     caller refills a, g and G in place; Linv and Rinv are updated in place
 *     (see "Factor state") and must hold symmetric matrices (initially I in
 *     the paper).
 *   - Writable buffers (Linv, Rinv, dW, stats) must not overlap any other
 *     buffer of any layer or the workspace.  Read-only inputs may be shared.
 *
 * Errors.  Every int-returning call returns MKOR_OK (0) or a negative status.
 * All argument checks run on the host before the first HIP call of a call.
 * Execution is asynchronous on `stream` (a hipStream_t passed as void*; NULL
 * is the default stream); device-side faults surface at the caller's next
 * synchronisation.  No call blocks on the device, and none prints.
 * mkor_last_error() returns a thread-local text describing the last failure.
 *
 * Calls that share a plan (or a workspace) must not run concurrently.
 */
#ifndef MKOR_H
#define MKOR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MKOR_ABI_VERSION 10

/* status codes */
#define MKOR_OK                   0
#define MKOR_INVALID_ARG         -1  /* null pointer, bad size, bad parameter, aliasing, misalignment */
#define MKOR_WORKSPACE_TOO_SMALL -2
#define MKOR_UNSUPPORTED         -3  /* e.g. an unknown gradient dtype */
#define MKOR_HIP_ERROR           -4  /* a HIP runtime call or kernel launch failed */

/* mkor_params.sm_variant */
#define MKOR_SM_EXACT      0
#define MKOR_SM_PAPER_EQ6  1
/* mkor_params.norm_kind */
#define MKOR_NORM_INF      0   /* max_i sum_j |P_ij| */
#define MKOR_NORM_MAXABS   1   /* max_ij |P_ij| */
/* mkor_layer.grad_dtype */
#define MKOR_DTYPE_F32     0
#define MKOR_DTYPE_BF16    1

/* kernels of one step, in launch order (mkor_run_stage) */
#define MKOR_STAGE_MEANS      0   /* a, g = row means of A, Gout (layers with rows > 0) */
#define MKOR_STAGE_SM_PASS    1   /* write pending term(s) into S (a lazy factor's: every other
                                     step); u_raw = P x, norm and s partials */
#define MKOR_STAGE_SM_FINALIZE 2  /* stabiliser decision, new pending rank-1 term */
#define MKOR_STAGE_GEMM_PREP  3   /* operands of the bf16 MFMA paths: bf16 copy of an fp32 G
                                     (bf16 factors), G^T (split path, bf16 G, d_in > d_out),
                                     (Q w) and ||G||^2 partials of the split path's first GEMM */
#define MKOR_STAGE_GEMM_XT    4   /* first GEMM: X^T = (Linv G)^T (fp32 MFMA), Y^T = Rinv G^T
                                     (bf16 MFMA paths) or X = Linv G (split path, bf16 G,
                                     d_in > d_out), ||G||^2 partials (the other paths) */
#define MKOR_STAGE_GEMM_DW    5   /* second GEMM: dW_hat = X Rinv or Linv Y, ||dW_hat||^2 partials */
#define MKOR_STAGE_RESCALE    6   /* rescale / first-order pass-through */
#define MKOR_NUM_STAGES       7

/* mkor_layer.gemm_path: how the preconditioning GEMMs of a layer with fp32
 * factors multiply.  Both paths give fp32 results to fp32 accuracy. */
#define MKOR_GEMM_AUTO     0   /* SPLIT where it applies, else FP32 */
#define MKOR_GEMM_FP32     1   /* fp32 MFMA (v_mfma_f32_32x32x2_f32), any d_in, d_out */
#define MKOR_GEMM_SPLIT    2   /* bf16 MFMA on an exact three-way bf16 split of each fp32
                                  operand (x = h + m + l), the three smallest of the nine
                                  partial products (below 2^-23 |x x'|) left out; needs
                                  d_in and d_out multiples of 64; exact for operand
                                  magnitudes in [2^-110, 3.396e38) */

/* largest supported d_in / d_out, and token rows of A / Gout */
#define MKOR_MAX_DIM       32768
#define MKOR_MAX_ROWS      (1 << 26)
#define MKOR_MAX_RANK      4
/* device workspace bytes mkor_step_noalloc can use (one array per GPU) */
#define MKOR_NOALLOC_MAX_BYTES (64u << 20)

typedef struct mkor_params {
    float   gamma;            /* momentum of Eq. 4/5, 0 < gamma < 1 */
    float   zeta;             /* stabiliser blend of Eq. 9/10, 0 < zeta <= 1 */
    float   stab_eps;         /* stabiliser threshold, >= 0; +INFINITY turns it off */
    int32_t norm_kind;        /* MKOR_NORM_INF or MKOR_NORM_MAXABS */
    int32_t sm_variant;       /* MKOR_SM_EXACT (default) or MKOR_SM_PAPER_EQ6 */
    int32_t rescale;          /* 1: rescale line of Algorithm 1 on; 0: dW = dW_hat */
    int32_t guard_nonfinite;  /* 1: a factor whose norm, s or update coefficient is
                                 not finite is left unchanged (and flagged in stats);
                                 0: non-finite values propagate */
} mkor_params;

/* mkor_opt_params.kind */
#define MKOR_OPT_SGD   1   /* d = dW + wd W, m = mu m + d, W -= lr m */
#define MKOR_OPT_LAMB  2   /* layer-wise adaptive moments, see mkor_step_opt */

/* Backend optimizer step fused with the rescale (mkor_step_opt). */
typedef struct mkor_opt_params {
    int32_t kind;          /* MKOR_OPT_SGD or MKOR_OPT_LAMB */
    int32_t step;          /* LAMB: t >= 1, the step count of the bias corrections */
    float   lr;            /* >= 0 */
    float   momentum;      /* SGD: 0 <= mu < 1 */
    float   beta1, beta2;  /* LAMB: 0 <= b < 1 */
    float   eps;           /* LAMB: > 0 */
    float   weight_decay;  /* >= 0 */
    int32_t store_dw;      /* 1: also write the rescaled dW into mkor_layer.dW
                              (layers without W always get dW) */
    int32_t reserved;      /* must be 0 */
} mkor_opt_params;

typedef struct mkor_layer {
    int32_t      d_in, d_out;   /* 1 .. MKOR_MAX_DIM */
    int32_t      second_order;  /* 1: MKOR branch; 0: dW = G (first-order layer) */
    int32_t      grad_dtype;    /* MKOR_DTYPE_F32 or MKOR_DTYPE_BF16 (element type of G) */
    void*        Linv;          /* d_in x d_in, in/out, factor_dtype elements (unused if second_order = 0) */
    void*        Rinv;          /* d_out x d_out, in/out, factor_dtype elements (unused if second_order = 0) */
    float*       a;             /* d_in x rank, mean activation(s): input, or output when rows > 0;
                                   vector l at a + l * d_in */
    float*       g;             /* d_out x rank, mean output gradient(s), vector l at g + l * d_out
                                   (a and g unused if second_order = 0) */
    const void*  G;             /* d_in x d_out gradient, grad_dtype elements */
    float*       dW;            /* d_in x d_out fp32 output */
    void*        stats;         /* optional device mkor_layer_stats*, may be NULL */
    /* Rank-1 approximation from token rows (Algorithm 1, its first two lines).
     * rows = 0: the caller supplies a and g.  rows > 0 (second-order layers
     * only): each step first sets a = mean of the rows of A and g = mean of
     * the rows of Gout (float64 sums, one fp32 rounding). */
    int32_t      rows;          /* 0 .. MKOR_MAX_ROWS */
    int32_t      act_dtype;     /* MKOR_DTYPE_F32 or MKOR_DTYPE_BF16 (elements of A and Gout) */
    const void*  A;             /* rows x d_in activations, row-major (rows > 0) */
    const void*  Gout;          /* rows x d_out output gradients, row-major (rows > 0) */
    /* Element type of Linv and Rinv.  MKOR_DTYPE_F32: fp32 factors (the
     * default), preconditioning as gemm_path selects.  MKOR_DTYPE_BF16: half-precision factors
     * (the paper's half-precision MKOR): the factors are stored in bf16, each
     * update is computed in fp32 from the stored values and rounded to bf16 (to
     * nearest, ties to even), and the preconditioning runs on bf16 MFMA with fp32
     * accumulation as dW_hat = Linv (G Rinv), G and the intermediate G Rinv
     * entering it in bf16.  Needs d_in and d_out to be multiples of 64. */
    int32_t      factor_dtype;
    /* Rank of the update (the paper's extension to higher ranks): 0 or 1 for
     * the rank-1 update; r in 2 .. MKOR_MAX_RANK applies the momentum
     * accumulation M_t = gamma M_hat + (1 - gamma) sum_l x_l x_l^T by r
     * sequential Sherman-Morrison updates, x_l the r vectors in a (Linv) and
     * g (Rinv).  r > 1 needs rows = 0, fp32 factors and, at call time, the
     * MKOR_SM_EXACT variant (MKOR_UNSUPPORTED otherwise).  A rank-r update is
     * written into Linv / Rinv within the step that computes it (one more
     * read and write of the factor), so it leaves no pending term. */
    int32_t      rank;
    /* Backend optimizer state (Algorithm 1, last line: the weights take an
     * optimizer step with dW), used by mkor_step_opt / mkor_precondition_opt
     * only; each d_in x d_out fp32, in/out, NULL when unused.  W: the layer's
     * weights.  opt_m: the SGD momentum buffer, or LAMB's first moment.
     * opt_v: LAMB's second moment.  Moments start at 0. */
    float*       W;
    float*       opt_m;
    float*       opt_v;
    /* MKOR_GEMM_AUTO (0), MKOR_GEMM_FP32 or MKOR_GEMM_SPLIT for fp32 factors;
     * must be MKOR_GEMM_AUTO for bf16 factors and first-order layers. */
    int32_t      gemm_path;
    int32_t      reserved0;     /* must be 0 */
} mkor_layer;

/* Per-layer observability record, written on the device when
 * mkor_layer.stats is not NULL.  Fields of a half that did not run keep their
 * previous contents. */
typedef struct mkor_layer_stats {
    float   nu_L, nu_R;        /* factor norms before this step's update */
    float   s_L, s_R;          /* x^T P_hat x */
    float   norm_G;            /* ||G||_F */
    float   norm_dW_hat;       /* ||Linv G Rinv||_F */
    float   scale;             /* rescale factor applied (1 when rescale = 0) */
    int32_t stab_L, stab_R;    /* 1 if the stabiliser fired */
    int32_t skip_L, skip_R;    /* 1 if nu, s or the coefficient was not finite */
    int32_t nonfinite_scale;   /* 1 if a rescale norm was not finite */
} mkor_layer_stats;

typedef struct mkor_plan mkor_plan;

/* MKOR_ABI_VERSION of the loaded library. */
int mkor_abi_version(void);

/* Static text for a status code. */
const char* mkor_status_string(int status);

/* Thread-local description of the last failure in this thread ("" if none). */
const char* mkor_last_error(void);

/* Checks a parameter block without touching the device. */
int mkor_params_check(const mkor_params* params);

/* Bytes of device workspace a plan over `layers[0..n)` needs (written to
 * *bytes).  Host-only. */
int mkor_workspace_size(const mkor_layer* layers, int32_t n, size_t* bytes);

/* Validates the layer list (sizes, pointers, alignment, aliasing), lays out
 * the workspace and uploads the grouped launch descriptors into it (one
 * synchronous host-to-device copy).  `layers` is copied; the caller may free
 * it afterwards.  n = 0 gives an empty plan whose calls are no-ops. */
int mkor_plan_create(const mkor_layer* layers, int32_t n, void* d_workspace,
                     size_t ws_bytes, mkor_plan** out);

/* Rank-1 means (layers with rows > 0), then stabiliser + SM update of Linv
 * and Rinv of every second-order layer (Algorithm 1, rank-1 approximation,
 * stabilisation and SM lines), in one grouped streaming pass plus one small
 * per-factor launch.  The update is left as the pending term (see "Factor
 * state").  Update frequency f (the paper updates every 10 iterations): call
 * mkor_step on update steps and mkor_precondition on the others, which
 * preconditions with the factors of the last update. */
int mkor_update_factors(mkor_plan* plan, const mkor_params* params, void* stream);

/* Preconditioning with the current factors (buffer + pending term), rescale,
 * and the first-order pass-through (Algorithm 1, precondition, rescale and
 * else lines). */
int mkor_precondition(mkor_plan* plan, const mkor_params* params, void* stream);

/* mkor_update_factors followed by mkor_precondition: one full step. */
int mkor_step(mkor_plan* plan, const mkor_params* params, void* stream);

/* Launches one kernel of a step (MKOR_STAGE_*), for profiling and per-kernel
 * timing.  Launching stages 0..MKOR_NUM_STAGES-1 in order on one stream is
 * exactly mkor_step; a stage launched out of that order reads whatever the
 * workspace holds from earlier launches. */
int mkor_run_stage(mkor_plan* plan, const mkor_params* params, int32_t stage, void* stream);

/* Writes the current value of every inverse factor (buffer + pending term)
 * into its buffer Linv / Rinv and clears the pending terms: one grouped
 * read + write of the factors that have a pending term.  Afterwards the
 * buffers hold exactly the factors the next step starts from.  Asynchronous
 * on `stream`; INVALID_ARG if plan is NULL. */
int mkor_sync_factors(mkor_plan* plan, void* stream);

/* Checks an optimizer parameter block without touching the device. */
int mkor_opt_params_check(const mkor_opt_params* opt);

/* mkor_step with the backend optimizer fused into the rescale (Algorithm 1,
 * rescale and last lines): for every layer with W the rescaled gradient g
 * (g = G for first-order layers) updates W in the same pass that scales it,
 *   MKOR_OPT_SGD:  d = g + wd W,  m = mu m + d,  W = W - lr m;
 *   MKOR_OPT_LAMB: m = b1 m + (1 - b1) g,  v = b2 v + (1 - b2) g^2,
 *                  r = (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps) + wd W,
 *                  W = W - lr (||W||_F / ||r||_F) r   per layer (ratio 1 if a
 *                  norm is 0), as LAMB's authors define it;
 * LAMB takes a second pass over m, v and W for the per-layer ratio.  Layers
 * without W get dW as in mkor_step.  Needs opt_m (SGD) or opt_m and opt_v
 * (LAMB) on every layer with W (INVALID_ARG otherwise). */
int mkor_step_opt(mkor_plan* plan, const mkor_params* params, const mkor_opt_params* opt, void* stream);

/* mkor_precondition with the same fused optimizer step (the steps between
 * factor updates of an update-every-f schedule). */
int mkor_precondition_opt(mkor_plan* plan, const mkor_params* params, const mkor_opt_params* opt,
                          void* stream);

/* ---- MKOR-H (the paper's "Hybrid MKOR" subsection): the second-order
 * branch early in training, the first-order one once the second-order
 * updates no longer speed up the decrease of the loss. */

/* Chooses each layer's branch of Algorithm 1 for the calls that follow on
 * the plan, without a new plan: flags[i] = 1 second-order (stabiliser, factor
 * update, preconditioning, rescale), 0 first-order (dW = G, and with
 * mkor_step_opt the optimizer steps with G; the layer's means, factor update
 * and GEMMs are skipped).  `flags` is a host array of the plan's n entries,
 * read before the call returns.  The mode words reach the workspace by a
 * small kernel launch on `stream`: calls enqueued after it on that stream see
 * them; the caller orders calls on other streams after it.  A layer planned
 * with second_order = 0 has no factors and must stay 0 (MKOR_INVALID_ARG,
 * nothing changed).  While a layer is first-order its factors (buffers and
 * pending terms) and its stats stay as they are; switching it back resumes
 * the updates from those factors.  mkor_sync_factors writes the pending terms
 * of every layer, whatever its mode.  A plan starts with every layer as
 * planned. */
int mkor_set_second_order(mkor_plan* plan, const int32_t* flags, void* stream);

/* *pending = 1 when a factor update ran on the plan since its creation or
 * its last mkor_sync_factors: the Linv / Rinv buffers of rank-1 layers may
 * then lag the current factors (see "Factor state"), and mkor_sync_factors is
 * needed before reading, saving or modifying them; else 0.  Host-side. */
int mkor_factors_pending(const mkor_plan* plan, int32_t* pending);

/* The switching rule (host-side).  The paper bases it on the rate at which
 * the loss decreases and gives no formula; this reading averages the loss
 * over consecutive windows of `window` iterations and, after each closed
 * window k >= max(1, warmup), forms the relative decrease of the window means
 *     r_k = (m_{k-1} - m_k) / |m_{k-1}|      (0 when m_{k-1} = 0);
 * after `patience` consecutive evaluated windows with r_k < threshold the
 * decision turns to first-order for the rest of training (the fallback the
 * paper describes; it never turns back). */
typedef struct mkor_hybrid_params {
    int32_t window;      /* iterations per window, >= 1 (e.g. the factor-update period) */
    int32_t patience;    /* consecutive slow windows before the switch, >= 1 */
    int32_t warmup;      /* closed windows before the first evaluation, >= 1 */
    float   threshold;   /* relative decrease per window below which a window is slow, finite, >= 0 */
} mkor_hybrid_params;

typedef struct mkor_hybrid_state {   /* caller-owned; fields are read-only outside the calls */
    mkor_hybrid_params params;
    double  sum;             /* losses of the open window */
    double  prev_mean;       /* mean loss of the last closed window */
    double  last_rate;       /* r_k of the last closed window (NaN before the second) */
    int64_t observed;        /* losses observed */
    int64_t switched_at;     /* value of `observed` when the decision turned to 0, or -1 */
    int32_t count;           /* losses in the open window */
    int32_t windows;         /* closed windows */
    int32_t slow;            /* consecutive evaluated windows below the threshold */
    int32_t second_order;    /* the decision: 1, then 0 after the switch */
} mkor_hybrid_state;

/* Validates `params` and starts a state (decision 1). */
int mkor_hybrid_init(const mkor_hybrid_params* params, mkor_hybrid_state* state);

/* Adds the loss of one iteration and writes the decision after it to
 * *second_order (may be NULL).  A non-finite loss is rejected
 * (MKOR_INVALID_ARG) and leaves the state unchanged. */
int mkor_hybrid_observe(mkor_hybrid_state* state, float loss, int32_t* second_order);

/* One full step for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * The same as creating a plan over layers[0..n) (a fresh one: no pending
 * term), mkor_step, mkor_sync_factors and mkor_plan_destroy, with the same
 * kernels and results, but with no workspace argument: the workspace lives in
 * a device array of MKOR_NOALLOC_MAX_BYTES that the library holds on each GPU
 * it runs on until the process ends.  The call allocates no device or pinned
 * memory.
 *   - Factors: Linv / Rinv are read, updated and written back within the
 *     call; afterwards they hold the updated factors (nothing is pending).
 *   - Size: a layer list whose mkor_workspace_size exceeds
 *     MKOR_NOALLOC_MAX_BYTES is rejected with MKOR_WORKSPACE_TOO_SMALL
 *     before any device work; use a plan for it.
 *   - Device and stream: the array of the current device (hipGetDevice) is
 *     used; `stream` must belong to that device.  The descriptor tables reach
 *     the array through small stream-ordered kernel launches (1 KiB each).
 *   - Concurrency: every call on one GPU shares that GPU's array and leaves
 *     it holding its own tables and partials.  Calls whose executions overlap
 *     on one GPU (other streams, other host threads) race and give undefined
 *     results: order them on one stream or with events.
 * Validation and errors as for mkor_plan_create and mkor_step. */
int mkor_step_noalloc(const mkor_layer* layers, int32_t n, const mkor_params* params, void* stream);

/* Frees the host-side plan (NULL is allowed).  The workspace stays the
 * caller's. */
void mkor_plan_destroy(mkor_plan* plan);

#ifdef __cplusplus
}
#endif

#endif /* MKOR_H */
