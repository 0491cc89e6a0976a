/*
 * forge.h -- C ABI of the MI355X (gfx950) fused weight-gradient + optimizer step.
 *
 * The operation (FORGE, Sec. 2.1-2.2, Eq. wgrad, Eq. tile, Algorithm 1): for a linear
 * layer Y = X W^T with weight W [d_out, d_in], activations X [T, d_in] and upstream
 * gradient dY [T, d_out], the weight gradient is G = dY^T X [d_out, d_in].  One call
 * forms G tile by tile in fp32 registers and applies AdamW to each tile right there:
 *
 *     m <- beta1 m + (1 - beta1) G
 *     v <- beta2 v + (1 - beta2) G*G
 *     W <- (1 - lr*wd) W - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 *
 * and writes back only W, m and v; G itself is never stored.
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 * - All tensors are row-major and contiguous.  bf16 is the 16-bit brain float (top half
 *   of an IEEE fp32).  Pointers are device pointers (HIP), owned by the caller; the
 *   library allocates no device memory and keeps no state between calls.
 * - W, m, v (and the int8 scales) are updated in place; X and dY are read only.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).  Calls only
 *   enqueue work: they return once the kernels are launched.  Faults inside a kernel
 *   surface at the caller's next synchronisation.
 * - Arguments are validated on the host before any HIP call, in this order: dtype codes,
 *   shapes (negative -> INVALID_SHAPE, unsupported -> UNSUPPORTED_SHAPE), the empty
 *   problem (d_in == 0 or d_out == 0 returns FORGE_OK with no launch), pointers,
 *   hyper-parameters, alignment, aliasing.  Validation never touches the GPU, so every
 *   error path can be exercised on a machine without one.
 * - Supported shapes: T >= 0 (T == 0 means a zero gradient), d_in and d_out multiples of
 *   8, and every tensor below 2^31 elements.  Ragged tiles (sizes not multiples of the
 *   tile) and ragged token counts are handled inside the kernels.
 * - NaN / Inf inputs are not checked; they propagate.
 * - Precondition (Algorithm 1, first line; the ordering remark of App. A): the layer's
 *   input gradient dX = dY W must already have been computed from the pre-update W.
 */
#ifndef FORGE_H
#define FORGE_H

#include <stdint.h>

/* Entry points are the library's only exported symbols (it is built with hidden default
   visibility). */
#if defined(__GNUC__) || defined(__clang__)
#define FORGE_API __attribute__((visibility("default")))
#else
#define FORGE_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Storage type of the optimizer moments m and v. */
typedef enum {
    FORGE_MOMENT_F32 = 0,  /* fp32 m and v */
    FORGE_MOMENT_BF16 = 1, /* bf16 m and v (round-to-nearest-even stores) */
    FORGE_MOMENT_I8 = 2,   /* int8 codes with one fp32 absmax scale per 256 rows of d_out and
                              per column: m = s_m * q_m, v = (s_v * q_v)^2 (the code stores
                              sqrt(v)); scales are [ceil(d_out/256), d_in] fp32.  The int8
                              block scheme follows App. B (re-quantised every step, second
                              moment kept away from zero: its codes are at least 1 in any
                              non-zero block). */
    FORGE_MOMENT_I8_ROW64 = 3, /* the paper's own int8 layout (App. B): one fp32 absmax scale
                              per 64 consecutive elements of a row (along d_in, a shorter last
                              block when d_in is not a multiple of 64): m = s_m * q_m and
                              v = s_v * q_v (v itself stored); scales are
                              [d_out, ceil(d_in/64)] fp32; same rounding and v floor as above.
                              forge_linear_step(_grouped), the backward calls and forge_adamw
                              accept it; forge_linear_step_opt does not. */
    FORGE_MOMENT_FP8 = 4   /* fp8 (OCP E4M3, largest finite 448, round to nearest even, values
                              clamped into range) codes of m and of sqrt(v), each tensor with
                              one delayed scale s = amax / 448: m = s_m * e4m3(q_m),
                              v = (s_v * e4m3(q_v))^2, and a sqrt(v) > 0 never stored as zero.
                              m_scale and v_scale each point to a ring of 4 fp32 amax slots
                              (16 bytes, caller-owned, all zero for a cold start with zero
                              codes).  Step t decodes with the scale of slot (t-2)%4, encodes
                              with slot (t-1)%4 (a scale of 1 while a slot is 0), records the
                              max |m'| and max sqrt(v') of its own values into slot t%4 and
                              clears slot (t+1)%4: consecutive calls on a tensor must pass
                              consecutive steps.  App. E's per-tensor delayed-scaled fp8 mode.
                              forge_linear_step(_grouped), the backward calls and
                              forge_linear_step_wfp8 accept it; forge_adamw and
                              forge_linear_step_unfused do not. */
} forge_moment_dtype;

/* Element type of a materialised gradient (only the two-kernel path stores one). */
typedef enum { FORGE_GRAD_BF16 = 0, FORGE_GRAD_F32 = 1 } forge_grad_dtype;

typedef enum {
    FORGE_OK = 0,
    FORGE_ERR_NULL_POINTER = 1,      /* a required pointer is NULL */
    FORGE_ERR_INVALID_SHAPE = 2,     /* a negative size */
    FORGE_ERR_UNSUPPORTED_SHAPE = 3, /* d_in or d_out not a multiple of 8, or a tensor >= 2^31 elements */
    FORGE_ERR_INVALID_HYPERPARAM = 4,/* step < 1, beta outside [0,1), eps <= 0, lr < 0, non-finite value */
    FORGE_ERR_INVALID_DTYPE = 5,     /* unknown moment or gradient dtype code */
    FORGE_ERR_MISALIGNED = 6,        /* a tensor pointer not 16-byte aligned */
    FORGE_ERR_ALIASING = 7,          /* an output overlaps another tensor */
    FORGE_ERR_NO_DEVICE = 8,         /* no usable gfx950 device is current */
    FORGE_ERR_LAUNCH = 9,            /* the kernel launch failed (hipGetLastError) */
    FORGE_ERR_INVALID_OPTIMIZER = 10,/* unknown optimizer code */
    FORGE_ERR_SCRATCH_LIMIT = 11     /* the problem needs more than the library's fixed
                                        FORGE_SCRATCH_BYTES buffer (forge_linear_step_unfused_noalloc) */
} forge_status;

/*
 * forge_linear_step -- the fused step (Algorithm 1 over every tile of W).
 *
 *   X        bf16 [T, d_in]            activations (may be NULL when T == 0)
 *   dY       bf16 [T, d_out]           upstream gradient (may be NULL when T == 0)
 *   W        bf16 [d_out, d_in]        weight, in/out
 *   m, v     [d_out, d_in] moments in `moment_dtype` (int8: codes), in/out
 *   m_scale, v_scale   int8 only: fp32 scales in the layout of `moment_dtype`, in/out;
 *            ignored otherwise
 *   step     t >= 1, the step being taken (bias corrections 1 - beta^t)
 *   lr, beta1, beta2, eps, weight_decay   AdamW hyper-parameters (Algorithm 1 notation
 *            eta, beta1, beta2, epsilon, lambda); decay is decoupled: W *= 1 - lr*wd.
 *
 * The gradient is accumulated in fp32 from bf16 products; the update runs in fp32; W is
 * stored to bf16 with round-to-nearest-even.  No gradient byte is written to memory.
 */
FORGE_API forge_status forge_linear_step(const void *X, const void *dY, void *W, void *m, void *v,
                               float *m_scale, float *v_scale, int64_t T, int64_t d_in,
                               int64_t d_out, int32_t moment_dtype, float lr, float beta1,
                               float beta2, float eps, float weight_decay, int64_t step,
                               void *stream);

/* Upper bound on the matrices of one forge_linear_step_grouped call. */
#define FORGE_MAX_GROUP 8

/* One matrix of a grouped step: the per-matrix arguments of forge_linear_step. */
typedef struct forge_matrix {
    const void *X;            /* bf16 [T, d_in] (may be NULL when T == 0) */
    const void *dY;           /* bf16 [T, d_out] (may be NULL when T == 0) */
    void *W;                  /* bf16 [d_out, d_in], in/out */
    void *m, *v;              /* [d_out, d_in] moments in the group's moment dtype, in/out */
    float *m_scale, *v_scale; /* int8 only: fp32 scales of the moment dtype's layout, in/out */
    int64_t d_in, d_out;
} forge_matrix;

/*
 * forge_linear_step_grouped -- forge_linear_step on n independent matrices in one launch.
 *
 * The weight gradients of one layer's projections that share an input and become
 * available together in the backward pass (for example q, k, v, or an MLP's gate and up)
 * can be stepped by one launch: the tiles of all matrices form one grid, so the machine
 * stays full across them.  Each matrix gets exactly the arithmetic of forge_linear_step
 * (the result is bit-identical to n separate calls): Algorithm 1 is tile-local (App. A,
 * Def. 1), so how tiles are grouped into launches does not change any value.
 *
 *   mats     host array of n descriptors, read during the call only (caller-owned)
 *   n        1 <= n <= FORGE_MAX_GROUP, else FORGE_ERR_INVALID_SHAPE
 *   T, moment_dtype, lr, beta1, beta2, eps, weight_decay, step, stream
 *            shared by all matrices, as in forge_linear_step
 *
 * Validation, in this order: the moment dtype; mats (NULL: FORGE_ERR_NULL_POINTER) and n;
 * each matrix in turn with forge_linear_step's shape, input-pointer and state-tensor rules;
 * the hyper-parameters; aliasing -- the state tensors (W, m, v and the scales) of all
 * matrices must be pairwise disjoint and disjoint from every matrix's X and dY
 * (FORGE_ERR_ALIASING; matrices may share X or dY); the device.  Matrices with d_in or
 * d_out == 0 are skipped; if all are empty the call returns FORGE_OK without a launch.
 */
FORGE_API forge_status forge_linear_step_grouped(const forge_matrix *mats, int32_t n, int64_t T,
                                       int32_t moment_dtype, float lr, float beta1, float beta2,
                                       float eps, float weight_decay, int64_t step, void *stream);

/*
 * Update rules of forge_linear_step_opt: the coordinate-wise optimizer families whose state
 * update reads only the gradient's own coordinate, so that they fuse into the tile epilogue
 * like AdamW (App. A, Def. 1; the family table of App. I), and Muon's momentum accumulate.
 * The paper does not restate these rules; each follows the reference implementation it was
 * checked against there (PyTorch's torch.optim for all but Lion, whose rule is that of its
 * authors).  G is the weight gradient, t the step, "gg" the gradient with coupled weight
 * decay added, gg = G + wd W; s1 and s2 are the state tensors.
 *
 *   FORGE_OPT_ADAMW          s1 = m, s2 = v: exactly forge_linear_step (decoupled decay)
 *   FORGE_OPT_SGD            no state: W -= lr gg
 *   FORGE_OPT_SGD_MOMENTUM   s1 = b: b = beta1 b + gg; W -= lr b       (beta1 = momentum)
 *   FORGE_OPT_ADAGRAD        s1 = sum: sum += gg^2; W -= clr gg / (sqrt(sum) + eps),
 *                            clr = lr / (1 + (t - 1) lr_decay)
 *   FORGE_OPT_RMSPROP        s1 = a: a = beta2 a + (1 - beta2) gg^2; W -= lr gg / (sqrt(a) + eps)
 *                            (beta2 = alpha)
 *   FORGE_OPT_LION           s1 = m: W = (1 - lr wd) W - lr sign(beta1 m + (1 - beta1) G);
 *                            m = beta2 m + (1 - beta2) G
 *   FORGE_OPT_NADAM          s1 = m, s2 = v (Adam moments of gg); with mu_i =
 *                            beta1 (1 - 0.5 * 0.96^(i momentum_decay)) and P_t = mu_1 ... mu_t:
 *                            W -= lr [(1 - mu_t)/(1 - P_t) gg + mu_{t+1}/(1 - P_t mu_{t+1}) m]
 *                                 / (sqrt(v / (1 - beta2^t)) + eps)
 *   FORGE_OPT_RADAM          s1 = m, s2 = v (Adam moments of gg); rho_inf = 2/(1 - beta2) - 1,
 *                            rho_t = rho_inf - 2 t beta2^t / (1 - beta2^t); if rho_t > 5:
 *                            W -= lr r (m / (1 - beta1^t)) sqrt(1 - beta2^t) / (sqrt(v) + eps),
 *                            r = sqrt((rho_t-4)(rho_t-2) rho_inf / ((rho_inf-4)(rho_inf-2) rho_t));
 *                            else W -= lr m / (1 - beta1^t)
 *   FORGE_OPT_ADAMAX         s1 = m, s2 = u: m = beta1 m + (1 - beta1) gg;
 *                            u = max(beta2 u, |gg| + eps); W -= lr / (1 - beta1^t) m / u
 *   FORGE_OPT_MUON_ACCUMULATE  s1 = B: B = beta1 B + G (the GEMM's beta; regime 2 of App. A).
 *                            W is neither read nor written (the orthogonalising weight update
 *                            reads B only and runs outside this call).  Over micro-batches of
 *                            one step pass beta1 = mu on the first and 1 on the others.
 */
typedef enum {
    FORGE_OPT_ADAMW = 0,
    FORGE_OPT_SGD = 1,
    FORGE_OPT_SGD_MOMENTUM = 2,
    FORGE_OPT_ADAGRAD = 3,
    FORGE_OPT_RMSPROP = 4,
    FORGE_OPT_LION = 5,
    FORGE_OPT_NADAM = 6,
    FORGE_OPT_RADAM = 7,
    FORGE_OPT_ADAMAX = 8,
    FORGE_OPT_MUON_ACCUMULATE = 9
} forge_optimizer;

/* Hyper-parameters of forge_linear_step_opt; a rule reads only the fields it names above. */
typedef struct forge_hparams {
    float lr;              /* >= 0 */
    float beta1;           /* [0, 1); Muon accumulate: [0, 1] */
    float beta2;           /* [0, 1) */
    float eps;             /* > 0 where used */
    float weight_decay;    /* finite */
    float lr_decay;        /* Adagrad: >= 0 */
    float momentum_decay;  /* NAdam: >= 0 (PyTorch's default is 0.004) */
} forge_hparams;

/*
 * forge_linear_step_opt -- the fused step with update rule `optimizer` on fp32 or bf16 state.
 *
 *   X, dY, T, d_in, d_out, step, stream   as in forge_linear_step
 *   W        bf16 [d_out, d_in], in/out (unused, may be NULL, for FORGE_OPT_MUON_ACCUMULATE)
 *   s1, s2   [d_out, d_in] state tensors in `state_dtype` (FORGE_MOMENT_F32 or _BF16), in/out;
 *            a rule with fewer states ignores the others (they may be NULL)
 *   hp       host pointer, read during the call only
 *
 * The tile mainloop is the one of forge_linear_step; only the epilogue differs, and W, the
 * states and the output roundings (bf16 / fp32, round-to-nearest-even) are handled as there.
 * Errors: FORGE_ERR_INVALID_OPTIMIZER for an unknown code; FORGE_ERR_INVALID_DTYPE for a
 * state dtype other than fp32 / bf16 (int8 moments: forge_linear_step); NULL hp:
 * FORGE_ERR_NULL_POINTER; out-of-range fields the rule reads: FORGE_ERR_INVALID_HYPERPARAM;
 * the other checks as in forge_linear_step.
 */
FORGE_API forge_status forge_linear_step_opt(const void *X, const void *dY, void *W, void *s1, void *s2,
                                             int64_t T, int64_t d_in, int64_t d_out, int32_t optimizer,
                                             int32_t state_dtype, const forge_hparams *hp, int64_t step,
                                             void *stream);

/*
 * forge_linear_step_wfp8 -- forge_linear_step with the weight stored in fp8: W holds OCP
 * E4M3 codes [d_out, d_in] (1 byte each) with a per-tensor delayed scale kept in the 4-slot
 * amax ring `w_amax` (the scheme of FORGE_MOMENT_FP8, applied to max |W'|).  The epilogue
 * decodes W, steps it in fp32 and encodes it again, so that weight quantisation costs no
 * pass of its own (Sec. 3, the FP8 weight and weight+moment recipes).
 *
 *   moment_dtype   FORGE_MOMENT_BF16 (m_amax, v_amax ignored) or FORGE_MOMENT_FP8
 *   other arguments as in forge_linear_step
 *
 * Errors as in forge_linear_step; FORGE_ERR_INVALID_DTYPE for another moment dtype; NULL
 * w_amax: FORGE_ERR_NULL_POINTER.
 */
FORGE_API forge_status forge_linear_step_wfp8(const void *X, const void *dY, void *W, float *w_amax, void *m,
                                              void *v, float *m_amax, float *v_amax, int64_t T, int64_t d_in,
                                              int64_t d_out, int32_t moment_dtype, float lr, float beta1,
                                              float beta2, float eps, float weight_decay, int64_t step,
                                              void *stream);

/*
 * forge_input_grad -- the layer's input gradient dX = dY W (Algorithm 1, first line; the
 * chain rule through Y = X W^T of Eq. fwd).
 *
 *   dY   bf16 [T, d_out]     upstream gradient (may be NULL when T, d_in or d_out is 0)
 *   W    bf16 [d_out, d_in]  weight (may be NULL when T, d_in or d_out is 0)
 *   dX   bf16 [T, d_in]      output, overwritten (may be NULL when T or d_in is 0)
 *
 * Products of bf16 inputs are accumulated in fp32 over d_out and rounded once to bf16
 * (round-to-nearest-even).  d_out == 0 (with T, d_in > 0) fills dX with zeros.  Shape
 * rules as in forge_linear_step; dX must not overlap dY or W (FORGE_ERR_ALIASING).
 */
FORGE_API forge_status forge_input_grad(const void *dY, const void *W, void *dX, int64_t T,
                                        int64_t d_in, int64_t d_out, void *stream);

/*
 * forge_linear_backward -- the layer-level backward of FORGE (Sec. 2.2; Algorithm 1): the
 * input gradient dX = dY W from the weight as it is before the step, then the fused step
 * forge_linear_step, both enqueued on `stream` in that order.  Because the step overwrites
 * W in place, dX has to be read off the pre-update weight (the ordering remark of App. A);
 * stream order guarantees it.  Weights read by more than one backward path within a step
 * (a tied embedding / LM head) must not use this call (same remark).
 *
 *   dX   bf16 [T, d_in], output (may be NULL when T or d_in is 0); other arguments as in
 *        forge_linear_step.
 *
 * Identical to forge_linear_backward_grouped with n == 1 (validation order included):
 * W, m, v end bit-identical to forge_linear_step's, dX bit-identical to forge_input_grad's
 * on the pre-update W.
 */
FORGE_API forge_status forge_linear_backward(const void *X, const void *dY, void *W, void *m, void *v,
                                             float *m_scale, float *v_scale, void *dX, int64_t T,
                                             int64_t d_in, int64_t d_out, int32_t moment_dtype,
                                             float lr, float beta1, float beta2, float eps,
                                             float weight_decay, int64_t step, void *stream);

/*
 * forge_linear_backward_grouped -- the layer-level backward of n projections of one input
 * (for example q, k and v, or an MLP's gate and up): that input's gradient is the sum of
 * their contributions, dX = sum_i dY_i W_i, formed in one launch from the pre-update
 * weights (fp32 accumulation over the concatenated d_out axes, one rounding to bf16), then
 * forge_linear_step_grouped on the n matrices, in stream order.
 *
 *   mats   n descriptors as for forge_linear_step_grouped; all must have the same d_in
 *          (else FORGE_ERR_INVALID_SHAPE); members with d_out == 0 add nothing to dX
 *   dX     bf16 [T, d_in], output (may be NULL when T or d_in is 0)
 *
 * Validation, in this order: the moment dtype; mats and n; equal d_in; then exactly as
 * forge_linear_step_grouped (each matrix, hyper-parameters, aliasing); then dX (NULL:
 * FORGE_ERR_NULL_POINTER, misaligned: FORGE_ERR_MISALIGNED, overlapping any member's X, dY
 * or state tensors: FORGE_ERR_ALIASING); the device.
 */
FORGE_API forge_status forge_linear_backward_grouped(const forge_matrix *mats, int32_t n, int64_t T,
                                                     void *dX, int32_t moment_dtype, float lr,
                                                     float beta1, float beta2, float eps,
                                                     float weight_decay, int64_t step, void *stream);

/*
 * forge_wgrad -- the weight-gradient GEMM alone, storing G = dY^T X (Eq. wgrad) to
 * `G` [d_out, d_in] in `grad_dtype` (bf16 with round-to-nearest-even, or fp32).  This is
 * the first kernel of the two-kernel comparison path and the store-G control of App. D.
 */
FORGE_API forge_status forge_wgrad(const void *X, const void *dY, void *G, int64_t T, int64_t d_in,
                         int64_t d_out, int32_t grad_dtype, void *stream);

/*
 * forge_adamw -- the stand-alone optimizer kernel: one AdamW step (Algorithm 1, state
 * update then weight update) reading a materialised gradient `G` [d_out, d_in] in
 * `grad_dtype`.  Arguments as in forge_linear_step.  G is read only.
 */
FORGE_API forge_status forge_adamw(const void *G, int32_t grad_dtype, void *W, void *m, void *v,
                         float *m_scale, float *v_scale, int64_t d_in, int64_t d_out,
                         int32_t moment_dtype, float lr, float beta1, float beta2, float eps,
                         float weight_decay, int64_t step, void *stream);

/*
 * forge_linear_step_unfused -- the same step as forge_linear_step done the conventional
 * way: forge_wgrad writes G into the caller's workspace `G_ws` (d_out*d_in elements of
 * `grad_dtype`), then forge_adamw consumes it, both on `stream`.  It exists to measure
 * the HBM traffic that fusion removes (Sec. 2.2, "Memory and bandwidth": the gradient's
 * write and read).  With a bf16 workspace the optimizer sees G rounded to bf16 (the
 * truncation discussed in App. B).
 */
FORGE_API forge_status forge_linear_step_unfused(const void *X, const void *dY, void *W, void *m,
                                       void *v, float *m_scale, float *v_scale, int64_t T,
                                       int64_t d_in, int64_t d_out, int32_t moment_dtype,
                                       float lr, float beta1, float beta2, float eps,
                                       float weight_decay, int64_t step, void *G_ws,
                                       int32_t grad_dtype, void *stream);

/* Size in bytes of the library's fixed device buffer (one per device, held from the
   library's load until the process ends). */
#define FORGE_SCRATCH_BYTES (64LL << 20)

/*
 * forge_linear_step_unfused_noalloc -- forge_linear_step_unfused for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation.  The gradient G goes to the library's fixed device buffer of
 * FORGE_SCRATCH_BYTES instead of a caller workspace; the call allocates nothing (no
 * hipMalloc, no allocating library routine) and otherwise behaves as
 * forge_linear_step_unfused with `grad_dtype` for G: the results are bit-identical.
 *
 *   arguments   as in forge_linear_step_unfused, without G_ws
 *
 * Errors: as forge_linear_step_unfused; d_in * d_out * (2 for bf16, 4 for fp32) above
 * FORGE_SCRATCH_BYTES: FORGE_ERR_SCRATCH_LIMIT (checked on the host after the shapes,
 * before any HIP call); FORGE_ERR_LAUNCH if the buffer's device address cannot be obtained.
 * The buffer is shared by every call on a device and keeps the last call's G: calls that
 * overlap on one device (two streams, two host threads) race and must be serialised by the
 * caller.  Nothing needs clearing between calls: the GEMM writes every element of G that
 * the optimizer kernel then reads.  Set-up: the first call on a device looks up the
 * buffer's device address (hipGetSymbolAddress, with that device current); the HIP
 * runtime may load the library's code object that holds the buffer at that moment (its
 * FORGE_SCRATCH_BYTES, held until the process ends), so a caller under graph capture or a
 * no-allocation harness makes one call outside it first.
 */
FORGE_API forge_status forge_linear_step_unfused_noalloc(const void *X, const void *dY, void *W, void *m,
                                                         void *v, float *m_scale, float *v_scale, int64_t T,
                                                         int64_t d_in, int64_t d_out, int32_t moment_dtype,
                                                         float lr, float beta1, float beta2, float eps,
                                                         float weight_decay, int64_t step, int32_t grad_dtype,
                                                         void *stream);

/* Static description of a status code (never NULL). */
FORGE_API const char *forge_status_string(int32_t status);

/*
 * forge_query_tile -- the tile geometry that the fused step uses on a matrix W [d_out, d_in]
 * with T tokens and `moment_dtype` state: rows of W (along d_out), columns (along d_in) and
 * tokens per pipeline chunk.  The fixed counterpart of App. H's per-shape tile choice:
 * 256x64 for int8 moments in 256-row blocks (one scale block per tile), 128x128 for every
 * other kind, at every shape.  Any output pointer may be NULL.  Returns
 * FORGE_ERR_INVALID_DTYPE for an unknown code and FORGE_ERR_INVALID_SHAPE for a negative size.
 */
FORGE_API forge_status forge_query_tile(int64_t T, int64_t d_in, int64_t d_out, int32_t moment_dtype,
                                        int32_t *tile_rows, int32_t *tile_cols, int32_t *tile_tokens);

#ifdef __cplusplus
}
#endif

#endif /* FORGE_H */
