/*
 * noble.h - C ABI of libnoble: the NOBLE-CosNet augmented linear layer on
 * AMD Instinct MI355X (gfx950).
 *
 * The layer (arXiv 2603.06492, Sec. 3.1 Eq. 1 with the CosNet nonlinearity of
 * Sec. 3.2 Eq. 2, restated in App. A), rows = tokens:
 *
 *   H  = x W_down                       [T, r]
 *   C1 = cos(H (.) omega1 + phi1)       [T, r]   (per-rank frequency/phase)
 *   H2 = C1 M                           [T, r]   (M stored [r_in, r_out])
 *   C2 = cos(H2 (.) omega2 + phi2)      [T, r]
 *   y  = x W + b + C2 W_up              [T, d_out]
 *
 * The backward computes every gradient of L = sum(dy (.) y) by the chain rule
 * (the paper prints none; d cos(u)/du = -sin(u)), recomputing the cosines from
 * the saved H instead of storing them.
 *
 * desc->activation selects the bottleneck nonlinearity among the variants of
 * the activation ablation (Sec. 4.4, Table 5): cos (the CosNet above), tanh,
 * LeakyReLU (negative slope 0.01) or GELU (exact, a Phi(a)), each either in
 * the two-application form above (f in place of cos, with M between) or as
 * one application C2 = f(H (.) omega1 + phi1), which has no M, omega2, phi2.
 * A third form, the 3-layer CosNet (last row of Table 5; Sec. 5), applies a
 * third cosine after a second mixing matrix M':
 *   C3 = cos((C2 M') (.) omega3 + phi3),   y = x W + b + C3 W_up
 * and stores its parameters stacked with the second layer's: M holds
 * [M ; M'] as [2, r, r], omega2 holds [omega2 ; omega3] and phi2
 * [phi2 ; phi3] as [2, r], and so do dM, domega2 and dphi2.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - All tensors are dense, row-major and contiguous, in device memory owned
 *    and allocated by the caller.  The library never allocates, frees or
 *    synchronises, and keeps no state between calls.
 *  - desc->dtype is the storage type of x, W, W_down, M, W_up, y, dy and dx.
 *    b, omega1, phi1, omega2, phi2 and every parameter gradient are float32.
 *    Arithmetic: bf16 operands with float32 accumulation on the bf16 path
 *    (cosine arguments, cos and sin in float32).  Of the branch's
 *    intermediates, C2 is rounded to bf16 where it feeds y and dW_up, and
 *    dH where it feeds dx; the mixing products (C1 M, dH2 M^T) and the
 *    gradient products dW_down = x^T dH and dM = C1^T dH2 take C1, dH2 and
 *    dH as a pair of bf16 values whose sum carries about 16 significant
 *    bits, so that those products are float32-accurate.  float32
 *    throughout on the f32 path.
 *  - Shapes: 0 <= T <= 2^31 - 4096; 8 <= d_in, d_out <= 2^20, multiples of
 *    8; r = 0 (plain linear: every branch pointer is ignored and may be NULL)
 *    or 8 <= r <= 256 (bf16) / 128 (f32, and the 3-layer form) with r a
 *    multiple of 8.  Each
 *    matrix product of a call must also fit one dispatch (2^32 - 1
 *    work-items): at most 8388607 output tiles of 256 x 256 (bf16) or
 *    16777215 of 128 x 128 (f32) in y = x W, dx and dW (plus, for dW, the
 *    rank gradients' tiles), which only layers far beyond a GPU's memory
 *    exceed.  Every pointer must be 16-byte aligned.  Outputs must not alias
 *    inputs or each other.
 *  - Groups (desc->groups = G, 1 to 4; 0 means 1): the d_out output columns
 *    form G equal blocks that share x, each with its own branch of rank r
 *    (Q, K and V of an attention block, each with its own CosNet,
 *    Sec. 4.1.1).  With d_g = d_out / G (a multiple of 8) and R = G r:
 *      W_down [d_in, R]   (group g: columns g r .. g r + r - 1)
 *      M [G, r, r], omega1/phi1/omega2/phi2 [R]   (group g: entries g r ..)
 *      (3-layer form: M [2, G, r, r], omega2/phi2 [2, R])
 *      W_up [R, d_g]      (group g: rows g r .., mapping onto y[:, g d_g ..])
 *    and the gradients have the same shapes.  G = 1 is the single layer.
 *  - Argument checking is complete before any HIP call: on any error the call
 *    returns a status and enqueues nothing.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream)
 *    and the call returns without waiting.  Device faults surface at the
 *    caller's next synchronisation.  Concurrent calls must use separate
 *    scratch buffers.
 *  - Only gfx950 devices are supported (NOBLE_ERR_UNSUPPORTED_DEVICE otherwise).
 */
#ifndef NOBLE_H
#define NOBLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum noble_dtype {
    NOBLE_BF16 = 0, /* bfloat16 storage, float32 accumulation */
    NOBLE_F32 = 1   /* float32 storage and arithmetic */
} noble_dtype;

typedef enum noble_status {
    NOBLE_OK = 0,
    NOBLE_ERR_NULL_ARG = 1,          /* a required pointer is NULL */
    NOBLE_ERR_BAD_SHAPE = 2,         /* dimension out of the ranges above */
    NOBLE_ERR_BAD_DTYPE = 3,         /* desc->dtype is not a noble_dtype */
    NOBLE_ERR_MISALIGNED = 4,        /* a pointer is not 16-byte aligned */
    NOBLE_ERR_WORKSPACE_TOO_SMALL = 5, /* scratch_bytes below the required size */
    NOBLE_ERR_UNSUPPORTED_DEVICE = 6,  /* current device is not gfx950 */
    NOBLE_ERR_HIP = 7,               /* a HIP runtime call or launch failed */
    NOBLE_ERR_BAD_ACTIVATION = 8     /* desc->activation is not a noble_activation */
} noble_status;

/* Bottleneck nonlinearity (Sec. 3.2 Eq. 2; variants of Sec. 4.4, Table 5).
 * The _M forms and COSNET apply f twice with M between them; the others
 * apply f once. */
typedef enum noble_activation {
    NOBLE_ACT_COSNET = 0,       /* cos(w2 (.) (cos(w1 (.) H + p1) M) + p2) */
    NOBLE_ACT_COS = 1,          /* cos(w1 (.) H + p1) */
    NOBLE_ACT_TANH = 2,
    NOBLE_ACT_TANH_M = 3,
    NOBLE_ACT_LEAKY_RELU = 4,
    NOBLE_ACT_LEAKY_RELU_M = 5,
    NOBLE_ACT_GELU = 6,
    NOBLE_ACT_GELU_M = 7,
    NOBLE_ACT_COSNET3 = 8       /* cos(w3 (.) (C2 M') + p3), C2 of COSNET; r <= 128 */
} noble_activation;

/* Problem description.  `dtype` holds a noble_dtype value and `activation`
 * a noble_activation (0, the CosNet, for a zero-initialised desc). */
typedef struct noble_linear_desc {
    int64_t T;      /* tokens (rows of x, y, dy, dx) */
    int64_t d_in;   /* input features */
    int64_t d_out;  /* output features */
    int64_t r;      /* bottleneck rank; 0 = plain linear */
    int32_t dtype;  /* noble_dtype */
    int32_t activation; /* noble_activation */
    int32_t groups;     /* output column groups, each with its own branch (0 = 1) */
    int32_t reserved;   /* must be 0 (NOBLE_ERR_BAD_SHAPE otherwise) */
} noble_linear_desc;

/* Sizes of the two caller-owned work buffers for `desc`.
 *   reserve_bytes: written by noble_linear_fwd (H = x W_down, float32 [T, R])
 *                  and read by the matching noble_linear_bwd; keep it intact
 *                  in between.  4*T*R bytes (R = groups * r).
 *   scratch_bytes: temporary space used within one call (fwd or bwd) only;
 *                  its contents need no initialisation.  The forward uses it
 *                  only when r > 0; the backward may use it also when r = 0
 *                  (split-K partial sums of dW), whenever scratch_bytes > 0.
 * Either output pointer may be NULL.  Returns NOBLE_ERR_NULL_ARG (desc NULL),
 * NOBLE_ERR_BAD_SHAPE, NOBLE_ERR_BAD_DTYPE or NOBLE_ERR_BAD_ACTIVATION;
 * makes no HIP call.  The 3-layer form's scratch is larger; the other
 * activations share one size. */
noble_status noble_linear_workspace_size(const noble_linear_desc* desc,
                                         size_t* reserve_bytes,
                                         size_t* scratch_bytes);

/* Scratch bytes the forward alone needs (at most the scratch_bytes of
 * noble_linear_workspace_size, which covers both calls): a forward-only or
 * inference caller may pass a buffer of this size to noble_linear_fwd.
 * Same errors as noble_linear_workspace_size; makes no HIP call. */
noble_status noble_linear_fwd_scratch_size(const noble_linear_desc* desc,
                                           size_t* scratch_bytes);

/* Forward, Eq. 1 with the CosNet of Eq. 2:
 *   y = x W + b + cos(omega2 (.) (cos(omega1 (.) (x W_down) + phi1) M) + phi2) W_up
 * Inputs : x [T, d_in], W [d_in, d_out], b [d_out] f32 (nullable = no bias),
 *          W_down [d_in, r], omega1/phi1/omega2/phi2 [r] f32, M [r, r],
 *          W_up [r, d_out].
 * Outputs: y [T, d_out]; reserve (>= reserve_bytes) receives H for the
 *          backward.  scratch must hold the bytes noble_linear_fwd_scratch_size
 *          gives (a buffer sized for both calls also serves).
 * reserve may be NULL: an inference-only forward that keeps no H (the
 * branch's permanent inference cost, Sec. 6); no backward can follow it.
 * With a one-application activation, M, omega2 and phi2 are not read and
 * may be NULL; the 3-layer form reads them in their stacked shapes. */
noble_status noble_linear_fwd(const noble_linear_desc* desc,
                              const void* x, const void* W, const float* b,
                              const void* W_down,
                              const float* omega1, const float* phi1,
                              const void* M,
                              const float* omega2, const float* phi2,
                              const void* W_up,
                              void* y, void* reserve,
                              void* scratch, size_t scratch_bytes,
                              void* stream);

/* The forward above without a scratch argument, for callers that cannot
 * allocate (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation).  It uses a scratch array that the library holds in
 * device memory: NOBLE_STATIC_SCRATCH_BYTES on each GPU it runs on, from the
 * first call on that GPU until the process ends.  It allocates nothing and
 * makes no allocating call.  Arguments, outputs and status codes are those of
 * noble_linear_fwd; a layer whose forward needs more scratch than the array
 * holds (noble_linear_fwd_scratch_size above NOBLE_STATIC_SCRATCH_BYTES;
 * at r = 128 that is beyond about 87000 tokens) returns
 * NOBLE_ERR_WORKSPACE_TOO_SMALL before any HIP call.  Every call on one GPU
 * shares that GPU's array: calls that overlap on one GPU (on different
 * streams, or from different threads without ordering) race on it and must
 * not be issued; calls ordered on one stream are safe.  The array's contents
 * are never read before being written within a call. */
#define NOBLE_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
noble_status noble_linear_fwd_static(const noble_linear_desc* desc,
                                     const void* x, const void* W, const float* b,
                                     const void* W_down,
                                     const float* omega1, const float* phi1,
                                     const void* M,
                                     const float* omega2, const float* phi2,
                                     const void* W_up,
                                     void* y, void* reserve,
                                     void* stream);

/* Backward of the forward above for upstream gradient dy [T, d_out], using
 * the reserve written by the matching forward (same inputs, same desc).
 * Every gradient buffer is overwritten (not accumulated):
 *   dx [T, d_in] (storage dtype), dW [d_in, d_out], db [d_out] (nullable =
 *   not computed), dW_down [d_in, r], dM [r, r], dW_up [r, d_out],
 *   domega1, dphi1, domega2, dphi2 [r]  (all float32; the 3-layer form's
 *   dM [2, r, r] and domega2, dphi2 [2, r]).
 * With T = 0 the parameter gradients are set to zero.  db and the four
 * omega / phi gradients are summed over tokens with float atomics, so they
 * may differ in the last bits between runs; dx, dW, dW_down, dM and dW_up
 * are reproducible (a token sum split into pieces stores per-piece partials
 * that are added in a fixed order).  scratch (>= scratch_bytes) may be NULL only when
 * scratch_bytes is 0 or T is 0.  With a one-application activation, M,
 * omega2 and phi2 are not read, and dM, domega2, dphi2 may be NULL; when
 * given they are set to zero (the function does not depend on them). */
noble_status noble_linear_bwd(const noble_linear_desc* desc,
                              const void* dy, const void* x, const void* W,
                              const void* W_down,
                              const float* omega1, const float* phi1,
                              const void* M,
                              const float* omega2, const float* phi2,
                              const void* W_up,
                              const void* reserve,
                              void* dx, float* dW, float* db,
                              float* dW_down, float* dM, float* dW_up,
                              float* domega1, float* dphi1,
                              float* domega2, float* dphi2,
                              void* scratch, size_t scratch_bytes,
                              void* stream);

/* Instrumentation, not needed to compute anything.  The next
 * noble_linear_bwd issued by the calling thread that reaches its
 * weight-gradient launch (the one grouped product computing dW, dW_down,
 * dW_up and dM, and db's column sums) records start_event and stop_event
 * (hipEvent_t values created by the caller, either may be NULL) on its
 * stream immediately before and after that launch, so that
 * hipEventElapsedTime gives the launch's duration, and stores the launch's
 * workgroup count in *workgroups (host memory; may be NULL) when it enqueues
 * it; the hook then clears itself.  Calling it again replaces the pending
 * request; NULL, NULL, NULL clears it.  A backward that fails validation, or
 * has T = 0, leaves it pending.  Returns NOBLE_OK; makes no HIP call. */
noble_status noble_profile_next_wgrad(void* start_event, void* stop_event, int64_t* workgroups);

/* ------------------------------------------------------------------------
 * Training recipe around the layer (Sec. 3.3 "Key Design Choices", App. A
 * "Hyperparameter Defaults").  Host-side values and one device fill; none
 * of it is on the forward/backward path.
 * ------------------------------------------------------------------------ */
typedef struct noble_recipe {
    double alpha;      /* W_up ~ N(0, (alpha / sqrt(r))^2); default 0.01 */
    double w_scale;    /* W ~ N(0, (w_scale / sqrt(d_in))^2); default 0.5 */
    double omega_min;  /* omega1, omega2 ~ U[omega_min, omega_max]; default 0.8 */
    double omega_max;  /* default 1.2 */
    double phi_std;    /* phi1, phi2 ~ N(0, phi_std^2); default 0.1 */
    double gamma;      /* lr(W_up) = lr (min(d_in, d_out) / r)^(2 gamma); default 0.3 */
    double gamma_M;    /* lr(M) = lr (min(d_in, d_out) / r)^gamma_M; default 0.45 */
    double omega_lr;   /* learning-rate multiplier of omega1, omega2; default 3.0 */
    double phi_lr;     /* learning-rate multiplier of phi1, phi2; default 5.0 */
} noble_recipe;

/* Fills *recipe with the defaults listed above (no-op for NULL). */
void noble_recipe_defaults(noble_recipe* recipe);

/* Learning-rate multipliers, relative to the base learning rate, of each
 * parameter of one layer (Sec. 3.3 Eqs. 3-4): W, b and W_down take the base
 * rate, W_up and M the elevated rates above, omega and phi the fixed
 * multipliers.  With r = 0 only W and b are meaningful (the rest are 0).
 * For a grouped layer the widths are those of one group (d_in, d_out / G). */
typedef struct noble_lr_mults {
    double W, b, W_down, W_up, M, omega, phi;
} noble_lr_mults;

/* Returns NOBLE_ERR_NULL_ARG (desc, recipe or out NULL), or the codes of
 * noble_linear_workspace_size for a bad desc; makes no HIP call. */
noble_status noble_lr_multipliers(const noble_linear_desc* desc,
                                  const noble_recipe* recipe,
                                  noble_lr_mults* out);

/* Initialises the layer's parameters on the device (Sec. 3.3 and App. A):
 *   W ~ N(0, (w_scale / sqrt(d_in))^2), b = 0,
 *   W_down ~ U(-1/sqrt(d_in), 1/sqrt(d_in))  (the paper gives no W_down
 *     init; this is the usual linear-layer default),
 *   omega1, omega2 ~ U[omega_min, omega_max], phi1, phi2 ~ N(0, phi_std^2),
 *   M ~ U(-sqrt(3 / r), sqrt(3 / r))  (Xavier uniform, fan_in = fan_out = r),
 *   W_up ~ N(0, (alpha / sqrt(r))^2).
 * Storage tensors (W, W_down, M, W_up) in desc->dtype, the rest float32;
 * shapes as in noble_linear_fwd (the 3-layer form's M' and omega3, phi3 are
 * drawn like M, omega2, phi2, as the second halves of those tensors).  A NULL pointer skips that tensor.
 * Random numbers: Philox4x32-10 (Salmon et al., SC 2011) keyed by `seed`
 * (key = low, high 32 bits); element e (row-major) of tensor t takes the
 * block at counter (e mod 2^32, e / 2^32, t, 0), t = 0 W, 1 W_down,
 * 2 omega1, 3 phi1, 4 M, 5 omega2, 6 phi2, 7 W_up.  With words x0, x1 and
 * u_i = (x_i + 1/2) 2^-32, a uniform draw on [lo, hi] is lo + (hi - lo) u0
 * and a normal draw is sqrt(-2 ln u0) cos(2 pi u1), both in double, then
 * rounded to float32 (and to bf16, nearest even, for bf16 storage).  The
 * values do not depend on the launch, so a layer is reproducible from its
 * seed.  Enqueued on `stream`; returns NOBLE_ERR_NULL_ARG (desc or recipe
 * NULL), a desc error, NOBLE_ERR_MISALIGNED (a pointer not aligned to its
 * element size) or NOBLE_ERR_HIP. */
noble_status noble_init_params(const noble_linear_desc* desc,
                               const noble_recipe* recipe, uint64_t seed,
                               void* W, float* b, void* W_down,
                               float* omega1, float* phi1, void* M,
                               float* omega2, float* phi2, void* W_up,
                               void* stream);

/* Static, human-readable name of a status code (never NULL). */
const char* noble_status_string(int status);

/* ABI version of this header (bumped on incompatible changes). */
int noble_abi_version(void);

#define NOBLE_ABI_VERSION 5

#ifdef __cplusplus
}
#endif

#endif /* NOBLE_H */
