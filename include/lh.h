/*
 * lh.h -- C ABI of the distilled modal recurrence on AMD MI355X (gfx950).
 *
 * The operation (Laughing Hyena distillation, Sec. 3.4 "Deploying the
 * recurrence", Proposition "modal_realization", App. B.1):
 *
 *   every channel c of a bank of D distilled filters carries d complex modes
 *   with poles lambda[c,n], residues R[c,n] and a real pass-through h0[c];
 *   its filter is h_0 = h0, h_t = Re sum_n R[c,n] lambda[c,n]^(t-1) (t >= 1,
 *   eq. "modal_impulse").  Its state-space form is A = diag(lambda), B = 1,
 *   C = R, D = h0 (eq. "dtssm"):
 *
 *       y_t     = Re( sum_n R[c,n] x_t[n] ) + h0[c] u_t      (reads x_t)
 *       x_{t+1} = lambda[c,n] x_t[n] + u_t                     (then updates)
 *
 *   so that, from x_0 = 0, y is the causal convolution of h with u
 *   (eq. "cnn") and x_T[n] = sum_{k<T} lambda[c,n]^(T-1-k) u_k.
 *
 * Prefill (lh_prefill) processes a prompt of T tokens: all outputs y_0..y_{T-1}
 * and the post-prompt state x_T.  Decode (lh_step) advances the state by one
 * token per call and returns that token's output; a step right after a prefill
 * of T tokens returns y_T.
 *
 * Layouts (all row-major, contiguous, caller-owned device memory):
 *   lambda, R : [D, d]    complex64, interleaved (re, im)        (lh_c32)
 *   h0        : [D]       float32
 *   u, y      : [B, T, D] float32 or bfloat16 (io_dtype), channel fastest
 *   state     : [B, D, d] complex64, mode fastest
 *   u_t, y_t  : [B, D]    float32 or bfloat16 (io_dtype)
 * All arithmetic is float32; bfloat16 inputs are widened exactly and bfloat16
 * outputs are rounded to nearest, ties to even.
 *
 * Ownership and execution: the library never allocates, frees or keeps a
 * pointer; it holds no state between calls and is re-entrant.  Work is enqueued
 * asynchronously on `stream` (a hipStream_t; NULL is the null stream) and the
 * call returns without synchronising.  Calls on the same buffers must be
 * ordered by the caller (same stream, or events).
 *
 * Errors: every argument is checked on the host before any device work is
 * enqueued; on a non-LH_OK status nothing has been enqueued and no buffer has
 * been touched.  Faults during execution surface at the caller's next
 * synchronisation of `stream`.  No call aborts and no C++ exception crosses
 * this interface.  lh_last_error() returns a thread-local description of the
 * most recent failure in the calling thread.
 */
#ifndef LH_H
#define LH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LH_ABI_VERSION 2

/* complex64, interleaved real and imaginary parts */
typedef struct lh_c32 {
    float re;
    float im;
} lh_c32;

/* element type of u / y (and u_t / y_t); lambda, R, h0 and the state are
 * always float32-based */
typedef enum lh_dtype {
    LH_F32 = 0,
    LH_BF16 = 1
} lh_dtype;

typedef enum lh_status {
    LH_OK = 0,
    LH_ERR_INVALID_ARG = 1,       /* null pointer, bad size, size overflow,
                                     pointer not accessible from the device */
    LH_ERR_OVERLAP = 2,           /* an output buffer overlaps another buffer */
    LH_ERR_UNSUPPORTED_DTYPE = 3, /* io_dtype is not LH_F32 or LH_BF16 */
    LH_ERR_NO_DEVICE = 4,         /* no HIP device is visible */
    LH_ERR_WORKSPACE = 5,         /* workspace null or smaller than required */
    LH_ERR_HIP = 6                /* the HIP runtime refused a launch */
} lh_status;

/* Largest supported number of modes per channel. */
#define LH_MAX_MODES 1024

/* LH_ABI_VERSION of the built library. */
int lh_abi_version(void);

/* Static description of a status code (never NULL). */
const char* lh_status_string(lh_status status);

/* Thread-local detail of the most recent non-LH_OK status returned in the
 * calling thread ("" if none). */
const char* lh_last_error(void);

/*
 * Workspace bytes lh_prefill needs for these sizes, for either input type
 * (the larger of the float32 and bfloat16 plans' needs).  Returns 0 when the
 * plan needs no workspace and (size_t)-1 when the arguments are invalid.
 * Pure function of its arguments; host only.
 */
size_t lh_prefill_workspace_bytes(int64_t B, int64_t D, int64_t d, int64_t T);

/*
 * Prefill (Sec. 3.4, "fast pre-filling"; states start at x_0 = 0): outputs
 * y[b,t,c] for t < T and the post-prompt state state[b,c,n] = x_T.
 *
 *   lambda, R, h0 : inputs as laid out above
 *   u             : [B,T,D] prompt inputs (io_dtype)
 *   B, D, d, T    : B >= 1, D >= 1, 1 <= d <= LH_MAX_MODES, T >= 0
 *   io_dtype      : LH_F32 or LH_BF16 (u and y)
 *   state         : out, [B,D,d] complex64 (overwritten, not read)
 *   y             : out, [B,T,D] (io_dtype); may be NULL only when T == 0
 *   workspace     : device scratch of at least
 *                   lh_prefill_workspace_bytes(B,D,d,T) bytes, 256-byte
 *                   aligned; may be NULL when that size is 0.  Its contents
 *                   on entry are ignored and on exit undefined.
 *
 * The library picks the plan (lh_prefill_plan with plan = LH_PREFILL_AUTO
 * reports which): the matrix-core chunked scan over the whole prompt where
 * its workgroups fill the GPU, the segmented matrix-core plan where the
 * prompt must be split in time to fill it, else the VALU chunked scan (see
 * lh_prefill_with_plan for what each computes and needs).  Every plan gives
 * the same results up to float32 rounding.
 * T == 0 zeroes the state and leaves y untouched.  y must not overlap u,
 * state, lambda, R, h0 or workspace; state must not overlap any input.
 */
lh_status lh_prefill(const lh_c32* lambda, const lh_c32* R, const float* h0,
                     const void* u, int64_t B, int64_t D, int64_t d, int64_t T,
                     lh_dtype io_dtype, lh_c32* state, void* y,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Scratch bytes lh_prefill_noalloc holds per GPU (64 MiB). */
#define LH_NOALLOC_SCRATCH_BYTES (UINT64_C(64) << 20)

/*
 * lh_prefill for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same results, arguments, plan, ownership and errors as lh_prefill, with no
 * workspace argument.  The plan's scratch is a static array of
 * LH_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends; this call allocates nothing and makes no
 * allocating runtime call.  Sizes whose plan needs more scratch than that
 * (lh_prefill_workspace_bytes(B,D,d,T) > LH_NOALLOC_SCRATCH_BYTES) return
 * LH_ERR_WORKSPACE before anything is enqueued.  Every call on one GPU shares
 * that GPU's array, which keeps the last call's contents (no plan reads
 * scratch it has not written in the same call): calls that overlap on one
 * GPU (on different streams, or from several threads without ordering) race
 * on it and must not be made.
 */
lh_status lh_prefill_noalloc(const lh_c32* lambda, const lh_c32* R, const float* h0,
                             const void* u, int64_t B, int64_t D, int64_t d, int64_t T,
                             lh_dtype io_dtype, lh_c32* state, void* y, void* stream);

/* Plan requests of lh_prefill_with_plan (values > 0 are VALU chunk lengths). */
#define LH_PREFILL_AUTO 0
#define LH_PREFILL_MFMA (-1)
#define LH_PREFILL_MFMA_SEG (-2)

/* Prefill plans (what a prefill runs). */
typedef enum {
    LH_PLAN_SCAN = 0,      /* VALU scan: one sequential pass or parallel time chunks */
    LH_PLAN_MFMA = 1,      /* matrix-core plan over the whole prompt */
    LH_PLAN_MFMA_SEG = 2   /* segmented matrix-core plan */
} lh_prefill_plan_kind;

/*
 * The plan a prefill takes for these sizes, plan request and input type when
 * u and y are 16-byte aligned (automatic matrix-core plans run the VALU scan,
 * with the same workspace, when they are not).  Returns an
 * lh_prefill_plan_kind, or -1 when the arguments are invalid or no plan
 * exists (as the prefill would fail).  Pure function of its arguments; host
 * only, no device call.
 */
int lh_prefill_plan(int64_t B, int64_t D, int64_t d, int64_t T, int64_t plan,
                    lh_dtype io_dtype);

/*
 * Workspace bytes of lh_prefill_with_plan for this plan request (as
 * lh_prefill_workspace_bytes; plan = LH_PREFILL_AUTO gives the same value).
 */
size_t lh_prefill_with_plan_workspace_bytes(int64_t B, int64_t D, int64_t d, int64_t T,
                                            int64_t plan);

/*
 * lh_prefill with the plan named by the caller instead of chosen by the
 * library: for callers that compare plans (tests, benchmarks).  Same results,
 * arguments, ownership and errors as lh_prefill, with
 *
 *   plan = LH_PREFILL_AUTO (0): the automatic plan (lh_prefill itself);
 *   plan > 0: the VALU chunked scan with this time-chunk length (the prompt
 *            is cut into ceil(T/plan) chunks processed in parallel: each
 *            chunk's end state from zero, a carry across chunks with
 *            lambda^plan formed in float64, then the outputs from each chunk's
 *            entry state; plan >= T means one sequential pass per row);
 *   plan = LH_PREFILL_MFMA: the matrix-core plan (chunks of 32 steps as dense
 *            contractions on the MFMA units: outputs Y = T U + W X_in, chunk
 *            end states S = P U and the carry X_in <- lambda^32 X_in + S; with
 *            the float32 operands split into bfloat16 terms: three with
 *            float32 u/y, two for the outputs and three for the state with
 *            bfloat16 u/y; d = 16 or 32 require D % 8 == 0, d = 64 requires
 *            float32 u/y and D % 4 == 0; always T >= 1 and 16-byte aligned u and
 *            y, else LH_ERR_INVALID_ARG).  The automatic plan uses it where
 *            supported and either ceil(D/16) * ceil(B/32) >= 256 (enough
 *            workgroups to fill the GPU without splitting the prompt in time)
 *            or an estimate of the chunk steps each compute unit walks puts
 *            it within 7/5 of the segmented plan below (the estimate depends
 *            on the input type, so float32 and bfloat16 calls may take
 *            different plans); at d = 64 also when T does not split into
 *            segments and B >= 4 or ceil(D/4) * ceil(B/16) >= 256, and never
 *            when B < 4 and B * T <= 1024 (the VALU scan is faster there);
 *   plan = LH_PREFILL_MFMA_SEG: the segmented matrix-core plan: the prompt is
 *            cut into 2^k segments of T / 2^k steps (a multiple of 32, at
 *            least 256), the fewest whose (batch row, segment) pairs fill the
 *            GPU; a matrix-core pass computes each segment's end state from
 *            zero, a carry gives each segment its entry state, and a second
 *            matrix-core pass computes the outputs (same operand splitting
 *            and requirements as LH_PREFILL_MFMA, and such a T).  The
 *            automatic plan takes it where the whole-prompt matrix-core plan
 *            is supported but not chosen and T splits this way (at d = 64
 *            only when B * T > 1024).
 * workspace: at least lh_prefill_with_plan_workspace_bytes(B,D,d,T,plan)
 * bytes.  A plan request the sizes do not support returns LH_ERR_INVALID_ARG.
 */
lh_status lh_prefill_with_plan(const lh_c32* lambda, const lh_c32* R, const float* h0,
                               const void* u, int64_t B, int64_t D, int64_t d, int64_t T,
                               lh_dtype io_dtype, lh_c32* state, void* y, int64_t plan,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Longest prompt lh_prefill_fft accepts (transforms of at most 2^20 points). */
#define LH_FFT_MAX_T (INT64_C(1) << 19)

/*
 * Workspace bytes lh_prefill_fft needs for these sizes; 0 when T == 0 and
 * (size_t)-1 when the arguments are invalid or T > LH_FFT_MAX_T.  Pure
 * function of its arguments.  About (2 + 2 ceil(B/2)) N D 4 bytes, with N the
 * transform length below, plus partial states and small tables.
 */
size_t lh_prefill_fft_workspace_bytes(int64_t B, int64_t D, int64_t d, int64_t T);

/*
 * Prefill by FFT convolution (Sec. 3.4, fast pre-filling "via convolutions"):
 * the same results as lh_prefill (outputs y[b,t,c] for t < T and state = x_T),
 * computed the other way the paper describes:
 *
 *   hhat_0 = h0[c],  hhat_t = Re sum_n R[c,n] lambda[c,n]^(t-1)   (t < T; the
 *       O(dT) evaluation of Lemma "ssmd_impulse")
 *   y[b,t,c]     = sum_{j<=t} hhat_{t-j} u[b,j,c]   (eq. "cnn"), by N-point
 *       FFTs with N the smallest power of two >= 2T - 1
 *   state[b,c,n] = sum_{k<T} lambda[c,n]^(T-1-k) u[b,k,c]  (Vandermonde
 *       contraction)
 *
 * Arguments, layouts, ownership and errors as lh_prefill, with
 *   T          : 0 <= T <= LH_FFT_MAX_T
 *   workspace  : at least lh_prefill_fft_workspace_bytes(B,D,d,T) bytes,
 *                256-byte aligned (NULL allowed when that size is 0)
 * The rounding differs from the scan's (float32 transforms: an error near
 * 1e-7 log2(N) of the largest outputs of a row, spread over the row).
 */
lh_status lh_prefill_fft(const lh_c32* lambda, const lh_c32* R, const float* h0,
                         const void* u, int64_t B, int64_t D, int64_t d, int64_t T,
                         lh_dtype io_dtype, lh_c32* state, void* y,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * Decode step (Proposition "modal_realization"; App. B.1 for the real part):
 *   y_t[b,c]     = Re(sum_n R[c,n] state[b,c,n]) + h0[c] u_t[b,c]
 *   state[b,c,n] = lambda[c,n] state[b,c,n] + u_t[b,c]      (in place)
 *
 *   state : in/out [B,D,d] complex64
 *   u_t   : [B,D] (io_dtype);  y_t : out [B,D] (io_dtype)
 * y_t must not overlap any other buffer; state must not overlap lambda, R,
 * h0 or u_t.  O(d) work per (b, c); one kernel launch; no workspace.
 */
lh_status lh_step(const lh_c32* lambda, const lh_c32* R, const float* h0,
                  lh_c32* state, const void* u_t, void* y_t,
                  int64_t B, int64_t D, int64_t d, lh_dtype io_dtype,
                  void* stream);

/* Largest modal order the companion form accepts (companion order 2d <= 32). */
#define LH_COMPANION_MAX_MODES 16

/*
 * Companion (rational) form of the distilled filters (App. "From Transfer
 * Function to State-Space", eq. "ssm_canon"; canonization of a modal SSM).
 * The real filter h_0 = h0, h_t = Re sum_n R_n lambda_n^(t-1) is the impulse
 * response of a real system of order 2d (each pole with its conjugate,
 * residues R_n / 2 and conj(R_n) / 2, App. B.1) whose transfer function in
 * w = z^-1 is
 *
 *   H(w) = h0 + (beta_1 w + ... + beta_2d w^2d) / (1 + a_1 w + ... + a_2d w^2d)
 *
 * This call writes, per channel, a[c, m-1] = a_m and beta[c, m-1] = beta_m
 * (m = 1..2d), computed in float64 from the complex64 poles and residues.
 *
 *   lambda, R : [D, d] complex64;  a, beta : out [D, 2d] float64
 *   D >= 1, 1 <= d <= LH_COMPANION_MAX_MODES
 * Outputs must not overlap each other or the inputs.  One kernel launch; no
 * workspace; same execution and error rules as lh_step.
 *
 * Numerical range: p's coefficients grow like binomial coefficients and the
 * companion state like the impulse response of 1/p, far beyond the outputs it
 * combines, so even in float64 the form meets a 1e-4 relative accuracy only
 * for small orders (measured over 1500 steps with pole angles spread over
 * [0, pi]: d <= 8 at pole radii up to 0.9999; d = 16 loses it near the unit
 * circle).  The modal calls above do not have this limit.
 */
lh_status lh_companion_coeffs(const lh_c32* lambda, const lh_c32* R, int64_t D, int64_t d,
                              double* a, double* beta, void* stream);

/*
 * Companion decode step (Lemma "efficient_recurrence"), per (b, c):
 *   y_t[b,c]      = sum_m beta[c,m] state[b,c,m] + h0[c] u_t[b,c]
 *   state[b,c,:]  = (u_t[b,c] - sum_m a[c,m] state[b,c,m], state[b,c,0], ...,
 *                    state[b,c,2d-2])                               (in place)
 * in float64, y_t rounded to io_dtype.
 *
 *   a, beta : [D, 2d] float64 (lh_companion_coeffs), 16-byte aligned
 *   h0      : [D] float32
 *   state   : in/out [B, D, 2d] float64, 16-byte aligned
 *   u_t, y_t: [B, D] (io_dtype)
 * y_t must not overlap any other buffer; state must not overlap a, beta, h0
 * or u_t.  One kernel launch; no workspace; same execution and error rules
 * as lh_step.
 */
lh_status lh_companion_step(const double* a, const double* beta, const float* h0,
                            double* state, const void* u_t, void* y_t,
                            int64_t B, int64_t D, int64_t d, lh_dtype io_dtype, void* stream);

/* Workspace bytes of lh_companion_init: T D 8 (the taps of 1/p); 0 when
 * T == 0, (size_t)-1 for invalid sizes. */
size_t lh_companion_init_workspace_bytes(int64_t D, int64_t d, int64_t T);

/*
 * Companion state after a prompt without stepping (Proposition "fast_init"):
 *   state[b,c,j] = v_{T-1-j},  v = g * u[b,:,c],  j = 0..2d-1
 * with g the impulse response of 1/p (g_0 = 1, g_t = -sum_m a_m g_{t-m}) and
 * v_t = 0 for t < 0; the state lh_companion_step reaches from zero after the
 * T prompt inputs.  Prompt outputs come from lh_prefill or lh_prefill_fft
 * (the same filter).
 *
 *   a        : [D, 2d] float64;  u : [B, T, D] (io_dtype)
 *   state    : out [B, D, 2d] float64, 16-byte aligned
 *   workspace: lh_companion_init_workspace_bytes(D, d, T) bytes, 256-byte
 *              aligned (NULL allowed when that is 0)
 *   T >= 0; T == 0 zeroes the state
 * state and workspace must not overlap each other or the inputs.  Two kernel
 * launches; same execution and error rules as lh_prefill.
 */
lh_status lh_companion_init(const double* a, const void* u, int64_t B, int64_t D, int64_t d,
                            int64_t T, lh_dtype io_dtype, double* state, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Multi-head decode step (Sec. 5, "Multi-head Long Convolutions": the
 * projections q, k, v of width D = M N are split into M heads of N channels;
 * per head the outer product z = k (x) v is convolved entry by entry with the
 * head's distilled filter and the result multiplies q).  Every entry (i, j)
 * of head m carries the d-mode state of Proposition "modal_realization":
 *
 *   z[i,j]          = k[b, mN+i] v[b, mN+j]
 *   y[b, mN+i]      = sum_j q[b, mN+j] ( Re(sum_n R[m,n] state[b,m,i,j,n])
 *                                        + h0[m] z[i,j] )          (reads state)
 *   state[b,m,i,j,n] = lambda[m,n] state[b,m,i,j,n] + z[i,j]       (in place)
 *
 * The q contraction runs over the second (value) index of z; exchanging the
 * k and v arguments gives the other orientation (q against the key index).
 *
 *   lambda, R : [M, d] complex64;  h0 : [M] float32 (one filter per head)
 *   state     : in/out [B, M, N, N, d] complex64, mode fastest
 *   q, k, v   : [B, M N] (io_dtype);  y : out [B, M N] (io_dtype)
 *   B, M, N   : >= 1;  1 <= d <= LH_MAX_MODES
 * y must not overlap any other buffer; state must not overlap lambda, R, h0,
 * q, k or v.  One kernel launch; no workspace; same execution and error
 * rules as lh_step.
 */
lh_status lh_mh_step(const lh_c32* lambda, const lh_c32* R, const float* h0,
                     lh_c32* state, const void* q, const void* k, const void* v, void* y,
                     int64_t B, int64_t M, int64_t N, int64_t d, lh_dtype io_dtype,
                     void* stream);

/*
 * Distillation objective of the modal form (Sec. 3.2, "Modal canonical
 * form"; the O(dL) filter evaluation of Lemma "ssmd_impulse").  Per channel c,
 * poles in polar form lambda = A e^{i theta} and residues R (cartesian) are
 * fitted to a real target filter h_1 .. h_L by the squared l2 interpolation
 * error:
 *
 *   hhat_t = Re sum_n R[c,n] lambda[c,n]^(t-1)   (t = 1..L)
 *   loss[c] = sum_t (hhat_t - h_t)^2
 *
 * with its gradients with respect to A, theta, Re R and Im R (dR holds
 * d/dRe R + i d/dIm R).  The pass-through h0 is matched by h_0 and is not
 * part of the objective.
 *
 *   A, theta : [D, d] float32 (polar poles);  R : [D, d] complex64
 *   target   : [D, L] float32, target[c, t-1] = h_t
 *   loss     : out [D];  dA, dtheta : out [D, d];  dR : out [D, d] complex64
 *   hhat     : out [D, L] (the materialised filter) or NULL
 *   D >= 1, 1 <= d <= LH_MAX_MODES, L >= 1
 * Outputs must not overlap each other or the inputs.  One kernel launch; no
 * workspace; same execution and error rules as lh_step.
 */
lh_status lh_distill(const float* A, const float* theta, const lh_c32* R, const float* target,
                     int64_t D, int64_t d, int64_t L, float* loss, float* dA, float* dtheta,
                     lh_c32* dR, float* hhat, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LH_H */
