/*
 * libmalt: the MALT / MALTER optimizer step for matrix parameters on AMD
 * Instinct MI355X (gfx950).
 *
 * The update rule is that of "MALT: Lightweight Curvature-Aware Muon via
 * Diagonal Preconditioning": Algorithm 1 (MALT) and Algorithm 2 (MALTER),
 * with the row/column preconditioners of Sec. 3.3 (Eq. dp_preconditioner),
 * Orth of Sec. 3.1 approximated by Newton-Schulz, and the norm grafting and
 * noise-adaptive stepsize of Sec. 3.5.  Per matrix W (m x n), one step does:
 *
 *   M <- mu1 M + (1-mu1) G                         momentum
 *   l <- mu2 l + (1-mu2) rowsum(G.G)               row squared norms
 *   r <- mu2 r + (1-mu2) colsum(G.G)               column squared norms
 *   L = Diag((l+eps)^(-1/8)),  R = Diag((r+eps)^(-1/8))
 *   Mt = L M R,  O = NS(Mt),  D = L O R
 *   MALTER: nu <- mu2 nu + (1-mu2) ||L G R||_F^2,
 *           alpha = sqrt(1-mu2^t)/(1-mu1^t+eps) * ||Mt||_F/(sqrt(nu)+eps)
 *   MALT:   alpha = 1
 *   W <- (1 - lr*weight_decay) W - lr * alpha * ||O||_F/(||D||_F+eps) * D
 *
 * NS is Muon's quintic Newton-Schulz iteration (the paper gives no
 * coefficients): X = Mt/(||Mt||_F + ns_eps) on the orientation with
 * rows <= cols, then ns_steps times  A = X X^T,  B = ns_b A + ns_c A A,
 * X <- ns_a X + B X.  It runs in bf16 on the matrix cores with fp32
 * accumulation; matrices whose shorter side is at most 32 run it in fp32
 * instead (only the final O is rounded to bf16).  Everything else is fp32
 * with fp64 scalar combines.
 *
 * Conventions shared by every entry point
 *  - Matrices are dense, row-major float32, `rows x cols`, 1 <= rows, cols <= 2^20,
 *    min(rows, cols) <= 32768 and rows*cols < 2^31, also with both dimensions
 *    rounded up to multiples of 256.  Device pointers must be 4-byte aligned; rows whose
 *    start is 16-byte aligned with cols % 4 == 0 take a vectorised path.
 *  - All device memory is owned by the caller.  The library never allocates
 *    device or pinned host memory; malt_init_state_scratch plans use the
 *    library's static scratch array instead of a caller workspace.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream).  Steps are
 *    enqueued asynchronously; argument errors are detected on the host before
 *    anything is enqueued and leave the state untouched.
 *  - One plan must not be used from two threads at once, and two steps of
 *    one plan must be enqueued on the same stream (they share the workspace).
 *  - NaN/Inf in gradients propagate; they are not checked.
 *  - Return codes are malt_status_t; malt_last_error() gives a message for
 *    the most recent failure on the calling thread.
 */
#ifndef LIBMALT_H
#define LIBMALT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MALT_OK = 0,
  MALT_ERR_INVALID_ARG = 1,     /* NULL pointer, bad count, hyper-parameter out of range */
  MALT_ERR_SHAPE = 2,           /* rows/cols < 1 or too large                        */
  MALT_ERR_ALIGNMENT = 3,       /* a device pointer is not 4-byte aligned             */
  MALT_ERR_STATE_MISMATCH = 4,  /* shapes or variant differ from those given at init  */
  MALT_ERR_HIP = 5,             /* a HIP runtime call failed                          */
  MALT_ERR_ALIAS = 6,           /* params / grads / state / workspace overlap          */
  MALT_ERR_SCRATCH_SIZE = 7,    /* workspace larger than the static scratch array      */
  MALT_ERR_BOUNDS = 8           /* malt_check_bounds found an address range outside its buffer */
} malt_status_t;

typedef enum { MALT_VARIANT_MALT = 0, MALT_VARIANT_MALTER = 1 } malt_variant_t;

/* One matrix, row-major. */
typedef struct {
  int64_t rows;
  int64_t cols;
} malt_shape_t;

/* Hyper-parameters of Algorithms 1 and 2 (eta, mu1, mu2, eps), the optional
 * decoupled weight decay (listed in the paper's hyper-parameter table, not in
 * the algorithms; 0 reproduces them exactly) and the Newton-Schulz reading.
 * Valid ranges: lr >= 0, 0 <= mu1 < 1, 0 <= mu2 < 1, eps > 0,
 * weight_decay >= 0, 1 <= ns_steps <= 64, ns_eps >= 0. */
typedef struct {
  double lr;
  double mu1;
  double mu2;
  double eps;
  double weight_decay;
  int32_t ns_steps;
  double ns_a, ns_b, ns_c;
  double ns_eps;
  int32_t precond_identity;    /* 1: L = R = I (the step is then Muon's, Sec. 3.1) */
} malt_hparams_t;

/* Defaults: lr 1.3e-3, mu1 0.95, mu2 0.99, eps 1e-8 (the paper's
 * hyper-parameter table), weight_decay 0 (a reading: the table lists 0.1 but
 * Algorithms 1 and 2 have no decay term; 0 reproduces them exactly),
 * ns_steps 5, (ns_a, ns_b, ns_c) = (3.4445, -4.7750, 2.0315), ns_eps 1e-7
 * (Muon's published Newton-Schulz settings; the paper gives none). */
void malt_hparams_default(malt_hparams_t* hp);

/* Opaque host-side plan: shapes, shape groups, device descriptor tables and
 * the step counter t.  Device buffers stay caller-owned. */
typedef struct malt_plan malt_plan_t;

/* Bytes of caller-provided device memory for `n` matrices.
 *  state_bytes: exactly 4 * sum(rows*cols + rows + cols), plus 4 per matrix
 *    for MALTER (the state sizes mn+m+n and mn+m+n+1 of the paper's
 *    memory-complexity table).  Layout (float32, contiguous, no padding):
 *    [M_0 .. M_{n-1} | l_0 .. l_{n-1} | r_0 .. r_{n-1} | nu_0 .. nu_{n-1}],
 *    M_i row-major rows x cols; malt_state_layout() gives the offsets.
 *  workspace_bytes: scratch for the preconditioner vectors, reduction
 *    partials, the bf16 Newton-Schulz buffers (padded to multiples of 256),
 *    the fp32 Newton-Schulz buffers of matrices with a short side of at most
 *    32, and the per-matrix scalar table.  Must be 256-byte aligned. */
malt_status_t malt_state_size(const malt_shape_t* shapes, int32_t n, malt_variant_t variant,
                              size_t* state_bytes, size_t* workspace_bytes);

/* Build a plan over `state_mem` / `workspace_mem` (device pointers of at least
 * the sizes above; state 16-byte aligned, workspace 256-byte aligned).
 * from_existing = 0: zero M, l, r, nu (the INITIALIZE line of Algorithms 1
 *   and 2) and set t = 0.
 * from_existing = 1: adopt the state already in `state_mem` (resume from a
 *   checkpoint) and set t = `step` (the number of steps already taken).
 * Uploads descriptor tables into the workspace on `stream` and synchronises
 * that stream before returning.  The device that owns the buffers and the
 * stream must be current (it also receives the kernels' LDS limit).  On
 * success *out owns a new plan. */
malt_status_t malt_init_state(malt_plan_t** out, const malt_shape_t* shapes, int32_t n,
                              malt_variant_t variant, void* state_mem, void* workspace_mem,
                              int32_t from_existing, int64_t step, void* stream);

/* Bytes of the library's static device scratch array (64 MiB). */
#define MALT_SCRATCH_BYTES (64ull << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same as
 * malt_init_state, but the workspace is a static array inside the library
 * (MALT_SCRATCH_BYTES per device, held until the process ends) instead of a
 * caller buffer.  Neither this call nor the steps of its plan call hipMalloc,
 * hipFree or any other allocating routine; the caller still allocates the
 * state and the parameters and gradients.
 * Errors: MALT_ERR_SCRATCH_SIZE when malt_state_size's workspace_bytes for these
 * shapes exceeds MALT_SCRATCH_BYTES (nothing is enqueued), plus those of
 * malt_init_state.
 * Sharing: every scratch plan on a device uses that device's one array.
 * Creating a scratch plan takes the array over (it zeroes it and writes its
 * tables there); steps of an older scratch plan on the same device then fail
 * with MALT_ERR_STATE_MISMATCH.  Work of two scratch plans that overlaps in
 * time on one device races on the array. */
malt_status_t malt_init_state_scratch(malt_plan_t** out, const malt_shape_t* shapes, int32_t n,
                                      malt_variant_t variant, void* state_mem, int32_t from_existing,
                                      int64_t step, void* stream);

/* Enqueue one step (Algorithm 1 or 2 by the plan's variant) on `stream`.
 * params[i]: device float32 rows x cols, updated in place.
 * grads[i]:  device float32 rows x cols, read only.
 * shapes/n must equal the init shapes (else MALT_ERR_STATE_MISMATCH).
 * Increments t on success; bias corrections use the new t.  Returns after
 * enqueueing, without waiting on the host for anything: the caller
 * synchronises `stream` before reading results.  When a param or grad pointer
 * differs from the previous step's, the plan's device pointer table is first
 * rewritten by small kernels on `stream` (the pointers travel as kernel
 * arguments). */
malt_status_t malt_step(malt_plan_t* plan, float* const* params, const float* const* grads,
                        const malt_shape_t* shapes, int32_t n, const malt_hparams_t* hp,
                        void* stream);

/* Float offsets (from state_mem) of matrix i's M, l, r, nu (nu = -1 for MALT). */
typedef struct {
  int64_t M, l, r, nu;
} malt_state_layout_t;
malt_status_t malt_state_layout(const malt_plan_t* plan, int32_t i, malt_state_layout_t* out);

/* Byte offsets into workspace_mem of matrix i's last-step intermediates,
 * for stage-by-stage checks:
 *  Lv, Rv:  float32 diagonals of L_t (rows) and R_t (cols);
 *  O:       bf16 Newton-Schulz output in the canonical orientation:
 *           min(rows,cols) x max(rows,cols), row pitch O_pitch elements; it is
 *           W's orientation when rows <= cols and its transpose otherwise
 *           (O_transposed = 1);
 *  X0:      bf16 L M R before normalisation, same layout; valid only after a
 *           step with ns_steps == 1 (later iterations reuse the buffer);
 *  scalars: float64 [s=||Mt||_F, sigma=1/(s+ns_eps), nu_t, alpha_t, ||O||^2,
 *           ||D||^2, graft=||O||/(||D||+eps), coef=lr*alpha*graft];
 *  A, B:    bf16 last Newton-Schulz iteration's A = X X^T and B' = a I + b A
 *           + c A A (symmetric, m' x m' padded to AB_pitch = a multiple of 256
 *           rows and columns); B holds [B'_hi | B'_lo] with row pitch
 *           2 AB_pitch when B_split = 1. Unused (0) for matrices with a short
 *           side of at most 32, whose Newton-Schulz runs in fp32. */
typedef struct {
  int64_t Lv, Rv, O, X0, scalars;
  int64_t O_pitch;
  int64_t O_transposed;
  int64_t A, B, AB_pitch, B_split;
} malt_debug_layout_t;
malt_status_t malt_debug_layout(const malt_plan_t* plan, int32_t i, malt_debug_layout_t* out);

/* Host-side proof that the kernels of a plan over these shapes stay inside
 * their buffers; for tests and for callers who want the check for their own
 * shapes.  Needs no plan and no device: it builds the work lists that
 * malt_init_state would build and, for every entry of every list (padding
 * entries of the XCD-ordered Newton-Schulz lists included), derives with the
 * kernels' own address functions the byte ranges the kernel can address: the
 * direct-load spans of both operands over the whole contraction, stores of
 * output tiles and mirrors, partial-slot indices, the layout of the workspace
 * regions.  The Newton-Schulz operand offsets, passed to the hardware as
 * 32-bit buffer offsets, must also stay below 4 GiB.
 * shrink_bytes >= 0 checks the Newton-Schulz operand and output buffers (the
 * ones read through buffer resources with the hardware range check off) as if
 * they were that many bytes shorter: with 16 it must fail, since the kernels
 * reach the last bytes of those buffers.
 * Returns MALT_OK with *ranges_checked = the number of checks made, or
 * MALT_ERR_BOUNDS with malt_last_error() naming the first kernel, matrix,
 * tile and byte range that does not fit (or the usual argument errors). */
malt_status_t malt_check_bounds(const malt_shape_t* shapes, int32_t n, malt_variant_t variant,
                                int64_t shrink_bytes, int64_t* ranges_checked);

/* Condition numbers of diag(l_t) and diag(r_t) for every matrix of the plan:
 * the quantity the paper's analysis of the diagonal preconditioners (Sec. 5.4,
 * the figure of preconditioner condition numbers per layer) reports for the
 * attention and MLP matrices, here for the state the last enqueued step left.
 * kappa(diag v) = max_i v_i / min_i v_i (v >= 0 is a running mean of squares);
 * +inf when min_i v_i = 0 (a zero row or column, or a plan that has not
 * stepped), NaN when an entry is NaN.
 * out: device float64 buffer of 2 * n values, 8-byte aligned, written as
 *   [kappa_l(0), kappa_r(0), kappa_l(1), kappa_r(1), ...]; caller-owned and
 *   not overlapping the state or workspace.
 * Enqueued on `stream` (one small kernel) after whatever is already there;
 * nothing waits on the host.  Errors: MALT_ERR_INVALID_ARG (NULL plan or
 * out), MALT_ERR_ALIGNMENT, MALT_ERR_ALIAS, MALT_ERR_STATE_MISMATCH (a
 * scratch plan whose array was taken over), MALT_ERR_HIP. */
malt_status_t malt_precond_condition(const malt_plan_t* plan, double* out, void* stream);

/* Step counter t (number of steps enqueued so far). */
int64_t malt_plan_step(const malt_plan_t* plan);

/* Per-phase device timing with HIP events recorded on the step's stream.
 * When enabled, every malt_step records an event pair around each phase;
 * malt_profile_read synchronises the last recorded event and reports the
 * summed milliseconds and launch counts since the last reset.
 * Phases: 0 momentum+row/col sums, 1 preconditioner finalise,
 * 2 scale+convert, 3 norm scalars, 4 NS Gram, 5 NS polynomial, 6 NS update,
 * 7 graft scalars, 8 back-map+write. */
#define MALT_NUM_PHASES 9
typedef struct {
  double ms[MALT_NUM_PHASES];
  int64_t launches[MALT_NUM_PHASES];
  double bytes[MALT_NUM_PHASES];   /* algorithmic HBM bytes per step, per phase */
  double flops[MALT_NUM_PHASES];   /* algorithmic flops per step, per phase     */
} malt_profile_t;
malt_status_t malt_profile_enable(malt_plan_t* plan, int32_t enable);
malt_status_t malt_profile_read(malt_plan_t* plan, malt_profile_t* out, int32_t reset);

/* Release the plan (host memory and profiling events only). */
void malt_destroy_state(malt_plan_t* plan);

const char* malt_status_string(malt_status_t status);
const char* malt_last_error(void);
const char* malt_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LIBMALT_H */
