/*
 * optima.h -- C ABI of the OPTIMA weight-update hot path on AMD MI355X (gfx950).
 *
 * OPTIMA (arXiv 2512.13886) rewrites the layer-wise weight reconstruction that
 * follows mask selection as one quadratic program per output column (Eq. (3)-(6)):
 *
 *     minimise  (w_j - w0_j)^T H (w_j - w0_j)   subject to  w_j[i] = 0 for every
 *     pruned entry i (mask[j][i] == 0),
 *
 * with one Hessian H = X^T X shared by all columns of the layer. The library
 * computes H from calibration tokens, damps it, estimates its spectral norm and
 * solves all column QPs together with a batched restarted accelerated
 * primal-dual hybrid gradient (rAPDHG) method (Section 3.3-3.4, Algorithm 1).
 *
 * Conventions shared by every call
 *   - Matrices are row-major. The weight and mask are stored [n_cols][d]: row j
 *     holds the QP of output column j (the PyTorch Linear layout; the paper
 *     writes W as d_in x d_out, Eq. (3)).
 *   - Mask bytes: 1 keeps the weight, 0 prunes it (Eq. (1)).
 *   - Every pointer argument is a device pointer owned by the caller unless
 *     stated otherwise; the library keeps no pointer after a call returns and
 *     allocates no device memory. Work buffers come from the caller through a
 *     `ws` argument sized by the matching *_workspace_bytes query.
 *   - All calls are ordered on `stream` (NULL = the default stream).
 *   - Errors are returned before any kernel is launched when they come from
 *     argument validation. HIP failures map to OPTIMA_E_HIP.
 */
#ifndef OPTIMA_H
#define OPTIMA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int optima_status;

#define OPTIMA_OK 0
#define OPTIMA_E_INVAL (-1)       /* NULL pointer, bad size, misaligned or aliased buffer */
#define OPTIMA_E_HIP (-2)         /* a HIP runtime call or kernel launch failed */
#define OPTIMA_E_NONFINITE (-3)   /* NaN or Inf in H, W0 or the spectral norm */
#define OPTIMA_E_WORKSPACE (-4)   /* ws NULL or smaller than the size query returned */
#define OPTIMA_E_UNSUPPORTED (-5) /* unsupported dtype, or the device is not gfx950 */

#define OPTIMA_DTYPE_F32 0
#define OPTIMA_DTYPE_BF16 1
#define OPTIMA_DTYPE_F64 2

/* Arithmetic of the solver's per-iteration H-products (optima_solver_opts).
 * FP32: v_mfma_f32_16x16x4_f32, fp32 products and sums.
 * BF16X3: every fp32 operand v is split into bf16 planes hi = rne(v),
 *   lo = rne(v - hi), and a*b is formed as hi*hi + hi*lo + lo*hi on
 *   v_mfma_f32_16x16x32_bf16 with fp32 accumulation; the dropped terms are
 *   below 3 * 2^-16 |a b| per product. The precision applies to every
 *   product of a solve, the setup products H w0 and H x0 included (with at
 *   most 8 active columns the iteration products stream H once per
 *   iteration through a 16-column MFMA kernel, with the same products). BF16X3 is
 *   the default: on the 4096-wide outlier layer its
 *   solutions differ from FP32's by under 1e-5 relative (Frobenius) and it
 *   runs the iteration about 2.5x faster. */
#define OPTIMA_PREC_FP32 0
#define OPTIMA_PREC_BF16X3 1

/* Solve method (optima_solver_opts.method).
 * RAPDHG: the paper's batched restarted accelerated method on the constrained
 *   form, Eq. (6) (described with optima_qp_solve_batched below).
 * CG: the unconstrained form of Eq. (7)-(11). With the pruned entries fixed
 *   at zero the optimum solves H_KK x_K = (H w0)_K for every column, which
 *   conjugate gradients reach without restarts or a step size: from
 *   x = sel(mask, w0, +0), r = P (H w0 - H x), p = r, each iteration forms
 *   q = H p (one batched product), alpha = r.r / p.q_K, x += alpha p,
 *   r -= alpha q_K, beta = r'.r' / r.r, p = r' + beta p, with x, r and p exactly
 *   zero off K. Columns are tested every check_every iterations with the same
 *   rule as RAPDHG, evaluated from the recurrence residual (r_d = 2 ||r_K||,
 *   gap = 2 |x.r|); lambda_max, the beta_* constants, step_safety and
 *   restarts are unused (lambda_max may be NULL). */
#define OPTIMA_METHOD_RAPDHG 0
#define OPTIMA_METHOD_CG 1

/* Human-readable name of a status code (static string, never NULL). */
const char* optima_status_string(optima_status status);

/* Library ABI version (increments on any signature change). */
int optima_abi_version(void);

/* ---------------------------------------------------------------------------
 * Hessian accumulation -- Section 3.4 "Hessian calculation", Algorithm 1.
 *
 * H[d][d] (fp32) = (accumulate ? H : 0) + X^T X, where X[n_tok][d] holds n_tok
 * calibration tokens (one or many 2048-token sequences; the paper sums
 * y_i^T y_i sequence by sequence, which gives the same matrix as stacking).
 * X is fp32 (dtype OPTIMA_DTYPE_F32) or bf16 (OPTIMA_DTYPE_BF16); products are
 * formed exactly and summed in fp32. Both triangles of H are written and the
 * result is exactly symmetric; with accumulate = 1 the lower triangle of the
 * incoming H is read and taken as the whole matrix. n_tok = 0 leaves H as it is
 * (accumulate = 1) or zeroes it. X must be 16-byte aligned (OPTIMA_E_INVAL
 * otherwise); H may alias nothing else. ws must hold
 * optima_hessian_workspace_bytes(n_tok, d, dtype) bytes: split-K partial sums,
 * plus a token-slab transpose buffer unless X is bf16 with d % 256 == 0 (then
 * token rows are read in place and only a 64-row tail buffer is needed).
 * ------------------------------------------------------------------------- */
size_t optima_hessian_workspace_bytes(int64_t n_tok, int64_t d, int dtype);
optima_status optima_hessian_accumulate(const void* X, int dtype, int64_t n_tok,
                                        int64_t d, float* H, int accumulate,
                                        void* ws, size_t ws_bytes,
                                        hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Damping. The paper's H = X^T X is only positive semi-definite (Eq. (6));
 * this call adds lambda * I with lambda = rel_damp * trace(H) / d, which makes
 * every column QP strictly convex so its optimum (Eq. (10)-(11)) is unique.
 * The trace is summed in fp64 on the device. lambda_out (device, one float,
 * required) receives lambda; if the trace is not finite, H is left unchanged
 * and lambda_out receives NaN (the solve then reports OPTIMA_E_NONFINITE).
 * ------------------------------------------------------------------------- */
optima_status optima_hessian_damp(float* H, int64_t d, float rel_damp,
                                  float* lambda_out, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Shared diagonal preconditioning (Jacobi). Not in the paper; a reading usual
 * for PDLP-family first-order solvers. One scaling serves all columns, so the
 * batching of Algorithm 1 is unchanged.
 *
 * H[d][d] fp32 (symmetric, damped) is replaced in place by D H D with
 * D_i = H_ii^(-1/2) (computed in fp64, rounded to fp32; 1 where H_ii is not
 * positive and finite), and scale_out[d] (device) receives D. The factor of
 * entry (i, j) is the fp32 product D_i D_j, so exact symmetry is kept. In the
 * coordinates y = D^-1 w every column QP of Eq. (6) keeps its zero pattern and
 * objective values, and its optimum is D^-1 w*. The outlier channels of
 * transformer layers make H badly scaled (condition numbers of 10^3 - 10^4);
 * D H D is well conditioned and the solvers need far fewer iterations.
 * Workflow: damp, optima_hessian_jacobi, optima_spectral_norm on the scaled H,
 * then optima_qp_solve_batched with opts.col_scale = scale_out: the solver
 * iterates on the scaled problem, tests termination with the gradient in the
 * original coordinates and writes W_out in the original coordinates.
 * ------------------------------------------------------------------------- */
optima_status optima_hessian_jacobi(float* H, int64_t d, float* scale_out,
                                    hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Spectral norm of H for the solver's step size (Section 3.3: the first-order
 * method's bottleneck is products with H; its step needs ||Q|| = 2 lambda_max).
 * H must be symmetric positive semi-definite (X^T X + lambda I is), [d][d]
 * fp32, 4-byte aligned (16-byte alignment and d % 4 == 0 enable vector loads).
 *
 * V0: [block][d] fp32 device array of start vectors (row a is vector a), not
 * modified; 1 <= block <= OPTIMA_SPECTRAL_MAX_BLOCK.
 *   block == 1: power iteration. Iteration i forms y = H v with v of unit
 *     length, rho_i = v^T y and v <- y / ||y||.
 *   block >= 2: subspace (orthogonal) iteration with Rayleigh-Ritz.
 *     Iteration i multiplies an orthonormal basis Q of the current block by
 *     H (Y = H Q, one pass over H) and takes rho_i = the largest Ritz value
 *     of span(Q), i.e. the largest eigenvalue of Q^T H Q; the next basis spans
 *     Y (Cholesky QR in fp64). Convergence goes as lambda_{block+1} /
 *     lambda_1 instead of lambda_2 / lambda_1, so Hessians whose top
 *     eigenvalues cluster (outlier channels) need a handful of passes. The
 *     b x b eigenvalue is found by repeated squaring, within 1e-8 relative.
 *     Directions that become numerically dependent (Cholesky pivot below
 *     1e-14 of the diagonal) are dropped.
 * Both stop once |rho_i - rho_{i-1}| <= tol * rho_i, or after max_iters
 * iterations. lambda_max (device, one float) receives the last rho (NaN if H
 * holds NaN/Inf and block >= 2); iters (device int32, may be NULL) the
 * iteration count. Blocking: the call synchronises `stream` a few times to
 * test convergence. ws: optima_spectral_norm_workspace_bytes(d, block) bytes.
 * ------------------------------------------------------------------------- */
#define OPTIMA_SPECTRAL_MAX_BLOCK 16
size_t optima_spectral_norm_workspace_bytes(int64_t d, int block);
optima_status optima_spectral_norm(const float* H, int64_t d, const float* V0,
                                   int block, int max_iters, float tol,
                                   void* ws, size_t ws_bytes, float* lambda_max,
                                   int32_t* iters, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * optima_spectral_norm for callers that cannot allocate memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, iterations, results and blocking behaviour as
 * optima_spectral_norm, without `ws`: the work buffer is a fixed array of
 * OPTIMA_SPECTRAL_NOALLOC_SCRATCH_BYTES inside the library, one copy per
 * device, held from the library's load until the process ends. It covers
 * every block size for d <= OPTIMA_SPECTRAL_NOALLOC_MAX_DIM; a larger d
 * returns OPTIMA_E_WORKSPACE before any launch. The call allocates nothing
 * (no device memory, no pinned host memory): its convergence polls copy into
 * host stack memory and synchronise `stream`. The first call on a device
 * looks up the array's device address once (hipGetSymbolAddress).
 * Every call on a device shares that device's array and leaves its contents
 * there: calls that overlap on one device (two streams, or two host threads)
 * race on it and must be serialised by the caller. Calls on different
 * devices are independent.
 * ------------------------------------------------------------------------- */
#define OPTIMA_SPECTRAL_NOALLOC_MAX_DIM 16384
#define OPTIMA_SPECTRAL_NOALLOC_SCRATCH_BYTES (8454144)
optima_status optima_spectral_norm_noalloc(const float* H, int64_t d, const float* V0,
                                           int block, int max_iters, float tol,
                                           float* lambda_max, int32_t* iters,
                                           hipStream_t stream);

/* ---------------------------------------------------------------------------
 * The same lambda_max (the step size of Section 3.3's first-order solver) by
 * the symmetric Lanczos process with full reorthogonalisation. Step j builds
 * q_j of an orthonormal basis of the Krylov space span{v0, H v0, ...,
 * H^(j-1) v0} from one product with H:
 *   w = H q_j, alpha_j = q_j^T w, w <- w - alpha_j q_j - beta_(j-1) q_(j-1),
 *   w <- w - Q (Q^T w), beta_j = ||w||, q_(j+1) = w / beta_j,
 * and rho_j = the largest eigenvalue of the j x j tridiagonal matrix
 * T = tridiag(beta; alpha; beta) = Q^T H Q (the largest Ritz value of the
 * Krylov space; never above lambda_max(H), non-decreasing in j). Its
 * convergence goes as a Chebyshev polynomial of the step count, so spectra
 * whose top has no gap (near-isotropic inputs, or H after diagonal scaling)
 * need far fewer passes over H than the subspace iteration of
 * optima_spectral_norm. The basis is fp32, all sums fp64; the eigenvalue of
 * T comes from Sturm-count bisection in fp64 (relative width 1e-15).
 *
 * H: [d][d] fp32, symmetric, 4-byte aligned (16-byte alignment and d % 4 ==
 * 0 enable vector loads). v0: [d] fp32 device start vector, not modified.
 * It stops once |rho_j - rho_(j-1)| <= tol * rho_j, once beta_j <= 1e-6 *
 * rho_j (the Krylov space is invariant: rho_j is an eigenvalue), or after
 * min(max_steps, d) steps, 1 <= max_steps <= OPTIMA_LANCZOS_MAX_STEPS.
 * Without a gap at the top of the spectrum the Ritz value rises by small
 * amounts long before it converges: there tol = 1e-7 stops within about
 * 1e-6 of lambda_max where 1e-6 can stop 3e-4 short.
 * lambda_max (device, one float) receives the last rho (0 for a zero v0, NaN
 * if H or v0 holds NaN/Inf); steps (device int32, may be NULL) the step
 * count. Blocking: the call synchronises `stream` every 8 steps to test
 * convergence. ws: optima_spectral_lanczos_workspace_bytes(d, max_steps)
 * bytes (about max_steps * d * 4 for the basis).
 * ------------------------------------------------------------------------- */
#define OPTIMA_LANCZOS_MAX_STEPS 256
size_t optima_spectral_lanczos_workspace_bytes(int64_t d, int max_steps);
optima_status optima_spectral_lanczos(const float* H, int64_t d, const float* v0,
                                      int max_steps, float tol, void* ws,
                                      size_t ws_bytes, float* lambda_max,
                                      int32_t* steps, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Wanda mask selection -- the mask M that the weight update starts from
 * (Algorithm 1 takes it from a selector; the configurations use the Wanda
 * saliency cited in Section 2, with the 2:4 pattern of Section 4).
 *
 * W0: [n_cols][d] fp32 (row j = column QP j), 4-byte aligned. col_sq: the
 * squared input norms c[i] = sum_t X[t][i]^2, element i at col_sq[i * stride],
 * fp32 (OPTIMA_DTYPE_F32) or fp64 (OPTIMA_DTYPE_F64); e.g. the diagonal of the
 * undamped Hessian is H with stride d + 1. mask: [n_cols][d] uint8 output
 * (1 keeps), 4-byte aligned, overlapping neither input.
 * score[j][i] = W0[j][i]^2 * c[i] in fp64 (the square of the saliency
 * |W0[j][i]| sqrt(c[i]), same order; exact square, one rounded product).
 * pattern OPTIMA_MASK_UNSTRUCTURED keeps the d - floor(sparsity * d) highest
 * scores of every row (0 <= sparsity <= 1); OPTIMA_MASK_2TO4 keeps the two
 * highest of every group [4g, 4g + 4) of a row (d % 4 == 0). Equal scores go
 * to the lower index; NaN scores rank below all others; -0 equals +0. The
 * result is a pure function of the input values: bit-exact against any IEEE
 * implementation of the same rule. Asynchronous on `stream`.
 * ------------------------------------------------------------------------- */
#define OPTIMA_MASK_UNSTRUCTURED 0
#define OPTIMA_MASK_2TO4 1
optima_status optima_wanda_mask(const float* W0, int64_t n_cols, int64_t d,
                                const void* col_sq, int col_sq_dtype,
                                int64_t col_sq_stride, int pattern,
                                double sparsity, uint8_t* mask,
                                hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Layer forward pass -- Algorithm 1: the layer outputs y = L(x) on the
 * calibration tokens, and the activations X <- L(X) handed to the next layer
 * once L is pruned. Also the squared output error between two weight sets.
 * The layer-wise error of Section 4 (MSE against the dense layer's outputs,
 * OPTIMA's over another method's) is a ratio of two such errors.
 *
 * Z[n_tok][d_out] = X W^T with X [n_tok][d_in] bf16 (row-major, 16-byte
 * aligned, d_in a multiple of 64) and W [d_out][d_in] fp32 rounded to bf16
 * on the device (round to nearest even), products exact, sums in fp32.
 * d_out must be a multiple of 4.
 * Y (nullable): act(Z), act OPTIMA_ACT_NONE or OPTIMA_ACT_SILU (z / (1 +
 *   e^-z) in fp32), stored as y_dtype OPTIMA_DTYPE_BF16 (round to nearest
 *   even, 8-byte aligned) or OPTIMA_DTYPE_F32 (16-byte aligned).
 * err_out (nullable, device double): receives the sum over all outputs of
 *   (Z - Y_ref)^2, accumulated in fp64 in a fixed order; Y_ref (fp32
 *   [n_tok][d_out], 16-byte aligned) is then required when n_tok > 0: a
 *   reference Z, e.g. the dense layer's from an earlier call with act NONE
 *   and fp32 Y. Y_ref without err_out, or neither Y nor err_out, is
 *   OPTIMA_E_INVAL. With n_tok = 0, X, Y and Y_ref are not read and
 *   err_out receives 0.
 * ws: optima_linear_forward_workspace_bytes(n_tok, d_in, d_out) bytes
 * (the bf16 weights and per-tile partial sums). The call synchronises the
 * stream once. It returns OPTIMA_E_NONFINITE if W holds a NaN or Inf.
 * ------------------------------------------------------------------------- */
#define OPTIMA_ACT_NONE 0
#define OPTIMA_ACT_SILU 1
size_t optima_linear_forward_workspace_bytes(int64_t n_tok, int64_t d_in, int64_t d_out);
optima_status optima_linear_forward(const void* X, int64_t n_tok, int64_t d_in,
                                    const float* W, int64_t d_out, int act, void* Y,
                                    int y_dtype, const float* Y_ref, double* err_out,
                                    void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Batched column-QP solve -- Eq. (6), Algorithm 1, Section 3.3-3.4.
 *
 * For every row j < n_cols of W0 (fp32 values) and mask (uint8), writes
 *   W_out[j] = argmin (w - W0[j])^T H (w - W0[j])  s.t. w[i] = +0.0 where
 *              mask[j][i] == 0,
 * reached with the batched rAPDHG iteration. The pruned entries are fixed
 * through equal lower and upper bounds (Section 3.4), i.e. the projection
 * keeps them at exactly +0.0 (bit pattern 0). Per column j, with
 * alpha_k = 2/(k+2), eta_k = (k+1)/(2L), L = 2 lambda_max (1 + step_safety):
 *   x_md = (1-alpha) x_ag + alpha x;  g = 2 H (x_md - w0);
 *   x = sel(mask, x - eta g, +0);     x_ag = (1-alpha) x_ag + alpha x,
 * starting from x = x_ag = sel(mask, w0, +0). Every check_every iterations
 * (and at max_iters) x and x_ag are scored by r_d = ||g restricted to kept
 * entries||, gap = |z^T g|, KKT = sqrt(r_d^2 + gap^2); the lower-KKT one is the
 * candidate (ties: x_ag). A column terminates (unless fixed_iters) when
 * r_d <= eps_abs + eps_rel ||2 H w0|| and gap <= eps_abs + eps_rel (|P| + |D|)
 * with P = f(cand), D = w0^T H w0 - cand^T H cand (Appendix D tolerances). It
 * restarts to the candidate on KKT decay by beta_sufficient, on decay by
 * beta_necessary without progress since the last check, or when the iterations
 * since the last restart reach beta_artificial times the total; a restart is
 * accepted only if it does not raise the objective above the previous restart
 * point's. Columns are fully independent: the result for a column does not
 * depend on the others in the batch (Algorithm 1 batching).
 *
 * H: [d][d] fp32, symmetric, 16-byte aligned. lambda_max: device float (from
 * optima_spectral_norm, optima_spectral_lanczos or the caller). W_out: [n_cols][d] fp32, must not
 * overlap W0. stats (host struct of device arrays, may be NULL; each array may
 * be NULL): per column iterations run, accepted restarts, convergence flag,
 * objective at the start point sel(mask, w0, 0), objective and KKT of W_out
 * (computed on the device from the maintained products). info (host, may be
 * NULL) receives run totals (for CG the timed window of each run of
 * iterations also covers their CG update kernels). ws:
 * optima_qp_workspace_bytes(d, n_cols) bytes.
 * Blocking: the call synchronises `stream` once per check to learn how many
 * columns are still active. Non-convergence is not an error; it is reported
 * per column. Returns OPTIMA_E_NONFINITE if H or W0 holds NaN/Inf,
 * lambda_max is not a positive finite number, or opts.col_scale holds an
 * entry that is not positive and finite.
 * ------------------------------------------------------------------------- */
typedef struct {
  int64_t max_iters;      /* >= 0; the paper uses 100000 (Table 8) */
  int32_t check_every;    /* >= 1; default 64 */
  int32_t fixed_iters;    /* 1: run exactly max_iters, checks only restart */
  float eps_rel;          /* default 0.01 (Table 8) */
  float eps_abs;          /* default 0.01 (Table 8) */
  float beta_sufficient;  /* default 0.2 */
  float beta_necessary;   /* default 0.8 */
  float beta_artificial;  /* default 0.36 */
  float step_safety;      /* default 1e-3 */
  int32_t restarts;       /* 0 disables restarts; default 1 */
  int32_t precision;      /* OPTIMA_PREC_BF16X3 (default) or OPTIMA_PREC_FP32 */
  int32_t method;         /* OPTIMA_METHOD_RAPDHG (default) or OPTIMA_METHOD_CG */
  const float* col_scale; /* NULL (default), or the [d] device diagonal D of a
                             preconditioned H = D H0 D (optima_hessian_jacobi);
                             see "Shared diagonal preconditioning" */
  int32_t sparse;         /* 1 (default): when precision is BF16X3, method is
                             RAPDHG and no mask row keeps more than 2 entries
                             of any group of 4 consecutive columns (a 2:4 mask,
                             Section 4), the iteration products take x
                             2:4-compressed and multiply on the sparse MFMA
                             (v_smfmac_f32_16x16x64_bf16), skipping the pruned
                             entries; the same products are formed, summed in
                             another order. 0: dense products always. */
  int32_t cooperative;    /* 1 (default): when at most 8 columns are still active
                             and d <= 4096, the iterations between two checks
                             run as one cooperative launch (hipLaunchCooperativeKernel)
                             that keeps H's split planes in registers and meets
                             at a grid barrier between iterations; the same
                             products and updates, bit for bit, as one launch
                             per iteration. 0: one launch per iteration (for
                             callers whose streams cannot take cooperative
                             launches). Falls back to per-iteration launches
                             by itself when the device refuses them. */
} optima_solver_opts;

typedef struct {
  int32_t* iters;
  int32_t* restarts;
  uint8_t* converged;
  float* f_initial;
  float* f_final;
  float* kkt_final;
} optima_solve_stats;

typedef struct {
  int64_t iterations;         /* iterations run by the longest-running column */
  int64_t gemm_calls;         /* H-product launches (including the two at setup) */
  int64_t row_products;       /* sum over those launches of the columns multiplied */
  int64_t checks;             /* check passes */
  int64_t timed_launches;     /* H-product launches between checks (the iteration loop) */
  int64_t timed_row_products; /* columns multiplied by those launches */
  double timed_product_ms;    /* their device time, from HIP events recorded on `stream`
                                 around each run of back-to-back product launches */
  int64_t sparse_products;    /* 1 if the iteration products ran 2:4-sparse (opts.sparse) */
  int64_t few_launches;       /* the timed launches that ran the few-column kernel (at most 8
                                 active columns with split planes: H streamed once per launch) */
  int64_t few_row_products;   /* columns multiplied by those launches */
  double few_product_ms;      /* their device time (included in timed_product_ms) */
  int64_t persistent_launches; /* blocks of few-column iterations (the iterations between two
                                  checks) that ran as one cooperative launch keeping H's planes
                                  in registers (d <= 4096); each counts all of its iterations in
                                  few_launches */
} optima_solve_info;

void optima_solver_opts_default(optima_solver_opts* opts);
size_t optima_qp_workspace_bytes(int64_t d, int64_t n_cols);
optima_status optima_qp_solve_batched(const float* H, int64_t d,
                                      const float* lambda_max, const float* W0,
                                      const uint8_t* mask, int64_t n_cols,
                                      const optima_solver_opts* opts, void* ws,
                                      size_t ws_bytes, float* W_out,
                                      const optima_solve_stats* stats,
                                      optima_solve_info* info,
                                      hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* OPTIMA_H */
