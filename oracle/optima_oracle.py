"""CPU oracle for the OPTIMA weight-update hot path.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or link
this module: only the tests, the smoke check and the benchmark's CPU-baseline
leg use it. It is a plain, slow, fp64 NumPy restatement of what the method
computes, written from the paper (OPTIMA, arXiv 2512.13886); it shares no code,
constants or helpers with the HIP library.

What each function follows
--------------------------
hessian          Section 3.4 "Hessian calculation": H = sum over calibration
                 sequences y_i of y_i^T y_i (the incremental form of Y^T Y).
damp             Not in the paper (it only states H = X^T X is PSD, Eq. (6)).
                 Reading: H + lambda I with lambda = rel * trace(H) / d, which
                 makes every column QP strictly convex (unique optimum).
power_iteration  Step size of the first-order solver (Section 3.3 names rAPDHG
                 but prints no step rule). Reading: Rayleigh quotient of the
                 power iteration started from a given vector.
subspace_iteration
                 The same quantity by block (orthogonal) iteration with
                 Rayleigh-Ritz, the textbook generalisation of the power
                 iteration to b vectors (Golub & Van Loan, "Matrix
                 Computations", orthogonal iteration; Saad, "Numerical Methods
                 for Large Eigenvalue Problems", subspace iteration). Its
                 convergence rate is lambda_{b+1}/lambda_1 instead of
                 lambda_2/lambda_1, which matters for Hessians whose top
                 eigenvalues cluster (outlier channels). b = 1 is
                 power_iteration.
lanczos          The same quantity by the Lanczos method with full
                 reorthogonalisation (Lanczos 1950; Golub & Van Loan, "Matrix
                 Computations", the symmetric Lanczos process; Parlett, "The
                 Symmetric Eigenvalue Problem"): the largest Ritz value of the
                 Krylov space of the start vector, from the tridiagonal matrix
                 of the three-term recurrence. It converges like a Chebyshev
                 polynomial of the step count, so spectra whose top has no gap
                 (near-isotropic inputs, or H after diagonal scaling) need far
                 fewer products with H than subspace_iteration.
wanda_mask       The mask the weight update starts from (Algorithm 1 takes M from
                 a selector; the configurations use Wanda, cited in Section 2,
                 with the 2:4 pattern of Section 4): score w0_ji^2 c_i in fp64
                 (the square of the saliency |w0_ji| sqrt(c_i), same order), per
                 row the d - floor(s d) highest scores, or the two highest of
                 every group of 4; ties go to the lower index, NaN scores last.
jacobi_scale     Shared diagonal preconditioning (not in the paper; a reading,
                 usual for PDLP-family solvers): D = diag(H)^(-1/2) and
                 H' = D H D. The column QPs in y = D^-1 w have Hessian H' and
                 anchors D^-1 w0, the same zero pattern, the same objective
                 values and optima y* = D^-1 w*. rapdhg and cg take D as
                 `scale`: they iterate on the scaled problem, test termination
                 in the original coordinates and return w = D y.
objective        Eq. (4)/(6): f_j = dw_j^T H dw_j with dw_j = w_j - w0_j.
closed_form      Eq. (10)-(11): the unconstrained QP over the kept set I has
                 Q = H_II, c = -2 H_IS w_S, so dw_I = H_II^{-1} H_IS w_S and
                 w_I = w0_I + H_II^{-1} H_IS w0_S, w_S = 0 (Cholesky of H_II).
kkt_solve        Eq. (6) solved through its KKT system (stationarity plus the
                 equality constraints of Eq. (5)) with a dense LU solve; used on
                 tiny d only, as an independent check of closed_form.
cg               Eq. (7)-(11): with the pruned entries fixed at zero the QP of
                 Eq. (6) becomes unconstrained in the kept entries, and its
                 stationarity condition is the linear system
                 H_KK x_K = (H w0)_K (Eq. (11) written for w instead of dw).
                 The paper describes this form but solves the constrained one;
                 this is the textbook conjugate-gradient method (Hestenes and
                 Stiefel) on that system, column by column, from the same start
                 point and with the same termination test as rapdhg.
rapdhg           Section 3.3 / 3.4: the batched restarted accelerated
                 primal-dual hybrid gradient solve of Eq. (6), with the pruned
                 entries fixed through equal lower and upper bounds (Section 3.4
                 "Equality constraints"). The paper only cites the algorithm, so
                 the iteration below is this module's reading of it for a QP
                 whose only constraints are bounds (the dual block is empty):
                   alpha_k = 2/(k+2), eta_k = (k+1)/(2L), L = 2 lambda_max (1+delta)
                   x_md = (1-alpha) x_ag + alpha x
                   g    = 2 H (x_md - w0)              (gradient of Eq. (6))
                   x    = sel(mask, x - eta g, 0)       (projection on the bounds)
                   x_ag = (1-alpha) x_ag + alpha x
                 Every `check_every` iterations (and at the last one) the
                 iterate x and the average x_ag are scored by
                   r_d = ||g_K||_2, gap = |z^T g|, KKT = sqrt(r_d^2 + gap^2)
                 and the lower-KKT one is the candidate (ties: x_ag). A column
                 terminates when r_d <= eps_abs + eps_rel ||2 H w0||_2 and
                 gap <= eps_abs + eps_rel (|P| + |D|), P = f(cand),
                 D = -cand^T H cand + w0^T H w0 (Appendix D tolerances). A
                 restart to the candidate happens on sufficient decay
                 (KKT <= 0.2 KKT_restart), on necessary decay without local
                 progress (KKT <= 0.8 KKT_restart and KKT > KKT_previous check),
                 or when the inner loop is long (k >= 0.36 t); it is accepted
                 only if it does not raise the objective above the last
                 restart point's. At max_iters every active column stops at
                 its candidate; no restart is applied or counted there.

Parity status
-------------
hessian, damp, objective, closed_form, kkt_solve: pinned by brute force, exact
rational arithmetic and closed forms in the CPU tests. power_iteration: pinned
by LAPACK eigenvalues. subspace_iteration: pinned by LAPACK eigenvalues of
matrices with known spectra, the Ritz upper bound, a hand-worked 2x2 case and
its reduction to power_iteration at b = 1. lanczos: pinned by the
recurrence coefficients of the discrete Chebyshev (Gram) polynomials (H =
diag(1..n), all-ones start), the Rayleigh-Ritz value of an explicitly built
Krylov basis, a hand-worked 2x2 case, breakdown on a two-eigenvalue spectrum,
the monotone Ritz bound, and LAPACK eigenvalues of the layer Hessians. wanda_mask: pinned by the rank
definition evaluated by brute force (an entry is kept iff fewer than k
entries beat it), hand-made ties and the keep counts. rapdhg: its fixed point is pinned by closed_form and its
iterates by the invariants (pruned entries exactly +0.0, accepted restarts never
raise the objective, the accelerated O(1/k^2) bound without restarts); the exact
trajectory (step schedule, restart constants) is the reading above and is
"parity unpinned": the paper prints no trajectory to compare against. cg:
pinned by finite termination (|K| steps reach the closed form in exact
arithmetic; fp64 on small systems to 1e-10), the one-step solution of the
hand-worked 2x2 case, A-conjugacy of the search directions and the monotone
decrease of the energy error. jacobi_scale: pinned by the unit diagonal of
D H D, and by the closed form of the original problem reached through the
scaled solve.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import scipy.linalg


# ----------------------------------------------------------------------------
# Hessian, damping, spectral norm
# ----------------------------------------------------------------------------

def hessian(chunks) -> np.ndarray:
    """H = sum_i y_i^T y_i over calibration sequences y_i (Section 3.4)."""
    H = None
    for y in chunks:
        y = np.asarray(y, dtype=np.float64)
        if H is None:
            H = np.zeros((y.shape[1], y.shape[1]))
        H += y.T @ y
    if H is None:
        raise ValueError("no calibration chunks")
    return H


def damp(H: np.ndarray, rel: float = 0.01):
    """Return (H + lambda I, lambda) with lambda = rel * trace(H) / d."""
    H = np.asarray(H, dtype=np.float64)
    lam = rel * np.trace(H) / H.shape[0]
    return H + lam * np.eye(H.shape[0]), lam


def jacobi_scale(H: np.ndarray):
    """Return (D H D, D) with D = diag(H)^(-1/2) (entries of H_ii <= 0 get 1)."""
    H = np.asarray(H, dtype=np.float64)
    h = np.diag(H)
    D = np.where(h > 0.0, 1.0 / np.sqrt(np.where(h > 0.0, h, 1.0)), 1.0)
    return H * np.outer(D, D), D


def power_iteration(H: np.ndarray, v0: np.ndarray, max_iters: int = 1000,
                    tol: float = 1e-6):
    """Largest eigenvalue of symmetric PSD H by power iteration.

    Iteration i computes y = H v (v of unit length), the Rayleigh quotient
    rho_i = v^T y, and v <- y / ||y||. It stops when
    |rho_i - rho_{i-1}| <= tol * rho_i, or after max_iters iterations.
    Returns (rho, iterations).
    """
    H = np.asarray(H, dtype=np.float64)
    v = np.asarray(v0, dtype=np.float64)
    v = v / np.linalg.norm(v)
    rho_prev = None
    rho = 0.0
    for it in range(1, max_iters + 1):
        y = H @ v
        rho = float(v @ y)
        ny = np.linalg.norm(y)
        if ny == 0.0:
            return 0.0, it
        v = y / ny
        if rho_prev is not None and abs(rho - rho_prev) <= tol * abs(rho):
            return rho, it
        rho_prev = rho
    return rho, max_iters


def subspace_iteration(H: np.ndarray, V0: np.ndarray, max_iters: int = 1000,
                       tol: float = 1e-6):
    """Largest eigenvalue of symmetric PSD H by subspace iteration.

    V0 holds b start vectors as rows, shape (b, d) (a 1-D array is one
    vector). Q starts as an orthonormal basis of the span of those vectors.
    Iteration i computes Y = H Q, the Rayleigh-Ritz matrix T = Q^T Y, its
    largest eigenvalue theta_i (the largest Ritz value of span(Q)), and then
    replaces Q by an orthonormal basis of span(Y) (Householder QR). It stops
    when |theta_i - theta_{i-1}| <= tol * theta_i, or after max_iters
    iterations. Ritz values never exceed lambda_max(H). Returns
    (theta, iterations).
    """
    H = np.asarray(H, dtype=np.float64)
    V = np.asarray(V0, dtype=np.float64)
    if V.ndim == 1:
        V = V[None, :]
    Q, _ = np.linalg.qr(V.T)
    theta_prev = None
    theta = 0.0
    for it in range(1, max_iters + 1):
        Y = H @ Q
        if not np.any(Y):
            return 0.0, it
        T = Q.T @ Y
        theta = float(np.linalg.eigvalsh(T)[-1])
        Q, _ = np.linalg.qr(Y)
        if theta_prev is not None and abs(theta - theta_prev) <= tol * abs(theta):
            return theta, it
        theta_prev = theta
    return theta, max_iters


# Relative size of beta_j below which the Krylov space counts as invariant.
LANCZOS_BREAKDOWN = 1e-6


def lanczos(H: np.ndarray, v0: np.ndarray, max_steps: int = 256, tol: float = 1e-6,
            tridiagonal: bool = False):
    """Largest eigenvalue of symmetric PSD H by the Lanczos method.

    Step j (1-based) extends the orthonormal basis q_1 = v0/||v0||, ..., q_j of
    the Krylov space K_j = span{v0, H v0, ..., H^(j-1) v0}:
      w = H q_j, alpha_j = q_j^T w,
      w <- w - alpha_j q_j - beta_(j-1) q_(j-1),
      w <- w - Q_j (Q_j^T w)   (full reorthogonalisation, once more),
      beta_j = ||w||, q_(j+1) = w / beta_j.
    T_j = tridiag(beta_(1..j-1); alpha_(1..j); beta_(1..j-1)) equals
    Q_j^T H Q_j, so theta_j = lambda_max(T_j) is the largest Ritz value of
    K_j. Ritz values never exceed lambda_max(H) and theta_j never decreases
    with j. It stops when |theta_j - theta_(j-1)| <= tol * theta_j, when
    beta_j <= LANCZOS_BREAKDOWN * theta_j (K_j is numerically invariant and
    theta_j an eigenvalue), or after max_steps steps (at most d).
    Returns (theta, steps), plus (alpha, beta) when `tridiagonal` is set.
    """
    H = np.asarray(H, dtype=np.float64)
    d = H.shape[0]
    q = np.asarray(v0, dtype=np.float64)
    q = q / np.linalg.norm(q)
    Q = [q]
    alpha: list[float] = []
    beta: list[float] = []
    theta = 0.0
    theta_prev = None
    steps = 0
    for j in range(1, min(max_steps, d) + 1):
        steps = j
        w = H @ Q[-1]
        alpha.append(float(Q[-1] @ w))
        w = w - alpha[-1] * Q[-1]
        if j > 1:
            w = w - beta[-1] * Q[-2]
        B = np.array(Q)
        w = w - B.T @ (B @ w)
        b = float(np.linalg.norm(w))
        T = np.diag(alpha) + np.diag(beta, 1) + np.diag(beta, -1)
        theta = float(np.linalg.eigvalsh(T)[-1])
        if theta_prev is not None and abs(theta - theta_prev) <= tol * abs(theta):
            break
        if b <= LANCZOS_BREAKDOWN * abs(theta):
            break
        theta_prev = theta
        beta.append(b)
        Q.append(w / b)
    if tridiagonal:
        return theta, steps, np.array(alpha), np.array(beta[:steps - 1])
    return theta, steps


# ----------------------------------------------------------------------------
# Mask selection (the input of the weight update)
# ----------------------------------------------------------------------------

def wanda_mask(W0: np.ndarray, col_sq: np.ndarray, pattern: str, sparsity: float = 0.5):
    """Wanda mask, rows of W0 = column QPs, uint8 (1 keeps).

    score[j][i] = W0[j][i]^2 * col_sq[i] in fp64 (W0[j][i]^2 is exact). pattern
    "unstructured" keeps the d - floor(sparsity * d) highest scores of every
    row; "2:4" keeps the two highest of every group [4g, 4g + 4) of a row.
    Among equal scores the lower index comes first; NaN scores come last.
    """
    W = np.asarray(W0, dtype=np.float64)
    c = np.asarray(col_sq, dtype=np.float64)
    score = (W * W) * c[None, :]
    n, d = W.shape
    mask = np.zeros((n, d), dtype=np.uint8)
    idx = np.arange(d)
    if pattern == "unstructured":
        keep = d - int(np.floor(sparsity * d))
        for j in range(n):
            order = np.lexsort((idx, -score[j]))  # by score descending, then index
            mask[j, order[:keep]] = 1
    elif pattern == "2:4":
        if d % 4:
            raise ValueError("2:4 needs d divisible by 4")
        for j in range(n):
            for g in range(0, d, 4):
                order = np.lexsort((idx[g:g + 4], -score[j, g:g + 4]))
                mask[j, g + order[:2]] = 1
    else:
        raise ValueError(pattern)
    return mask


# ----------------------------------------------------------------------------
# The column QPs: objective, closed form, KKT
# ----------------------------------------------------------------------------

def objective(H: np.ndarray, W0: np.ndarray, W: np.ndarray) -> np.ndarray:
    """f_j = (w_j - w0_j)^T H (w_j - w0_j) for every row j (Eq. (4))."""
    D = np.asarray(W, dtype=np.float64) - np.asarray(W0, dtype=np.float64)
    return np.einsum("ij,ij->i", D @ np.asarray(H, dtype=np.float64), D)


def closed_form(H: np.ndarray, W0: np.ndarray, mask: np.ndarray) -> np.ndarray:
    """Unique optimum of every column QP (Eq. (10)-(11)), via Cholesky of H_II."""
    H = np.asarray(H, dtype=np.float64)
    W0 = np.asarray(W0, dtype=np.float64)
    keep = np.asarray(mask) != 0
    W = np.zeros_like(W0)
    for j in range(W0.shape[0]):
        I = np.flatnonzero(keep[j])
        S = np.flatnonzero(~keep[j])
        if I.size == 0:
            continue
        rhs = H[np.ix_(I, S)] @ W0[j, S]
        dw = scipy.linalg.cho_solve(scipy.linalg.cho_factor(H[np.ix_(I, I)]), rhs)
        W[j, I] = W0[j, I] + dw
    return W


def kkt_solve(H: np.ndarray, W0: np.ndarray, mask: np.ndarray) -> np.ndarray:
    """Optimum of Eq. (6) from its KKT system, one dense solve per column.

    Unknowns (dw, nu): stationarity 2 H dw + E_S^T nu = 0 and feasibility
    E_S dw = -w0_S (Eq. (5)), E_S selecting the pruned entries.
    """
    H = np.asarray(H, dtype=np.float64)
    W0 = np.asarray(W0, dtype=np.float64)
    keep = np.asarray(mask) != 0
    n, d = W0.shape
    W = np.zeros_like(W0)
    for j in range(n):
        S = np.flatnonzero(~keep[j])
        m = S.size
        K = np.zeros((d + m, d + m))
        K[:d, :d] = 2.0 * H
        E = np.zeros((m, d))
        E[np.arange(m), S] = 1.0
        K[:d, d:] = E.T
        K[d:, :d] = E
        rhs = np.concatenate([np.zeros(d), -W0[j, S]])
        sol = np.linalg.solve(K, rhs)
        W[j] = W0[j] + sol[:d]
        W[j, S] = 0.0  # the constraint holds exactly
    return W


# ----------------------------------------------------------------------------
# rAPDHG
# ----------------------------------------------------------------------------

@dataclass
class SolverOptions:
    max_iters: int = 100_000
    check_every: int = 64
    fixed_iters: bool = False      # run exactly max_iters (checks still restart)
    eps_rel: float = 0.01
    eps_abs: float = 0.01
    beta_sufficient: float = 0.2
    beta_necessary: float = 0.8
    beta_artificial: float = 0.36
    step_safety: float = 1e-3      # L = 2 lambda_max (1 + step_safety)
    restarts: bool = True


@dataclass
class SolveResult:
    W: np.ndarray
    iters: np.ndarray
    restarts: np.ndarray
    converged: np.ndarray
    f_initial: np.ndarray
    f_final: np.ndarray
    kkt_final: np.ndarray
    anchors: list = field(default_factory=list)  # per column: f at each accepted restart


def _score(H, W0, keep, Z, D=None):
    """Per-row r_d, gap, KKT, f and z^T H z of candidate rows Z.

    With a diagonal scaling D (H, W0 and Z in scaled coordinates), r_d is the
    norm of the gradient in the original coordinates, D^-1 g; gap, f and
    z^T H z are the same in both coordinates.
    """
    dZ = Z - W0
    HdZ = dZ @ H                      # rows of H (z - w0); H is symmetric
    G = 2.0 * HdZ
    Go = G if D is None else G / D[None, :]
    rd = np.sqrt(np.sum(np.where(keep, Go, 0.0) ** 2, axis=1))
    gap = np.abs(np.sum(Z * G, axis=1))
    f = np.sum(dZ * HdZ, axis=1)
    zHz = np.sum(Z * (Z @ H), axis=1)
    return {"rd": rd, "gap": gap, "kkt": np.hypot(rd, gap), "f": f, "zHz": zHz}


def anchor_terms(H, W0, D=None):
    """Per-row quantities of the termination test that depend on the anchors
    only: H w0 (rows), c_norm = ||2 H w0||_2 (the gradient of Eq. (6) at
    w = 0, in the original coordinates when a scaling D is given) and
    w0^T H w0 (the constant of the QP form of Eq. (6))."""
    Hw0 = W0 @ H
    c_norm = np.linalg.norm(2.0 * (Hw0 if D is None else Hw0 / D[None, :]), axis=1)
    w0Hw0 = np.sum(W0 * Hw0, axis=1)
    return Hw0, c_norm, w0Hw0


def termination(s: dict, c_norm, w0Hw0, opts: SolverOptions):
    """Appendix D test of scored rows s (from _score): returns (converged, P, D).

    P = f(z) is the primal objective. D = w0^T H w0 - z^T H z is the dual
    objective of the QP form 1/2 z^T Q z + c^T z + w0^T H w0 (Q = 2H,
    c = -2 H w0) with bounds only: -1/2 z^T Q z plus the constant, the bound
    terms vanishing because every bound is 0. P - D = z^T g, so the gap
    |z^T g| is |P - D|. A row passes when r_d <= eps_abs + eps_rel c_norm and
    gap <= eps_abs + eps_rel (|P| + |D|).
    """
    P = s["f"]
    D = w0Hw0 - s["zHz"]
    conv = ((s["rd"] <= opts.eps_abs + opts.eps_rel * c_norm)
            & (s["gap"] <= opts.eps_abs + opts.eps_rel * (np.abs(P) + np.abs(D))))
    return conv, P, D


def check_decision(s_x: dict, s_a: dict, kkt_restart, kkt_prev, f_anchor, k, t,
                   c_norm, w0Hw0, opts: SolverOptions):
    """Candidate choice, termination test and restart test at one check.

    Returns (use_x, converged, restart, s_cand). All inputs are per-column arrays.
    """
    use_x = s_x["kkt"] < s_a["kkt"]  # ties go to the average
    s_c = {key: np.where(use_x, s_x[key], s_a[key]) for key in s_x}
    converged, _, _ = termination(s_c, c_norm, w0Hw0, opts)
    kc = s_c["kkt"]
    cond = ((kc <= opts.beta_sufficient * kkt_restart)
            | ((kc <= opts.beta_necessary * kkt_restart) & (kc > kkt_prev))
            | (k >= opts.beta_artificial * t))
    restart = cond & (s_c["f"] <= f_anchor) if opts.restarts else np.zeros_like(cond)
    return use_x, converged, restart, s_c


def cg(H: np.ndarray, W0: np.ndarray, mask: np.ndarray, opts: SolverOptions | None = None,
       observer=None, scale=None) -> SolveResult:
    """Conjugate gradients on H_KK x_K = (H w0)_K for every row of W0.

    Start x = sel(mask, w0, 0), r = P (H w0 - H x), p = r (P keeps the kept
    entries). Iteration: q = P H p, alpha = r.r / p.q, x += alpha p,
    r -= alpha q, beta = r'.r' / r.r, p = r' + beta p (alpha = beta = 0 once
    r.r = 0). Every `check_every` iterations and at max_iters, x is tested with
    rapdhg's termination rule (r_d, gap against the Appendix D tolerances).
    Only max_iters, check_every, fixed_iters, eps_rel and eps_abs of `opts`
    apply. `observer(t, x, p)` sees the iterates after every iteration. `scale`
    works as in rapdhg.
    """
    opts = opts or SolverOptions()
    H = np.asarray(H, dtype=np.float64)
    D = None if scale is None else np.asarray(scale, dtype=np.float64)
    W0 = np.asarray(W0, dtype=np.float64)
    if D is not None:
        W0 = W0 / D[None, :]
    keep = np.asarray(mask) != 0
    n, d = W0.shape

    x = np.where(keep, W0, 0.0)
    Hw0, c_norm, w0Hw0 = anchor_terms(H, W0, D)
    r = np.where(keep, Hw0 - x @ H, 0.0)
    p = r.copy()
    rr = np.sum(r * r, axis=1)

    done = np.zeros(n, dtype=bool)
    out = {"W": np.zeros_like(W0), "iters": np.zeros(n, dtype=np.int64),
           "converged": np.zeros(n, dtype=bool), "f_final": np.zeros(n),
           "kkt_final": np.zeros(n)}

    def test(Z):
        s = _score(H, W0, keep, Z, D)
        return s, termination(s, c_norm, w0Hw0, opts)[0]

    def finish(rows, s, t, conv):
        out["W"][rows] = (x if D is None else x * D[None, :])[rows]
        out["iters"][rows] = t
        out["converged"][rows] = conv[rows]
        out["f_final"][rows] = s["f"][rows]
        out["kkt_final"][rows] = s["kkt"][rows]
        done[rows] = True

    s0, conv0 = test(x)
    f_initial = s0["f"].copy()
    if opts.max_iters <= 0:
        finish(np.ones(n, dtype=bool), s0, 0, conv0)
    elif not opts.fixed_iters:
        finish(conv0, s0, 0, conv0)

    t = 0
    while t < opts.max_iters and not done.all():
        act = ~done
        q = np.where(keep, p @ H, 0.0)
        pq = np.sum(p * q, axis=1)
        alpha = np.where(rr > 0.0, rr / np.where(pq > 0.0, pq, 1.0), 0.0)
        x_new = x + alpha[:, None] * p
        r_new = r - alpha[:, None] * q
        rr_new = np.sum(r_new * r_new, axis=1)
        beta = np.where(rr > 0.0, rr_new / np.where(rr > 0.0, rr, 1.0), 0.0)
        p_new = r_new + beta[:, None] * p
        x[act], r[act], p[act], rr[act] = x_new[act], r_new[act], p_new[act], rr_new[act]
        t += 1
        if observer is not None:
            observer(t, x, p)
        if t % opts.check_every and t != opts.max_iters:
            continue
        s, conv = test(x)
        if not opts.fixed_iters:
            stop = act & conv
            finish(stop, s, t, conv)
            act = act & ~stop
        if t == opts.max_iters:
            finish(act, s, t, conv)

    return SolveResult(W=out["W"], iters=out["iters"], restarts=np.zeros(n, dtype=np.int64),
                       converged=out["converged"], f_initial=f_initial,
                       f_final=out["f_final"], kkt_final=out["kkt_final"])


def rapdhg(H: np.ndarray, W0: np.ndarray, mask: np.ndarray, lambda_max: float,
           opts: SolverOptions | None = None, observer=None, scale=None) -> SolveResult:
    """Solve all column QPs of Eq. (6) side by side (one row of W0 per QP).

    `observer(t, x, x_ag)`, if given, sees the iterates after every iteration
    (before that iteration's check); it must not modify them. With `scale` = D
    (see jacobi_scale), H is the scaled D H0 D, lambda_max its largest
    eigenvalue, W0 and the result stay in the original coordinates.
    """
    opts = opts or SolverOptions()
    H = np.asarray(H, dtype=np.float64)
    D = None if scale is None else np.asarray(scale, dtype=np.float64)
    W0_orig = np.asarray(W0, dtype=np.float64)
    W0 = W0_orig if D is None else W0_orig / D[None, :]
    keep = np.asarray(mask) != 0
    n, d = W0.shape
    L = 2.0 * float(lambda_max) * (1.0 + opts.step_safety)

    def sel(V):
        return np.where(keep, V, 0.0)

    x = sel(W0)
    xa = x.copy()
    _, c_norm, w0Hw0 = anchor_terms(H, W0, D)

    k = np.zeros(n, dtype=np.int64)
    done = np.zeros(n, dtype=bool)
    out = {"W": np.zeros_like(W0), "iters": np.zeros(n, dtype=np.int64),
           "restarts": np.zeros(n, dtype=np.int64),
           "converged": np.zeros(n, dtype=bool), "f_final": np.zeros(n),
           "kkt_final": np.zeros(n)}
    anchors = [[] for _ in range(n)]

    s0 = _score(H, W0, keep, x, D)
    f_initial = s0["f"].copy()
    kkt_restart = s0["kkt"].copy()
    kkt_prev = s0["kkt"].copy()
    f_anchor = s0["f"].copy()

    def finish(rows, Z, s, t, conv):
        out["W"][rows] = (Z if D is None else Z * D[None, :])[rows]
        out["iters"][rows] = t
        out["converged"][rows] = conv[rows]
        out["f_final"][rows] = s["f"][rows]
        out["kkt_final"][rows] = s["kkt"][rows]
        done[rows] = True

    # Termination test at the start point (all-kept or all-pruned columns, or
    # a start that already meets the tolerances).
    conv0, _, _ = termination(s0, c_norm, w0Hw0, opts)
    if opts.max_iters <= 0:
        finish(np.ones(n, dtype=bool), x, s0, 0, conv0)
    elif not opts.fixed_iters:
        finish(conv0, x, s0, 0, conv0)

    t = 0
    while t < opts.max_iters and not done.all():
        act = ~done
        alpha = (2.0 / (k + 2.0))[:, None]
        eta = ((k + 1.0) / (2.0 * L))[:, None]
        x_md = (1.0 - alpha) * xa + alpha * x
        g = 2.0 * ((x_md - W0) @ H)
        x_new = sel(x - eta * g)
        xa_new = (1.0 - alpha) * xa + alpha * x_new
        x[act] = x_new[act]
        xa[act] = xa_new[act]
        k[act] += 1
        t += 1
        if observer is not None:
            observer(t, x, xa)
        if t % opts.check_every and t != opts.max_iters:
            continue
        s_x = _score(H, W0, keep, x, D)
        s_a = _score(H, W0, keep, xa, D)
        use_x, conv, restart, s_c = check_decision(
            s_x, s_a, kkt_restart, kkt_prev, f_anchor, k, t, c_norm, w0Hw0, opts)
        cand = np.where(use_x[:, None], x, xa)
        if not opts.fixed_iters:
            stop = act & conv
            finish(stop, cand, s_c, t, conv)
            act = act & ~stop
        if t == opts.max_iters:
            # The iteration budget ends here: every active column stops at its
            # candidate, and a restart that would never run is not counted.
            finish(act, cand, s_c, t, conv)
            break
        acc = act & restart
        x[acc] = cand[acc]
        xa[acc] = cand[acc]
        k[acc] = 0
        kkt_restart[acc] = s_c["kkt"][acc]
        f_anchor[acc] = s_c["f"][acc]
        out["restarts"][acc] += 1
        for j in np.flatnonzero(acc):
            anchors[j].append(float(s_c["f"][j]))
        kkt_prev[act] = s_c["kkt"][act]

    return SolveResult(W=out["W"], iters=out["iters"], restarts=out["restarts"],
                       converged=out["converged"], f_initial=f_initial,
                       f_final=out["f_final"], kkt_final=out["kkt_final"],
                       anchors=anchors)
