"""fp64 CPU oracle of the Periodic Row-wise Muon (PRM) optimizer step.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package.  The product path (``paper_2608_20818_amd`` and ``libprm.so``) never
imports it and shares no code, constant table or helper with it.

Everything here is plain NumPy in float64 and follows the paper
("Scaling Muon for Diffusion Transformers") in its own order and notation:

* refresh indicator  rho_t = 1[t mod K = 0]           -- Sec. 3.3, eq. (periodic-direction); Alg. 1
* orientation        O(M) = M if m <= n else M^T      -- Sec. 3.1 (complementary geometries)
* RowNorm_eps        X_i / max(||X_i||_2, eps)        -- eq. (rownorm), eq. (app-rownorm-eps)
* NS5 map Phi_5      G = X X^T; B = bG + cG^2;        -- eq. (app-ns-recurrence), coefficients
                     X <- aX + BX, five times            (a,b,c) = (3.4445, -4.7750, 2.0315) from
                                                         App. "Optimizer and Training Hyperparameters"
* direction          D~ = NS5(M~) if rho_t else gamma * RowNorm(M~)
                     D  = s(W) * O^{-1}(D~)           -- eq. (periodic-direction); Alg. 1
* parameter write    W <- (1 - eta*lambda) W - eta*D  -- eq. (finite_ns5), eq. (periodic-direction)

Readings of what the paper leaves open (each one is listed, with its
reason, in the design notes of the repository):

* momentum update   M <- beta*M + G (heavy-ball); optional dampening
                    M <- beta*M + (1-beta)*G and optional Nesterov input
                    U = G + beta*M.  Alg. 1 defers the momentum update to Sec. 2,
                    which never writes it out; beta = 0.95 (hyperparameter table).
* NS input scaling  X0 = M~ / (||M~||_F + eps_ns), eps_ns = 1e-7 > 0 (App. "Per-matrix
                    arithmetic" names an input normalization without its form).
* ablations         Table 3a: RowNorm on every step (never_refresh) and the
                    scalar-controlled variant (gamma on both branches).
* eps of RowNorm    1e-8 (the only epsilon the paper prints).
* shape scale s(W)  sqrt(max(1, m/n)) by default (the paper scales the update
                    by a factor that depends on the shape, without a formula).
                    PARITY UNPINNED BY THE PAPER: s(W) is a convention that
                    both sides read from the same configuration; the tests pin
                    only its stated definition (update RMS = 1/sqrt(n) for an
                    exactly orthogonal direction).
* weight decay      always uses eta_t (not gamma*eta_t), as eq.
                    (periodic-direction) writes it.

Auxiliary AdamW group (the non-matrix parameters: Sec. 2, "Muon" setup, and
App. "Optimizer and Training Hyperparameters" -- biases, normalization and
other non-matrix parameters stay on AdamW with decoupled weight decay;
optimizer-hyperparameter table: LR 1e-4, betas (0.9, 0.95), eps 1e-8, weight
decay 0.01).  The paper cites AdamW (decoupled weight decay) without writing
it out; ``adamw_step`` follows that method as published:

* moments           m <- beta1 m + (1 - beta1) g;  v <- beta2 v + (1 - beta2) g^2
* bias correction   m^ = m / (1 - beta1^t), v^ = v / (1 - beta2^t), t >= 1 the
                    update count including this one
* parameter write   p <- p - eta (m^ / (sqrt(v^) + eps) + lambda p)
                    (decay uses the old p and is not normalized by v^)

Also provided for the pins (not part of the method):
``ns5_closed_form`` (U phi5(S/(||M||_F+eps)) V^T, from an SVD), ``polar``
(U V^T) and ``ns5_rows_closed_form`` (selected oriented rows of NS5 through an
eigendecomposition of the Gram matrix; used to check sampled rows of large
matrices, where running the full five-iteration map would take minutes).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

# App. "Optimizer and Training Hyperparameters": the fixed quintic coefficients.
NS_COEFFS = (3.4445, -4.7750, 2.0315)
NS_ITERS = 5  # J_NS = 5 (Sec. 2, eq. finite_ns5)

SCALE_ONE = 0
SCALE_SQRT_ASPECT = 1
SCALE_RMS_0P2 = 2


# --------------------------------------------------------------------------
# schedule
# --------------------------------------------------------------------------
def refresh_indicator(t: int, K: int) -> int:
    """rho_t = 1[t mod K = 0] for 0-based t and K >= 1 (Sec. 3.3; Alg. 1)."""
    if K < 1:
        raise ValueError("K must be >= 1")
    if t < 0:
        raise ValueError("t must be >= 0")
    return 1 if t % K == 0 else 0


# --------------------------------------------------------------------------
# orientation (Sec. 3.1)
# --------------------------------------------------------------------------
def orient(M: np.ndarray) -> np.ndarray:
    """O(M): M itself when m <= n (square counts as wide), else M^T."""
    m, n = M.shape
    return M if m <= n else M.T


def orient_inv(Xt: np.ndarray, m: int, n: int) -> np.ndarray:
    """O^{-1}: map an oriented r x c direction back to the stored m x n shape."""
    return Xt if m <= n else Xt.T


# --------------------------------------------------------------------------
# momentum (a reading: Alg. 1 refers the momentum update to Sec. 2)
# --------------------------------------------------------------------------
def momentum_update(M: np.ndarray, G: np.ndarray, beta: float,
                    dampening: bool = False) -> np.ndarray:
    """Heavy-ball M <- beta*M + G; with dampening M <- beta*M + (1-beta)*G."""
    if dampening:
        return beta * M + (1.0 - beta) * G
    return beta * M + G


def momentum_direction_input(M_new: np.ndarray, G: np.ndarray, beta: float,
                             nesterov: bool = False) -> np.ndarray:
    """The matrix that the direction map consumes: M_t, or G + beta*M_t (Nesterov)."""
    if nesterov:
        return G + beta * M_new
    return M_new


# --------------------------------------------------------------------------
# RowNorm (eq. rownorm / eq. app-rownorm-eps)
# --------------------------------------------------------------------------
def rownorm(X: np.ndarray, eps: float) -> np.ndarray:
    """Each row divided by max(||row||_2, eps); the clamp comes after the square root."""
    X = np.asarray(X, dtype=np.float64)
    nu = np.sqrt(np.sum(X * X, axis=1))
    nu = np.maximum(nu, eps)
    return X / nu[:, None]


# --------------------------------------------------------------------------
# NS5 (eq. app-ns-recurrence)
# --------------------------------------------------------------------------
def ns_normalize(X: np.ndarray, eps_ns: float) -> np.ndarray:
    """Input normalization X / (||X||_F + eps_ns)."""
    return X / (np.linalg.norm(X) + eps_ns)


def ns5(X: np.ndarray, eps_ns: float = 1e-7, coeffs=NS_COEFFS,
        iters: int = NS_ITERS) -> np.ndarray:
    """Finite Newton-Schulz map Phi_5 on an oriented r x c matrix (r <= c).

    G_j = X_j X_j^T;  B_j = b G_j + c G_j^2;  X_{j+1} = a X_j + B_j X_j.
    This is the implemented finite map, not the polar factor.
    """
    a, b, c = coeffs
    X = ns_normalize(np.asarray(X, dtype=np.float64), eps_ns)
    for _ in range(iters):
        G = X @ X.T
        B = b * G + c * (G @ G)
        X = a * X + B @ X
    return X


def quintic(x, coeffs=NS_COEFFS):
    """The scalar map p(x) = a x + b x^3 + c x^5 that one NS iteration applies to
    every singular value."""
    a, b, c = coeffs
    return a * x + b * x ** 3 + c * x ** 5


def phi5(x, coeffs=NS_COEFFS, iters: int = NS_ITERS):
    """Five-fold composition of the scalar quintic."""
    y = np.asarray(x, dtype=np.float64)
    for _ in range(iters):
        y = quintic(y, coeffs)
    return y


def ns5_closed_form(X: np.ndarray, eps_ns: float = 1e-7, coeffs=NS_COEFFS,
                    iters: int = NS_ITERS) -> np.ndarray:
    """NS5 through the SVD: U phi5(S / (||X||_F + eps)) V^T.

    Every NS iterate is an odd matrix polynomial of X, so with X = U S V^T one
    iteration maps S to p(S) and keeps U, V.
    """
    X = np.asarray(X, dtype=np.float64)
    U, S, Vt = np.linalg.svd(X, full_matrices=False)
    Sh = S / (np.linalg.norm(X) + eps_ns)
    return (U * phi5(Sh, coeffs, iters)) @ Vt


def ns5_rows_closed_form(X: np.ndarray, rows, eps_ns: float = 1e-7,
                         coeffs=NS_COEFFS, iters: int = NS_ITERS) -> np.ndarray:
    """Selected rows of NS5(X) for an oriented X (r <= c).

    With X0 = X/(||X||_F+eps) and X0 X0^T = Q diag(lam) Q^T, NS5(X) =
    Q diag(phi5(sqrt(lam))/sqrt(lam)) Q^T X0; phi5(x)/x is a polynomial in
    x^2, so the zero eigenvalues are handled by its limit a^iters.
    """
    X = np.asarray(X, dtype=np.float64)
    X0 = ns_normalize(X, eps_ns)
    A = X0 @ X0.T
    lam, Q = np.linalg.eigh(A)
    lam = np.clip(lam, 0.0, None)
    x = np.sqrt(lam)
    g = np.empty_like(x)
    small = x < 1e-150
    g[~small] = phi5(x[~small], coeffs, iters) / x[~small]
    g[small] = coeffs[0] ** iters
    rows = np.asarray(rows)
    T = (Q[rows, :] * g) @ Q.T
    return T @ X0


def polar(X: np.ndarray) -> np.ndarray:
    """Exact polar factor U V^T of an oriented matrix (eq. polar-geometry)."""
    U, _, Vt = np.linalg.svd(np.asarray(X, dtype=np.float64), full_matrices=False)
    return U @ Vt


# --------------------------------------------------------------------------
# shape scale (reading; parity unpinned by the paper)
# --------------------------------------------------------------------------
def shape_scale(m: int, n: int, mode: int = SCALE_SQRT_ASPECT) -> float:
    if mode == SCALE_ONE:
        return 1.0
    if mode == SCALE_SQRT_ASPECT:
        return math.sqrt(max(1.0, m / n))
    if mode == SCALE_RMS_0P2:
        return 0.2 * math.sqrt(max(m, n))
    raise ValueError(f"unknown scale mode {mode}")


# --------------------------------------------------------------------------
# the optimizer step (Alg. 1, one matrix)
# --------------------------------------------------------------------------
@dataclass
class PRMConfig:
    K: int = 3                 # refresh period (hyperparameter table: K = 3)
    beta: float = 0.95         # momentum (hyperparameter table)
    lr: float = 5e-3           # eta_t
    wd: float = 0.01           # lambda (hyperparameter table caption)
    gamma: float = 0.15        # RowNorm multiplier (hyperparameter table)
    eps_rownorm: float = 1e-8
    eps_ns: float = 1e-7
    nesterov: bool = False
    ema_dampening: bool = False
    scale_mode: int = SCALE_SQRT_ASPECT
    never_refresh: bool = False     # ablation: RowNorm at every step
    gamma_on_refresh: bool = False  # ablation: scalar-controlled (gamma on both branches)
    coeffs: tuple = field(default=NS_COEFFS)

    def __post_init__(self):
        # both clamps must be positive: a zero momentum (or a zero row) then
        # gives a zero direction instead of 0/0
        if self.K < 1 or not self.eps_rownorm > 0 or not self.eps_ns > 0:
            raise ValueError("need K >= 1, eps_rownorm > 0 and eps_ns > 0")


def direction(U: np.ndarray, t: int, cfg: PRMConfig) -> tuple[np.ndarray, int]:
    """D_t = s(W) O^{-1}(D~_t) for one matrix, and rho_t (eq. periodic-direction)."""
    m, n = U.shape
    rho = 0 if cfg.never_refresh else refresh_indicator(t, cfg.K)
    Xt = orient(np.asarray(U, dtype=np.float64))
    if rho:
        Dt = ns5(Xt, cfg.eps_ns, cfg.coeffs)
        if cfg.gamma_on_refresh:
            Dt = cfg.gamma * Dt
    else:
        Dt = cfg.gamma * rownorm(Xt, cfg.eps_rownorm)
    return shape_scale(m, n, cfg.scale_mode) * orient_inv(Dt, m, n), rho


def step_matrix(W: np.ndarray, M: np.ndarray, G: np.ndarray, t: int,
                cfg: PRMConfig, lr: float | None = None):
    """One PRM step on one matrix.  Returns (W_new, M_new, D, rho).

    Alg. 1: momentum, rho_t, orientation, NS5 or gamma*RowNorm, shape scale,
    decoupled weight decay with eta_t.
    """
    eta = cfg.lr if lr is None else lr
    W = np.asarray(W, dtype=np.float64)
    M = np.asarray(M, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    M_new = momentum_update(M, G, cfg.beta, cfg.ema_dampening)
    U = momentum_direction_input(M_new, G, cfg.beta, cfg.nesterov)
    D, rho = direction(U, t, cfg)
    W_new = (1.0 - eta * cfg.wd) * W - eta * D
    return W_new, M_new, D, rho


def step(Ws, Ms, Gs, t: int, cfg: PRMConfig, lr: float | None = None):
    """One PRM step over a list of matrices (the loop over W_M in Alg. 1)."""
    out_W, out_M, out_D = [], [], []
    rho = None
    for W, M, G in zip(Ws, Ms, Gs):
        Wn, Mn, D, r = step_matrix(W, M, G, t, cfg, lr)
        out_W.append(Wn)
        out_M.append(Mn)
        out_D.append(D)
        rho = r
    if rho is None:
        rho = 0 if cfg.never_refresh else refresh_indicator(t, cfg.K)
    return out_W, out_M, out_D, rho


# --------------------------------------------------------------------------
# auxiliary AdamW group
# --------------------------------------------------------------------------
@dataclass
class AdamWConfig:
    """Aux AdamW settings of the optimizer-hyperparameter table (LR 1e-4,
    betas (0.9, 0.95)) and its caption (eps 1e-8, weight decay 0.01)."""
    lr: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    wd: float = 0.01


def adamw_step(p: np.ndarray, g: np.ndarray, m: np.ndarray, v: np.ndarray, t: int,
               cfg: AdamWConfig, lr: float | None = None):
    """One AdamW update of one tensor.  Returns (p_new, m_new, v_new).

    Adam's first and second moment estimates with their bias corrections,
    then the decoupled weight-decay write (the update the paper keeps for its
    non-matrix parameters, App. "Optimizer and Training Hyperparameters").
    ``t`` is the 1-based number of this update.
    """
    if t < 1:
        raise ValueError("t must be >= 1")
    eta = cfg.lr if lr is None else lr
    p = np.asarray(p, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m = np.asarray(m, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    # first and second raw moment estimates
    m_new = cfg.beta1 * m + (1.0 - cfg.beta1) * g
    v_new = cfg.beta2 * v + (1.0 - cfg.beta2) * (g * g)
    # bias-corrected estimates
    m_hat = m_new / (1.0 - cfg.beta1 ** t)
    v_hat = v_new / (1.0 - cfg.beta2 ** t)
    # decoupled weight decay on the old parameter, plus the normalized step
    p_new = p - eta * (m_hat / (np.sqrt(v_hat) + cfg.eps) + cfg.wd * p)
    return p_new, m_new, v_new


def adamw_bytes_per_element(param_bytes: int, grad_bytes: int) -> int:
    """Algorithmic HBM bytes of one AdamW element: p, g, m, v read once; p, m, v
    written once (m and v fp32)."""
    return 2 * param_bytes + grad_bytes + 2 * 4 + 2 * 4


# --------------------------------------------------------------------------
# arithmetic model (App. "Per-matrix arithmetic")
# --------------------------------------------------------------------------
def ns5_flops(m: int, n: int) -> int:
    """Leading-order FLOPs of NS5 on one oriented r x c matrix: 20 r^2 c + 10 r^3."""
    r, c = min(m, n), max(m, n)
    return 20 * r * r * c + 10 * r ** 3
