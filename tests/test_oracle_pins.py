"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these re-types the oracle's formula: each checks it against a closed
form reached by another route (SVD, eigendecomposition, scalar recursion),
an invariant the paper states, a brute-force search, or a value the paper
prints.  A plausible mistake in the oracle (dropped term, wrong sign, wrong
orientation, wrong clamp) fails at least one of them; the mutation tests at
the end plant such mistakes in the oracle, on the CPU, and check that.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import prm_oracle as po

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def rand_lowrank(rng, m, n, k=None, noise=0.01):
    k = min(m, n) if k is None else k
    U, _ = np.linalg.qr(rng.standard_normal((m, k)))
    V, _ = np.linalg.qr(rng.standard_normal((n, k)))
    s = 1.0 / np.arange(1, k + 1)
    return (U * s) @ V.T + noise * rng.standard_normal((m, n))


# ----------------------------------------------------------------- constants
def test_defaults_match_paper_tables():
    assert tuple(GOLD["ns_coefficients"]["value"]) == po.NS_COEFFS
    assert GOLD["ns_iterations"]["value"] == po.NS_ITERS
    cfg = po.PRMConfig()
    assert cfg.beta == GOLD["momentum_beta"]["value"]
    assert cfg.gamma == GOLD["rownorm_gamma"]["value"]
    assert cfg.K == GOLD["refresh_period_K"]["value"]
    assert cfg.wd == GOLD["weight_decay"]["value"]


def test_flop_model_matches_paper_gemm_counts():
    # App. 'Per-matrix arithmetic': 2r^2c + 2r^3 + 2r^2c per iteration, 5 iterations.
    g = GOLD["ns5_gemm_flops_per_iteration"]["value"]
    for (m, n) in [(256, 1024), (1024, 256), (3072, 9216), (12288, 3072), (77, 77)]:
        r, c = min(m, n), max(m, n)
        per_iter = g["gram_r2c"] * r * r * c + g["square_r3"] * r ** 3 + g["apply_r2c"] * r * r * c
        assert po.ns5_flops(m, n) == 5 * per_iter
        f = GOLD["ns5_flop_model"]["value"]
        assert po.ns5_flops(m, n) == f["r2c"] * r * r * c + f["r3"] * r ** 3


# ----------------------------------------------------------------- schedule
@pytest.mark.parametrize("K", list(range(1, 13)))
def test_schedule_exhaustive(K):
    # Alg. 1: t = 0..T-1 and rho_t = 1[t mod K = 0]; the refresh steps are
    # exactly 0, K, 2K, ... (built here by striding, not by the modulus).
    T = 1000
    got = {t for t in range(T) if po.refresh_indicator(t, K) == 1}
    assert got == set(range(0, T, K))
    assert po.refresh_indicator(0, K) == 1  # the first step always refreshes


def test_schedule_rejects_bad_args():
    with pytest.raises(ValueError):
        po.refresh_indicator(0, 0)
    with pytest.raises(ValueError):
        po.refresh_indicator(-1, 3)


def test_never_refresh_variant_has_no_ns5():
    cfg = po.PRMConfig(K=1, never_refresh=True)
    rng = np.random.default_rng(0)
    U = rng.standard_normal((8, 12))
    for t in range(10):
        D, rho = po.direction(U, t, cfg)
        assert rho == 0
        np.testing.assert_allclose(np.linalg.norm(D / cfg.gamma, axis=1), 1.0, rtol=1e-12)


# ----------------------------------------------------------------- momentum
def test_momentum_closed_form_after_three_steps():
    rng = np.random.default_rng(1)
    beta = 0.95
    G = [rng.standard_normal((5, 7)) for _ in range(3)]
    M = np.zeros((5, 7))
    for g in G:
        M = po.momentum_update(M, g, beta)
    np.testing.assert_allclose(M, beta ** 2 * G[0] + beta * G[1] + G[2], rtol=1e-14, atol=1e-14)
    Md = np.zeros((5, 7))
    for g in G:
        Md = po.momentum_update(Md, g, beta, dampening=True)
    np.testing.assert_allclose(Md, (1 - beta) * (beta ** 2 * G[0] + beta * G[1] + G[2]),
                               rtol=1e-13, atol=1e-14)


def _quintic5(y):
    """phi5 by a plain scalar loop over the paper's printed coefficients."""
    a, b, c = GOLD["ns_coefficients"]["value"]
    for _ in range(5):
        y = a * y + b * y ** 3 + c * y ** 5
    return y


def _unit_rows(E):
    return E / np.linalg.norm(E, axis=1, keepdims=True)


def pin_nesterov_zero_momentum():
    """With M_0 = 0 the Nesterov input is G + beta * G = (1 + beta) G, a positive
    multiple of the plain input M_1 = G; both direction maps are positively
    homogeneous, so every direction must equal the non-Nesterov one."""
    rng = np.random.default_rng(2)
    for (m, n) in [(6, 14), (14, 6)]:
        W = rng.standard_normal((m, n))
        G = rng.standard_normal((m, n))
        for t in (0, 1):
            c0 = po.PRMConfig(K=2, beta=0.9)
            c1 = po.PRMConfig(K=2, beta=0.9, nesterov=True)
            _, M0, D0, _ = po.step_matrix(W, np.zeros((m, n)), G, t, c0)
            _, M1, D1, _ = po.step_matrix(W, np.zeros((m, n)), G, t, c1)
            np.testing.assert_array_equal(M1, M0)          # the state does not see Nesterov
            assert rel(D1, D0) < 1e-6, (m, n, t)


def pin_nesterov_lookahead():
    """Nesterov as a look-ahead: since M_t = beta M_{t-1} + G_t, the input
    G_t + beta M_t equals the extrapolation M_t + beta (M_t - M_{t-1}).  Over a
    trajectory, every Nesterov direction must be the direction of that
    extrapolation of the momenta the (separately pinned) momentum recursion
    produced: through the SVD closed form on refresh steps, rows scaled to unit
    norm on row-wise steps."""
    rng = np.random.default_rng(21)
    beta = 0.9
    for (m, n) in [(8, 20), (20, 8)]:
        cfg = po.PRMConfig(K=3, beta=beta, nesterov=True, lr=0.01)
        W = rng.standard_normal((m, n))
        M = rng.standard_normal((m, n))
        s = po.shape_scale(m, n)
        for t in range(6):
            G = rng.standard_normal((m, n))
            W, M_new, D, rho = po.step_matrix(W, M, G, t, cfg)
            E = po.orient(M_new + beta * (M_new - M))
            if rho:
                want = s * po.orient_inv(po.ns5_closed_form(E, cfg.eps_ns), m, n)
            else:
                want = s * po.orient_inv(cfg.gamma * _unit_rows(E), m, n)
            assert rel(D, want) < 1e-11, (m, n, t, rel(D, want))
            M = M_new


def pin_nesterov_constructed_target():
    """Choose the Nesterov input: for a target U* = sigma u v^T and any M_0, the
    gradient G = (U* - beta^2 M_0) / (1 + beta) makes G + beta (beta M_0 + G) = U*.
    A rank-one input has closed-form directions: phi5 of its normalized single
    singular value times u v^T (refresh), and sign(u_i) v / ||v|| per stored row
    of a wide matrix (row-wise)."""
    rng = np.random.default_rng(22)
    beta, gamma = 0.8, 0.3
    m, n = 7, 12
    u, v = rng.standard_normal(m), rng.standard_normal(n)
    Ustar = 1.7 * np.outer(u, v)
    M0 = rng.standard_normal((m, n))
    G = (Ustar - beta ** 2 * M0) / (1 + beta)
    cfg = po.PRMConfig(K=2, beta=beta, gamma=gamma, nesterov=True)
    nf = np.linalg.norm(Ustar)
    y = _quintic5(nf / (nf + cfg.eps_ns))
    _, _, D, rho = po.step_matrix(np.zeros((m, n)), M0, G, 0, cfg)
    assert rho == 1
    assert rel(D, y * np.outer(u / np.linalg.norm(u), v / np.linalg.norm(v))) < 1e-10
    _, _, D, rho = po.step_matrix(np.zeros((m, n)), M0, G, 1, cfg)
    assert rho == 0
    assert rel(D, gamma * np.outer(np.sign(u), v / np.linalg.norm(v))) < 1e-12


def test_nesterov_zero_momentum():
    pin_nesterov_zero_momentum()


def test_nesterov_lookahead():
    pin_nesterov_lookahead()


def test_nesterov_constructed_target():
    pin_nesterov_constructed_target()


# ----------------------------------------------------------------- RowNorm
def test_rownorm_rows_have_unit_norm_and_direction():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((16, 40)) * rng.uniform(0.1, 10, size=(16, 1))
    R = po.rownorm(X, 1e-8)
    np.testing.assert_allclose(np.linalg.norm(R, axis=1), 1.0, rtol=1e-14)
    # each row keeps its direction: R_i is a positive multiple of X_i
    cos = np.sum(R * X, axis=1) / (np.linalg.norm(X, axis=1))
    np.testing.assert_allclose(cos, 1.0, rtol=1e-14)


def pin_rownorm_eps_clamp_after_sqrt():
    """eq. (rownorm): denominator max(||X_i||, eps).  A zero row stays zero; a
    row with norm below eps is divided by eps (not by sqrt(eps) or eps^2)."""
    eps = 1e-2
    X = np.zeros((3, 4))
    X[1] = [3e-3, 4e-3, 0, 0]          # norm 5e-3 < eps
    X[2] = [3.0, 4.0, 0, 0]            # norm 5
    R = po.rownorm(X, eps)
    np.testing.assert_array_equal(R[0], 0.0)
    np.testing.assert_allclose(R[1], [0.3, 0.4, 0, 0], rtol=1e-14)
    np.testing.assert_allclose(R[2], [0.6, 0.8, 0, 0], rtol=1e-15)


def test_rownorm_eps_clamp_after_sqrt():
    pin_rownorm_eps_clamp_after_sqrt()


def test_rownorm_frobenius_and_inner_product_identities():
    # Sec. 3.3: a RowNorm direction with nonzero rows has Frobenius norm sqrt(r);
    # App. A: <X, RN(X)> = sum_i ||X_i||.
    rng = np.random.default_rng(4)
    X = rng.standard_normal((24, 60))
    R = po.rownorm(X, 1e-8)
    assert abs(np.linalg.norm(R) - math.sqrt(24)) < 1e-12
    assert abs(np.sum(X * R) - np.sum(np.linalg.norm(X, axis=1))) < 1e-10


def test_rownorm_variational_lemma_brute_force():
    # Lemma (row-wise variational characterization): RN(X) maximizes <X, U>
    # over ||U||_{2,inf} <= 1; no random feasible U beats it.
    rng = np.random.default_rng(5)
    X = rng.standard_normal((6, 9))
    best = np.sum(X * po.rownorm(X, 1e-8))
    for _ in range(10000):
        U = rng.standard_normal((6, 9))
        U /= np.maximum(np.linalg.norm(U, axis=1, keepdims=True), 1.0) * rng.uniform(1, 3, (6, 1))
        assert np.sum(X * U) <= best + 1e-12


def test_rownorm_equivariances():
    rng = np.random.default_rng(6)
    X = rng.standard_normal((10, 30))
    R = po.rownorm(X, 1e-8)
    D = np.diag(rng.uniform(0.5, 5, 10) * rng.choice([-1, 1], 10))
    np.testing.assert_allclose(po.rownorm(D @ X, 1e-8), np.sign(D) @ R, rtol=1e-13, atol=1e-15)
    Q, _ = np.linalg.qr(rng.standard_normal((30, 30)))
    np.testing.assert_allclose(po.rownorm(X @ Q, 1e-8), R @ Q, rtol=1e-12, atol=1e-13)


def pin_sharded_tall_rownorm():
    """Prop. (sharded RowNorm): for a tall M the oriented rows are the stored
    columns, and per-shard column sums of squares, summed over any row split,
    give their norms.  The oracle's step on a tall matrix must produce exactly
    those column-normalized directions."""
    rng = np.random.default_rng(7)
    M = rng.standard_normal((96, 20))
    eps = 1e-8
    cfg = po.PRMConfig(K=2, beta=0.0, gamma=1.0, eps_rownorm=eps, scale_mode=po.SCALE_ONE)
    _, _, dense, rho = po.step_matrix(np.zeros_like(M), np.zeros_like(M), M, 1, cfg)
    assert rho == 0
    for p in (1, 2, 3, 7):
        shards = np.array_split(np.arange(96), p)
        q = sum(np.sum(M[s] ** 2, axis=0) for s in shards)
        nu = np.maximum(np.sqrt(q), eps)
        np.testing.assert_allclose(dense, M / nu[None, :], rtol=1e-13)


def test_sharded_tall_rownorm_equivalence():
    pin_sharded_tall_rownorm()


# ----------------------------------------------------------------- NS5
NS5_SHAPES = [(8, 8), (16, 48), (32, 64), (24, 100), (5, 300)]


@pytest.mark.parametrize("shape", NS5_SHAPES)
def test_ns5_matches_svd_closed_form(shape):
    rng = np.random.default_rng(sum(shape))
    X = rand_lowrank(rng, *shape)
    a = po.ns5(X)
    b = po.ns5_closed_form(X)
    assert rel(a, b) < 1e-12


def test_ns5_scalar_recursion_on_diagonal_input():
    # X = sigma [I 0]: every singular value is 1/sqrt(r) after normalization, so
    # NS5(X) = phi5(1/sqrt(r)) [I 0] where phi5 is the scalar quintic applied
    # five times, here by a plain Python loop.
    r, c = 4, 6
    X = np.zeros((r, c))
    X[:, :r] = 3.7 * np.eye(r)
    y = 1.0 / math.sqrt(r) * (3.7 * math.sqrt(r)) / (3.7 * math.sqrt(r) + 1e-7)
    a, b, cc = GOLD["ns_coefficients"]["value"]
    for _ in range(5):
        y = a * y + b * y ** 3 + cc * y ** 5
    out = po.ns5(X)
    np.testing.assert_allclose(out[:, :r], y * np.eye(r), rtol=1e-13, atol=1e-15)
    np.testing.assert_array_equal(out[:, r:], 0.0)


def test_ns5_zero_matrix_gives_zero():
    np.testing.assert_array_equal(po.ns5(np.zeros((4, 9))), 0.0)


def _band():
    # the scalar map's range over [1.6e-3, 1], by dense evaluation
    x = np.logspace(np.log10(1.6e-3), 0, 200001)
    y = x.copy()
    a, b, c = GOLD["ns_coefficients"]["value"]
    for _ in range(5):
        y = a * y + b * y ** 3 + c * y ** 5
    return y.min(), y.max()


def test_ns5_singular_values_lie_in_band():
    lo, hi = _band()
    assert 0.68 < lo < 0.69 and 1.19 < hi < 1.21
    rng = np.random.default_rng(11)
    for shape in [(64, 192), (32, 128), (48, 48)]:
        X = rand_lowrank(rng, *shape)
        S = np.linalg.svd(X, compute_uv=False)
        sh = S / np.linalg.norm(X)
        So = np.linalg.svd(po.ns5(X), compute_uv=False)
        # singular values keep their order (phi5 is increasing on [0, ~0.3])
        keep = sh >= 1.6e-3
        assert np.all(So[keep] >= lo - 1e-12) and np.all(So[keep] <= hi + 1e-12)


def test_ns5_distance_to_polar_is_bounded_not_zero():
    # NS5 is not the polar factor (Sec. 2): its distance to U V^T equals
    # sqrt(sum (phi5(s_i) - 1)^2), nonzero but within the band.
    rng = np.random.default_rng(12)
    X = rand_lowrank(rng, 32, 96)
    N = po.ns5(X)
    P = po.polar(X)
    S = np.linalg.svd(X, compute_uv=False) / np.linalg.norm(X)
    lo, hi = _band()
    d = np.linalg.norm(N - P)
    assert d > 1e-3
    assert d <= math.sqrt(len(S)) * max(1 - lo, hi - 1) + 1e-12


def test_ns5_orthogonal_equivariance():
    rng = np.random.default_rng(13)
    X = rand_lowrank(rng, 16, 40)
    Q, _ = np.linalg.qr(rng.standard_normal((16, 16)))
    P, _ = np.linalg.qr(rng.standard_normal((40, 40)))
    N = po.ns5(X)
    assert rel(po.ns5(Q @ X), Q @ N) < 1e-12
    assert rel(po.ns5(X @ P), N @ P) < 1e-12
    assert rel(po.ns5(X.T), N.T) < 1e-12
    assert rel(po.ns5(37.0 * X), N) < 1e-6   # scale invariant up to eps_ns


def test_ns5_rows_closed_form_matches_iteration():
    rng = np.random.default_rng(14)
    X = rand_lowrank(rng, 40, 130)
    rows = [0, 3, 17, 39]
    assert rel(po.ns5_rows_closed_form(X, rows), po.ns5(X)[rows]) < 1e-11
    Z = np.zeros((6, 10))
    Z[:3] = rng.standard_normal((3, 10))          # rank deficient: zero eigenvalues
    assert rel(po.ns5_rows_closed_form(Z, range(6)), po.ns5(Z)) < 1e-11


# ----------------------------------------------------------------- polar reference
def test_polar_reference_properties():
    rng = np.random.default_rng(15)
    X = rng.standard_normal((12, 30))
    P = po.polar(X)
    np.testing.assert_allclose(P @ P.T, np.eye(12), atol=1e-13)           # eq. (app-polar-definition)
    S = np.linalg.svd(X, compute_uv=False)
    assert abs(np.sum(X * P) - S.sum()) < 1e-11                            # optimum = nuclear norm
    lam, Q = np.linalg.eigh(X @ X.T)
    P2 = (Q / np.sqrt(lam)) @ Q.T @ X                                      # (XX^T)^{-1/2} X
    assert rel(P, P2) < 1e-12
    # eq. (polar-perturbation) on random pairs
    for _ in range(20):
        A = rng.standard_normal((8, 20))
        B = A + 0.1 * rng.standard_normal((8, 20))
        smin = np.linalg.svd(A, compute_uv=False)[-1] + np.linalg.svd(B, compute_uv=False)[-1]
        assert np.linalg.norm(po.polar(A) - po.polar(B)) <= 2 * np.linalg.norm(A - B) / smin + 1e-12


# ----------------------------------------------------------------- shape scale
def test_shape_scale_rms_convention():
    # s = sqrt(max(1, m/n)) makes s * polar(O(M)) have RMS 1/sqrt(n) for both
    # wide and tall matrices (parity unpinned by the paper; this pins the stated rule).
    rng = np.random.default_rng(16)
    for (m, n) in [(16, 48), (48, 16), (32, 32)]:
        M = rng.standard_normal((m, n))
        D = po.shape_scale(m, n) * po.orient_inv(po.polar(po.orient(M)), m, n)
        assert abs(np.sqrt(np.mean(D * D)) - 1 / math.sqrt(n)) < 1e-12
    assert po.shape_scale(10, 20, po.SCALE_ONE) == 1.0


# ----------------------------------------------------------------- whole step
def pin_step_rank_one_closed_forms(gamma_on_refresh=False):
    """M0 = 0 and G = sigma u v^T: M1 = G; a rank-one matrix has one singular
    value, equal to its Frobenius norm, so refresh gives phi5(~1) u v^T
    (unit u, v); the row-wise branch maps every oriented row to sign times a
    unit vector.  With the scalar-controlled ablation (Table 3a: gamma on both
    branches) the refresh direction is gamma times the plain one and the
    row-wise one is unchanged."""
    rng = np.random.default_rng(17)
    for (m, n) in [(6, 10), (10, 6)]:
        u = rng.standard_normal(m)
        v = rng.standard_normal(n)
        G = 2.5 * np.outer(u, v)
        W = rng.standard_normal((m, n))
        cfg = po.PRMConfig(K=2, beta=0.9, gamma=0.3, wd=0.1, lr=0.05, gamma_on_refresh=gamma_on_refresh)
        s = math.sqrt(max(1.0, m / n))
        nf = np.linalg.norm(G)
        y = _quintic5(nf / (nf + 1e-7))
        g_ref = 0.3 if gamma_on_refresh else 1.0
        Wn, Mn, D, rho = po.step_matrix(W, np.zeros((m, n)), G, 0, cfg)
        assert rho == 1
        np.testing.assert_allclose(Mn, G)
        expect_D = g_ref * s * y * np.outer(u / np.linalg.norm(u), v / np.linalg.norm(v))
        np.testing.assert_allclose(D, expect_D, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(Wn, (1 - 0.05 * 0.1) * W - 0.05 * expect_D, rtol=1e-12)
        Wn, Mn, D, rho = po.step_matrix(W, np.zeros((m, n)), G, 1, cfg)
        assert rho == 0
        if m <= n:   # oriented rows are stored rows: each row is sign(u_i) v/||v||
            expect = 0.3 * s * np.outer(np.sign(u), v / np.linalg.norm(v))
        else:        # tall: oriented rows are stored columns: u/||u|| sign(v_j)
            expect = 0.3 * s * np.outer(u / np.linalg.norm(u), np.sign(v))
        np.testing.assert_allclose(D, expect, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(Wn, (1 - 0.05 * 0.1) * W - 0.05 * expect, rtol=1e-12)


def test_step_rank_one_closed_forms():
    pin_step_rank_one_closed_forms()


def test_scalar_controlled_ablation_closed_forms():
    pin_step_rank_one_closed_forms(gamma_on_refresh=True)


def pin_scalar_controlled_scales_refresh_only():
    """Scalar-controlled ablation on a full-rank input: over a trajectory, the
    refresh directions are exactly gamma times those of the paper's method and
    the row-wise directions are identical (the state never depends on D)."""
    rng = np.random.default_rng(23)
    for (m, n) in [(12, 30), (30, 12)]:
        a = po.PRMConfig(K=3, gamma=0.15)
        b = po.PRMConfig(K=3, gamma=0.15, gamma_on_refresh=True)
        Wa = Wb = rng.standard_normal((m, n))
        Ma = Mb = rng.standard_normal((m, n))
        for t in range(6):
            G = rng.standard_normal((m, n))
            Wa, Ma, Da, ra = po.step_matrix(Wa, Ma, G, t, a)
            Wb, Mb, Db, rb = po.step_matrix(Wb, Mb, G, t, b)
            assert ra == rb == (1 if t % 3 == 0 else 0)
            np.testing.assert_array_equal(Mb, Ma)
            np.testing.assert_allclose(Db, (0.15 if ra else 1.0) * Da, rtol=1e-13, atol=1e-16)


def test_scalar_controlled_scales_refresh_only():
    pin_scalar_controlled_scales_refresh_only()


def test_gamma_only_on_rownorm_branch_and_wd_uses_eta():
    # eq. (periodic-direction) and Alg. 2: gamma scales only the RowNorm output;
    # weight decay always uses eta_t.
    rng = np.random.default_rng(18)
    W = rng.standard_normal((8, 16))
    M = rng.standard_normal((8, 16))
    G = rng.standard_normal((8, 16))
    c1 = po.PRMConfig(K=2, gamma=0.15)
    c2 = po.PRMConfig(K=2, gamma=0.9)
    _, _, D1, _ = po.step_matrix(W, M, G, 0, c1)
    _, _, D2, _ = po.step_matrix(W, M, G, 0, c2)
    np.testing.assert_allclose(D1, D2)
    W1, _, Dr, _ = po.step_matrix(W, M, G, 1, c1, lr=0.0)
    np.testing.assert_allclose(W1, W)                # eta = 0: no decay, no update
    Wz, _, _, _ = po.step_matrix(W, M, np.zeros_like(G), 1, po.PRMConfig(K=2, beta=0.0), lr=0.1)
    np.testing.assert_allclose(Wz, (1 - 0.1 * 0.01) * W)  # zero momentum -> pure decay


def test_trajectory_schedule_over_period():
    rng = np.random.default_rng(19)
    shapes = [(8, 24), (24, 8)]
    Ws = [rng.standard_normal(s) for s in shapes]
    Ms = [np.zeros(s) for s in shapes]
    cfg = po.PRMConfig(K=4)
    rhos = []
    for t in range(9):
        Gs = [rng.standard_normal(s) for s in shapes]
        Ws, Ms, Ds, rho = po.step(Ws, Ms, Gs, t, cfg)
        rhos.append(rho)
    assert rhos == [1, 0, 0, 0, 1, 0, 0, 0, 1]


# ----------------------------------------------------------------- mutations
def test_mutations_are_caught(monkeypatch):
    """Plant plausible mistakes in the oracle (on the CPU) and check a pin fails."""
    rng = np.random.default_rng(20)
    X = rand_lowrank(rng, 16, 48)

    def svd_pin_holds():
        return rel(po.ns5(X), po.ns5_closed_form(X, coeffs=tuple(GOLD["ns_coefficients"]["value"]))) < 1e-12

    assert svd_pin_holds()
    # wrong sign of b
    monkeypatch.setattr(po, "NS_COEFFS", (3.4445, 4.7750, 2.0315))
    monkeypatch.setattr(po.ns5, "__defaults__", (1e-7, (3.4445, 4.7750, 2.0315), 5))
    assert not svd_pin_holds()
    # dropped quintic term
    monkeypatch.setattr(po.ns5, "__defaults__", (1e-7, (3.4445, -4.7750, 0.0), 5))
    assert not svd_pin_holds()
    # four iterations instead of five
    monkeypatch.setattr(po.ns5, "__defaults__", (1e-7, (3.4445, -4.7750, 2.0315), 4))
    assert not svd_pin_holds()
    monkeypatch.undo()
    assert svd_pin_holds()


def _raises(pin, *args):
    try:
        pin(*args)
    except AssertionError:
        return True
    return False


def test_rownorm_mutations_fail_their_pins(monkeypatch):
    """RowNorm mistakes planted into the oracle itself."""
    pin_rownorm_eps_clamp_after_sqrt()
    pin_sharded_tall_rownorm()
    real = po.rownorm

    # the clamp taken before the square root: max(||x||^2, eps)
    def clamp_before_sqrt(X, eps):
        X = np.asarray(X, dtype=np.float64)
        return X / np.sqrt(np.maximum(np.sum(X * X, axis=1), eps))[:, None]
    monkeypatch.setattr(po, "rownorm", clamp_before_sqrt)
    assert _raises(pin_rownorm_eps_clamp_after_sqrt)
    # the clamp dropped
    monkeypatch.setattr(po, "rownorm", lambda X, eps: X / np.linalg.norm(X, axis=1, keepdims=True))
    assert _raises(pin_rownorm_eps_clamp_after_sqrt)
    # the squared norm in the denominator
    monkeypatch.setattr(po, "rownorm", lambda X, eps: X / np.maximum(np.sum(X * X, axis=1), eps)[:, None])
    assert _raises(pin_rownorm_eps_clamp_after_sqrt)
    monkeypatch.setattr(po, "rownorm", real)
    # a tall matrix normalized along its stored rows (no orientation)
    monkeypatch.setattr(po, "orient", lambda M: M)
    monkeypatch.setattr(po, "orient_inv", lambda X, m, n: X)
    assert _raises(pin_sharded_tall_rownorm)
    assert _raises(pin_step_rank_one_closed_forms)
    monkeypatch.undo()
    pin_sharded_tall_rownorm()
    pin_step_rank_one_closed_forms()


def _step_with(U_of):
    """step_matrix with the direction input replaced by U_of(M_old, M_new, G, cfg)."""
    def step_matrix(W, M, G, t, cfg, lr=None):
        eta = cfg.lr if lr is None else lr
        W, M, G = (np.asarray(x, dtype=np.float64) for x in (W, M, G))
        M_new = po.momentum_update(M, G, cfg.beta, cfg.ema_dampening)
        D, rho = po.direction(U_of(M, M_new, G, cfg), t, cfg)
        return (1.0 - eta * cfg.wd) * W - eta * D, M_new, D, rho
    return step_matrix


def test_nesterov_mutations_fail_their_pins(monkeypatch):
    """Nesterov mistakes planted into the oracle's step."""
    pin_nesterov_lookahead()
    pin_nesterov_constructed_target()
    # the look-ahead built from the momentum before this step's update
    monkeypatch.setattr(po, "step_matrix",
                        _step_with(lambda Mo, Mn, G, c: G + c.beta * Mo if c.nesterov else Mn))
    assert _raises(pin_nesterov_lookahead)
    assert _raises(pin_nesterov_constructed_target)
    # beta dropped from the look-ahead
    monkeypatch.setattr(po, "step_matrix", _step_with(lambda Mo, Mn, G, c: G + Mn if c.nesterov else Mn))
    assert _raises(pin_nesterov_lookahead)
    assert _raises(pin_nesterov_constructed_target)
    # the flag ignored
    monkeypatch.setattr(po, "step_matrix", _step_with(lambda Mo, Mn, G, c: Mn))
    assert _raises(pin_nesterov_lookahead)
    assert _raises(pin_nesterov_constructed_target)
    # the correct form passes through the same wrapper
    monkeypatch.setattr(po, "step_matrix",
                        _step_with(lambda Mo, Mn, G, c: G + c.beta * Mn if c.nesterov else Mn))
    pin_nesterov_lookahead()
    pin_nesterov_constructed_target()


def test_scalar_controlled_mutations_fail_their_pins(monkeypatch):
    """gamma mistakes planted into the oracle's direction map."""
    pin_step_rank_one_closed_forms(True)
    pin_scalar_controlled_scales_refresh_only()
    real = po.direction

    def with_refresh_gamma(g_of):
        def direction(U, t, cfg):
            D, rho = real(U, t, po.PRMConfig(**{**cfg.__dict__, "gamma_on_refresh": False}))
            return (g_of(cfg) * D if rho else D), rho
        return direction
    # the ablation flag ignored (no gamma on the refresh branch)
    monkeypatch.setattr(po, "direction", with_refresh_gamma(lambda c: 1.0))
    assert _raises(pin_step_rank_one_closed_forms, True)
    assert _raises(pin_scalar_controlled_scales_refresh_only)
    # gamma applied twice
    monkeypatch.setattr(po, "direction", with_refresh_gamma(lambda c: c.gamma ** 2 if c.gamma_on_refresh else 1.0))
    assert _raises(pin_step_rank_one_closed_forms, True)
    assert _raises(pin_scalar_controlled_scales_refresh_only)
    # gamma on the refresh branch of the paper's method too
    monkeypatch.setattr(po, "direction", with_refresh_gamma(lambda c: c.gamma))
    assert _raises(pin_step_rank_one_closed_forms)
    # the correct rule passes through the same wrapper
    monkeypatch.setattr(po, "direction", with_refresh_gamma(lambda c: c.gamma if c.gamma_on_refresh else 1.0))
    pin_step_rank_one_closed_forms(True)
    pin_step_rank_one_closed_forms()
    pin_scalar_controlled_scales_refresh_only()


def test_config_rejects_nonpositive_clamps():
    # a zero eps_ns would turn a zero momentum into 0/0 in the input scaling
    for kw in ({"eps_ns": 0.0}, {"eps_rownorm": 0.0}, {"K": 0}):
        with pytest.raises(ValueError):
            po.PRMConfig(**kw)
    cfg = po.PRMConfig(K=1, beta=0.0)
    _, _, D, rho = po.step_matrix(np.ones((3, 5)), np.zeros((3, 5)), np.zeros((3, 5)), 0, cfg)
    assert rho == 1
    np.testing.assert_array_equal(D, 0.0)
