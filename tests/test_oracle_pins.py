"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test ties the oracle to something other than itself: the coefficients the
paper prints (Eq. 6), the exact inverse fourth root of Shampoo's EMA factor
(Eq. 2 and Algorithm 1) within the truncation error of the series (Eq. 5),
spectral closed forms in the commuting case, a similarity identity that holds
for any state, exact special cases (G = 0), invariants (symmetry, grafting
norm, orthogonal equivariance, transpose duality, the update interval) and a
50-digit mpmath evaluation on tiny inputs.
"""
import os
from fractions import Fraction

import mpmath
import numpy as np
import pytest

from oracle import (BETA_CLAMPED, BETA_DYNAMIC, BETA_FIXED, SERIES_C1, SERIES_C2, SERIES_C3,
                    JorgeOracle, beta_select, gram_factors, init_factor, update_factor,
                    update_weights)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_orth(rng, d):
    q, r = np.linalg.qr(rng.standard_normal((d, d)))
    return q * np.sign(np.diag(r))


def rand_spd(rng, d, lo=0.5, hi=2.0):
    q = rand_orth(rng, d)
    s = (q * rng.uniform(lo, hi, d)) @ q.T
    return 0.5 * (s + s.T)                      # bitwise symmetric


# Series coefficients of (1 + a)^(-1/4), independently of the oracle.
_TAYLOR = [float(c) for c in mpmath.taylor(lambda a: (1 + a) ** mpmath.mpf(-0.25), 0, 4)]


# ---------------------------------------------------------------- series coefficients
def test_series_coefficients_match_paper_and_taylor():
    vals = {}
    with open(os.path.join(GOLDEN, "series_coefficients.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, num, den = line.split()
                vals[name] = Fraction(int(num), int(den))
    assert SERIES_C1 == float(vals["linear"]) == _TAYLOR[1]
    assert SERIES_C2 == float(vals["quadratic"]) == _TAYLOR[2]
    # The cubic term that Section 3 drops (kept by series_order=3): Eq. 5's general term.
    assert SERIES_C3 == _TAYLOR[3] == -15.0 / 128.0


# ---------------------------------------------------------------- step 1 vs exact
def _first_step_case(rng, m, n, sigma, beta2, mode, eps=1e-6, series_order=2):
    G = rng.standard_normal((m, n)) * sigma
    M = G @ G.T
    L1, diag = update_factor(init_factor(m, eps), M, beta2, mode, symmetrize=True,
                             series_order=series_order)
    lam, U = np.linalg.eigh(M)
    lam = np.clip(lam, 0.0, None)
    l0 = eps ** -0.25
    nu = l0 ** 4 * np.sqrt(np.sum(lam ** 2))        # ||X||_F with X = l0^4 M
    if mode == BETA_FIXED or (mode == BETA_CLAMPED and nu / (nu + 1) <= beta2):
        beta = beta2
    else:
        beta = nu / (nu + 1)
    return G, M, L1, diag, lam, U, l0, nu, beta


@pytest.mark.parametrize("mode,sigma,beta2,dynamic", [
    (BETA_FIXED, 3e-4, 0.9, False),     # ||cX|| < 1 with the user beta
    (BETA_DYNAMIC, 1e-2, 0.9, True),
    (BETA_DYNAMIC, 1e-4, 0.9, True),    # small nu: still nu/(nu+1)
    (BETA_CLAMPED, 1e-2, 0.9, True),    # clamps to the dynamic value
    (BETA_CLAMPED, 2.5e-4, 0.9, False), # 1/9 < nu < 9: stays on beta2
    (BETA_CLAMPED, 1e-4, 0.5, False),   # stays on beta2
])
def test_step1_within_truncation_bound_of_exact_inverse_root(mode, sigma, beta2, dynamic):
    rng = np.random.default_rng(1)
    m, n, eps = 7, 11, 1e-6
    G, M, L1, diag, lam, U, l0, nu, beta = _first_step_case(rng, m, n, sigma, beta2, mode, eps)
    assert (beta != beta2) == dynamic
    assert diag["nu"] == pytest.approx(nu, rel=1e-12)
    assert diag["beta_eff"] == pytest.approx(beta, rel=1e-12)
    # Shampoo's EMA factor after one step from L_0 = eps I (Eq. 2), exact inverse 4th root.
    L_exact_eigs = (beta * eps + (1 - beta) * lam) ** -0.25
    s = beta ** -0.25
    a = (1 - beta) / beta * l0 ** 4 * lam
    assert np.all(a <= 1 + 1e-12)
    # At t = 1 the oracle's factor is diagonal in the eigenbasis of G G^T.
    D = U.T @ L1 @ U
    scale = np.abs(np.diag(D)).max()
    assert np.abs(D - np.diag(np.diag(D))).max() <= 1e-12 * scale
    err = np.diag(D) - L_exact_eigs
    bound = s * l0 * (-_TAYLOR[3]) * a ** 3
    # Alternating series: truncation leaves the first omitted (negative) term's sign.
    assert np.all(err >= -1e-12 * scale)
    assert np.all(err <= bound * (1 + 1e-9) + 1e-12 * scale)
    # The spectral form of the truncated update itself (Eq. 6 with p = 1/4).
    series = s * l0 * (1 + _TAYLOR[1] * a + _TAYLOR[2] * a ** 2)
    np.testing.assert_allclose(np.diag(D), series, rtol=1e-12, atol=1e-12 * scale)


@pytest.mark.parametrize("mode,sigma,beta2", [
    (BETA_DYNAMIC, 1e-2, 0.9),          # c X normalised: eigenvalues of c X up to 1
    (BETA_CLAMPED, 1e-2, 0.9),
    (BETA_FIXED, 3e-4, 0.9),
])
def test_step1_cubic_series_within_quartic_bound(mode, sigma, beta2):
    """series_order=3 keeps Eq. 5's cubic term: the error against the exact
    inverse fourth root then has the sign of the quartic term and at most its
    size, and it is smaller than the quadratic truncation's wherever a > 0."""
    rng = np.random.default_rng(1)
    m, n, eps = 7, 11, 1e-6
    G, M, L3, diag, lam, U, l0, nu, beta = _first_step_case(rng, m, n, sigma, beta2, mode, eps,
                                                           series_order=3)
    L2, _ = update_factor(init_factor(m, eps), M, beta2, mode, symmetrize=True)
    L_exact_eigs = (beta * eps + (1 - beta) * lam) ** -0.25
    s = beta ** -0.25
    a = (1 - beta) / beta * l0 ** 4 * lam
    assert np.all(a <= 1 + 1e-12) and a.max() > 0.05
    D3, D2 = U.T @ L3 @ U, U.T @ L2 @ U
    scale = np.abs(np.diag(D3)).max()
    assert np.abs(D3 - np.diag(np.diag(D3))).max() <= 1e-12 * scale
    err3 = np.diag(D3) - L_exact_eigs
    err2 = np.diag(D2) - L_exact_eigs
    assert np.all(err3 <= 1e-12 * scale)
    assert np.all(err3 >= -s * l0 * _TAYLOR[4] * a ** 4 * (1 + 1e-9) - 1e-12 * scale)
    big = a > 0.05
    assert np.all(np.abs(err3[big]) < np.abs(err2[big]))
    series = s * l0 * (1 + _TAYLOR[1] * a + _TAYLOR[2] * a ** 2 + _TAYLOR[3] * a ** 3)
    np.testing.assert_allclose(np.diag(D3), series, rtol=1e-12, atol=1e-12 * scale)


# ---------------------------------------------------------------- commuting closed form
def _beta_paper(nu, beta2, mode):
    if mode == BETA_FIXED or nu == 0:
        return (1 - beta2) / beta2, beta2 ** -0.25
    if mode == BETA_CLAMPED and nu <= beta2 / (1 - beta2):
        return (1 - beta2) / beta2, beta2 ** -0.25
    return 1.0 / nu, ((nu + 1.0) / nu) ** 0.25          # Eq. 9


@pytest.mark.parametrize("series_order", [2, 3])
@pytest.mark.parametrize("mode,sigma,beta2", [(BETA_FIXED, 3e-4, 0.99),
                                              (BETA_CLAMPED, 1e-2, 0.9),
                                              (BETA_DYNAMIC, 1e-3, 0.9)])
def test_commuting_gradients_follow_scalar_recurrence(mode, sigma, beta2, series_order):
    """G_t = U diag(sigma_t) V^T with fixed U, V: each factor stays diagonal in U (V)."""
    rng = np.random.default_rng(2)
    m, n, eps, steps = 5, 8, 1e-6, 6
    U, V = rand_orth(rng, m), rand_orth(rng, n)
    orc = JorgeOracle([(m, n)], eps=eps, beta_mode=mode, series_order=series_order)
    lL = np.full(m, eps ** -0.25)
    lR = np.full(n, eps ** -0.25)
    for t in range(steps):
        sig = rng.uniform(0.2, 1.0, m) * sigma
        G = U @ np.diag(sig) @ V[:, :m].T
        orc.step([np.zeros((m, n))], [G], 0.1, beta2, 0.9, 0.0)
        for lam_vals, l in ((np.concatenate([sig ** 2]), lL),
                            (np.concatenate([sig ** 2, np.zeros(n - m)]), lR)):
            x = l ** 4 * lam_vals
            c, s = _beta_paper(np.sqrt(np.sum(x ** 2)), beta2, mode)
            cubic = -15 * (c * x) ** 3 / 128 if series_order == 3 else 0.0
            l *= s * (1 - c * x / 4 + 5 * c * c * x * x / 32 + cubic)
        st = orc.layers[0]
        np.testing.assert_allclose(st.L, (U * lL) @ U.T, rtol=0, atol=1e-12 * lL.max())
        np.testing.assert_allclose(st.R, (V * lR) @ V.T, rtol=0, atol=1e-12 * lR.max())


# ---------------------------------------------------------------- any state: similarity
@pytest.mark.parametrize("series_order", [2, 3])
@pytest.mark.parametrize("mode", [BETA_FIXED, BETA_CLAMPED])
def test_update_similarity_identity_noncommuting(mode, series_order):
    """For X = A^4 M: A^-3 Z A^2 = s P(K) with K = A^2 M A^2 symmetric.

    X = A^2 K A^-2, so the literal update Z = s A P(X) satisfies the identity;
    the opposite orientation M A^4 (or P A) does not. nu is checked against
    the spectral form ||X||_F^2 = sum_i l_i^8 ||(U^T M)_i||^2.
    """
    rng = np.random.default_rng(3)
    d = 6
    A = rand_spd(rng, d, 0.6, 1.4)
    Gm = rng.standard_normal((d, 9)) * 0.05
    M = Gm @ Gm.T
    Z, diag = update_factor(A, M, 0.9, mode, symmetrize=False, series_order=series_order)
    l, U = np.linalg.eigh(A)
    nu_spec = np.sqrt(np.sum(l ** 8 * np.sum((U.T @ M) ** 2, axis=1)))
    assert diag["nu"] == pytest.approx(nu_spec, rel=1e-12)
    A2 = (U * l ** 2) @ U.T
    K = A2 @ M @ A2
    c, s = diag["c"], diag["s"]
    PK = np.eye(d) + _TAYLOR[1] * c * K + _TAYLOR[2] * c * c * (K @ K)
    if series_order == 3:
        PK = PK + _TAYLOR[3] * c ** 3 * (K @ K @ K)
    Ainv3 = (U * l ** -3.0) @ U.T
    lhs = Ainv3 @ Z @ A2
    np.testing.assert_allclose(lhs, s * PK, rtol=0, atol=1e-11 * np.abs(PK).max())
    # symmetrize=True is exactly the symmetric part of the literal update.
    Zs, _ = update_factor(A, M, 0.9, mode, symmetrize=True, series_order=series_order)
    np.testing.assert_array_equal(Zs, 0.5 * (Z + Z.T))


# ---------------------------------------------------------------- exact special cases
@pytest.mark.parametrize("series_order", [2, 3])
@pytest.mark.parametrize("mode", [BETA_FIXED, BETA_CLAMPED])
def test_zero_gradient_is_pure_beta_scaling(mode, series_order):
    rng = np.random.default_rng(4)
    m, n = 4, 6
    orc = JorgeOracle([(m, n)], beta_mode=mode, series_order=series_order)
    st = orc.layers[0]
    st.L, st.R = rand_spd(rng, m), rand_spd(rng, n)
    st.m, st.m_sgd = rng.standard_normal((m, n)), rng.standard_normal((m, n))
    L0, R0, m0, s0 = st.L.copy(), st.R.copy(), st.m.copy(), st.m_sgd.copy()
    beta2, beta1, lr, wd = 0.8, 0.7, 0.3, 0.01
    theta0 = rng.standard_normal((m, n))
    (theta1,) = orc.step([theta0], [np.zeros((m, n))], lr, beta2, beta1, wd)
    assert np.array_equal(st.L, 0.5 * ((beta2 ** -0.25 * L0) + (beta2 ** -0.25 * L0).T))
    np.testing.assert_allclose(st.L, beta2 ** -0.25 * L0, rtol=1e-15, atol=0)
    np.testing.assert_allclose(st.R, beta2 ** -0.25 * R0, rtol=1e-15, atol=0)
    np.testing.assert_allclose(st.m, beta1 * m0, rtol=1e-15)
    np.testing.assert_allclose(st.m_sgd, beta1 * s0, rtol=1e-15)
    g = lr * np.linalg.norm(beta1 * s0) / np.linalg.norm(beta1 * m0)
    np.testing.assert_allclose(theta1, theta0 * (1 - lr * wd) - g * beta1 * m0, rtol=1e-14)
    # From zero momenta the parameters only decay.
    orc2 = JorgeOracle([(m, n)], beta_mode=mode)
    (theta1,) = orc2.step([theta0], [np.zeros((m, n))], lr, beta2, beta1, wd)
    np.testing.assert_array_equal(theta1, theta0 * (1 - lr * wd))


def test_beta_select_modes():
    # DYNAMIC/CLAMPED branch keeps ||c X|| = 1 (Eq. 8 with equality); FIXED uses beta2.
    c, s, b = beta_select(50.0, 0.9, BETA_DYNAMIC)
    assert c * 50.0 == pytest.approx(1.0, rel=1e-15) and b == pytest.approx(50 / 51)
    assert s == pytest.approx(b ** -0.25, rel=1e-14)
    assert beta_select(0.0, 0.9, BETA_DYNAMIC)[:2] == beta_select(0.0, 0.9, BETA_FIXED)[:2]
    # CLAMPED is continuous at the switch nu = beta2/(1-beta2).
    nu0 = 0.9 / 0.1
    lo = beta_select(nu0 * (1 - 1e-12), 0.9, BETA_CLAMPED)
    hi = beta_select(nu0 * (1 + 1e-12), 0.9, BETA_CLAMPED)
    assert lo[0] == pytest.approx(hi[0], rel=1e-10) and lo[1] == pytest.approx(hi[1], rel=1e-10)
    with pytest.raises(ValueError):
        beta_select(1.0, 0.9, 7)


@pytest.mark.parametrize("mode", [BETA_DYNAMIC, BETA_CLAMPED])
def test_dynamic_branch_normalises_cX(mode):
    rng = np.random.default_rng(5)
    A = rand_spd(rng, 5) * 10
    G = rng.standard_normal((5, 7))
    _, diag = update_factor(A, G @ G.T, 0.9, mode)
    assert diag["nu"] > 9
    assert np.linalg.norm(diag["c"] * diag["X"]) == pytest.approx(1.0, rel=1e-14)


# ---------------------------------------------------------------- invariants
def _random_run(rng, m, n, steps, mode=BETA_CLAMPED, transform=None, graft=True, k=1):
    orc = JorgeOracle([(m, n)], beta_mode=mode, graft=graft, precond_interval=k)
    theta = rng.standard_normal((m, n))
    grads = [rng.standard_normal((m, n)) * 10 ** rng.uniform(-3, -1) for _ in range(steps)]
    for G in grads:
        if transform is not None:
            G = transform(G)
        (theta,) = orc.step([theta], [G], 0.05, 0.9, 0.9, 1e-3)
    return orc, theta


def test_factors_stay_exactly_symmetric():
    orc, _ = _random_run(np.random.default_rng(6), 5, 9, 8)
    st = orc.layers[0]
    assert np.array_equal(st.L, st.L.T) and np.array_equal(st.R, st.R.T)


def test_orthogonal_equivariance():
    """G -> Q G P gives L -> Q L Q^T, R -> P^T R P, m -> Q m P (isotropic init)."""
    m, n, steps = 5, 7, 6
    rng = np.random.default_rng(7)
    Q, P = rand_orth(rng, m), rand_orth(rng, n)
    grads = [rng.standard_normal((m, n)) * 10 ** rng.uniform(-3, -1) for _ in range(steps)]
    a = JorgeOracle([(m, n)])
    b = JorgeOracle([(m, n)])
    ta, tb = np.zeros((m, n)), np.zeros((m, n))
    for G in grads:
        (ta,) = a.step([ta], [G], 0.05, 0.9, 0.9, 1e-3)
        (tb,) = b.step([tb], [Q @ G @ P], 0.05, 0.9, 0.9, 1e-3)
    sa, sb = a.layers[0], b.layers[0]
    for x, y in ((Q @ sa.L @ Q.T, sb.L), (P.T @ sa.R @ P, sb.R), (Q @ sa.m @ P, sb.m),
                 (Q @ ta @ P, tb)):
        np.testing.assert_allclose(y, x, rtol=0, atol=1e-10 * np.abs(x).max())


def test_transpose_duality():
    """A run on G^T is the transposed run, with the roles of L_hat and R_hat swapped."""
    m, n, steps = 4, 7, 6
    rng = np.random.default_rng(8)
    grads = [rng.standard_normal((m, n)) * 10 ** rng.uniform(-3, -1) for _ in range(steps)]
    theta0 = rng.standard_normal((m, n))
    a, b = JorgeOracle([(m, n)]), JorgeOracle([(n, m)])
    ta, tb = theta0, theta0.T.copy()
    for G in grads:
        (ta,) = a.step([ta], [G], 0.05, 0.9, 0.9, 1e-3)
        (tb,) = b.step([tb], [G.T.copy()], 0.05, 0.9, 0.9, 1e-3)
    np.testing.assert_allclose(b.layers[0].L, a.layers[0].R, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b.layers[0].R, a.layers[0].L, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(tb, ta.T, rtol=1e-12, atol=1e-14)


def test_graft_norm_identity():
    rng = np.random.default_rng(9)
    m, n = 6, 5
    orc = JorgeOracle([(m, n)])
    theta = rng.standard_normal((m, n))
    lr, wd = 0.07, 3e-3
    for _ in range(5):
        G = rng.standard_normal((m, n)) * 1e-2
        (new,) = orc.step([theta], [G], lr, 0.9, 0.9, wd)
        step = new - theta * (1 - lr * wd)
        assert np.linalg.norm(step) == pytest.approx(lr * np.linalg.norm(orc.layers[0].m_sgd),
                                                     rel=1e-12)
        theta = new


def test_update_interval_and_momentum_closed_forms():
    """k larger than the run: factors update once, then stay bitwise fixed.

    With a constant G the momenta have closed forms:
    m_SGD,t = G (1 - b^t)/(1 - b) and m_t = (1 - b^t) L_1 G R_1; without
    grafting theta_t = theta_{t-1} (1 - lr wd) - lr m_t.
    """
    rng = np.random.default_rng(10)
    m, n, b, lr, wd = 4, 6, 0.8, 0.1, 0.02
    G = rng.standard_normal((m, n)) * 1e-2
    orc = JorgeOracle([(m, n)], precond_interval=100, graft=False)
    theta = rng.standard_normal((m, n))
    (theta,) = orc.step([theta], [G], lr, 0.9, b, wd)
    st = orc.layers[0]
    L1, R1 = st.L.copy(), st.R.copy()
    Gt = L1 @ G @ R1
    for t in range(2, 8):
        prev = theta
        (theta,) = orc.step([theta], [G], lr, 0.9, b, wd)
        assert np.array_equal(st.L, L1) and np.array_equal(st.R, R1)
        np.testing.assert_allclose(st.m_sgd, G * (1 - b ** t) / (1 - b), rtol=1e-13)
        np.testing.assert_allclose(st.m, (1 - b ** t) * Gt, rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(theta, prev * (1 - lr * wd) - lr * st.m, rtol=1e-13)
    # k = 3: updates on steps 1, 4, 7, ...
    orc = JorgeOracle([(m, n)], precond_interval=3)
    seen = []
    for t in range(1, 8):
        before = orc.layers[0].L.copy()
        orc.step([np.zeros((m, n))], [G * t], lr, 0.9, b, wd)
        seen.append(not np.array_equal(before, orc.layers[0].L))
    assert seen == [True, False, False, True, False, False, True]


# ---------------------------------------------------------------- full first step, SVD form
@pytest.mark.parametrize("graft", [True, False])
def test_first_step_svd_closed_form(graft):
    """From the isotropic start, step 1 has a closed form in the SVD G = U S V^T.

    Both statistics share the nonzero eigenvalues S^2, so nu_L = nu_R; the
    factors are U f_L U^T and V f_R V^T and G_tilde = U f_L S f_R V^T.
    """
    rng = np.random.default_rng(11)
    m, n, eps, beta2, beta1, lr, wd = 5, 8, 1e-6, 0.9, 0.9, 0.1, 1e-3
    G = rng.standard_normal((m, n)) * 1e-2
    theta0 = rng.standard_normal((m, n))
    orc = JorgeOracle([(m, n)], eps=eps, graft=graft)
    (theta1,) = orc.step([theta0], [G], lr, beta2, beta1, wd)
    U, S, Vt = np.linalg.svd(G)
    l0 = eps ** -0.25
    x = l0 ** 4 * S ** 2
    nu = np.sqrt(np.sum(x ** 2))
    c, s = 1.0 / nu, ((nu + 1) / nu) ** 0.25           # clamps to the dynamic branch
    assert nu > beta2 / (1 - beta2)
    f = s * l0 * (1 + _TAYLOR[1] * c * x + _TAYLOR[2] * (c * x) ** 2)
    fR = np.full(n, s * l0)
    fR[:m] = f
    st = orc.layers[0]
    np.testing.assert_allclose(st.L, (U * f) @ U.T, rtol=0, atol=1e-12 * l0)
    np.testing.assert_allclose(st.R, (Vt.T * fR) @ Vt, rtol=0, atol=1e-12 * l0)
    Gt = (U * (f * S * f)) @ Vt[:m]
    m1 = (1 - beta1) * Gt
    np.testing.assert_allclose(st.m, m1, rtol=0, atol=1e-12 * np.abs(m1).max())
    g = lr * np.linalg.norm(G) / np.linalg.norm(m1) if graft else lr
    np.testing.assert_allclose(theta1, theta0 * (1 - lr * wd) - g * m1, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- 50-digit evaluation
def _mp_step(Lh, Rh, mom, msgd, theta, G, lr, beta2, beta1, wd):
    def upd(A, M):
        d = A.rows
        X = A * A * A * A * M
        nu = mpmath.sqrt(sum(X[i, j] ** 2 for i in range(d) for j in range(d)))
        if nu > beta2 / (1 - beta2):
            c, s = 1 / nu, (1 + 1 / nu) ** mpmath.mpf(0.25)
        else:
            c, s = (1 - beta2) / beta2, beta2 ** mpmath.mpf(-0.25)
        P = mpmath.eye(d) - (c / 4) * X + (5 * c * c / 32) * (X * X)
        Z = s * (A * P)
        return (Z + Z.T) / 2
    Lh = upd(Lh, G * G.T)
    Rh = upd(Rh, G.T * G)
    mom = beta1 * mom + (1 - beta1) * (Lh * G * Rh)
    msgd = beta1 * msgd + G
    g = lr * mpmath.mnorm(msgd, "f") / mpmath.mnorm(mom, "f")
    theta = theta * (1 - lr * wd) - g * mom
    return Lh, Rh, mom, msgd, theta


def test_oracle_rounding_against_mpmath():
    mpmath.mp.dps = 50
    rng = np.random.default_rng(12)
    for (m, n) in ((2, 3), (3, 2)):
        orc = JorgeOracle([(m, n)])
        theta = rng.standard_normal((m, n))
        mp = [mpmath.matrix(init_factor(m, 1e-6).tolist()), mpmath.matrix(init_factor(n, 1e-6).tolist()),
              mpmath.zeros(m, n), mpmath.zeros(m, n), mpmath.matrix(theta.tolist())]
        mp[0] = mpmath.eye(m) * mpmath.mpf(10) ** mpmath.mpf(1.5)
        mp[1] = mpmath.eye(n) * mpmath.mpf(10) ** mpmath.mpf(1.5)
        for _ in range(5):
            G = rng.standard_normal((m, n)) * 1e-2
            (theta,) = orc.step([theta], [G], 0.1, 0.9, 0.9, 1e-3)
            mp = list(_mp_step(*mp, mpmath.matrix(G.tolist()), mpmath.mpf(0.1), mpmath.mpf(0.9),
                               mpmath.mpf(0.9), mpmath.mpf(1e-3)))
        st = orc.layers[0]
        for ours, ref in ((st.L, mp[0]), (st.R, mp[1]), (st.m, mp[2]), (theta, mp[4])):
            ref = np.array(ref.tolist(), dtype=np.float64)
            assert np.linalg.norm(ours - ref) <= 1e-12 * np.linalg.norm(ref)


def test_gram_factors_shapes_and_symmetry():
    G = np.arange(12.0).reshape(3, 4)
    ML, MR = gram_factors(G)
    assert ML.shape == (3, 3) and MR.shape == (4, 4)
    assert np.array_equal(ML, ML.T) and ML[0, 1] == sum(G[0] * G[1])
    assert MR[1, 2] == sum(G[:, 1] * G[:, 2])


def test_update_weights_no_graft_zero_norm():
    z = np.zeros((2, 2))
    theta, m, msgd, info = update_weights(np.ones((2, 2)), z, z, z, z, 0.1, 0.9, 0.5, graft=True)
    assert info["g"] == 0.0 and np.array_equal(theta, np.full((2, 2), 0.95))
