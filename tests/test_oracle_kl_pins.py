"""Pins of the oracle's KL-Shampoo factor accumulation (CPU only).

The KL-SOAP step of Algorithm 2 replaces the factor EMA by an update that
weighs each factor's new term by the inverse of the other factor, estimated
from its eigenvalues in the current eigenbasis.  The pins, each chosen so that
a plausible slip fails at least one of them:

* exact basis: when Q_R diagonalises R, the estimates are R's eigenvalues and
  the accumulation is the KL-Shampoo rule with the true inverse (R + eps I)^-1,
  computed by a linear solve (catches the exponent's sign, the basis the
  estimates act in, a transposed Q, the 1/out and 1/in normalisations, eps);
* the fixed point of Appendix A.3: L = U (S / sqrt(n)) U^T, R = V (S / sqrt(n))
  V^T with aligned bases is left unchanged (square G = U S V^T);
* the whole KL-SOAP iteration on a constant square gradient, started with
  bases aligned to U and V, converges to that fixed point, so the factor's
  condition number is the square root of the plain (Shampoo) factor's (the
  equation of Section 5.4.3); with beta_kron = 1/2 the eigenvalue recursion is
  Heron's square-root iteration;
* started from identity bases it ends on the KL-Shampoo fixed point with true
  inverses, L = G R^-1 G^T / n, R = G^T L^-1 G / n;
* identity start: with Q = I and unit-diagonal factors the accumulation is the
  plain factor EMA (pinned in test_oracle_pins) of G / sqrt(out), G^T / sqrt(in);
* one nonzero per gradient row and column keeps both factors diagonal, so the
  bases stay exactly I and KL-SOAP is AdamW (Section 2).
"""
import numpy as np
import pytest

import oracle

HP = dict(beta1=0.95, beta2=0.95, eps=1e-8, lr=1e-3, weight_decay=0.1)


def rel(x, y):
    return np.linalg.norm(x - y) / max(np.linalg.norm(y), 1e-300)


def _orthogonal(rng, n):
    Q, R = np.linalg.qr(rng.standard_normal((n, n)))
    return Q * np.sign(np.diag(R))


def test_eigenvalue_estimates_exact_in_eigenbasis():
    rng = np.random.default_rng(1)
    Q = _orthogonal(rng, 6)
    mu = rng.uniform(0.5, 3.0, 6)
    F = Q @ np.diag(mu) @ Q.T
    lam = oracle.eigenvalue_estimates(F, Q)
    assert np.max(np.abs(lam - mu)) <= 1e-13
    # in another basis the estimates are F's diagonal there, and they sum to the trace
    lam_i = oracle.eigenvalue_estimates(F, np.eye(6))
    assert np.array_equal(lam_i, np.diag(F))
    assert abs(lam.sum() - np.trace(F)) <= 1e-12


@pytest.mark.parametrize("m,n,eps", [(3, 5, 0.0), (5, 3, 1e-3), (4, 4, 0.25)])
def test_exact_basis_is_kl_shampoo_with_true_inverse(m, n, eps):
    rng = np.random.default_rng(m * 10 + n)
    QL, QR = _orthogonal(rng, m), _orthogonal(rng, n)
    L = QL @ np.diag(rng.uniform(0.5, 2.0, m)) @ QL.T
    R = QR @ np.diag(rng.uniform(0.5, 2.0, n)) @ QR.T
    G = rng.standard_normal((m, n))
    beta = 0.7
    L1, R1, lam_L, lam_R = oracle.kl_factors(L, R, QL, QR, G, beta, eps)
    want_L = beta * L + (1 - beta) / n * G @ np.linalg.solve(R + eps * np.eye(n), G.T)
    want_R = beta * R + (1 - beta) / m * G.T @ np.linalg.solve(L + eps * np.eye(m), G)
    assert rel(L1, want_L) <= 1e-12
    assert rel(R1, want_R) <= 1e-12
    assert np.array_equal(L1, L1.T) and np.array_equal(R1, R1.T)


@pytest.mark.parametrize("beta", [0.3, 0.95])
def test_appendix_fixed_point_is_stationary(beta):
    n = 5
    rng = np.random.default_rng(7)
    U, V = _orthogonal(rng, n), _orthogonal(rng, n)
    s = np.array([3.0, 2.0, 1.5, 0.7, 0.2])
    G = U @ np.diag(s) @ V.T
    L = U @ np.diag(s / np.sqrt(n)) @ U.T
    R = V @ np.diag(s / np.sqrt(n)) @ V.T
    L1, R1, lam_L, lam_R = oracle.kl_factors(L, R, U, V, G, beta, 0.0)
    assert rel(L1, L) <= 1e-13 and rel(R1, R) <= 1e-13
    assert np.max(np.abs(lam_R - s / np.sqrt(n))) <= 1e-13
    # the plain factor EMA does not stop there: it heads for U S^2 U^T
    Lp = oracle.factor_ema(L, G, beta)
    assert rel(Lp, L) > 1e-2


def _square_problem(n=4):
    rng = np.random.default_rng(3)
    U, V = _orthogonal(rng, n), _orthogonal(rng, n)
    s = np.array([8.0, 4.0, 2.0, 1.0])[:n]
    return U, V, s, U @ np.diag(s) @ V.T


@pytest.mark.parametrize("beta_kron,steps", [(0.5, 60), (0.95, 700)])
def test_kl_soap_converges_to_singular_values(beta_kron, steps):
    """Constant square G = U S V^T, factors started at I with the bases aligned
    to U and V (the assumption of Appendix A.3): the factor eigenvalues converge
    to S / sqrt(n), so kappa(L) = sqrt(kappa(G G^T)) (Section 5.4.3), and the
    refresh keeps the bases at U and V."""
    n = 4
    U, V, s, G = _square_problem(n)
    st = oracle.init_state(np.zeros((n, n)))
    st.QL, st.QR = U.copy(), V.copy()
    hp = dict(HP, eps=0.0)
    for t in range(1, steps + 1):
        st = oracle.kl_soap_step(st, G, t, beta_kron=beta_kron, **hp)
    evL = np.sort(np.linalg.eigvalsh(st.L))[::-1]
    evR = np.sort(np.linalg.eigvalsh(st.R))[::-1]
    assert np.max(np.abs(evL - s / np.sqrt(n))) <= 1e-12
    assert np.max(np.abs(evR - s / np.sqrt(n))) <= 1e-12
    kappa_kl = np.linalg.cond(st.L)
    kappa_shampoo = np.linalg.cond(G @ G.T)
    assert abs(kappa_kl - np.sqrt(kappa_shampoo)) <= 1e-10 * kappa_kl
    assert np.max(np.abs(st.QL - U)) <= 1e-12
    assert np.max(np.abs(st.QR - V)) <= 1e-12


@pytest.mark.parametrize("beta_kron,steps", [(0.5, 80), (0.95, 900)])
def test_kl_soap_from_identity_reaches_kl_shampoo_fixed_point(beta_kron, steps):
    """From identity bases the iteration still ends where the bases diagonalise
    the factors, so the estimated inverses are exact there and the limit obeys
    the KL-Shampoo rule of Appendix A.3 with true inverses:
    L = G R^-1 G^T / n and R = G^T L^-1 G / n.  (The spectra need not be the
    balanced S / sqrt(n) of the aligned start: every such pair is stationary.)"""
    n = 4
    U, V, s, G = _square_problem(n)
    st = oracle.init_state(np.zeros((n, n)))
    hp = dict(HP, eps=0.0)
    for t in range(1, steps + 1):
        st = oracle.kl_soap_step(st, G, t, beta_kron=beta_kron, **hp)
    L, R = st.L, st.R
    assert rel(L, G @ np.linalg.solve(R, G.T) / n) <= 1e-12
    assert rel(R, G.T @ np.linalg.solve(L, G) / n) <= 1e-12
    for F, Q in ((L, st.QL), (R, st.QR)):
        D = Q.T @ F @ Q
        assert np.linalg.norm(D - np.diag(np.diag(D))) <= 1e-12 * np.linalg.norm(D)
    # the product of the two factors' determinants is fixed by G alone
    assert abs(np.linalg.det(L) * np.linalg.det(R) - np.prod(s) ** 2 / n ** n) <= 1e-10


def test_heron_recursion_of_the_eigenvalues():
    """With aligned bases each eigenvalue pair follows a <- b a + (1-b) s^2 / (n a'),
    and from L = R = I the two sides stay equal; for b = 1/2 that is Heron's
    iteration for s / sqrt(n).  Checked step by step against the scalar recursion."""
    n = 3
    rng = np.random.default_rng(5)
    U, V = _orthogonal(rng, n), _orthogonal(rng, n)
    s = np.array([2.0, 1.0, 0.5])
    G = U @ np.diag(s) @ V.T
    L, R = U @ U.T, V @ V.T
    a = np.ones(n)
    for _ in range(8):
        L, R, _, _ = oracle.kl_factors(L, R, U, V, G, 0.5, 0.0)
        a = 0.5 * a + 0.5 * s * s / (n * a)
        assert np.max(np.abs(np.diag(U.T @ L @ U) - a)) <= 1e-13
        assert np.max(np.abs(np.diag(V.T @ R @ V) - a)) <= 1e-13
    assert np.max(np.abs(a - s / np.sqrt(n))) <= 1e-15


def test_identity_start_is_plain_ema_of_scaled_gradient():
    m, n = 3, 5
    rng = np.random.default_rng(9)
    G = rng.standard_normal((m, n))
    L1, R1, _, _ = oracle.kl_factors(np.eye(m), np.eye(n), np.eye(m), np.eye(n), G, 0.95, 0.0)
    assert rel(L1, oracle.factor_ema(np.eye(m), G / np.sqrt(n), 0.95)) <= 1e-15
    assert rel(R1, oracle.factor_ema(np.eye(n), G.T / np.sqrt(m), 0.95)) <= 1e-15


def _adamw_textbook(W, G, m, v, t, beta1, beta2, eps, lr, weight_decay):
    m = beta1 * m + (1 - beta1) * G
    v = beta2 * v + (1 - beta2) * G * G
    W = W - lr * weight_decay * W - lr * (m / (1 - beta1 ** t)) / (np.sqrt(v / (1 - beta2 ** t)) + eps)
    return W, m, v


def test_kl_identity_eigenbasis_reduces_to_adamw():
    from synth.gradients import permutation_gradient
    m, n = 5, 7
    rng = np.random.default_rng(10)
    W0 = rng.standard_normal((m, n))
    st = oracle.init_state(W0)
    Wa, ma, va = W0.copy(), np.zeros((m, n)), np.zeros((m, n))
    for t in range(1, 11):
        G = permutation_gradient(m, n, 3, t).astype(np.float64)
        st = oracle.kl_soap_step(st, G, t, beta_kron=0.95, **HP)
        Wa, ma, va = _adamw_textbook(Wa, G, ma, va, t, **HP)
        assert np.array_equal(st.QL, np.eye(m)) and np.array_equal(st.QR, np.eye(n))
        assert np.array_equal(np.diag(np.diag(st.L)), st.L)
        assert np.array_equal(np.diag(np.diag(st.R)), st.R)
        assert rel(st.W, Wa) <= 1e-14


def test_kl_step_keeps_factors_positive_definite():
    rng = np.random.default_rng(12)
    st = oracle.init_state(rng.standard_normal((6, 9)))
    for t in range(1, 6):
        st = oracle.kl_soap_step(st, rng.standard_normal((6, 9)), t, beta_kron=0.95, **HP)
        np.linalg.cholesky(st.L)
        np.linalg.cholesky(st.R)
        assert np.array_equal(st.L, st.L.T) and np.array_equal(st.R, st.R.T)
