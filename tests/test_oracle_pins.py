"""Pins the fp64 oracle to things other than itself (CPU only).

Each pin is chosen so that a plausible slip in the oracle (a dropped term, a
wrong sign or index, a transposed operand, a misplaced EMA coefficient) fails
at least one test:

* QR: residuals, LAPACK agreement after the sign fix, closed forms (2x2,
  diagonal, triangular, orthogonal input), rank-deficient input; the
  refresh's LAPACK route for large factors against the textbook code.
* Products: numpy's matmul against plain triple loops.
* Factor EMA: brute-force loops, exact symmetry, positive definiteness.
* Rotations: the identity map and norm preservation.
* Adam: a 1x1 closed form.
* Whole step: the paper's reduction to AdamW for identity eigenbases
  (Section 2), the update-RMS identity (Section 5.2), Algorithm 2's literal
  eigenbasis-resident momentum, the polar-factor limit (Appendix A.1) and a
  full step in 50-digit decimal arithmetic with a different QR algorithm.
"""
import decimal
from decimal import Decimal

import numpy as np
import pytest

import oracle
from oracle import soap_oracle as so

HP = dict(beta1=0.95, beta2=0.95, eps=1e-8, lr=1e-3, weight_decay=0.1)


def rel(x, y):
    return np.linalg.norm(x - y) / max(np.linalg.norm(y), 1e-300)


# ----------------------------------------------------------------------------- QR
@pytest.mark.parametrize("n", [1, 2, 3, 7, 33, 100, 257])
def test_qr_residuals(n):
    rng = np.random.default_rng(n)
    A = rng.standard_normal((n, n))
    Q, R = oracle.householder_qr(A, with_r=True)
    assert np.linalg.norm(Q @ R - A) / np.linalg.norm(A) <= 1e-12
    assert np.linalg.norm(Q.T @ Q - np.eye(n)) / np.sqrt(n) <= 1e-12
    assert np.all(np.diag(R) >= 0)
    assert np.all(np.tril(R, -1) == 0)


@pytest.mark.parametrize("n", [2, 5, 64, 300])
def test_qr_matches_lapack_after_sign_fix(n):
    rng = np.random.default_rng(100 + n)
    A = rng.standard_normal((n, n)) + 3 * np.eye(n)
    Ql, Rl = np.linalg.qr(A)          # LAPACK dgeqrf + dorgqr
    d = np.sign(np.diag(Rl))
    Ql = Ql * d
    Q = oracle.householder_qr(A)
    assert rel(Q, Ql) <= 1e-12


def test_qr_2x2_closed_form():
    for a, b, c, d in [(3.0, 1.0, 4.0, 2.0), (-1.0, 2.0, 0.5, -3.0), (0.0, 1.0, 2.0, 0.0)]:
        A = np.array([[a, b], [c, d]])
        r = np.hypot(a, c)
        q1 = np.array([a, c]) / r
        det = a * d - b * c
        q2 = np.array([-c, a]) / r * (1.0 if det > 0 else -1.0)
        Q = oracle.householder_qr(A)
        assert np.allclose(Q[:, 0], q1, atol=1e-15, rtol=0)
        assert np.allclose(Q[:, 1], q2, atol=1e-15, rtol=0)


def test_qr_diagonal_and_triangular_give_exact_identity():
    D = np.diag([3.0, 1e-3, 7.0, 2.0])
    assert np.array_equal(oracle.householder_qr(D), np.eye(4))
    U = np.triu(np.random.default_rng(1).standard_normal((6, 6))) + 5 * np.eye(6)
    assert np.array_equal(oracle.householder_qr(U), np.eye(6))
    # negative diagonal entries flip exactly the matching columns
    Dn = np.diag([2.0, -1.0, 3.0])
    assert np.array_equal(oracle.householder_qr(Dn), np.diag([1.0, -1.0, 1.0]))


def test_qr_of_orthogonal_matrix_is_itself():
    rng = np.random.default_rng(5)
    Q0, R0 = np.linalg.qr(rng.standard_normal((40, 40)))
    Q0 = Q0 * np.sign(np.diag(R0))
    assert np.max(np.abs(oracle.householder_qr(Q0) - Q0)) <= 1e-13


def test_qr_rank_deficient():
    rng = np.random.default_rng(6)
    A = rng.standard_normal((8, 8))
    A[:, 3] = 0.0
    A[:, 5] = A[:, 1]
    Q, R = oracle.householder_qr(A, with_r=True)
    assert np.linalg.norm(Q @ R - A) / np.linalg.norm(A) <= 1e-13
    assert np.linalg.norm(Q.T @ Q - np.eye(8)) <= 1e-13
    assert np.all(np.diag(R) >= 0)


@pytest.mark.parametrize("n", [1, 2, 5, 64, 300, 1000])
def test_lapack_route_matches_textbook_householder(n):
    """The refresh's LAPACK route (blocked Householder, dgeqrf + dorgqr) reaches
    the same unique Q as the unblocked textbook C code, with the same sign
    convention, and meets the fp64 residual bars on its own."""
    rng = np.random.default_rng(200 + n)
    A = rng.standard_normal((n, n)) + 2 * np.eye(n)
    Ql = oracle.lapack_qr(A)
    assert rel(Ql, oracle.householder_qr(A)) <= 1e-12
    assert np.linalg.norm(Ql.T @ Ql - np.eye(n)) / np.sqrt(n) <= 1e-12
    R = Ql.T @ A
    assert np.linalg.norm(Ql @ np.triu(R) - A) / np.linalg.norm(A) <= 1e-12
    assert np.all(np.diag(R) >= -1e-12 * np.linalg.norm(A))


def test_lapack_route_closed_forms():
    for a, b, c, d in [(3.0, 1.0, 4.0, 2.0), (-1.0, 2.0, 0.5, -3.0)]:
        A = np.array([[a, b], [c, d]])
        r = np.hypot(a, c)
        Q = oracle.lapack_qr(A)
        assert np.allclose(Q[:, 0], np.array([a, c]) / r, atol=1e-15, rtol=0)
        assert np.allclose(Q[:, 1], np.array([-c, a]) / r * np.sign(a * d - b * c),
                           atol=1e-15, rtol=0)
    assert np.array_equal(oracle.lapack_qr(np.diag([3.0, 1e-3, 7.0])), np.eye(3))
    assert np.array_equal(oracle.lapack_qr(np.diag([2.0, -1.0, 3.0])), np.diag([1.0, -1.0, 1.0]))


def test_refresh_takes_the_textbook_route_up_to_its_limit(monkeypatch):
    rng = np.random.default_rng(11)
    A = rng.standard_normal((50, 50)) + 3 * np.eye(50)
    calls = []
    monkeypatch.setattr(so, "householder_qr", lambda X: calls.append("textbook") or np.eye(50))
    monkeypatch.setattr(so, "lapack_qr", lambda X: calls.append("lapack") or np.eye(50))
    so.refresh_qr(A)
    monkeypatch.setattr(so, "TEXTBOOK_QR_MAX", 49)
    so.refresh_qr(A)
    assert calls == ["textbook", "lapack"]


def test_matrix_products_against_naive_loops():
    """The oracle's products (numpy's matmul, a library primitive) against
    plain triple loops: the power product F Q, both rotations, and the
    factor products G G^T, G^T G."""
    rng = np.random.default_rng(12)
    m, n = 5, 7
    G = rng.standard_normal((m, n))
    QL = np.linalg.qr(rng.standard_normal((m, m)))[0]
    QR = np.linalg.qr(rng.standard_normal((n, n)))[0]
    S = rng.standard_normal((n, n))
    F = S + S.T

    def mm(A, B):
        return np.array([[sum(A[i][k] * B[k][j] for k in range(len(B)))
                          for j in range(len(B[0]))] for i in range(len(A))])

    def tr(A):
        return [list(r) for r in zip(*A)]

    assert np.max(np.abs(F @ QR - mm(F, QR))) <= 1e-13
    assert np.max(np.abs(oracle.rotate_in(QL, G, QR) - mm(mm(tr(QL), G), QR))) <= 1e-13
    assert np.max(np.abs(oracle.rotate_out(QL, G, QR) - mm(mm(QL, G), tr(QR)))) <= 1e-13
    assert np.max(np.abs(oracle.factor_ema(np.zeros((m, m)), G, 0.0) - mm(G, tr(G)))) <= 1e-13
    assert np.max(np.abs(oracle.factor_ema(np.zeros((n, n)), G.T, 0.0) - mm(tr(G), G))) <= 1e-13


# ------------------------------------------------------------------ factor EMA
def test_factor_ema_brute_force():
    rng = np.random.default_rng(7)
    G = rng.standard_normal((3, 4))
    S = rng.standard_normal((3, 3))
    F = S + S.T
    beta = 0.8
    want = [[beta * F[i][j] + (1 - beta) * sum(G[i][k] * G[j][k] for k in range(4))
             for j in range(3)] for i in range(3)]
    assert np.max(np.abs(oracle.factor_ema(F, G, beta) - np.array(want))) <= 1e-14
    S4 = rng.standard_normal((4, 4))
    F4 = S4 + S4.T
    want_r = [[beta * F4[i][j] + (1 - beta) * sum(G[k][i] * G[k][j] for k in range(3))
               for j in range(4)] for i in range(4)]
    assert np.max(np.abs(oracle.factor_ema(F4, G.T, beta) - np.array(want_r))) <= 1e-14


def test_factor_ema_symmetric_and_positive_definite():
    rng = np.random.default_rng(8)
    L = np.eye(20)
    beta = 0.95
    for t in range(1, 16):
        L = oracle.factor_ema(L, rng.standard_normal((20, 5)), beta)
        assert np.array_equal(L, L.T)
        np.linalg.cholesky(L)
        # identity start: L - beta^t I is a sum of PSD terms
        assert np.min(np.linalg.eigvalsh(L - beta ** t * np.eye(20))) >= -1e-12


# ------------------------------------------------------------------ rotations
def test_rotations_identity_and_norm():
    rng = np.random.default_rng(9)
    X = rng.standard_normal((6, 9))
    assert np.array_equal(oracle.rotate_in(np.eye(6), X, np.eye(9)), X)
    assert np.array_equal(oracle.rotate_out(np.eye(6), X, np.eye(9)), X)
    QL = np.linalg.qr(rng.standard_normal((6, 6)))[0]
    QR = np.linalg.qr(rng.standard_normal((9, 9)))[0]
    Y = oracle.rotate_in(QL, X, QR)
    assert abs(np.linalg.norm(Y) - np.linalg.norm(X)) <= 1e-13 * np.linalg.norm(X)
    assert rel(oracle.rotate_out(QL, Y, QR), X) <= 1e-14
    # rotate_in must be Q_L^T X Q_R, not Q_L X Q_R^T
    assert rel(Y, QL.T @ X @ QR) <= 1e-14
    assert rel(Y, QL @ X @ QR.T) > 1e-3


# ------------------------------------------------------------------- Adam 1x1
def test_adam_scalar_closed_form():
    # beta2 = 0.5, V = 0, g' = 2 -> V = 2; t = 1: c2 = 0.5 -> sqrt(V/c2) = 2
    # m' = 1, c1 = 0.5 -> m'/c1 = 2 -> N = 2 / (2 + eps)
    V, N = oracle.adam_eigenbasis(np.array([[2.0]]), np.array([[1.0]]), np.array([[0.0]]),
                                  0.5, 1e-8, 0.5, 0.5)
    assert V[0, 0] == 2.0
    assert N[0, 0] == 2.0 / (2.0 + 1e-8)
    c1, c2 = oracle.bias_corrections(0.9, 0.95, 3, True)
    assert c1 == 1 - 0.9 ** 3 and c2 == 1 - 0.95 ** 3
    assert oracle.bias_corrections(0.9, 0.95, 3, False) == (1.0, 1.0)


# --------------------------------------------------------------- whole step
def _adamw_textbook(W, G, m, v, t, beta1, beta2, eps, lr, weight_decay):
    m = beta1 * m + (1 - beta1) * G
    v = beta2 * v + (1 - beta2) * G * G
    mhat = m / (1 - beta1 ** t)
    vhat = v / (1 - beta2 ** t)
    W = W - lr * weight_decay * W - lr * mhat / (np.sqrt(vhat) + eps)
    return W, m, v


def test_identity_eigenbasis_reduces_to_adamw():
    """Section 2: with identity eigenvectors SOAP is AdamW.  Gradients with one
    nonzero per row and column keep L and R diagonal, so Q stays exactly I."""
    from synth.gradients import permutation_gradient
    m, n = 5, 7
    rng = np.random.default_rng(10)
    W0 = rng.standard_normal((m, n))
    st = oracle.init_state(W0)
    Wa, ma, va = W0.copy(), np.zeros((m, n)), np.zeros((m, n))
    for t in range(1, 11):
        G = permutation_gradient(m, n, 3, t).astype(np.float64)
        st = oracle.soap_step(st, G, t, **HP)
        Wa, ma, va = _adamw_textbook(Wa, G, ma, va, t, **HP)
        assert np.array_equal(st.QL, np.eye(m)) and np.array_equal(st.QR, np.eye(n))
        assert np.array_equal(np.diag(np.diag(st.L)), st.L)
        assert rel(st.W, Wa) <= 1e-14
        assert rel(st.M, ma) <= 1e-15
        assert rel(st.V, va) <= 1e-15


def test_update_rms_identity():
    """Section 5.2: ||Delta W||_F = ||N||_F because the rotations are orthogonal."""
    rng = np.random.default_rng(11)
    st = oracle.init_state(rng.standard_normal((12, 20)))
    for t in range(1, 4):
        st, d = oracle.soap_step(st, rng.standard_normal((12, 20)), t, diagnostics=True, **HP)
        assert abs(np.linalg.norm(d["dW"]) - np.linalg.norm(d["N"])) <= 1e-12 * np.linalg.norm(d["N"])


def _sign_fixed_lapack_q(A):
    Q, R = np.linalg.qr(A)
    return Q * np.where(np.diag(R) < 0, -1.0, 1.0)


def test_weight_space_momentum_equals_algorithm2_literal():
    """Algorithm 2 keeps m in the eigenbasis and re-rotates it at each refresh
    (rotate back with the old Q, forward with the new Q).  With F = 1 this must
    equal the weight-space momentum used by the oracle."""
    rng = np.random.default_rng(12)
    m, n = 9, 14
    b1, b2, eps, lr, wd = 0.9, 0.95, 1e-8, 1e-2, 0.1
    W = rng.standard_normal((m, n))
    st = oracle.init_state(W)
    L, R, QL, QR = np.eye(m), np.eye(n), np.eye(m), np.eye(n)
    me, v, Wl = np.zeros((m, n)), np.zeros((m, n)), W.copy()
    for t in range(1, 7):
        G = rng.standard_normal((m, n))
        st = oracle.soap_step(st, G, t, beta1=b1, beta2=b2, eps=eps, lr=lr, weight_decay=wd)
        # Algorithm 2, beta on the old state, LAPACK QR with the sign fix
        L = b2 * L + (1 - b2) * G @ G.T
        R = b2 * R + (1 - b2) * G.T @ G
        mhat = QL @ me @ QR.T
        QL = _sign_fixed_lapack_q(L @ QL)
        QR = _sign_fixed_lapack_q(R @ QR)
        me = QL.T @ mhat @ QR
        Gp = QL.T @ G @ QR
        me = b1 * me + (1 - b1) * Gp
        v = b2 * v + (1 - b2) * Gp * Gp
        N = (me / (1 - b1 ** t)) / (np.sqrt(v / (1 - b2 ** t)) + eps)
        Wl = (1 - lr * wd) * Wl - lr * QL @ N @ QR.T
        assert rel(st.QL, QL) <= 1e-12 and rel(st.QR, QR) <= 1e-12
        assert rel(st.V, v) <= 1e-11
        assert rel(st.W, Wl) <= 1e-12


def test_polar_factor_limit():
    """Appendix A.1: with the EMAs off, the eigenbases converge to the singular
    vectors of a fixed G, Adam tends to sign(Sigma), and Delta W -> U V^T."""
    rng = np.random.default_rng(13)
    n = 4
    U = _sign_fixed_lapack_q(rng.standard_normal((n, n)))
    Vt = _sign_fixed_lapack_q(rng.standard_normal((n, n))).T
    G = U @ np.diag([8.0, 4.0, 2.0, 1.0]) @ Vt
    Us, _, Vts = np.linalg.svd(G)
    polar = Us @ Vts
    st = oracle.init_state(np.zeros((n, n)))
    for t in range(1, 31):
        st, d = oracle.soap_step(st, G, t, beta1=0.0, beta2=0.0, eps=1e-8, lr=1.0,
                                 weight_decay=0.0, diagnostics=True)
    assert rel(d["dW"], polar) <= 1e-6
    # a transposed rotation would not converge to the polar factor
    assert rel(d["dW"].T, polar) > 1e-2


# -------------------------------------------------- 50-digit brute force step
decimal.getcontext().prec = 50


def _D(x):
    return [[Decimal(float(v)) for v in row] for row in np.asarray(x)]


def _mm(A, B):
    return [[sum((A[i][k] * B[k][j] for k in range(len(B))), Decimal(0))
             for j in range(len(B[0]))] for i in range(len(A))]


def _T(A):
    return [list(r) for r in zip(*A)]


def _mgs_q(A):
    """Modified Gram-Schmidt (a different algorithm than Householder) in 50
    digits; for nonsingular A it yields the unique Q with positive diag(R)."""
    n = len(A)
    cols = [[A[i][j] for i in range(n)] for j in range(n)]
    qs = []
    for j in range(n):
        v = cols[j][:]
        for q in qs:
            r = sum((q[i] * v[i] for i in range(n)), Decimal(0))
            v = [v[i] - r * q[i] for i in range(n)]
        nrm = sum((x * x for x in v), Decimal(0)).sqrt()
        qs.append([x / nrm for x in v])
    return [[qs[j][i] for j in range(n)] for i in range(n)]


def test_full_step_against_50_digit_brute_force():
    rng = np.random.default_rng(14)
    m, n = 3, 4
    b1, b2, eps, lr, wd, t = 0.9, 0.95, 1e-8, 1e-2, 0.1, 3
    G = rng.standard_normal((m, n))
    W = rng.standard_normal((m, n))
    Ls = rng.standard_normal((m, m)); L = Ls @ Ls.T + np.eye(m)
    Rs = rng.standard_normal((n, n)); R = Rs @ Rs.T + np.eye(n)
    QL = _sign_fixed_lapack_q(rng.standard_normal((m, m)))
    QR = _sign_fixed_lapack_q(rng.standard_normal((n, n)))
    M = rng.standard_normal((m, n))
    V = rng.random((m, n))
    st = oracle.OracleState(W, L, R, QL, QR, M, V)
    new = oracle.soap_step(st, G, t, beta1=b1, beta2=b2, eps=eps, lr=lr, weight_decay=wd)

    one = Decimal(1)
    B1, B2, E, LR, WD = (Decimal(x) for x in (b1, b2, eps, lr, wd))
    Gd, Wd, Ld, Rd, QLd, QRd, Md, Vd = map(_D, (G, W, L, R, QL, QR, M, V))
    GGt, GtG = _mm(Gd, _T(Gd)), _mm(_T(Gd), Gd)
    Ld = [[B2 * Ld[i][j] + (one - B2) * GGt[i][j] for j in range(m)] for i in range(m)]
    Rd = [[B2 * Rd[i][j] + (one - B2) * GtG[i][j] for j in range(n)] for i in range(n)]
    QLd = _mgs_q(_mm(Ld, QLd))
    QRd = _mgs_q(_mm(Rd, QRd))
    Md = [[B1 * Md[i][j] + (one - B1) * Gd[i][j] for j in range(n)] for i in range(m)]
    Gp = _mm(_mm(_T(QLd), Gd), QRd)
    Mp = _mm(_mm(_T(QLd), Md), QRd)
    c1 = one - B1 ** t
    c2 = one - B2 ** t
    Vd = [[B2 * Vd[i][j] + (one - B2) * Gp[i][j] * Gp[i][j] for j in range(n)] for i in range(m)]
    Nd = [[(Mp[i][j] / c1) / ((Vd[i][j] / c2).sqrt() + E) for j in range(n)] for i in range(m)]
    dW = _mm(_mm(QLd, Nd), _T(QRd))
    Wd = [[(one - LR * WD) * Wd[i][j] - LR * dW[i][j] for j in range(n)] for i in range(m)]

    def f(X):
        return np.array([[float(v) for v in row] for row in X])

    for got, want in [(new.L, Ld), (new.R, Rd), (new.QL, QLd), (new.QR, QRd), (new.M, Md),
                      (new.V, Vd), (new.W, Wd)]:
        assert rel(got, f(want)) <= 1e-13


# ------------------------------------------- refresh period and stale refresh
@pytest.mark.parametrize("F", [2, 3])
def test_refresh_period_equals_algorithm2_literal(F):
    """Algorithm 2 with t mod F gating: the eigenbasis-resident m is rotated
    back and forward only at a refresh, V never.  The oracle's weight-space
    momentum must give the same step for any F."""
    rng = np.random.default_rng(40 + F)
    m, n = 7, 11
    b1, b2, eps, lr, wd = 0.9, 0.95, 1e-8, 1e-2, 0.1
    W = rng.standard_normal((m, n))
    st = oracle.init_state(W)
    L, R, QL, QR = np.eye(m), np.eye(n), np.eye(m), np.eye(n)
    me, v, Wl = np.zeros((m, n)), np.zeros((m, n)), W.copy()
    for t in range(1, 9):
        G = rng.standard_normal((m, n))
        st = oracle.soap_step(st, G, t, beta1=b1, beta2=b2, eps=eps, lr=lr, weight_decay=wd,
                              refresh_every=F)
        L = b2 * L + (1 - b2) * G @ G.T
        R = b2 * R + (1 - b2) * G.T @ G
        if t % F == 0:
            mhat = QL @ me @ QR.T
            QL = _sign_fixed_lapack_q(L @ QL)
            QR = _sign_fixed_lapack_q(R @ QR)
            me = QL.T @ mhat @ QR
        Gp = QL.T @ G @ QR
        me = b1 * me + (1 - b1) * Gp
        v = b2 * v + (1 - b2) * Gp * Gp
        N = (me / (1 - b1 ** t)) / (np.sqrt(v / (1 - b2 ** t)) + eps)
        Wl = (1 - lr * wd) * Wl - lr * QL @ N @ QR.T
        assert rel(st.QL, QL) <= 1e-12 and rel(st.QR, QR) <= 1e-12
        assert rel(st.V, v) <= 1e-11
        assert rel(st.W, Wl) <= 1e-12
        if t < F:
            assert np.array_equal(st.QL, np.eye(m)) and np.array_equal(st.QR, np.eye(n))


def test_stale_refresh_uses_the_previous_factors():
    """Sections 5.4.1-5.4.2: the stale variant refreshes from the factors before
    the current gradient enters them.  From the identity start its first
    refresh is QR(I Q) = I exactly; afterwards each refresh equals the
    sign-fixed LAPACK QR of L_{t-1} Q_{t-1}, R_{t-1} Q_{t-1}."""
    rng = np.random.default_rng(44)
    m, n = 6, 9
    st = oracle.init_state(rng.standard_normal((m, n)))
    for t in range(1, 6):
        prev = st
        st = oracle.soap_step(prev, rng.standard_normal((m, n)), t, stale_refresh=True, **HP)
        if t == 1:
            assert np.array_equal(st.QL, np.eye(m)) and np.array_equal(st.QR, np.eye(n))
        assert rel(st.QL, _sign_fixed_lapack_q(prev.L @ prev.QL)) <= 1e-12
        assert rel(st.QR, _sign_fixed_lapack_q(prev.R @ prev.QR)) <= 1e-12
    # the KL variant refreshes from the same pre-gradient factors
    st = oracle.init_state(rng.standard_normal((m, n)))
    for t in range(1, 4):
        prev = st
        st = oracle.kl_soap_step(prev, rng.standard_normal((m, n)), t, beta_kron=0.95,
                                 stale_refresh=True, **HP)
        assert rel(st.QL, _sign_fixed_lapack_q(prev.L @ prev.QL)) <= 1e-12
        assert rel(st.QR, _sign_fixed_lapack_q(prev.R @ prev.QR)) <= 1e-12


def test_fresh_refresh_sees_the_new_gradient_first():
    """The point of Section 5.4.2: after the gradient switches to a new
    direction u2, the fresh refresh brings u2 into the leading two basis
    vectors in the very next step; the stale one does so exactly one step
    later (its refresh at step t is the fresh refresh of step t - 1)."""
    m, n = 5, 8
    rng = np.random.default_rng(45)
    U, _ = np.linalg.qr(rng.standard_normal((m, m)))
    u1, u2 = U[:, 0], U[:, 1]
    v1 = rng.standard_normal(n)
    v1 /= np.linalg.norm(v1)
    hp = dict(HP, beta2=0.5)
    fresh, stale = oracle.init_state(np.zeros((m, n))), oracle.init_state(np.zeros((m, n)))
    for t in range(1, 6):
        G = np.outer(u1, v1)
        fresh = oracle.soap_step(fresh, G, t, **hp)
        stale = oracle.soap_step(stale, G, t, stale_refresh=True, **hp)
    reach = lambda Q: np.linalg.norm(Q[:, :2].T @ u2)
    assert reach(fresh.QL) < 0.2 and reach(stale.QL) < 0.2
    G = 10.0 * np.outer(u2, v1)
    fresh = oracle.soap_step(fresh, G, 6, **hp)
    stale = oracle.soap_step(stale, G, 6, stale_refresh=True, **hp)
    assert reach(fresh.QL) > 0.9999 and reach(stale.QL) < 0.2
    stale = oracle.soap_step(stale, G, 7, stale_refresh=True, **hp)
    assert reach(stale.QL) > 0.9999
