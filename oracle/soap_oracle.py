"""fp64 oracle of one SOAP optimizer step (TEST INFRASTRUCTURE ONLY).

Only tests/, the smoke check and the bench's CPU-baseline leg may import this
module.  Every input is the exact fp32 array handed to the GPU, promoted to fp64.

The step follows the paper's KL-SOAP listing (Algorithm 2, "KL-SOAP used in
experiments") with the plain-EMA Kronecker factors of the Shampoo primer
(Section 2), refresh frequency F = 1 (hyperparameter table of Section 5.4) and
the real-time refresh of Section 5.4.2 (the current gradient enters the factors
before the eigenbasis is recomputed).  Readings where the paper is silent or
inconsistent:

  * EMA coefficients multiply the OLD state (Section 2 primer, Muon Algorithm 1,
    the hyperparameter table's "EMA coefficient" wording); Algorithm 2's
    placement of beta on the new term is read as a notation slip.
  * The first moment is kept in weight space and rotated every step,
    M' = Q_L^T M Q_R (Eq. 1).  With F = 1 and orthogonal Q this equals Algorithm
    2's rotate-back / rotate-in of an eigenbasis-resident m (pinned in tests).
  * V lives in the eigenbasis and is not re-rotated at a refresh (Algorithm 2
    touches only m there).
  * Adam bias correction is on by default (c1 = 1 - beta1^t, c2 = 1 - beta2^t),
    eps is added to sqrt(V / c2); with the flag off the step is Algorithm 2
    literally.  Identity eigenbases then reproduce AdamW (Section 2).
  * One beta2 serves the factor EMA and V (the table gives both 0.95).
  * QR(.).Q means the Q factor with non-negative diagonal R (unique for
    nonsingular input).
  * Initial state: L = R = Q_L = Q_R = I, M = V = 0.

kl_soap_step is the KL-SOAP variant the paper recommends (Sections 5.4.3 and
7): the factors are accumulated by the KL-Shampoo rule of Algorithm 2
(readings in kl_factor_update), the rest of the step is unchanged.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Dict, Optional, Tuple

import numpy as np

from . import build as _build

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = _build.build()
        lib = ctypes.CDLL(path)
        lib.oracle_householder_qr.restype = ctypes.c_int
        lib.oracle_householder_qr.argtypes = [
            ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
        _LIB = lib
    return _LIB


def _threads() -> int:
    return int(os.environ.get("OMP_NUM_THREADS", "0") or 0)


@dataclasses.dataclass
class OracleState:
    """Per-matrix SOAP state (Algorithm 2 "Optimizer States"), fp64.

    W, M, V: m x n (M in weight space, V in the eigenbasis); L, Q_L: m x m;
    R, Q_R: n x n.
    """
    W: np.ndarray
    L: np.ndarray
    R: np.ndarray
    QL: np.ndarray
    QR: np.ndarray
    M: np.ndarray
    V: np.ndarray

    def copy(self) -> "OracleState":
        return OracleState(*(np.array(getattr(self, f.name), copy=True)
                             for f in dataclasses.fields(self)))


def init_state(W: np.ndarray) -> OracleState:
    """L = R = Q_L = Q_R = I and M = V = 0 (initial state; the paper gives none)."""
    m, n = W.shape
    return OracleState(np.array(W, dtype=np.float64), np.eye(m), np.eye(n), np.eye(m),
                       np.eye(n), np.zeros((m, n)), np.zeros((m, n)))


def factor_ema(F: np.ndarray, X: np.ndarray, beta: float) -> np.ndarray:
    """Kronecker-factor EMA of the Shampoo primer (Section 2):
    F <- beta F + (1 - beta) X X^T.  For L pass X = G, for R pass X = G^T.

    The result is symmetric by definition; it is formed from its lower triangle
    (the old F is read only there) and mirrored."""
    S = beta * np.asarray(F, dtype=np.float64) + (1.0 - beta) * (X @ X.T)
    low = np.tril(S)
    return low + np.tril(low, -1).T


def householder_qr(A: np.ndarray, with_r: bool = False):
    """Q of A = QR with non-negative diag(R), by textbook unblocked Householder
    (see householder.c).  Algorithm 2's eigenbasis refresh applies this to
    L_t Q_L and R_t Q_R."""
    A = np.ascontiguousarray(A, dtype=np.float64)
    n = A.shape[0]
    if A.shape != (n, n):
        raise ValueError("square matrices only")
    Q = np.empty((n, n))
    R = np.empty((n, n)) if with_r else None
    rc = _lib().oracle_householder_qr(n, A.ctypes.data, Q.ctypes.data,
                                      R.ctypes.data if with_r else None, _threads())
    if rc != 0:
        raise RuntimeError("oracle QR failed")
    return (Q, R) if with_r else Q


def lapack_qr(A: np.ndarray) -> np.ndarray:
    """Q of A = QR with non-negative diag(R) through LAPACK's blocked Householder
    QR (dgeqrf, then dorgqr for the explicit Q: a library primitive) and the
    same column-sign fix as householder.c (a column whose R diagonal is
    negative is negated; a zero diagonal keeps its sign).  Same unique Q as
    householder_qr for nonsingular A, reached by a different summation order;
    the pins hold the two within 1e-12 of each other."""
    from scipy.linalg import lapack
    A = np.asfortranarray(A, dtype=np.float64)
    n = A.shape[0]
    if A.shape != (n, n):
        raise ValueError("square matrices only")
    lwork = max(1, 256 * n)
    qr, tau, _, info = lapack.dgeqrf(A, lwork=lwork)
    if info != 0:
        raise RuntimeError("dgeqrf failed")
    sgn = np.where(np.diag(qr) < 0.0, -1.0, 1.0)
    Q, _, info = lapack.dorgqr(qr, tau, lwork=lwork, overwrite_a=True)
    if info != 0:
        raise RuntimeError("dorgqr failed")
    return np.ascontiguousarray(Q * sgn[None, :])


# Largest factor dimension whose refresh runs the textbook C Householder QR;
# above it (its memory-bound rank-1 updates would take minutes) the refresh
# takes LAPACK's blocked route to the same unique Q.
TEXTBOOK_QR_MAX = 4096


def refresh_qr(A: np.ndarray) -> np.ndarray:
    """The eigenbasis refresh's QR(.).Q (Algorithm 2): householder_qr up to
    TEXTBOOK_QR_MAX, lapack_qr above."""
    return householder_qr(A) if A.shape[0] <= TEXTBOOK_QR_MAX else lapack_qr(A)


def momentum_ema(M: np.ndarray, G: np.ndarray, beta1: float) -> np.ndarray:
    """First-moment EMA in weight space (Section 2 primer; Eq. 1 rotates m_t):
    M <- beta1 M + (1 - beta1) G."""
    return beta1 * M + (1.0 - beta1) * G


def rotate_in(QL: np.ndarray, X: np.ndarray, QR: np.ndarray) -> np.ndarray:
    """Rotation into the eigenbasis, Q_L^T X Q_R (Algorithm 2, "Rotate gradient
    into eigenbasis"; Eq. 1 for the first moment).  Evaluated as (Q_L^T X) Q_R."""
    return (QL.T @ X) @ QR


def bias_corrections(beta1: float, beta2: float, t: int, enabled: bool) -> Tuple[float, float]:
    """Adam bias corrections c1 = 1 - beta1^t, c2 = 1 - beta2^t (1, 1 when off)."""
    if not enabled:
        return 1.0, 1.0
    return 1.0 - beta1 ** t, 1.0 - beta2 ** t


def adam_eigenbasis(Gp: np.ndarray, Mp: np.ndarray, V: np.ndarray, beta2: float,
                    eps: float, c1: float, c2: float) -> Tuple[np.ndarray, np.ndarray]:
    """Adam in the eigenbasis (Algorithm 2, "Calculate Adam update"):
    V <- beta2 V + (1 - beta2) G' * G';  N = (M'/c1) / (sqrt(V/c2) + eps)."""
    V = beta2 * V + (1.0 - beta2) * Gp * Gp
    N = (Mp / c1) / (np.sqrt(V / c2) + eps)
    return V, N


def rotate_out(QL: np.ndarray, N: np.ndarray, QR: np.ndarray) -> np.ndarray:
    """Rotation back, Delta W = Q_L N Q_R^T (Algorithm 2, "Rotate update out of
    eigenbasis").  Evaluated as (Q_L N) Q_R^T."""
    return (QL @ N) @ QR.T


def weight_update(W: np.ndarray, dW: np.ndarray, lr: float, wd: float) -> np.ndarray:
    """Decoupled weight decay and update (Algorithm 2, last step):
    W <- (1 - lr wd) W - lr Delta W."""
    return (1.0 - lr * wd) * W - lr * dW


def eigenvalue_estimates(F: np.ndarray, Q: np.ndarray) -> np.ndarray:
    """Approximate eigenvalues of a Kronecker factor in the current eigenbasis
    (Algorithm 2, KL-Shampoo accumulation): lambda = diag(Q^T F Q), with the
    factor and basis of the previous step."""
    return np.diag(Q.T @ F @ Q).copy()


def kl_factor_update(F: np.ndarray, X: np.ndarray, Q_other: np.ndarray, lam_other: np.ndarray,
                     beta_kron: float, eps: float, count: int) -> np.ndarray:
    """KL-Shampoo accumulation of one Kronecker factor (Algorithm 2; the
    KL-Shampoo rule restated in Appendix A.3):

        F <- beta_kron F + (1 - beta_kron) / count * X S^{-1} X^T,
        S^{-1} = Q_other diag(1 / (lam_other + eps)) Q_other^T.

    For L pass X = G (m x n), the R-side basis and eigenvalue estimates and
    count = n ("out"); for R pass X = G^T, the L-side ones and count = m
    ("in").  Readings: beta_kron multiplies the old factor, like every EMA of
    the Section 2 primer; the exponent applied to (lambda + eps) is -1, the
    inverse the appendix's rule uses; and the eigenvalue estimates act in the
    basis they were measured in, so S^{-1} is the inverse of the other factor
    as that basis diagonalises it.  The result is symmetric by definition; it
    is formed from its lower triangle and mirrored."""
    Sinv = Q_other @ np.diag(1.0 / (lam_other + eps)) @ Q_other.T
    S = beta_kron * np.asarray(F, dtype=np.float64) + ((1.0 - beta_kron) / count) * (X @ Sinv @ X.T)
    low = np.tril(S)
    return low + np.tril(low, -1).T


def refresh_due(t: int, refresh_every: int) -> bool:
    """Algorithm 2 recomputes the eigenbasis when t mod F = 0 (t is 1-based,
    so F = 1 refreshes every step)."""
    if refresh_every < 1:
        raise ValueError("the refresh period F must be >= 1")
    return t % refresh_every == 0


def _refresh_and_update(s: OracleState, G: np.ndarray, t: int, beta1: float, beta2: float,
                        eps: float, lr: float, weight_decay: float, bias_correction: bool,
                        diagnostics: bool, FL: Optional[np.ndarray], FR: Optional[np.ndarray]):
    """The part of the step after the factor update: power product and QR
    refresh from the factors FL, FR (skipped when they are None: the bases are
    kept), first-moment EMA, rotation in, Adam, rotation out, weight update
    (Algorithm 2).  The first moment lives in weight space, so a refresh needs
    no re-rotation of it: rotating it in with whichever bases are current is
    Algorithm 2's rotate-back / rotate-in of an eigenbasis-resident m."""
    AL = AR = None
    if FL is not None:
        AL = FL @ s.QL
        AR = FR @ s.QR
        s.QL = refresh_qr(AL)
        s.QR = refresh_qr(AR)
    s.M = momentum_ema(s.M, G, beta1)
    Gp = rotate_in(s.QL, G, s.QR)
    Mp = rotate_in(s.QL, s.M, s.QR)
    c1, c2 = bias_corrections(beta1, beta2, t, bias_correction)
    s.V, N = adam_eigenbasis(Gp, Mp, s.V, beta2, eps, c1, c2)
    dW = rotate_out(s.QL, N, s.QR)
    s.W = weight_update(s.W, dW, lr, weight_decay)
    if diagnostics:
        return s, {"AL": AL, "AR": AR, "Gp": Gp, "Mp": Mp, "N": N, "dW": dW}
    return s


def soap_step(state: OracleState, G: np.ndarray, t: int, beta1: float, beta2: float,
              eps: float, lr: float, weight_decay: float, bias_correction: bool = True,
              diagnostics: bool = False, refresh_every: int = 1, stale_refresh: bool = False):
    """One SOAP step on one matrix (Algorithm 2).

    Order: factor EMA with the current G, power product and QR refresh, first
    moment EMA, rotation in, Adam, rotation out, weight update.  The refresh
    runs when t mod refresh_every = 0 (Algorithm 2's F; F = 1 is the paper's
    setting).  stale_refresh takes the power product from the factors as they
    were before this step's gradient was added: the lagging preconditioner that
    Section 5.4.1 shows unstable and Section 5.4.2 replaces (an ablation).
    Returns the new state (and a dict of intermediates when ``diagnostics``)."""
    if t < 1:
        raise ValueError("step t is 1-based")
    G = np.asarray(G, dtype=np.float64)
    s = state.copy()
    L_old, R_old = s.L, s.R
    s.L = factor_ema(s.L, G, beta2)
    s.R = factor_ema(s.R, G.T, beta2)
    FL, FR = (L_old, R_old) if stale_refresh else (s.L, s.R)
    if not refresh_due(t, refresh_every):
        FL = FR = None
    return _refresh_and_update(s, G, t, beta1, beta2, eps, lr, weight_decay, bias_correction,
                               diagnostics, FL, FR)


def kl_factors(L: np.ndarray, R: np.ndarray, QL: np.ndarray, QR: np.ndarray, G: np.ndarray,
               beta_kron: float, eps: float):
    """Both KL-Shampoo factor updates of Algorithm 2 from the previous step's
    L, R, Q_L, Q_R: the eigenvalue estimates of both factors are taken first,
    then each factor is accumulated with the other side's estimates.  Returns
    (L_new, R_new, lam_L, lam_R)."""
    G = np.asarray(G, dtype=np.float64)
    m, n = G.shape
    lam_L = eigenvalue_estimates(L, QL)
    lam_R = eigenvalue_estimates(R, QR)
    L_new = kl_factor_update(L, G, QR, lam_R, beta_kron, eps, n)
    R_new = kl_factor_update(R, G.T, QL, lam_L, beta_kron, eps, m)
    return L_new, R_new, lam_L, lam_R


def kl_soap_step(state: OracleState, G: np.ndarray, t: int, beta1: float, beta2: float,
                 beta_kron: float, eps: float, lr: float, weight_decay: float,
                 bias_correction: bool = True, diagnostics: bool = False,
                 refresh_every: int = 1, stale_refresh: bool = False):
    """One KL-SOAP step (Algorithm 2): the factor EMA of soap_step is replaced
    by the KL-Shampoo accumulation (kl_factors); the same eps serves the
    eigenvalue floor and Adam (hyperparameter table of Section 5.4).
    Everything after the accumulation, including refresh_every and
    stale_refresh, is soap_step's."""
    if t < 1:
        raise ValueError("step t is 1-based")
    G = np.asarray(G, dtype=np.float64)
    s = state.copy()
    L_old, R_old = s.L, s.R
    s.L, s.R, lam_L, lam_R = kl_factors(s.L, s.R, s.QL, s.QR, G, beta_kron, eps)
    FL, FR = (L_old, R_old) if stale_refresh else (s.L, s.R)
    if not refresh_due(t, refresh_every):
        FL = FR = None
    out = _refresh_and_update(s, G, t, beta1, beta2, eps, lr, weight_decay, bias_correction,
                              diagnostics, FL, FR)
    if diagnostics:
        out[1]["lam_L"], out[1]["lam_R"] = lam_L, lam_R
    return out


def soap_step_batched(states, Gs, t: int, **hp):
    """The batched entry point is B independent single-matrix steps."""
    return [soap_step(st, G, t, **hp) for st, G in zip(states, Gs)]


def kl_soap_step_batched(states, Gs, t: int, **hp):
    """The batched KL entry point is B independent single-matrix KL steps."""
    return [kl_soap_step(st, G, t, **hp) for st, G in zip(states, Gs)]
