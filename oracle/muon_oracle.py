"""fp64 oracle of one Muon optimizer step (TEST INFRASTRUCTURE ONLY).

Only tests/, the smoke check and the bench's CPU-baseline leg may import this
module.  It follows the paper's Muon listing (Algorithm 1, "MomentUm
Orthogonalized by Newton-Schulz with Weight Decay") step by step:

    M <- beta1 M + (1 - beta1) G
    X_0 = M / max(||M||_F, eps)
    for i = 1..n:  A = X X^T,  B = b_i A + c_i A^2,  X <- a_i X + B X
    Delta W = X_n * sqrt(max(in, out))
    W <- (1 - lr wd) W - lr Delta W

The coefficient triples (a_i, b_i, c_i) are inputs: the paper uses the
PolarExpress schedule without printing it (hyperparameter table of Section
5.3), so callers pass their own.  Readings: beta1 multiplies the old momentum
(Algorithm 1 as printed); "in" and "out" are the two dimensions of the m x n
weight (Algorithm 1's states are in x out).
"""
from __future__ import annotations

import numpy as np


def momentum_ema(M: np.ndarray, G: np.ndarray, beta1: float) -> np.ndarray:
    """Algorithm 1, momentum buffer: M <- beta1 M + (1 - beta1) G."""
    return beta1 * M + (1.0 - beta1) * G


def newton_schulz(M: np.ndarray, coeffs, eps: float) -> np.ndarray:
    """Algorithm 1's orthogonalisation: X_0 = M / max(||M||_F, eps), then one
    polynomial step X <- a X + (b A + c A^2) X with A = X X^T per triple."""
    X = M / max(np.linalg.norm(M), eps)
    for a, b, c in coeffs:
        A = X @ X.T
        B = b * A + c * (A @ A)
        X = a * X + B @ X
    return X


def muon_step(W: np.ndarray, M: np.ndarray, G: np.ndarray, beta1: float, lr: float,
              weight_decay: float, eps: float, coeffs, diagnostics: bool = False):
    """One Muon step on one m x n matrix (Algorithm 1).  Returns (W, M) and,
    with ``diagnostics``, a dict holding the orthogonalised direction O and
    Delta W."""
    W = np.asarray(W, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    M = momentum_ema(np.asarray(M, dtype=np.float64), G, beta1)
    O = newton_schulz(M, coeffs, eps)
    dW = O * np.sqrt(max(W.shape))
    W = (1.0 - lr * weight_decay) * W - lr * dW
    if diagnostics:
        return W, M, {"O": O, "dW": dW}
    return W, M
