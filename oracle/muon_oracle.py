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

Precision.  The paper runs the Newton-Schulz iterations in bfloat16 (its
discussion of orthogonalisation accuracy in the conclusion) and the rest of
the step in fp32.  ``newton_schulz(..., precision="bf16")`` states that
reading: X_0, every A, every B and every X are bfloat16 values, each the
correctly rounded (nearest, ties to even) result of the exact operation on
bfloat16 operands -- the product, the linear combination -- taken in fp64
here.  Hardware that accumulates a product in fp32 before rounding it once
to bfloat16 lands on the same value except where the exact result is within
an fp32 accumulation error of a rounding boundary.
"""
from __future__ import annotations

import numpy as np


def momentum_ema(M: np.ndarray, G: np.ndarray, beta1: float) -> np.ndarray:
    """Algorithm 1, momentum buffer: M <- beta1 M + (1 - beta1) G."""
    return beta1 * M + (1.0 - beta1) * G


BF16_MANT = 8          # significant bits of bfloat16 (7 stored + the implicit one)
BF16_EMIN = -126       # smallest normal exponent (as fp32): 2^-126
BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127


def round_bf16(x) -> np.ndarray:
    """Nearest bfloat16 value of each entry (ties to even), as fp64.

    bfloat16 is fp32's sign and 8-bit exponent with 8 significant bits, so a
    normal value v = f 2^e (0.5 <= |f| < 1) rounds to rint(f 2^8) 2^(e-8);
    below 2^-126 the spacing stays 2^-133 (subnormals); past the largest
    finite value, rounding gives +-inf; NaN stays NaN."""
    x = np.asarray(x, dtype=np.float64)
    f, e = np.frexp(x)
    e = np.maximum(e, BF16_EMIN + 1)          # subnormal range keeps spacing 2^-133
    q = np.ldexp(np.rint(np.ldexp(x, BF16_MANT - e)), e - BF16_MANT)
    # past the largest finite value: ties and beyond go to infinity
    big = np.abs(q) > BF16_MAX
    q = np.where(big, np.copysign(np.inf, x), q)
    return np.where(np.isnan(x), np.nan, q)


def newton_schulz(M: np.ndarray, coeffs, eps: float, precision: str = "fp64") -> np.ndarray:
    """Algorithm 1's orthogonalisation: X_0 = M / max(||M||_F, eps), then one
    polynomial step X <- a X + (b A + c A^2) X with A = X X^T per triple.
    precision "bf16": X_0, A, B and X are rounded to bfloat16 after each
    operation (module docstring)."""
    if precision not in ("fp64", "bf16"):
        raise ValueError(precision)
    r = round_bf16 if precision == "bf16" else (lambda v: v)
    X = r(M / max(np.linalg.norm(M), eps))
    for a, b, c in coeffs:
        A = r(X @ X.T)
        B = r(b * A + c * (A @ A))
        X = r(a * X + B @ X)
    return X


def muon_step(W: np.ndarray, M: np.ndarray, G: np.ndarray, beta1: float, lr: float,
              weight_decay: float, eps: float, coeffs, diagnostics: bool = False,
              precision: str = "fp64"):
    """One Muon step on one m x n matrix (Algorithm 1).  Returns (W, M) and,
    with ``diagnostics``, a dict holding the orthogonalised direction O and
    Delta W.  ``precision`` applies to the Newton-Schulz iterations only."""
    W = np.asarray(W, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    M = momentum_ema(np.asarray(M, dtype=np.float64), G, beta1)
    O = newton_schulz(M, coeffs, eps, precision)
    dW = O * np.sqrt(max(W.shape))
    W = (1.0 - lr * weight_decay) * W - lr * dW
    if diagnostics:
        return W, M, {"O": O, "dW": dW}
    return W, M
