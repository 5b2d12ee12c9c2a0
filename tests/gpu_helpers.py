"""Helpers shared by the GPU tests: host<->device copies and error metrics."""
import numpy as np


def dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().astype(np.float64)


def rel(x, y):
    """Relative Frobenius error ||x - y||_F / ||y||_F (y is the reference)."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    d = np.linalg.norm(x - y)
    ny = np.linalg.norm(y)
    return d / ny if ny > 0 else d


def column_signs_agree(Qg, Qo):
    """Q factors compared as subspaces: every column of the GPU Q must point the
    same way as the oracle's (no flipped columns)."""
    d = np.einsum("ij,ij->j", np.asarray(Qg, np.float64), np.asarray(Qo, np.float64))
    return bool(np.all(d > 0))


def log(msg):
    print(msg, flush=True)


U32 = 2.0 ** -24   # unit roundoff of fp32


def adam_fp32_bound(N_ora, Vhat_ora, g_scale, eps, factor=64.0):
    """First-order fp32 error bound of N = Mhat / (sqrt(Vhat) + eps) per entry.

    Mhat = M'/c1 and Vhat = V/c2 come from fp32 rotations by orthogonal Q_L,
    Q_R, so each carries an absolute error of order u * ||G||_2 (g_scale: the
    largest spectral norm of the gradients so far).  Propagated through the
    quotient this gives u * g_scale * (1 + |N|) / (sqrt(Vhat) + eps); the
    factor covers the accumulated rounding of the GEMMs and the QR.  Where this
    bound is O(|N|) the entry is a sign-like decision that fp32 -- the paper's
    precision for the optimizer step -- cannot take reliably (at t = 1, N is
    sign(G') smoothed by eps)."""
    return factor * U32 * g_scale * (1.0 + np.abs(N_ora)) / (np.sqrt(np.maximum(Vhat_ora, 0.0)) + eps)


def update_from_weights(W_prev, W_new, QL, QR, lr, wd):
    """N recovered from two consecutive fp32 weights: the step wrote
    W_new = (1 - lr wd) W_prev - lr Q_L N Q_R^T."""
    beta_w = float(np.float32(1.0) - np.float32(lr) * np.float32(wd))
    dW = (beta_w * W_prev - W_new) / float(np.float32(lr))
    return QL.T @ dW @ QR
