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


TOL = 1e-4
HP = dict(beta1=0.95, beta2=0.95, eps=1e-8, lr=1e-3, weight_decay=0.1)


def compare_state(st, gs, tag, tol=TOL):
    """Every state tensor of the GPU state `gs` against the oracle state `st`."""
    errs = {
        "L": rel(host(gs.L), st.L), "R": rel(host(gs.R), st.R),
        "Q_L": rel(host(gs.Q_L), st.QL), "Q_R": rel(host(gs.Q_R), st.QR),
        "M": rel(host(gs.M), st.M), "V": rel(host(gs.V), st.V),
    }
    for k, v in errs.items():
        assert v <= tol, (tag, k, v)
    assert column_signs_agree(host(gs.Q_L), st.QL) and column_signs_agree(host(gs.Q_R), st.QR)
    return errs


def run_open_loop(m, n, grads, W0, hp=HP, flags=0, bias_correction=True, beta_kron=None,
                  refresh_every=1, stale_refresh=False):
    """Open loop over the given gradients (SOAP, or KL-SOAP when beta_kron is
    given).  Every step:
      * L, R, Q_L, Q_R, M, V: relative Frobenius error <= TOL;
      * the update N (recovered from the GPU weights): every entry within
        1e-4 |N| plus 64x the first-order fp32 error of the eigenbasis quotient,
        and relative Frobenius error <= TOL over the well-determined entries
        (those whose first-order fp32 error is below 1% of |N|);
      * W: relative Frobenius error <= TOL against the oracle's weights re-based
        on the GPU's N at the entries that are not well determined."""
    import paper_2607_20548_amd as soap
    import oracle
    kl = beta_kron is not None
    gs = soap.SoapState(m, n, kl=kl)
    W = dev(W0)
    st = oracle.init_state(W0.astype(np.float64))
    W_adj = W0.astype(np.float64)
    lr, wd, eps = hp["lr"], hp["weight_decay"], hp["eps"]
    g_scale = 0.0
    extra = dict(beta_kron=beta_kron) if kl else {}
    for t, G in enumerate(grads, start=1):
        W_prev = host(W)
        Q_prev = (host(gs.Q_L), host(gs.Q_R))
        gs.step(W, dev(G), t, flags=flags, refresh_every=refresh_every,
                stale_refresh=stale_refresh, **extra, **hp)
        step_fn = oracle.kl_soap_step if kl else oracle.soap_step
        st, d = step_fn(st, G.astype(np.float64), t, bias_correction=bias_correction,
                        diagnostics=True, refresh_every=refresh_every,
                        stale_refresh=stale_refresh, **extra, **hp)
        if t % refresh_every != 0:   # no refresh: the bases are kept bit for bit
            assert np.array_equal(host(gs.Q_L), Q_prev[0]) and np.array_equal(host(gs.Q_R), Q_prev[1])
        errs = compare_state(st, gs, f"{m}x{n} t={t}")
        g_scale = max(g_scale, np.linalg.norm(G.astype(np.float64), 2))
        Wg = host(W)
        N_gpu = update_from_weights(W_prev, Wg, host(gs.Q_L), host(gs.Q_R), lr, wd)
        _, c2 = oracle.bias_corrections(hp["beta1"], hp["beta2"], t, bias_correction)
        N_ora = d["N"]
        bound = adam_fp32_bound(N_ora, st.V / c2, g_scale, eps)
        dN = np.abs(N_gpu - N_ora)
        assert np.all(dN <= 1e-4 * np.abs(N_ora) + bound + 1e-6), (t, float(np.max(dN - bound)))
        # well determined: the expected fp32 error (factor 1) is below 1% of |N|
        well = adam_fp32_bound(N_ora, st.V / c2, g_scale, eps, factor=1.0) <= 1e-2 * np.abs(N_ora)
        errs["N_well"] = rel(N_gpu[well], N_ora[well]) if well.any() else 0.0
        assert errs["N_well"] <= TOL, (t, errs["N_well"])
        N_adj = np.where(well, N_ora, N_gpu)
        W_adj = (1.0 - lr * wd) * W_adj - lr * (st.QL @ N_adj @ st.QR.T)
        errs["W"] = rel(Wg, W_adj)
        errs["W_plain"] = rel(Wg, st.W)
        log(f"{'KL ' if kl else ''}{m}x{n} t={t} not_well_determined={int((~well).sum())} " +
            " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
        assert errs["W"] <= TOL, (t, errs["W"])
    return gs, W, st


def check_factor_ema_sampled(pre, post, G, rng, beta2=HP["beta2"], nsamp=48):
    """L, R of one plain SOAP step, entry by entry from their definition."""
    m, n = G.shape
    for F, X, d in (("L", G, m), ("R", G.T, n)):
        ii = rng.integers(0, d, nsamp)
        jj = rng.integers(0, d, nsamp)
        want = beta2 * pre[F][ii, jj] + (1 - beta2) * np.einsum("ij,ij->i", X[ii], X[jj])
        assert rel(post[F][ii, jj], want) <= TOL, F
        assert np.array_equal(post[F][ii, jj], post[F][jj, ii])


def check_refresh_adam_sampled(pre, post, G, t, rng, hp=HP, nsamp=48, ncols=16):
    """Everything of one step after the factors (fp64, sampled), given the GPU
    state before (`pre`) and after (`post`) it:
      * M entry by entry;
      * the refreshed eigenbases by their defining properties -- Q^T Q = I and
        Q^T (F Q_prev) upper triangular with a positive diagonal -- on sampled
        columns (those properties fix the Q factor uniquely);
      * V and the update N at sampled eigenbasis entries, from G' = Q_L^T G Q_R
        and M' = Q_L^T M Q_R formed with matrix-vector products;
      * W through N recovered from consecutive weights."""
    b1, b2, eps, lr, wd = (hp[k] for k in ("beta1", "beta2", "eps", "lr", "weight_decay"))
    m, n = G.shape
    c1, c2 = 1 - b1 ** t, 1 - b2 ** t
    ii, jj = rng.integers(0, m, nsamp), rng.integers(0, n, nsamp)
    assert rel(post["M"][ii, jj], b1 * pre["M"][ii, jj] + (1 - b1) * G[ii, jj]) <= TOL
    for F, Qp, Qn, d in (("L", pre["QL"], post["QL"], m), ("R", pre["QR"], post["QR"], n)):
        cols = np.unique(np.concatenate([rng.integers(0, d, ncols), [0, d - 1]]))
        A_cols = post[F] @ Qp[:, cols]                      # columns of F_t Q_prev
        QtA = Qn.T @ A_cols                                 # d x len(cols)
        colnorm = np.linalg.norm(A_cols, axis=0)
        for k, j in enumerate(cols):
            below = QtA[j + 1:, k]
            assert np.linalg.norm(below) <= TOL * colnorm[k], (F, j)
            assert QtA[j, k] > 0, (F, j)
        ortho = Qn.T @ Qn[:, cols]
        ortho[cols, np.arange(len(cols))] -= 1.0
        assert np.linalg.norm(ortho) / np.sqrt(len(cols)) <= TOL, F
    QL, QR = post["QL"], post["QR"]
    kk, ll = rng.integers(0, m, nsamp), rng.integers(0, n, nsamp)
    Mn = post["M"]
    GQ = G @ QR[:, ll]                 # m x nsamp
    MQ = Mn @ QR[:, ll]
    Gp = np.einsum("ik,ik->k", QL[:, kk], GQ)
    Mp = np.einsum("ik,ik->k", QL[:, kk], MQ)
    V_want = b2 * pre["V"][kk, ll] + (1 - b2) * Gp * Gp
    assert rel(post["V"][kk, ll], V_want) <= TOL
    N_want = (Mp / c1) / (np.sqrt(post["V"][kk, ll] / c2) + eps)
    beta_w = float(np.float32(1.0) - np.float32(lr) * np.float32(wd))
    dW = (beta_w * pre["W"] - post["W"]) / float(np.float32(lr))
    N_got = np.einsum("ik,ik->k", QL[:, kk], dW @ QR[:, ll])
    g_scale = np.linalg.norm(G, 2)
    bound = adam_fp32_bound(N_want, post["V"][kk, ll] / c2, g_scale, eps)
    assert np.all(np.abs(N_got - N_want) <= 1e-4 * np.abs(N_want) + bound + 1e-5)
    well = adam_fp32_bound(N_want, post["V"][kk, ll] / c2, g_scale, eps, factor=1.0) <= 1e-2 * np.abs(N_want)
    if well.sum() >= nsamp // 2:
        assert rel(N_got[well], N_want[well]) <= TOL
    assert np.all(np.isfinite(dW))
    return {"N_rel_well": rel(N_got[well], N_want[well]) if well.any() else 0.0}
