"""The QR's give-up path and checkpoint/resume.

Give-up: the resident block factorizations wait for each other with bounded
waits; when one gives up, the library keeps that side's eigenbasis, runs the
rest of the step with it (the step then equals one whose refresh of that side
was skipped) and reports it in the workspace's status word.  The tests force
the path from the host (soap_test_force_qr_give_up raises the abort flags
before the block kernels start, so every bounded wait ends at once and every
kernel exits normally) and compare with the oracle.

Checkpoint/resume: the library keeps no optimizer state between calls, so
copying the state tensors out after k steps and into freshly allocated ones
(new workspace) must continue the run bit for bit.
"""
import numpy as np
import pytest

from tests.gpu_helpers import dev, host, log, compare_state, UpdateCheck, HP, rel, recipe_grads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_20548_amd as soap
    soap.lib()
    yield
    soap.soap_test_force_qr_give_up(0)


def _grads(m, n, steps, seed, batch=None):
    return recipe_grads(m, n, steps, 31 + seed, batch=batch)


def _oracle_one_side_kept(st, G, t, keep_left, hp=HP):
    """One SOAP step written out with the oracle's functions, refreshing only
    one eigenbasis (the other is kept): the expected result of a step whose
    other QR gave up."""
    import oracle
    b1, b2, eps, lr, wd = (hp[k] for k in ("beta1", "beta2", "eps", "lr", "weight_decay"))
    s = st.copy()
    s.L = oracle.factor_ema(s.L, G, b2)
    s.R = oracle.factor_ema(s.R, G.T, b2)
    if keep_left:
        s.QR = oracle.refresh_qr(s.R @ s.QR)
    else:
        s.QL = oracle.refresh_qr(s.L @ s.QL)
    s.M = oracle.momentum_ema(s.M, G, b1)
    Gp = oracle.rotate_in(s.QL, G, s.QR)
    Mp = oracle.rotate_in(s.QL, s.M, s.QR)
    c1, c2 = oracle.bias_corrections(b1, b2, t, True)
    s.V, N = oracle.adam_eigenbasis(Gp, Mp, s.V, b2, eps, c1, c2)
    s.W = oracle.weight_update(s.W, oracle.rotate_out(s.QL, N, s.QR), lr, wd)
    return s, N


@pytest.mark.parametrize("kl", [False, True])
def test_forced_give_up_of_both_qrs_keeps_the_bases(kl):
    """Steps 1, 2 and 4 refresh; at step 3 both QRs are made to give up: the
    status word reports both sides, Q_L and Q_R are bit for bit those of step
    2, and the step equals the oracle's step with the refresh skipped."""
    import paper_2607_20548_amd as soap
    import oracle
    m, n = 300, 600
    grads = _grads(m, n, 4, int(kl))
    W0 = (0.02 * np.random.default_rng(5).standard_normal((m, n))).astype(np.float32)
    gs = soap.SoapState(m, n, kl=kl)
    W = dev(W0)
    st = oracle.init_state(W0.astype(np.float64))
    chk = UpdateCheck(HP)
    extra = dict(beta_kron=0.95) if kl else {}
    step_fn = oracle.kl_soap_step if kl else oracle.soap_step
    for t, G in enumerate(grads, start=1):
        forced = t == 3
        Q_prev = (host(gs.Q_L), host(gs.Q_R))
        W_prev = host(W)
        soap.soap_test_force_qr_give_up(soap.SOAP_STATUS_QR_L | soap.SOAP_STATUS_QR_R if forced else 0)
        gs.step(W, dev(G), t, **extra, **HP)
        soap.soap_test_force_qr_give_up(0)
        code, word = gs.status()
        if forced:
            assert (code, word) == (soap.SOAP_ERR_QR_GAVE_UP, soap.SOAP_STATUS_QR_L | soap.SOAP_STATUS_QR_R)
            assert "both factors" in soap.soap_last_error()
            assert np.array_equal(host(gs.Q_L), Q_prev[0]) and np.array_equal(host(gs.Q_R), Q_prev[1])
        else:
            assert (code, word) == (soap.SOAP_OK, 0)
        # the oracle skips the refresh at t = 3 (t mod 2 != 0)
        st, d = step_fn(st, G.astype(np.float64), t, diagnostics=True,
                        refresh_every=2 if forced else 1, **extra, **HP)
        errs = compare_state(st, gs, f"t={t}")
        errs.update(chk(t, G, host(gs.update()), d["N"], st.V, host(W), st.W, f"t={t}",
                        chain=(W_prev, host(gs.Q_L), host(gs.Q_R))))
        log(f"{'KL ' if kl else ''}give-up t={t} forced={forced} " +
            " ".join(f"{k}={v:.2e}" if isinstance(v, float) else f"{k}={v}" for k, v in errs.items()))


@pytest.mark.parametrize("m,n", [(300, 600), (320, 320), (1100, 300)])
@pytest.mark.parametrize("side", ["L", "R"])
def test_forced_give_up_of_one_qr_keeps_only_that_basis(side, m, n):
    """One side's QR gives up (320 x 320: both QRs are one call over two
    matrices, and the give-up of one half keeps only that half's basis;
    1100 x 300: the larger factor on the L side)."""
    import paper_2607_20548_amd as soap
    import oracle
    grads = _grads(m, n, 3, 7)
    W0 = (0.02 * np.random.default_rng(6).standard_normal((m, n))).astype(np.float32)
    gs = soap.SoapState(m, n)
    W = dev(W0)
    st = oracle.init_state(W0.astype(np.float64))
    chk = UpdateCheck(HP)
    bit = soap.SOAP_STATUS_QR_L if side == "L" else soap.SOAP_STATUS_QR_R
    for t, G in enumerate(grads, start=1):
        forced = t == 3
        Q_prev = (host(gs.Q_L), host(gs.Q_R))
        W_prev = host(W)
        soap.soap_test_force_qr_give_up(bit if forced else 0)
        gs.step(W, dev(G), t, **HP)
        soap.soap_test_force_qr_give_up(0)
        assert gs.status() == ((soap.SOAP_ERR_QR_GAVE_UP, bit) if forced else (soap.SOAP_OK, 0))
        if forced:
            kept = Q_prev[0] if side == "L" else Q_prev[1]
            assert np.array_equal(host(gs.Q_L if side == "L" else gs.Q_R), kept)
            st, N = _oracle_one_side_kept(st, G.astype(np.float64), t, keep_left=side == "L")
        else:
            st, d = oracle.soap_step(st, G.astype(np.float64), t, diagnostics=True, **HP)
            N = d["N"]
        errs = compare_state(st, gs, f"{side} t={t}")
        errs.update(chk(t, G, host(gs.update()), N, st.V, host(W), st.W, f"{side} t={t}",
                        chain=(W_prev, host(gs.Q_L), host(gs.Q_R))))
        log(f"give-up {side} t={t} forced={forced} " + " ".join(
            f"{k}={v:.2e}" if isinstance(v, float) else f"{k}={v}" for k, v in errs.items()))


@pytest.mark.parametrize("m,n", [(256, 1024), (200, 1100)])
def test_forced_give_up_of_r_at_wider_orders(m, n):
    """n >= 2m with several reflector groups in the R-side QR: when that QR
    gives up, the step rotates by the kept Q_R and equals the oracle's step
    with the refresh of Q_R skipped."""
    import paper_2607_20548_amd as soap
    import oracle
    grads = _grads(m, n, 3, 12)
    W0 = (0.02 * np.random.default_rng(13).standard_normal((m, n))).astype(np.float32)
    gs = soap.SoapState(m, n)
    W = dev(W0)
    st = oracle.init_state(W0.astype(np.float64))
    chk = UpdateCheck(HP)
    bit = soap.SOAP_STATUS_QR_R
    for t, G in enumerate(grads, start=1):
        forced = t == 3
        QR_prev = host(gs.Q_R)
        W_prev = host(W)
        soap.soap_test_force_qr_give_up(bit if forced else 0)
        gs.step(W, dev(G), t, **HP)
        soap.soap_test_force_qr_give_up(0)
        assert gs.status() == ((soap.SOAP_ERR_QR_GAVE_UP, bit) if forced else (soap.SOAP_OK, 0))
        if forced:
            assert np.array_equal(host(gs.Q_R), QR_prev)
            st, N = _oracle_one_side_kept(st, G.astype(np.float64), t, keep_left=False)
        else:
            st, d = oracle.soap_step(st, G.astype(np.float64), t, diagnostics=True, **HP)
            N = d["N"]
        errs = compare_state(st, gs, f"{m}x{n} t={t}")
        errs.update(chk(t, G, host(gs.update()), N, st.V, host(W), st.W, f"{m}x{n} t={t}",
                        chain=(W_prev, host(gs.Q_L), host(gs.Q_R))))
        log(f"give-up R {m}x{n} t={t} forced={forced} " + " ".join(
            f"{k}={v:.2e}" if isinstance(v, float) else f"{k}={v}" for k, v in errs.items()))


def test_forced_give_up_batched_keeps_every_entry():
    """Three matrices through soap_step_batched: a forced give-up of the n x n
    QR keeps Q_R of every entry; the next step refreshes normally."""
    import paper_2607_20548_amd as soap
    import oracle
    B, m, n = 3, 300, 600
    grads = _grads(m, n, 3, 8, batch=B)
    W0 = (0.02 * np.random.default_rng(7).standard_normal((B, m, n))).astype(np.float32)
    gs = soap.SoapState(m, n, batch=B)
    W = dev(W0)
    sts = [oracle.init_state(W0[b].astype(np.float64)) for b in range(B)]
    for t, G in enumerate(grads, start=1):
        forced = t == 2
        QR_prev = host(gs.Q_R)
        soap.soap_test_force_qr_give_up(soap.SOAP_STATUS_QR_R if forced else 0)
        gs.step(W, dev(G), t, **HP)
        soap.soap_test_force_qr_give_up(0)
        assert gs.status() == ((soap.SOAP_ERR_QR_GAVE_UP, soap.SOAP_STATUS_QR_R) if forced
                               else (soap.SOAP_OK, 0))
        if forced:
            assert np.array_equal(host(gs.Q_R), QR_prev)
        for b in range(B):
            if forced:
                sts[b], _ = _oracle_one_side_kept(sts[b], G[b].astype(np.float64), t, keep_left=False)
            else:
                sts[b] = oracle.soap_step(sts[b], G[b].astype(np.float64), t, **HP)
            compare_state(sts[b], gs, f"entry {b} t={t}", b=b)
            assert rel(host(W)[b], sts[b].W) <= 1e-4


@pytest.mark.parametrize("side", ["L", "R"])
def test_forced_give_up_batched_square_keeps_that_side(side):
    """Three 320 x 320 matrices: both sides' QRs are one call over six
    matrices; a forced give-up of one side keeps that side's basis in every
    entry and refreshes the other side's."""
    import paper_2607_20548_amd as soap
    B, m = 3, 320
    grads = _grads(m, m, 2, 9, batch=B)
    W0 = (0.02 * np.random.default_rng(8).standard_normal((B, m, m))).astype(np.float32)
    gs = soap.SoapState(m, m, batch=B)
    W = dev(W0)
    import oracle
    sts = [oracle.init_state(W0[b].astype(np.float64)) for b in range(B)]
    bit = soap.SOAP_STATUS_QR_L if side == "L" else soap.SOAP_STATUS_QR_R
    for t, G in enumerate(grads, start=1):
        forced = t == 2
        Q_prev = (host(gs.Q_L), host(gs.Q_R))
        soap.soap_test_force_qr_give_up(bit if forced else 0)
        gs.step(W, dev(G), t, **HP)
        soap.soap_test_force_qr_give_up(0)
        assert gs.status() == ((soap.SOAP_ERR_QR_GAVE_UP, bit) if forced else (soap.SOAP_OK, 0))
        if forced:
            assert np.array_equal(host(gs.Q_L if side == "L" else gs.Q_R),
                                  Q_prev[0] if side == "L" else Q_prev[1])
        for b in range(B):
            if forced:
                sts[b], _ = _oracle_one_side_kept(sts[b], G[b].astype(np.float64), t,
                                                  keep_left=side == "L")
            else:
                sts[b] = oracle.soap_step(sts[b], G[b].astype(np.float64), t, **HP)
            compare_state(sts[b], gs, f"square {side} entry {b} t={t}", b=b)
            assert rel(host(W)[b], sts[b].W) <= 1e-4


def test_forced_give_up_of_the_qr_stage():
    """soap_qr_f32: a forced give-up leaves Q as it was and is reported; the
    next call factors normally and reports nothing."""
    import torch
    import paper_2607_20548_amd as soap
    import oracle
    n = 700
    A = np.random.default_rng(9).standard_normal((n, n)).astype(np.float32) + 3 * np.eye(n, dtype=np.float32)
    nb = soap.soap_qr_workspace_bytes(n)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    Ad = dev(A)
    marker = np.full((n, n), 0.25, np.float32)
    Q = dev(marker)
    soap.soap_test_force_qr_give_up(soap.SOAP_STATUS_QR_L)
    soap.soap_qr_f32(n, Ad, Q, None, ws, nb)
    soap.soap_test_force_qr_give_up(0)
    assert soap.soap_workspace_status(ws) == (soap.SOAP_ERR_QR_GAVE_UP, soap.SOAP_STATUS_QR_L)
    assert np.array_equal(host(Q), marker)
    soap.soap_qr_f32(n, Ad, Q, None, ws, nb)
    assert soap.soap_workspace_status(ws) == (soap.SOAP_OK, 0)
    Qo = oracle.householder_qr(A.astype(np.float64))
    assert rel(host(Q), Qo) <= 1e-4


@pytest.mark.parametrize("kl,batch", [(False, 1), (True, 1), (False, 3)])
def test_checkpoint_resume_is_bitwise(kl, batch):
    """k steps, the state copied to the host and into newly allocated tensors
    (new workspace), then the remaining steps: bit for bit the uninterrupted
    run."""
    import torch
    import paper_2607_20548_amd as soap
    m, n, steps, k = 200, 330, 6, 3
    grads = _grads(m, n, steps, 10 + int(kl), batch=None if batch == 1 else batch)
    shp = (m, n) if batch == 1 else (batch, m, n)
    W0 = (0.02 * np.random.default_rng(11).standard_normal(shp)).astype(np.float32)
    extra = dict(beta_kron=0.95) if kl else {}
    names = ("L", "R", "Q_L", "Q_R", "M", "V")

    def run(stop=None):
        gs = soap.SoapState(m, n, batch=batch, kl=kl)
        W = dev(W0)
        for t in range(1, steps + 1):
            gs.step(W, dev(grads[t - 1]), t, **extra, **HP)
            if t == stop:
                torch.cuda.synchronize()
                saved = {k2: getattr(gs, k2).cpu().numpy().copy() for k2 in names}
                saved["W"] = W.cpu().numpy().copy()
                del gs, W
                torch.cuda.empty_cache()
                gs = soap.SoapState(m, n, batch=batch, kl=kl)   # fresh identity state, new workspace
                for k2 in names:
                    getattr(gs, k2).copy_(torch.from_numpy(saved[k2]))
                W = torch.from_numpy(saved["W"]).cuda()
        torch.cuda.synchronize()
        return {k2: getattr(gs, k2).cpu().numpy() for k2 in names} | {"W": W.cpu().numpy()}

    a, b = run(), run(stop=k)
    for key in a:
        assert np.array_equal(a[key], b[key]), key
