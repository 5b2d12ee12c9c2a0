"""End-to-end parity of soap_step / soap_step_batched with the fp64 oracle.

Open loop: the GPU state and the oracle state evolve independently from the
same fp32 inputs; every state tensor is compared each step with the relative
Frobenius metric at tolerance 1e-4 (the eigenbases also column by column for
sign)."""
import numpy as np
import pytest

from tests.gpu_helpers import (dev, host, rel, column_signs_agree, log, adam_fp32_bound,
                                update_from_weights)

pytestmark = pytest.mark.gpu

TOL = 1e-4
HP = dict(beta1=0.95, beta2=0.95, eps=1e-8, lr=1e-3, weight_decay=0.1)


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_20548_amd as soap
    soap.lib()


def _compare(st, gs, tag):
    errs = {
        "L": rel(host(gs.L), st.L), "R": rel(host(gs.R), st.R),
        "Q_L": rel(host(gs.Q_L), st.QL), "Q_R": rel(host(gs.Q_R), st.QR),
        "M": rel(host(gs.M), st.M), "V": rel(host(gs.V), st.V),
    }
    for k, v in errs.items():
        assert v <= TOL, (tag, k, v)
    assert column_signs_agree(host(gs.Q_L), st.QL) and column_signs_agree(host(gs.Q_R), st.QR)
    return errs


def _run_open_loop(m, n, grads, W0, hp=HP, flags=0, bias_correction=True):
    """Open loop over the given gradients.  Every step:
      * L, R, Q_L, Q_R, M, V: relative Frobenius error <= TOL;
      * the update N (recovered from the GPU weights): every entry within
        1e-4 |N| plus 64x the first-order fp32 error of the eigenbasis quotient,
        and relative Frobenius error <= TOL over the well-determined entries
        (those whose first-order fp32 error is below 1% of |N|);
      * W: relative Frobenius error <= TOL against the oracle's weights re-based
        on the GPU's N at the entries that are not well determined."""
    import paper_2607_20548_amd as soap
    import oracle
    gs = soap.SoapState(m, n)
    W = dev(W0)
    st = oracle.init_state(W0.astype(np.float64))
    W_adj = W0.astype(np.float64)
    lr, wd, eps = hp["lr"], hp["weight_decay"], hp["eps"]
    g_scale = 0.0
    for t, G in enumerate(grads, start=1):
        W_prev = host(W)
        gs.step(W, dev(G), t, flags=flags, **hp)
        st, d = oracle.soap_step(st, G.astype(np.float64), t, bias_correction=bias_correction,
                                 diagnostics=True, **hp)
        errs = _compare(st, gs, f"{m}x{n} t={t}")
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
        log(f"{m}x{n} t={t} not_well_determined={int((~well).sum())} " +
            " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
        assert errs["W"] <= TOL, (t, errs["W"])
    return gs, W, st


def test_workload0_ten_steps_open_loop():
    """The 256x512 workload: rank-16 signal + N(0, 1e-3) noise, 10 steps."""
    from synth import gradients as sg
    spec = sg.workload(0).matrices[0]
    grads = list(sg.make_matrix_stream(spec, 0, 10))
    _run_open_loop(256, 512, grads, sg.initial_weight(spec, 0))


@pytest.mark.parametrize("m,n", [(1, 1), (3, 5), (37, 70), (130, 129), (200, 257)])
def test_ragged_shapes(m, n):
    rng = np.random.default_rng([m, n, 21])
    grads = [rng.standard_normal((m, n)).astype(np.float32) for _ in range(3)]
    _run_open_loop(m, n, grads, (0.02 * rng.standard_normal((m, n))).astype(np.float32))


def test_no_bias_correction_flag():
    import paper_2607_20548_amd as soap
    rng = np.random.default_rng(22)
    grads = [rng.standard_normal((40, 24)).astype(np.float32) for _ in range(3)]
    _run_open_loop(40, 24, grads, np.zeros((40, 24), np.float32),
                   flags=soap.SOAP_FLAG_NO_BIAS_CORRECTION, bias_correction=False)


def test_identity_eigenbasis_is_adamw():
    """Gradients with one nonzero per row and column keep L, R diagonal: the
    eigenbases stay exactly I and the step is elementwise AdamW."""
    import paper_2607_20548_amd as soap
    from synth.gradients import permutation_gradient
    m, n = 64, 96
    gs = soap.SoapState(m, n)
    W0 = (0.02 * np.random.default_rng(23).standard_normal((m, n))).astype(np.float32)
    W = dev(W0)
    Wa = W0.astype(np.float32)
    W_prev = W0.astype(np.float32)
    ma = np.zeros((m, n), np.float32)
    va = np.zeros((m, n), np.float32)
    b1, b2, eps, lr, wd = (np.float32(x) for x in (0.95, 0.95, 1e-8, 1e-3, 0.1))
    for t in range(1, 8):
        G = permutation_gradient(m, n, 5, t)
        gs.step(W, dev(G), t, **HP)
        assert np.array_equal(host(gs.Q_L), np.eye(m)) and np.array_equal(host(gs.Q_R), np.eye(n))
        ma = b1 * ma + (np.float32(1) - b1) * G
        va = b2 * va + (np.float32(1) - b2) * G * G
        # bias corrections as the library forms them: from the fp32 betas, in double
        c1 = np.float32(1.0 - float(np.float32(0.95)) ** t)
        c2 = c1
        upd = (ma / c1) / (np.sqrt(va / c2) + eps)
        Wa = (np.float32(1) - lr * wd) * Wa - lr * upd
        Wg = host(W).astype(np.float32)
        # Same arithmetic, different rounding (fused multiply-adds on the GPU,
        # separately rounded numpy): W may differ by a couple of ulp of the
        # operands, plus the update by the EMA rounding drift (about t ulp of
        # M and V; where M cancels, ulps of its terms, which are O(1) in units
        # of the Adam-normalised update).
        bound = (2 * np.spacing(np.abs(W_prev).astype(np.float32))
                 + 2 * np.spacing(np.abs(Wa).astype(np.float32))
                 + float(lr) * 2e-6 * (1.0 + np.abs(upd)))
        err = np.abs(Wg.astype(np.float64) - Wa)
        assert np.all(err <= bound), (t, float(np.max(err / bound)))
        W_prev = Wg


def test_batched_matches_single_and_oracle():
    import paper_2607_20548_amd as soap
    import oracle
    import torch
    B, m, n = 5, 37, 70
    rng = np.random.default_rng(24)
    W0 = (0.02 * rng.standard_normal((B, m, n))).astype(np.float32)
    grads = [rng.standard_normal((B, m, n)).astype(np.float32) for _ in range(3)]
    gb = soap.SoapState(m, n, batch=B)
    Wb = dev(W0)
    singles = [soap.SoapState(m, n) for _ in range(B)]
    Ws = [dev(W0[b]) for b in range(B)]
    sts = [oracle.init_state(W0[b].astype(np.float64)) for b in range(B)]
    for t, G in enumerate(grads, start=1):
        gb.step(Wb, dev(G), t, **HP)
        for b in range(B):
            singles[b].step(Ws[b], dev(G[b]), t, **HP)
            sts[b] = oracle.soap_step(sts[b], G[b].astype(np.float64), t, **HP)
        Wbh = host(Wb)
        for b in range(B):
            assert rel(Wbh[b], host(Ws[b])) <= 1e-6
            assert rel(host(gb.Q_R)[b], host(singles[b].Q_R)) <= 1e-6
            assert rel(Wbh[b], sts[b].W) <= TOL
            assert rel(host(gb.Q_L)[b], sts[b].QL) <= TOL
            assert rel(host(gb.V)[b], sts[b].V) <= TOL


def test_two_runs_are_bitwise_identical():
    import paper_2607_20548_amd as soap
    rng = np.random.default_rng(25)
    m, n = 300, 520
    grads = [rng.standard_normal((m, n)).astype(np.float32) for _ in range(2)]
    outs = []
    for _ in range(2):
        gs = soap.SoapState(m, n)
        W = dev(np.zeros((m, n), np.float32))
        for t, G in enumerate(grads, start=1):
            gs.step(W, dev(G), t, **HP)
        outs.append([host(x) for x in (W, gs.L, gs.R, gs.Q_L, gs.Q_R, gs.M, gs.V)])
    for a, b in zip(*outs):
        assert np.array_equal(a, b)
