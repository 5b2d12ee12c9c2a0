"""End-to-end parity of soap_step / soap_step_batched with the fp64 oracle.

Open loop: the GPU state and the oracle state evolve independently from the
same fp32 inputs; every state tensor is compared each step with the relative
Frobenius metric at tolerance 1e-4 (the eigenbases also column by column for
sign)."""
import numpy as np
import pytest

from tests.gpu_helpers import dev, host, rel, run_open_loop, recipe_grads

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


def _run_open_loop(m, n, grads, W0, hp=HP, flags=0, bias_correction=True, strict=True):
    return run_open_loop(m, n, grads, W0, hp=hp, flags=flags, bias_correction=bias_correction,
                         strict=strict)


def test_workload0_ten_steps_open_loop():
    """The 256x512 workload: rank-16 signal + N(0, 1e-3) noise, 10 steps."""
    from synth import gradients as sg
    spec = sg.workload(0).matrices[0]
    grads = list(sg.make_matrix_stream(spec, 0, 10))
    _run_open_loop(256, 512, grads, sg.initial_weight(spec, 0))


@pytest.mark.parametrize("m,n", [(1, 1), (3, 5), (37, 70), (130, 129), (200, 257), (300, 600),
                                 (600, 300), (1100, 200)])
def test_ragged_shapes(m, n):
    """Shapes that are not multiples of the tiles, with gradients of the
    workloads' recipe (low-rank signal + 10% noise)."""
    rng = np.random.default_rng([m, n, 21])
    _run_open_loop(m, n, recipe_grads(m, n, 3, 21),
                   (0.02 * rng.standard_normal((m, n))).astype(np.float32))


@pytest.mark.parametrize("m,n", [(256, 1024), (200, 1100), (128, 2100), (300, 2300)])
def test_wide_shapes_several_reflector_groups(m, n):
    """n >= 2m at orders where the R-side QR forms several quads of blocks
    (rank-512 Q formation, pair updates of the far columns, a ragged last
    block), with the L side's QR started from inside the R side's loop."""
    rng = np.random.default_rng([m, n, 23])
    _run_open_loop(m, n, recipe_grads(m, n, 3, 23),
                   (0.02 * rng.standard_normal((m, n))).astype(np.float32))


@pytest.mark.parametrize("m,n", [(200, 200), (520, 520), (1100, 1100), (4104, 4104)])
def test_square_shapes(m, n):
    """Square weights: both factors' QRs run as one call over two matrices
    when A_L, A_R (and T_G, T_M) lie back to back in the workspace (m^2 a
    multiple of 64: 200, 520 with Q formed forwards; 4104, past the forward
    threshold, with Q formed backwards in the call's buffer); 1100 takes two
    separate QRs."""
    rng = np.random.default_rng([m, n, 26])
    _run_open_loop(m, n, recipe_grads(m, n, 3, 26),
                   (0.02 * rng.standard_normal((m, n))).astype(np.float32))


@pytest.mark.parametrize("m,n", [(37, 70), (200, 257)])
def test_ragged_shapes_gaussian_stress(m, n):
    """Full-rank Gaussian gradients: ill-conditioned factors, checked with the
    conditioning-aware fp32 intervals (UpdateCheck, strict=False)."""
    rng = np.random.default_rng([m, n, 21])
    grads = [rng.standard_normal((m, n)).astype(np.float32) for _ in range(3)]
    _run_open_loop(m, n, grads, (0.02 * rng.standard_normal((m, n))).astype(np.float32),
                   strict=False)


def test_no_bias_correction_flag():
    import paper_2607_20548_amd as soap
    _run_open_loop(40, 24, recipe_grads(40, 24, 3, 22), np.zeros((40, 24), np.float32),
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


def test_batched_square_matches_single_and_oracle():
    """Three square matrices through soap_step_batched: one QR call over the
    six factors; every entry's bases and weight follow the oracle and equal
    the single-matrix steps' (one QR call over two factors each)."""
    import paper_2607_20548_amd as soap
    import oracle
    B, m = 3, 200
    rng = np.random.default_rng(27)
    W0 = (0.02 * rng.standard_normal((B, m, m))).astype(np.float32)
    grads = recipe_grads(m, m, 3, 27, batch=B)
    gb = soap.SoapState(m, m, batch=B)
    Wb = dev(W0)
    singles = [soap.SoapState(m, m) for _ in range(B)]
    Ws = [dev(W0[b]) for b in range(B)]
    sts = [oracle.init_state(W0[b].astype(np.float64)) for b in range(B)]
    for t, G in enumerate(grads, start=1):
        gb.step(Wb, dev(G), t, **HP)
        assert gb.status() == (soap.SOAP_OK, 0)
        for b in range(B):
            singles[b].step(Ws[b], dev(G[b]), t, **HP)
            sts[b] = oracle.soap_step(sts[b], G[b].astype(np.float64), t, **HP)
        Wbh, QLb, QRb = host(Wb), host(gb.Q_L), host(gb.Q_R)
        for b in range(B):
            assert rel(Wbh[b], host(Ws[b])) <= 1e-6
            assert rel(QLb[b], host(singles[b].Q_L)) <= 1e-6
            assert rel(QRb[b], host(singles[b].Q_R)) <= 1e-6
            assert rel(Wbh[b], sts[b].W) <= TOL
            assert rel(QLb[b], sts[b].QL) <= TOL and rel(QRb[b], sts[b].QR) <= TOL
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


@pytest.mark.parametrize("F,stale", [(3, False), (1, True), (2, True)])
def test_refresh_period_and_stale_refresh(F, stale):
    """Algorithm 2's refresh every F steps (bases kept bit for bit in between)
    and the stale-refresh ablation, against the oracle."""
    rng = np.random.default_rng([F, int(stale), 26])
    m, n = 96, 160
    run_open_loop(m, n, recipe_grads(m, n, 6, 26 + F + 10 * int(stale)),
                  (0.02 * rng.standard_normal((m, n))).astype(np.float32),
                  refresh_every=F, stale_refresh=stale)
