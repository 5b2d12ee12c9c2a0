"""Parity of the KL-SOAP path (soap_kl_factors_f32, soap_kl_step,
soap_kl_step_batched) with the fp64 oracle.

* The KL-Shampoo accumulation alone: L, R and the eigenvalue estimates
  against oracle.kl_factors on random symmetric positive definite factors and
  random orthogonal bases, over shapes that span several 64- and 128-wide
  tiles with ragged tails.
* The whole step open-loop against oracle.kl_soap_step (every state tensor
  each step, relative Frobenius error <= 1e-4), ragged shapes, the batched
  entry point, and the AdamW reduction.
* At the bench shape 4096 x 14336, one closed-loop step checked on sampled
  entries from the GPU's own pre-step state (the estimates in fp64 in full,
  the factors entry by entry, the rest as for plain SOAP).
"""
import numpy as np
import pytest

from tests.gpu_helpers import (dev, host, rel, log, run_open_loop, recipe_grads,
                                check_refresh_adam_sampled,
                               HP, TOL)

pytestmark = pytest.mark.gpu

BK = 0.95


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_20548_amd as soap
    soap.lib()


def _orthogonal(rng, n):
    Q, R = np.linalg.qr(rng.standard_normal((n, n)))
    return Q * np.where(np.diag(R) < 0, -1.0, 1.0)


def _spd(rng, n):
    X = rng.standard_normal((n, n + 3))
    return X @ X.T / (n + 3) + 0.1 * np.eye(n)


@pytest.mark.parametrize("m,n", [(1, 1), (3, 5), (64, 64), (65, 130), (130, 70), (129, 257),
                                 (300, 128), (256, 512)])
@pytest.mark.parametrize("eps", [1e-8, 0.05])
def test_kl_factors_match_oracle(m, n, eps):
    import torch
    import paper_2607_20548_amd as soap
    import oracle
    rng = np.random.default_rng([m, n, 31])
    L0, R0 = _spd(rng, m).astype(np.float32), _spd(rng, n).astype(np.float32)
    QL, QR = _orthogonal(rng, m).astype(np.float32), _orthogonal(rng, n).astype(np.float32)
    G = rng.standard_normal((m, n)).astype(np.float32)
    L, R = dev(L0), dev(R0)
    lamL = torch.empty(m, dtype=torch.float32, device="cuda")
    lamR = torch.empty(n, dtype=torch.float32, device="cuda")
    wsb = soap.soap_kl_factors_workspace_bytes(m, n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    log(f"kl_factors {m}x{n} eps={eps}")
    soap.soap_kl_factors_f32(m, n, dev(G), L, R, dev(QL), dev(QR), BK, eps, lamL, lamR, ws, wsb)
    L1, R1, lam_L, lam_R = oracle.kl_factors(L0.astype(np.float64), R0.astype(np.float64),
                                             QL.astype(np.float64), QR.astype(np.float64),
                                             G.astype(np.float64), BK, eps)
    errs = dict(L=rel(host(L), L1), R=rel(host(R), R1), lam_L=rel(host(lamL), lam_L),
                lam_R=rel(host(lamR), lam_R))
    log("  " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for k, v in errs.items():
        assert v <= TOL, (k, v)
    Lh, Rh = host(L), host(R)
    assert np.array_equal(Lh, Lh.T) and np.array_equal(Rh, Rh.T)


def test_kl_workload0_ten_steps_open_loop():
    """The 256 x 512 workload (rank-16 signal + N(0, 1e-3) noise), 10 KL steps."""
    from synth import gradients as sg
    spec = sg.workload(0).matrices[0]
    grads = list(sg.make_matrix_stream(spec, 0, 10))
    run_open_loop(256, 512, grads, sg.initial_weight(spec, 0), beta_kron=BK)


@pytest.mark.parametrize("m,n", [(1, 1), (3, 5), (37, 70), (130, 129), (200, 257), (257, 200)])
def test_kl_ragged_shapes(m, n):
    rng = np.random.default_rng([m, n, 33])
    run_open_loop(m, n, recipe_grads(m, n, 3, 33),
                  (0.02 * rng.standard_normal((m, n))).astype(np.float32), beta_kron=BK)


@pytest.mark.parametrize("m,n", [(37, 70), (200, 257)])
def test_kl_ragged_shapes_gaussian_stress(m, n):
    """Full-rank Gaussian gradients, conditioning-aware fp32 intervals."""
    rng = np.random.default_rng([m, n, 33])
    grads = [rng.standard_normal((m, n)).astype(np.float32) for _ in range(3)]
    run_open_loop(m, n, grads, (0.02 * rng.standard_normal((m, n))).astype(np.float32),
                  beta_kron=BK, strict=False)


@pytest.mark.parametrize("m,n", [(1, 3), (3, 1), (37, 80), (130, 300), (300, 130)])
def test_kl_low_rank_power_update_shapes(m, n):
    """Shapes where one side is more than twice the other: that side's power
    product is formed from Q^T F_old plus the rank-(other side) update."""
    rng = np.random.default_rng([m, n, 38])
    run_open_loop(m, n, recipe_grads(m, n, 3, 38),
                  (0.02 * rng.standard_normal((m, n))).astype(np.float32), beta_kron=BK)


@pytest.mark.parametrize("m,n", [(2400, 100), (100, 2400)])
def test_kl_capped_side_products(m, n):
    """Large enough that the factor updates beside the other side's QR run as
    capped (tile-looping) launches, with the low-rank power update."""
    rng = np.random.default_rng([m, n, 39])
    grads = [(np.float32(1e-2) * G) for G in recipe_grads(m, n, 2, 39)]
    run_open_loop(m, n, grads, (0.02 * rng.standard_normal((m, n))).astype(np.float32),
                  beta_kron=BK)


def test_kl_beta_kron_half_no_bias_correction():
    import paper_2607_20548_amd as soap
    run_open_loop(48, 80, recipe_grads(48, 80, 4, 34), np.zeros((48, 80), np.float32),
                  beta_kron=0.5,
                  flags=soap.SOAP_FLAG_NO_BIAS_CORRECTION, bias_correction=False)


def test_kl_identity_eigenbasis_is_adamw():
    """One nonzero per gradient row and column keeps both factors diagonal
    under the KL accumulation too: the bases stay exactly I."""
    import paper_2607_20548_amd as soap
    from synth.gradients import permutation_gradient
    m, n = 64, 96
    gs = soap.SoapState(m, n, kl=True)
    W = dev(np.zeros((m, n), np.float32))
    for t in range(1, 6):
        gs.step(W, dev(permutation_gradient(m, n, 5, t)), t, beta_kron=BK, **HP)
        assert np.array_equal(host(gs.Q_L), np.eye(m)) and np.array_equal(host(gs.Q_R), np.eye(n))
        Lh, Rh = host(gs.L), host(gs.R)
        assert np.array_equal(np.diag(np.diag(Lh)), Lh) and np.array_equal(np.diag(np.diag(Rh)), Rh)


@pytest.mark.parametrize("m,n", [(37, 70), (37, 80), (90, 40)])
def test_kl_batched_matches_single_and_oracle(m, n):
    import paper_2607_20548_amd as soap
    import oracle
    B = 4
    rng = np.random.default_rng([m, n, 35])
    W0 = (0.02 * rng.standard_normal((B, m, n))).astype(np.float32)
    grads = [rng.standard_normal((B, m, n)).astype(np.float32) for _ in range(3)]
    gb = soap.SoapState(m, n, batch=B, kl=True)
    Wb = dev(W0)
    singles = [soap.SoapState(m, n, kl=True) for _ in range(B)]
    Ws = [dev(W0[b]) for b in range(B)]
    sts = [oracle.init_state(W0[b].astype(np.float64)) for b in range(B)]
    for t, G in enumerate(grads, start=1):
        gb.step(Wb, dev(G), t, beta_kron=BK, **HP)
        for b in range(B):
            singles[b].step(Ws[b], dev(G[b]), t, beta_kron=BK, **HP)
            sts[b] = oracle.kl_soap_step(sts[b], G[b].astype(np.float64), t, beta_kron=BK, **HP)
        Wbh = host(Wb)
        for b in range(B):
            assert rel(Wbh[b], host(Ws[b])) <= 1e-6
            assert rel(host(gb.R)[b], host(singles[b].R)) <= 1e-6
            assert rel(Wbh[b], sts[b].W) <= TOL
            assert rel(host(gb.L)[b], sts[b].L) <= TOL
            assert rel(host(gb.R)[b], sts[b].R) <= TOL
            assert rel(host(gb.Q_R)[b], sts[b].QR) <= TOL


def test_kl_two_runs_are_bitwise_identical():
    import paper_2607_20548_amd as soap
    rng = np.random.default_rng(36)
    m, n = 300, 520
    grads = [rng.standard_normal((m, n)).astype(np.float32) for _ in range(2)]
    outs = []
    for _ in range(2):
        gs = soap.SoapState(m, n, kl=True)
        W = dev(np.zeros((m, n), np.float32))
        for t, G in enumerate(grads, start=1):
            gs.step(W, dev(G), t, beta_kron=BK, **HP)
        outs.append([host(x) for x in (W, gs.L, gs.R, gs.Q_L, gs.Q_R, gs.M, gs.V)])
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


def _check_kl_factors_sampled(pre, post, G, rng, nsamp=48):
    """L and R of one KL step entry by entry: the estimates in full (fp64),
    then L[i,j] = bk L[i,j] + (1-bk)/n sum_k Y_R[i,k] Y_R[j,k] / (lam_R[k]+eps)
    with Y_R = G Q_R, and R likewise with Y_L = Q_L^T G and 1/m."""
    eps = HP["eps"]
    m, n = G.shape
    lam_L = np.einsum("ik,ik->k", pre["QL"], pre["L"] @ pre["QL"])
    lam_R = np.einsum("ik,ik->k", pre["QR"], pre["R"] @ pre["QR"])
    ii, jj = rng.integers(0, m, nsamp), rng.integers(0, m, nsamp)
    YRi, YRj = G[ii] @ pre["QR"], G[jj] @ pre["QR"]
    want = BK * pre["L"][ii, jj] + (1 - BK) / n * np.einsum("ik,ik->i", YRi / (lam_R + eps), YRj)
    eL = rel(post["L"][ii, jj], want)
    ii, jj = rng.integers(0, n, nsamp), rng.integers(0, n, nsamp)
    YLi, YLj = pre["QL"].T @ G[:, ii], pre["QL"].T @ G[:, jj]
    want = BK * pre["R"][ii, jj] + (1 - BK) / m * np.einsum("ki,ki->i", YLi / (lam_L + eps)[:, None], YLj)
    eR = rel(post["R"][ii, jj], want)
    log(f"  KL factors sampled: L={eL:.2e} R={eR:.2e}")
    assert eL <= TOL and eR <= TOL
    assert np.array_equal(post["R"][ii, jj], post["R"][jj, ii])


def test_kl_bench_shape_sampled_closed_loop():
    """4096 x 14336 (the bench workload): 2 KL steps, then one more checked on
    sampled entries from the GPU's pre-step state."""
    import paper_2607_20548_amd as soap
    from synth import gradients as sg
    spec = sg.workload(2).matrices[0]
    m, n = spec.m, spec.n
    grads = list(sg.make_matrix_stream(spec, 2, 3))
    gs = soap.SoapState(m, n, kl=True)
    W = dev(sg.initial_weight(spec, 2))
    for t in (1, 2):
        gs.step(W, dev(grads[t - 1]), t, beta_kron=BK, **HP)
    snap = lambda: {k: host(v) for k, v in dict(W=W, L=gs.L, R=gs.R, QL=gs.Q_L, QR=gs.Q_R,
                                                   M=gs.M, V=gs.V).items()}
    pre = snap()
    gs.step(W, dev(grads[2]), 3, beta_kron=BK, **HP)
    post = snap()
    G = grads[2].astype(np.float64)
    log(f"KL closed-loop step at {m}x{n}")
    rng = np.random.default_rng(37)
    _check_kl_factors_sampled(pre, post, G, rng)
    info = check_refresh_adam_sampled(pre, post, G, 3, rng)
    log(f"  ok {info}")


@pytest.mark.parametrize("m,n,F,stale", [(64, 96, 2, False), (37, 80, 3, False), (37, 80, 1, True),
                                         (90, 40, 2, True)])
def test_kl_refresh_period_and_stale_refresh(m, n, F, stale):
    rng = np.random.default_rng([m, n, F, int(stale), 40])
    run_open_loop(m, n, recipe_grads(m, n, 5, 40 + F + 10 * int(stale)),
                  (0.02 * rng.standard_normal((m, n))).astype(np.float32),
                  beta_kron=BK, refresh_every=F, stale_refresh=stale)
