"""Parity of the Muon step (soap_muon_step, soap_muon_step_batched) with the
fp64 oracle of Algorithm 1.

The paper's PolarExpress coefficients are not printed, so the schedules here
are the textbook ones and a steeper made-up one: the quintic from the Taylor
series of (1 - z)^(-1/2), (15/8, -5/4, 3/8), 16 times (the paper's n); the
cubic (1.5, -0.5, 0), which takes the library's c = 0 path; and three steep
steps (3, -3.2, 1.2) followed by the quintic.  Open loop: W and M are
compared every step with the relative Frobenius metric at 1e-4.
"""
import numpy as np
import pytest

from tests.gpu_helpers import dev, host, rel, log, TOL

pytestmark = pytest.mark.gpu

QUINTIC = [(15 / 8, -5 / 4, 3 / 8)] * 16
CUBIC = [(1.5, -0.5, 0.0)] * 16
STEEP = [(3.0, -3.2, 1.2)] * 3 + [(15 / 8, -5 / 4, 3 / 8)] * 13
HPM = dict(beta1=0.9, lr=2e-2, weight_decay=0.1, eps=1e-7)


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_20548_amd as soap
    soap.lib()


def _run(m, n, grads, W0, coeffs, batch=None, tag=""):
    import paper_2607_20548_amd as soap
    import oracle
    ms = soap.MuonState(m, n, batch=batch or 1)
    W = dev(W0)
    Wo = W0.astype(np.float64)
    Mo = np.zeros(W0.shape)
    for t, G in enumerate(grads, start=1):
        ms.step(W, dev(G), coeffs, **HPM)
        if batch:
            outs = [oracle.muon_step(Wo[b], Mo[b], G[b], coeffs=coeffs, **HPM) for b in range(batch)]
            Wo = np.stack([o[0] for o in outs])
            Mo = np.stack([o[1] for o in outs])
        else:
            Wo, Mo = oracle.muon_step(Wo, Mo, G, coeffs=coeffs, **HPM)
        eW, eM = rel(host(W), Wo), rel(host(ms.M), Mo)
        log(f"muon {tag} {m}x{n} t={t}: W={eW:.2e} M={eM:.2e}")
        assert eW <= TOL and eM <= TOL, (t, eW, eM)
    return W, ms


@pytest.mark.parametrize("m,n", [(1, 1), (3, 5), (5, 3), (64, 200), (200, 64), (129, 257),
                                 (300, 300)])
@pytest.mark.parametrize("name", ["quintic", "cubic", "steep"])
def test_muon_matches_oracle(m, n, name):
    coeffs = dict(quintic=QUINTIC, cubic=CUBIC, steep=STEEP)[name]
    rng = np.random.default_rng([m, n, len(name)])
    grads = [rng.standard_normal((m, n)).astype(np.float32) for _ in range(3)]
    _run(m, n, grads, (0.02 * rng.standard_normal((m, n))).astype(np.float32), coeffs, tag=name)


def test_muon_update_direction_matches():
    """The update alone (weights start at zero, no decay), so that a small
    relative error in W cannot hide a wrong direction."""
    import paper_2607_20548_amd as soap
    import oracle
    m, n = 96, 160
    rng = np.random.default_rng(50)
    G = rng.standard_normal((m, n)).astype(np.float32)
    ms = soap.MuonState(m, n)
    W = dev(np.zeros((m, n), np.float32))
    ms.step(W, dev(G), QUINTIC, beta1=0.0, lr=1.0, weight_decay=0.0, eps=1e-7)
    Wo, _, d = oracle.muon_step(np.zeros((m, n)), np.zeros((m, n)), G, 0.0, 1.0, 0.0, 1e-7,
                                QUINTIC, diagnostics=True)
    assert rel(-host(W), d["dW"]) <= TOL
    # the quintic drives all singular values of the direction near 1
    sv = np.linalg.svd(-host(W) / np.sqrt(n), compute_uv=False)
    assert np.all(np.abs(sv - 1) < 0.05)


def test_muon_zero_gradient_only_decays():
    import paper_2607_20548_amd as soap
    m, n = 40, 24
    W0 = np.random.default_rng(51).standard_normal((m, n)).astype(np.float32)
    ms = soap.MuonState(m, n)
    W = dev(W0)
    ms.step(W, dev(np.zeros((m, n), np.float32)), QUINTIC, **HPM)
    want = (np.float32(1) - np.float32(HPM["lr"]) * np.float32(HPM["weight_decay"])) * W0
    assert np.array_equal(host(W).astype(np.float32), want.astype(np.float32))


def test_muon_batched_matches_single_and_oracle():
    import paper_2607_20548_amd as soap
    B, m, n = 4, 37, 70
    rng = np.random.default_rng(52)
    W0 = (0.02 * rng.standard_normal((B, m, n))).astype(np.float32)
    grads = [rng.standard_normal((B, m, n)).astype(np.float32) for _ in range(2)]
    Wb, _ = _run(m, n, grads, W0, QUINTIC, batch=B, tag="batched")
    for b in range(B):
        ms = soap.MuonState(m, n)
        W = dev(W0[b])
        for G in grads:
            ms.step(W, dev(G[b]), QUINTIC, **HPM)
        assert rel(host(Wb)[b], host(W)) <= 1e-6


@pytest.mark.parametrize("m,n", [(2048, 8192), (8192, 2048)])
def test_muon_layer_shapes(m, n):
    """Two shapes of the 24-layer dense model, one full oracle step each
    (rank-128 signal, Student-t noise at 5%)."""
    from synth import gradients as sg
    spec = next(s for s in sg.workload(4).matrices if (s.m, s.n) == (m, n))
    G = next(sg.make_matrix_stream(spec, 4, 1))
    _run(m, n, [G], sg.initial_weight(spec, 4), QUINTIC, tag="layer")


def test_muon_bench_shape():
    """4096 x 14336 (the bench workload), one full oracle step."""
    from synth import gradients as sg
    spec = sg.workload(2).matrices[0]
    G = next(sg.make_matrix_stream(spec, 2, 1))
    _run(spec.m, spec.n, [G], sg.initial_weight(spec, 2), QUINTIC, tag="bench")
