"""Parity at the full sizes of the benchmark workloads, in the launch
configuration the bench uses (soap_step / soap_step_batched on the real
shapes).

The fp64 oracle cannot run many full steps at 4096..14336, so these tests
check ONE step closed-loop: the GPU takes a few steps, its state is copied to
the host, the GPU takes one more step, and every updated quantity with a
plain definition is recomputed in fp64 on sampled entries from the GPU's own
pre-step state:
  * L, R (factor EMA) and M (momentum EMA) entry by entry;
  * the refreshed eigenbases by their defining properties -- Q^T Q = I and
    Q^T (L Q_prev) upper triangular with a positive diagonal -- on sampled
    columns (those properties fix the Q factor uniquely);
  * V and the update N at sampled eigenbasis entries, from G' = Q_L^T G Q_R
    and M' = Q_L^T M Q_R formed with matrix-vector products;
  * W through N recovered from consecutive weights.
The 4096 x 4096 shape also gets one full oracle step (all tensors), and the
expert bank full oracle parity on two experts.
"""
import numpy as np
import pytest

from tests.gpu_helpers import (dev, host, rel, log, column_signs_agree, check_factor_ema_sampled,
                                check_refresh_adam_sampled)

pytestmark = pytest.mark.gpu

HP = dict(beta1=0.95, beta2=0.95, eps=1e-8, lr=1e-3, weight_decay=0.1)
TOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_20548_amd as soap
    soap.lib()


def _snap(gs, W, b=None):
    sel = (lambda x: x[b]) if b is not None else (lambda x: x)
    return {k: sel(host(v)) for k, v in dict(W=W, L=gs.L, R=gs.R, QL=gs.Q_L, QR=gs.Q_R,
                                               M=gs.M, V=gs.V).items()}


def _sampled_step_checks(pre, post, G, t, rng, nsamp=48, ncols=16):
    """All checks of one step from the GPU state `pre` to `post` (fp64 arrays)."""
    check_factor_ema_sampled(pre, post, G, rng, HP["beta2"], nsamp)
    return check_refresh_adam_sampled(pre, post, G, t, rng, HP, nsamp, ncols)


def _run_single(spec, cfg, steps_before, seed=0):
    import paper_2607_20548_amd as soap
    from synth import gradients as sg
    m, n = spec.m, spec.n
    grads = list(sg.make_matrix_stream(spec, cfg, steps_before + 1, seed=seed))
    gs = soap.SoapState(m, n)
    W = dev(sg.initial_weight(spec, cfg, seed=seed))
    for t in range(1, steps_before + 1):
        gs.step(W, dev(grads[t - 1]), t, **HP)
    pre = _snap(gs, W)
    t = steps_before + 1
    gs.step(W, dev(grads[-1]), t, **HP)
    post = _snap(gs, W)
    return pre, post, grads[-1].astype(np.float64), t


@pytest.mark.parametrize("cfg,steps_before", [(2, 2), (1, 3)])
def test_single_matrix_workloads_sampled(cfg, steps_before):
    from synth import gradients as sg
    spec = sg.workload(cfg).matrices[0]
    log(f"workload {spec.m}x{spec.n}: {steps_before} steps, then a sampled closed-loop step")
    pre, post, G, t = _run_single(spec, cfg, steps_before)
    info = _sampled_step_checks(pre, post, G, t, np.random.default_rng(cfg))
    log(f"  ok {info}")


@pytest.mark.parametrize("shape", [(2048, 6144), (2048, 2048), (2048, 8192), (8192, 2048)])
def test_transformer_layer_shapes_sampled(shape):
    """The four matrix shapes of the 24-layer dense model (h 2048, FFN 8192),
    Student-t(3) noise at 5% of the signal."""
    from synth import gradients as sg
    spec = next(s for s in sg.workload(4).matrices if (s.m, s.n) == shape)
    log(f"layer shape {shape}")
    pre, post, G, t = _run_single(spec, 4, 2)
    info = _sampled_step_checks(pre, post, G, t, np.random.default_rng(shape[0] + shape[1]))
    log(f"  ok {info}")


def test_layer_shape_batched_rank1024_q_formation():
    """Two 2048 x 8192 matrices through soap_step_batched: the R-side QR
    (n = 8192) forms Q by rank-1024 updates, each of whose products starts
    from the head block of W = Y^T Q taken from diag(d), for every batch
    entry.  One step, then the sampled closed-loop checks of a second step
    on both entries."""
    import paper_2607_20548_amd as soap
    from synth import gradients as sg
    spec = next(s for s in sg.workload(4).matrices if (s.m, s.n) == (2048, 8192))
    B, steps = 2, 2
    log(f"batched layer shape {spec.m}x{spec.n} x{B}")
    grads = np.stack([np.stack(list(sg.make_matrix_stream(spec, 4, steps, seed=b)))
                      for b in range(B)], axis=1)                       # steps x B x m x n
    W = dev(np.stack([sg.initial_weight(spec, 4, seed=b) for b in range(B)]))
    gs = soap.SoapState(spec.m, spec.n, batch=B)
    for t in range(1, steps):
        gs.step(W, dev(grads[t - 1]), t, **HP)
    pre_all = _snap(gs, W)
    gs.step(W, dev(grads[steps - 1]), steps, **HP)
    post_all = _snap(gs, W)
    rng = np.random.default_rng(8192)
    for b in range(B):
        pre = {k: v[b] for k, v in pre_all.items()}
        post = {k: v[b] for k, v in post_all.items()}
        info = _sampled_step_checks(pre, post, grads[steps - 1, b].astype(np.float64), steps, rng)
        log(f"  entry {b} ok {info}")


def test_workload_4096_full_oracle_step():
    """One full closed-loop oracle step at 4096 x 4096 (every tensor)."""
    import oracle
    from synth import gradients as sg
    spec = sg.workload(1).matrices[0]
    pre, post, G, t = _run_single(spec, 1, 2)
    st = oracle.OracleState(pre["W"], pre["L"], pre["R"], pre["QL"], pre["QR"], pre["M"], pre["V"])
    st, d = oracle.soap_step(st, G, t, diagnostics=True, **HP)
    errs = {k: rel(post[k], getattr(st, a)) for k, a in
            [("L", "L"), ("R", "R"), ("QL", "QL"), ("QR", "QR"), ("M", "M"), ("V", "V"), ("W", "W")]}
    log("4096x4096 closed-loop step: " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for k, v in errs.items():
        assert v <= TOL, (k, v)
    assert column_signs_agree(post["QL"], st.QL) and column_signs_agree(post["QR"], st.QR)


def test_expert_bank_batched():
    """64 experts of 2048 x 768 through soap_step_batched, per-expert scale
    10^U(-4,-2).  Two experts get full oracle parity (open loop over the first
    steps), every expert the sampled closed-loop checks of the last step."""
    import paper_2607_20548_amd as soap
    import oracle
    from synth import gradients as sg
    wl = sg.workload(3)
    B, m, n = len(wl.matrices), 2048, 768
    steps = 3
    scales = sg.expert_scales(0, 3, B)
    grads = np.stack([np.stack(list(sg.make_matrix_stream(s, 3, steps, scale=scales[e])))
                      for e, s in enumerate(wl.matrices)], axis=1)      # steps x B x m x n
    W0 = np.stack([sg.initial_weight(s, 3) for s in wl.matrices])
    gs = soap.SoapState(m, n, batch=B)
    W = dev(W0)
    check = [0, 37]
    sts = {e: oracle.init_state(W0[e].astype(np.float64)) for e in check}
    for t in range(1, steps + 1):
        if t == steps:
            pre_all = {k: v for k, v in dict(W=host(W), L=host(gs.L), R=host(gs.R), QL=host(gs.Q_L),
                                               QR=host(gs.Q_R), M=host(gs.M), V=host(gs.V)).items()}
        gs.step(W, dev(grads[t - 1]), t, **HP)
        for e in check:
            sts[e] = oracle.soap_step(sts[e], grads[t - 1, e].astype(np.float64), t, **HP)
            for k, a in [("L", "L"), ("R", "R"), ("Q_L", "QL"), ("Q_R", "QR"), ("M", "M"), ("V", "V")]:
                err = rel(host(getattr(gs, k)[e]), getattr(sts[e], a))
                assert err <= TOL, (e, t, k, err)
            assert rel(host(W[e]), sts[e].W) <= TOL
    post_all = dict(W=host(W), L=host(gs.L), R=host(gs.R), QL=host(gs.Q_L), QR=host(gs.Q_R),
                    M=host(gs.M), V=host(gs.V))
    rng = np.random.default_rng(3)
    for e in range(0, B, 9):
        pre = {k: v[e] for k, v in pre_all.items()}
        post = {k: v[e] for k, v in post_all.items()}
        _sampled_step_checks(pre, post, grads[steps - 1, e].astype(np.float64), steps, rng,
                             nsamp=32, ncols=8)
    log("expert bank ok")
