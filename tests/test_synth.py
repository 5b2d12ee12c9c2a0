"""The seeded generator: determinism, spectra and noise levels (CPU only)."""
import numpy as np

from synth import gradients as g


def test_deterministic_bits():
    spec = g.workload(0).matrices[0]
    a = list(g.make_matrix_stream(spec, 0, 3, seed=0))
    b = list(g.make_matrix_stream(spec, 0, 3, seed=0))
    for x, y in zip(a, b):
        assert x.dtype == np.float32 and np.array_equal(x, y)
    c = list(g.make_matrix_stream(spec, 0, 1, seed=1))
    assert not np.array_equal(a[0], c[0])
    # a stream started later reproduces the same step
    d = list(g.make_matrix_stream(spec, 0, 1, seed=0, start_step=3))
    assert np.array_equal(a[2], d[0])


def test_low_rank_signal_spectrum_and_noise_levels():
    spec = g.MatrixSpec("x", 300, 200, 16, "rel", 0.10)
    G = next(g.make_matrix_stream(spec, 1, 1)).astype(np.float64)
    s = np.linalg.svd(G, compute_uv=False)
    # leading singular values follow 1/i up to the 10% noise
    assert abs(s[0] - 1.0) < 0.1 and abs(s[1] - 0.5) < 0.1
    S_norm = np.sqrt(np.sum(1.0 / np.arange(1, 17) ** 2))
    # ||G||^2 = ||S||^2 + ||E||^2 (+ a small cross term)
    assert abs(np.linalg.norm(G) ** 2 - 1.01 * S_norm ** 2) < 0.02 * S_norm ** 2
    spec0 = g.workload(0).matrices[0]
    G0 = next(g.make_matrix_stream(spec0, 0, 1)).astype(np.float64)
    resid = G0 - np.linalg.svd(G0)[0][:, :16] @ np.diag(np.linalg.svd(G0)[1][:16]) @ np.linalg.svd(G0)[2][:16]
    assert 0.8e-3 < np.std(resid) < 1.2e-3


def test_workload_shapes():
    assert [(s.m, s.n) for s in g.workload(1).matrices] == [(4096, 4096)]
    assert [(s.m, s.n) for s in g.workload(2).matrices] == [(4096, 14336)]
    w3 = g.workload(3)
    assert len(w3.matrices) == 64 and w3.batched and {(s.m, s.n) for s in w3.matrices} == {(2048, 768)}
    w4 = g.workload(4)
    assert len(w4.matrices) == 96 and w4.steps == 5
    sc = g.expert_scales(0, 3, 64)
    assert np.all(sc >= 1e-4) and np.all(sc <= 1e-2)


def test_permutation_gradient_has_diagonal_factors():
    G = g.permutation_gradient(5, 7, 0, 1).astype(np.float64)
    for F in (G @ G.T, G.T @ G):
        assert np.array_equal(F, np.diag(np.diag(F)))
