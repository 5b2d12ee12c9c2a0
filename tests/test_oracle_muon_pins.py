"""Pins of the oracle's Muon step (Algorithm 1), CPU only.

* Each Newton-Schulz step acts on the singular values alone:
  X = U S V^T  ->  U (a S + b S^3 + c S^5) V^T, checked against numpy's SVD
  (catches a swapped b / c, a wrong power, a product on the wrong side).
* The textbook cubic (1.5, -0.5, 0) and the quintic from the Taylor series of
  (1 - z)^(-1/2), (15/8, -5/4, 3/8), converge to the polar factor U V^T of
  the momentum (SVD), which Section 5.3's orthogonalisation approximates.
* Frobenius normalisation: the direction ignores the scale of M; M = 0 gives
  X_0 = 0 through the eps floor, so only the weight decay acts.
* The update scale sqrt(max(in, out)) and the decoupled weight decay on an
  orthogonal gradient, and the momentum EMA with beta1 on the old buffer.
"""
import numpy as np
import pytest

import oracle

CUBIC = (1.5, -0.5, 0.0)
QUINTIC = (15 / 8, -5 / 4, 3 / 8)


def rel(x, y):
    return np.linalg.norm(x - y) / max(np.linalg.norm(y), 1e-300)


def _with_singular_values(rng, m, n, s):
    U, _ = np.linalg.qr(rng.standard_normal((m, m)))
    V, _ = np.linalg.qr(rng.standard_normal((n, n)))
    k = len(s)
    return U[:, :k] @ np.diag(s) @ V[:, :k].T, U[:, :k], V[:, :k]


@pytest.mark.parametrize("m,n", [(4, 7), (7, 4), (5, 5)])
@pytest.mark.parametrize("abc", [(3.0, -3.2, 1.2), (2.0, -1.5, 0.5), QUINTIC])
def test_one_step_maps_singular_values(m, n, abc):
    rng = np.random.default_rng(m * 10 + n)
    k = min(m, n)
    s = np.sort(rng.uniform(0.05, 1.0, k))[::-1]
    s /= np.linalg.norm(s)             # already unit Frobenius norm: X_0 = M
    M, U, V = _with_singular_values(rng, m, n, s)
    X = oracle.newton_schulz(M, [abc], 1e-7)
    a, b, c = abc
    p = a * s + b * s ** 3 + c * s ** 5
    want = U @ np.diag(p) @ V.T
    assert rel(X, want) <= 1e-13
    got_s = np.sort(np.linalg.svd(X, compute_uv=False))[::-1]
    assert np.max(np.abs(got_s - np.sort(np.abs(p))[::-1])) <= 1e-13


@pytest.mark.parametrize("abc,iters", [(CUBIC, 60), (QUINTIC, 30)])
@pytest.mark.parametrize("m,n", [(6, 9), (9, 6)])
def test_iteration_converges_to_polar_factor(abc, iters, m, n):
    rng = np.random.default_rng(m + n)
    M = rng.standard_normal((m, n))
    X = oracle.newton_schulz(M, [abc] * iters, 1e-7)
    U, _, Vt = np.linalg.svd(M, full_matrices=False)
    assert rel(X, U @ Vt) <= 1e-12


def test_normalisation_and_eps_floor():
    rng = np.random.default_rng(3)
    M = rng.standard_normal((5, 8))
    X1 = oracle.newton_schulz(M, [QUINTIC] * 5, 1e-7)
    X2 = oracle.newton_schulz(1e4 * M, [QUINTIC] * 5, 1e-7)
    assert rel(X2, X1) <= 1e-14
    assert np.array_equal(oracle.newton_schulz(np.zeros((5, 8)), [QUINTIC] * 5, 1e-7),
                          np.zeros((5, 8)))
    W0 = rng.standard_normal((5, 8))
    W, Mn = oracle.muon_step(W0, np.zeros((5, 8)), np.zeros((5, 8)), 0.9, 0.01, 0.1, 1e-7,
                             [QUINTIC] * 3)
    assert np.array_equal(W, (1 - 0.01 * 0.1) * W0) and np.array_equal(Mn, np.zeros((5, 8)))
    # below eps the floor replaces the norm: X_0 = M / eps
    tiny = 1e-9 * np.eye(3)
    assert np.allclose(oracle.newton_schulz(tiny, [], 1e-7), tiny / 1e-7, rtol=1e-15, atol=0)


def test_update_scale_and_weight_decay_on_orthogonal_gradient():
    """beta1 = 0 and an orthogonal square G: the normalised momentum has all
    singular values 1/sqrt(n), the cubic iteration drives them to 1, and the
    update is sqrt(n) G."""
    n = 4
    rng = np.random.default_rng(4)
    Q, _ = np.linalg.qr(rng.standard_normal((n, n)))
    W0 = rng.standard_normal((n, n))
    lr, wd = 0.02, 0.1
    W, M, d = oracle.muon_step(W0, np.zeros((n, n)), Q, 0.0, lr, wd, 1e-7, [CUBIC] * 40,
                               diagnostics=True)
    assert rel(d["O"], Q) <= 1e-13
    assert rel(W, (1 - lr * wd) * W0 - lr * np.sqrt(n) * Q) <= 1e-13
    # rectangular: the scale is sqrt of the larger dimension
    G = rng.standard_normal((3, 7))
    _, _, d = oracle.muon_step(np.zeros((3, 7)), np.zeros((3, 7)), G, 0.0, lr, wd, 1e-7,
                               [CUBIC] * 60, diagnostics=True)
    assert rel(d["dW"], np.sqrt(7) * d["O"]) <= 1e-15


def test_momentum_beta_on_old_buffer():
    rng = np.random.default_rng(5)
    M0, G = rng.standard_normal((3, 4)), rng.standard_normal((3, 4))
    _, M = oracle.muon_step(np.zeros((3, 4)), M0, G, 0.9, 0.0, 0.0, 1e-7, [])
    assert rel(M, 0.9 * M0 + 0.1 * G) <= 1e-15


# ---- bfloat16 Newton-Schulz (the paper's precision for the iterations) ----

def _bf16_by_bits(x32):
    """Round-to-nearest-even to bfloat16 on the fp32 bit pattern: add 0x7FFF
    plus the lowest kept bit, keep the upper 16 bits (NaN passed through)."""
    u = np.asarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).astype(np.float64)
    return np.where(np.isnan(x32), np.nan, out)


def test_round_bf16_worked_values():
    r = oracle.round_bf16
    assert r(1.0) == 1.0
    assert r(1 + 2.0 ** -8) == 1.0                    # tie: to the even neighbour 1
    assert r(1 + 3 * 2.0 ** -8) == 1 + 2.0 ** -6      # tie: up to the even mantissa
    assert r(1 + 2.0 ** -8 + 2.0 ** -30) == 1 + 2.0 ** -7
    assert r(1 / 3) == 0.333984375                    # 0x3EAB
    assert r(-2.0 ** -133) == -2.0 ** -133            # smallest subnormal
    assert r(2.0 ** -134) == 0.0                      # half the smallest subnormal: tie to 0
    assert np.isinf(r(3.5e38)) and np.isnan(r(np.nan))


def test_round_bf16_matches_bit_definition_and_torch():
    import torch
    rng = np.random.default_rng(3)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
        (1 + (2 * rng.integers(0, 127, 2000) + 1) * 2.0 ** -8) * 2.0 ** rng.integers(-20, 20, 2000),
        rng.uniform(-1, 1, 2000) * 2.0 ** -126,        # subnormal range
        [0.0, -0.0, 2.0 ** -133, 3.0e38, -3.3e38]]).astype(np.float32)
    ours = oracle.round_bf16(x.astype(np.float64))
    assert np.array_equal(ours, _bf16_by_bits(x))
    tb = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, tb)


def _ns_fp32_accumulate(M, coeffs, eps):
    """The hardware model: products and linear combinations in fp32 on
    bfloat16 operands, each result rounded once to bfloat16 (torch's
    conversion)."""
    import torch
    bf = lambda t: t.to(torch.bfloat16).to(torch.float32)
    Mt = torch.from_numpy(M.astype(np.float32))
    X = bf(Mt / max(float(np.linalg.norm(M)), eps))
    for a, b, c in coeffs:
        A = bf(X @ X.T)
        B = bf(b * A + c * (A @ A))
        X = bf(a * X + B @ X)
    return X.double().numpy()


@pytest.mark.parametrize("m,n", [(24, 40), (40, 24), (32, 32)])
def test_bf16_newton_schulz_matches_fp32_accumulating_model(m, n):
    """The oracle (exact operation, one rounding) and the fp32-accumulating
    model round differently only next to rounding boundaries; over 16 quintic
    steps that keeps them within a few bfloat16 units in Frobenius norm."""
    rng = np.random.default_rng(m * 100 + n)
    M = rng.standard_normal((m, n))
    coeffs = [QUINTIC] * 16
    if m > n:   # the library orthogonalises the transpose of a tall matrix
        ours = oracle.newton_schulz(M.T, coeffs, 1e-7, "bf16").T
        model = _ns_fp32_accumulate(M.T, coeffs, 1e-7).T
    else:
        ours = oracle.newton_schulz(M, coeffs, 1e-7, "bf16")
        model = _ns_fp32_accumulate(M, coeffs, 1e-7)
    assert np.array_equal(oracle.round_bf16(ours), ours)     # every entry is a bfloat16 value
    assert rel(ours, model) <= 8 * 2.0 ** -8
    exact = oracle.newton_schulz(M.T if m > n else M, coeffs, 1e-7)
    exact = exact.T if m > n else exact
    assert rel(ours, exact) <= 0.1                           # bfloat16 noise, not a different map
    assert rel(ours, exact) > 1e-4                           # ... and the rounding did happen
