"""Parity of the bfloat16 Newton-Schulz form of the Muon step
(SOAP_MUON_BF16) with the oracle's bfloat16 reading of Algorithm 1.

The oracle rounds the exact result of every operation once to bfloat16; the
GPU accumulates each product in fp32 on the matrix cores and then rounds
once, so the two agree except where an exact result lies within the fp32
accumulation error of a bfloat16 rounding boundary, and such a difference is
one bfloat16 unit.  The checks:

* one step with lr sqrt(max(m, n)) ~ 1 and W = 0, so that -W is the
  orthogonalised direction O itself (recovered exactly: O is a bfloat16
  value and the fp32 scaling moves it by far less than half a unit): after
  0 and 1 iterations almost every entry of O is bit-identical to the
  oracle's, and none is more than two units (at its own size, or the
  entries' RMS size when it is smaller) away -- one for its own rounding,
  one for a boundary case in a large entry of B, which shifts a whole row of
  B X -- also at 2048 x 16384;
* 16 quintic iterations (the paper's n) over three steps, wide, tall, square
  and batched: every entry of O is a bfloat16 value, O is within
  8 units (8 x 2^-8) of the oracle in relative Frobenius norm -- the spread
  that two correctly rounded bfloat16 evaluations show once a boundary case
  is amplified by the iteration (pinned on the CPU against an
  fp32-accumulating model) -- and within bfloat16 noise (0.1) of the fp64
  iteration; the momentum (fp32) matches to 1e-6;
* 4096 x 14336 (the bench workload): the bfloat16 direction against the
  fp32 path's, which is checked against the fp64 oracle at smaller sizes.
"""
import numpy as np
import pytest

from tests.gpu_helpers import dev, host, rel, log

pytestmark = pytest.mark.gpu

QUINTIC = [(15 / 8, -5 / 4, 3 / 8)] * 16
CUBIC = [(1.5, -0.5, 0.0)] * 16
U8 = 2.0 ** -8          # half the spacing of bfloat16 at 1 (relative unit)


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_20548_amd as soap
    soap.lib()


def _direction(m, n, G, coeffs, batch=None):
    """O of one bf16 Muon step from W = 0, M = 0, beta1 = 0 (so M = G):
    W = -lr sqrt(max(m, n)) O with lr = 1 / sqrt(max(m, n))."""
    import paper_2607_20548_amd as soap
    s = float(np.sqrt(max(m, n)))
    ms = soap.MuonState(m, n, batch=batch or 1)
    W = dev(np.zeros(G.shape, np.float32))
    ms.step(W, dev(G), coeffs, beta1=0.0, lr=1.0 / s, weight_decay=0.0, eps=1e-7, bf16=True)
    import oracle
    lr32 = float(np.float32(1.0 / s))
    return oracle.round_bf16(-host(W) / (lr32 * s))


def _oracle_direction(G, coeffs, precision="bf16"):
    import oracle
    G = G.astype(np.float64)
    if G.shape[0] > G.shape[1]:      # the library orthogonalises the transpose of a tall matrix
        return oracle.newton_schulz(G.T, coeffs, 1e-7, precision).T
    return oracle.newton_schulz(G, coeffs, 1e-7, precision)


def _units_apart(x, y):
    """|x - y| in units of the bfloat16 spacing at max(|x|, |y|, RMS of y).
    (The RMS floor: an entry whose value cancels to far below the size of its
    terms carries the fp32 accumulation error of those terms, not just the
    rounding of the result.)"""
    rms = float(np.sqrt(np.mean(np.square(y)))) or 1.0
    big = np.maximum(np.maximum(np.abs(x), np.abs(y)), rms)
    spacing = np.ldexp(1.0, np.frexp(big)[1] - 8)
    return np.abs(x - y) / spacing


@pytest.mark.parametrize("m,n", [(64, 200), (200, 64), (128, 128), (136, 264), (8, 8)])
@pytest.mark.parametrize("iters", [0, 1])
def test_bf16_first_iterations_are_correctly_rounded(m, n, iters):
    rng = np.random.default_rng([m, n, iters, 16])
    G = rng.standard_normal((m, n)).astype(np.float32)
    O = _direction(m, n, G, QUINTIC[:iters])
    Oo = _oracle_direction(G, QUINTIC[:iters])
    same = np.mean(O == Oo)
    units = _units_apart(O, Oo)
    log(f"bf16 NS {m}x{n} iters={iters}: identical {same:.5f}, max units {units.max():.2f}")
    assert np.array_equal(oracle_round(O), O)
    assert same >= 0.99
    assert units.max() <= 2.0


def test_bf16_first_iteration_large():
    """2048 x 16384 (2048 tiles in the update product, K = 16384 in the Gram
    product): one iteration against the oracle, entry by entry."""
    m, n = 2048, 16384
    rng = np.random.default_rng(20)
    G = rng.standard_normal((m, n)).astype(np.float32)
    O = _direction(m, n, G, QUINTIC[:1])
    Oo = _oracle_direction(G, QUINTIC[:1])
    same = np.mean(O == Oo)
    units = _units_apart(O, Oo)
    log(f"bf16 NS {m}x{n} iters=1: identical {same:.5f}, max units {units.max():.2f}")
    assert same >= 0.99
    assert units.max() <= 2.0


def oracle_round(x):
    import oracle
    return oracle.round_bf16(x)


@pytest.mark.parametrize("m,n", [(64, 200), (200, 64), (256, 256), (136, 520), (520, 136)])
@pytest.mark.parametrize("name", ["quintic", "cubic"])
def test_bf16_muon_matches_oracle(m, n, name):
    import paper_2607_20548_amd as soap
    import oracle
    coeffs = dict(quintic=QUINTIC, cubic=CUBIC)[name]
    rng = np.random.default_rng([m, n, len(name), 17])
    W0 = (0.02 * rng.standard_normal((m, n))).astype(np.float32)
    hp = dict(beta1=0.9, lr=2e-2, weight_decay=0.1, eps=1e-7)
    ms = soap.MuonState(m, n)
    W = dev(W0)
    Mo = np.zeros((m, n))
    for t in range(1, 4):
        G = rng.standard_normal((m, n)).astype(np.float32)
        W_prev = host(W)
        ms.step(W, dev(G), coeffs, bf16=True, **hp)
        Mo = oracle.muon_step(W_prev, Mo, G, coeffs=coeffs, precision="bf16", **hp)[1]
        assert rel(host(ms.M), Mo) <= 1e-6
        # O from the weights: W = (1 - lr wd) W_prev - lr sqrt(max(m, n)) O
        bw = float(np.float32(1.0) - np.float32(hp["lr"]) * np.float32(hp["weight_decay"]))
        O = oracle.round_bf16((bw * W_prev - host(W)) / (hp["lr"] * np.sqrt(max(m, n))))
        Mb = host(ms.M)
        Oo = _oracle_direction(Mb, coeffs)
        Of = _oracle_direction(Mb, coeffs, "fp64")
        e_bf, e_64 = rel(O, Oo), rel(O, Of)
        log(f"bf16 muon {name} {m}x{n} t={t}: vs bf16 oracle {e_bf:.2e}, vs fp64 {e_64:.2e}")
        assert e_bf <= 8 * U8, (t, e_bf)
        assert e_64 <= 0.1, (t, e_64)


def test_bf16_muon_batched_matches_single():
    """The batched call is the single call per matrix, bit for bit."""
    import paper_2607_20548_amd as soap
    rng = np.random.default_rng(18)
    B, m, n = 3, 136, 264
    G = rng.standard_normal((B, m, n)).astype(np.float32)
    W0 = (0.02 * rng.standard_normal((B, m, n))).astype(np.float32)
    hp = dict(beta1=0.9, lr=2e-2, weight_decay=0.1, eps=1e-7)
    mb = soap.MuonState(m, n, batch=B)
    Wb = dev(W0)
    mb.step(Wb, dev(G), QUINTIC, bf16=True, **hp)
    for b in range(B):
        ms = soap.MuonState(m, n)
        W = dev(W0[b])
        ms.step(W, dev(G[b]), QUINTIC, bf16=True, **hp)
        assert np.array_equal(host(W), host(Wb)[b])


def test_bf16_muon_rejects_ragged_shapes():
    import paper_2607_20548_amd as soap
    ms = soap.MuonState(12, 20)
    W = dev(np.zeros((12, 20), np.float32))
    with pytest.raises(RuntimeError, match="multiples of 8"):
        ms.step(W, dev(np.ones((12, 20), np.float32)), QUINTIC, bf16=True)


def test_bf16_muon_fullsize_against_fp32_path():
    """4096 x 14336: the bf16 direction against the fp32 path's (both from
    the same momentum), to bfloat16 noise."""
    import paper_2607_20548_amd as soap
    import torch
    m, n = 4096, 14336
    g = torch.Generator(device="cuda").manual_seed(19)
    G = torch.randn((m, n), device="cuda", generator=g)
    s = float(np.sqrt(n))
    out = {}
    for bf in (False, True):
        ms = soap.MuonState(m, n)
        W = torch.zeros((m, n), device="cuda")
        ms.step(W, G, QUINTIC, beta1=0.0, lr=1.0 / s, weight_decay=0.0, eps=1e-7, bf16=bf)
        torch.cuda.synchronize()
        out[bf] = W
    e = (torch.linalg.norm(out[True] - out[False]) / torch.linalg.norm(out[False])).item()
    log(f"bf16 vs fp32 Newton-Schulz at 4096x14336: {e:.3e}")
    assert e <= 0.1
    assert torch.isfinite(out[True]).all().item()
