"""Stage parity on the GPU: each kernel family alone against the plain
definition (fp64) or the fp64 oracle, on ragged shapes that span several
tiles and a partial tail."""
import numpy as np
import pytest

from tests.gpu_helpers import dev, host, rel, column_signs_agree, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_20548_amd as soap
    soap.lib()


GEMM_SHAPES = [(1, 1, 1), (3, 5, 7), (128, 128, 16), (127, 129, 130), (257, 300, 513),
               (64, 1000, 37), (512, 256, 1024)]


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_matches_definition(ta, tb, M, N, K):
    import paper_2607_20548_amd as soap
    log(f"gemm ta={ta} tb={tb} M={M} N={N} K={K}")
    rng = np.random.default_rng([M, N, K, ta, tb])
    A = rng.standard_normal((K, M) if ta else (M, K)).astype(np.float32)
    B = rng.standard_normal((N, K) if tb else (K, N)).astype(np.float32)
    C0 = rng.standard_normal((M, N)).astype(np.float32)
    opA = A.T.astype(np.float64) if ta else A.astype(np.float64)
    opB = B.T.astype(np.float64) if tb else B.astype(np.float64)
    for alpha, beta in [(1.0, 0.0), (-0.5, 1.0), (2.0, 0.25)]:
        Ad, Bd, Cd = dev(A), dev(B), dev(C0)
        soap.soap_gemm_f32(ta, tb, M, N, K, alpha, Ad, A.shape[1], Bd, B.shape[1], beta, Cd, N)
        want = alpha * (opA @ opB) + beta * C0.astype(np.float64)
        assert rel(host(Cd), want) <= 2e-6, (alpha, beta)


def test_gemm_leading_dimensions_and_submatrix():
    """A product on sub-blocks of larger row-major arrays (lda, ldb, ldc > cols)."""
    import paper_2607_20548_amd as soap
    rng = np.random.default_rng(3)
    big = rng.standard_normal((300, 301)).astype(np.float32)
    C = np.zeros((200, 211), np.float32)
    Bd, Cd = dev(big), dev(C)
    # C[0:150, 0:90] = big[10:160, 5:105] @ big[20:120, 7:97]
    off_a = (10 * 301 + 5) * 4
    off_b = (20 * 301 + 7) * 4
    soap.soap_gemm_f32(0, 0, 150, 90, 100, 1.0, Bd.data_ptr() + off_a, 301,
                       Bd.data_ptr() + off_b, 301, 0.0, Cd, 211)
    got = host(Cd)
    want = big[10:160, 5:105].astype(np.float64) @ big[20:120, 7:97].astype(np.float64)
    assert rel(got[:150, :90], want) <= 2e-6
    assert np.all(got[150:, :] == 0) and np.all(got[:, 90:] == 0)


@pytest.mark.parametrize("trans", [0, 1])
@pytest.mark.parametrize("m,n", [(1, 1), (3, 5), (130, 70), (129, 257), (300, 128), (256, 512)])
def test_factor_ema_matches_oracle(trans, m, n):
    import paper_2607_20548_amd as soap
    import oracle
    log(f"factor_ema trans={trans} m={m} n={n}")
    rng = np.random.default_rng([m, n, trans])
    G = rng.standard_normal((m, n)).astype(np.float32)
    d = n if trans else m
    S = rng.standard_normal((d, d))
    F0 = (S @ S.T / d + np.eye(d)).astype(np.float32)
    F0 = np.tril(F0) + np.tril(F0, -1).T
    Fd = dev(F0)
    soap.soap_factor_ema_f32(trans, m, n, dev(G), Fd, 0.95)
    got = host(Fd)
    X = G.T.astype(np.float64) if trans else G.astype(np.float64)
    want = oracle.factor_ema(F0.astype(np.float64), X, 0.95)
    assert rel(got, want) <= 1e-6
    assert np.array_equal(got, got.T)


def _well_conditioned(n, seed):
    """A = L Q with L symmetric positive definite and Q orthogonal, like the
    power products of the step."""
    rng = np.random.default_rng([n, seed, 5])
    X = rng.standard_normal((n, max(4, n // 4)))
    Lm = np.eye(n) + X @ X.T / X.shape[1]
    Q, R = np.linalg.qr(rng.standard_normal((n, n)))
    return (Lm @ (Q * np.sign(np.diag(R)))).astype(np.float32)


QR_SIZES = [1, 2, 3, 5, 16, 17, 31, 100, 127, 128, 129, 255, 256, 257, 300, 640, 1000, 1500]


@pytest.mark.parametrize("n", QR_SIZES)
def test_qr_matches_oracle(n):
    import paper_2607_20548_amd as soap
    import oracle
    import torch
    log(f"qr n={n}")
    A = _well_conditioned(n, 1)
    Ad = dev(A)
    Qd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    Rd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    wsb = soap.soap_qr_workspace_bytes(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    soap.soap_qr_f32(n, Ad, Qd, Rd, ws, wsb)
    Q, R = host(Qd), host(Rd)
    A64 = A.astype(np.float64)
    Qo = oracle.householder_qr(A64)
    assert column_signs_agree(Q, Qo)
    assert rel(Q, Qo) <= 1e-4
    assert np.linalg.norm(Q @ R - A64) / np.linalg.norm(A64) <= 1e-5
    assert np.linalg.norm(Q.T @ Q - np.eye(n)) / np.sqrt(n) <= 1e-5
    assert np.all(np.tril(R, -1) == 0) and np.all(np.diag(R) >= 0)
    assert np.array_equal(host(Ad), A)   # input untouched


@pytest.mark.parametrize("n", [3300, 4500])
def test_qr_matches_oracle_32_row_blocks(n):
    """Orders whose first blocks take 32 rows per thread: eight-column rounds
    up to 16 workgroups (n = 3300: two blocks of 13; n = 4500: 16 down to 13
    after four blocks of 18 and 17 workgroups with four-column rounds), then
    the 16-row kernel."""
    import paper_2607_20548_amd as soap
    import oracle
    import torch
    log(f"qr n={n}")
    A = _well_conditioned(n, 3)
    Ad = dev(A)
    Qd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    Rd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    wsb = soap.soap_qr_workspace_bytes(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    soap.soap_qr_f32(n, Ad, Qd, Rd, ws, wsb)
    Q, R = host(Qd), host(Rd)
    A64 = A.astype(np.float64)
    Qo = oracle.householder_qr(A64)
    assert column_signs_agree(Q, Qo)
    assert rel(Q, Qo) <= 1e-4
    assert np.linalg.norm(Q @ R - A64) / np.linalg.norm(A64) <= 1e-5
    assert np.linalg.norm(Q.T @ Q - np.eye(n)) / np.sqrt(n) <= 1e-5
    assert np.all(np.tril(R, -1) == 0) and np.all(np.diag(R) >= 0)


@pytest.mark.parametrize("n", [255, 256, 257, 300, 640, 1000, 1500])
def test_qr_q_only_matches_oracle(n):
    """Without an R output (the SOAP step's call): the same Q as with one, to
    the oracle's bar."""
    import paper_2607_20548_amd as soap
    import oracle
    import torch
    log(f"qr q-only n={n}")
    A = _well_conditioned(n, 2)
    Ad = dev(A)
    Qd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    Rd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    wsb = soap.soap_qr_workspace_bytes(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    soap.soap_qr_f32(n, Ad, Qd, None, ws, wsb)
    Q = host(Qd)
    soap.soap_qr_f32(n, Ad, Qd, Rd, ws, wsb)   # with R
    Qb, R = host(Qd), host(Rd)
    A64 = A.astype(np.float64)
    Qo = oracle.householder_qr(A64)
    assert column_signs_agree(Q, Qo)
    assert rel(Q, Qo) <= 1e-4
    assert rel(Q, Qb) <= 1e-5
    assert np.linalg.norm(Q @ R - A64) / np.linalg.norm(A64) <= 1e-5
    assert np.linalg.norm(Q.T @ Q - np.eye(n)) / np.sqrt(n) <= 1e-5


@pytest.mark.parametrize("n", [300, 640, 3300])
def test_qr_nearly_dependent_neighbour_columns(n):
    """Every third column is 1.5 x its left neighbour plus 5% of a fresh
    direction: the reflector of the left column removes most of it, so the
    block factorization ends a round right before that column, at every
    alignment within the rounds (n = 3300: also in the 32-row kernel with
    eight-column rounds).  Q against the oracle and the residuals at the
    usual bar."""
    import paper_2607_20548_amd as soap
    import oracle
    import torch
    log(f"qr nearly dependent n={n}")
    B = _well_conditioned(n, 3).astype(np.float64)
    A = B.copy()
    for j in range(0, n - 1, 3):
        A[:, j + 1] = 1.5 * A[:, j] + 0.05 * B[:, j + 1]
    A = A.astype(np.float32)
    Qd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    Rd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    wsb = soap.soap_qr_workspace_bytes(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    soap.soap_qr_f32(n, dev(A), Qd, Rd, ws, wsb)
    Q, R = host(Qd), host(Rd)
    A64 = A.astype(np.float64)
    Qo = oracle.householder_qr(A64)
    assert column_signs_agree(Q, Qo)
    assert rel(Q, Qo) <= 1e-4
    assert np.linalg.norm(Q @ R - A64) / np.linalg.norm(A64) <= 1e-5
    assert np.linalg.norm(Q.T @ Q - np.eye(n)) / np.sqrt(n) <= 1e-5
    assert np.all(np.tril(R, -1) == 0) and np.all(np.diag(R) >= 0)


def test_qr_large_residuals_rank1024_q_formation():
    """n = 8576 = 67 blocks: Q formed by rank-1024 updates (8 octs) plus a
    leftover pair and block; residuals computed in fp64 on the GPU."""
    import paper_2607_20548_amd as soap
    import torch
    n = 8576
    g = torch.Generator(device="cuda").manual_seed(21)
    A = (torch.eye(n, device="cuda") + 0.1 * torch.randn((n, n), device="cuda", generator=g) / n ** 0.5)
    Q = torch.empty((n, n), device="cuda")
    R = torch.empty((n, n), device="cuda")
    wsb = soap.soap_qr_workspace_bytes(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    soap.soap_qr_f32(n, A, Q, R, ws, wsb)
    Q2 = torch.empty_like(Q)
    soap.soap_qr_f32(n, A, Q2, None, ws, wsb)
    torch.cuda.synchronize()
    assert torch.equal(Q, Q2)
    Qd, Rd, Ad = Q.double(), R.double(), A.double()
    orth = (torch.linalg.norm(Qd.T @ Qd - torch.eye(n, device="cuda", dtype=torch.float64)) / n ** 0.5).item()
    rec = (torch.linalg.norm(Qd @ Rd - Ad) / torch.linalg.norm(Ad)).item()
    log(f"qr n={n}: orth {orth:.2e} rec {rec:.2e}")
    assert orth <= 1e-5 and rec <= 1e-5
    assert torch.equal(torch.tril(R, -1), torch.zeros_like(R))
    assert bool((torch.diagonal(R) >= 0).all())


def test_qr_random_gaussian_residuals():
    """Ill-conditioned (Gaussian) input: Q is less determined, residuals still tiny."""
    import paper_2607_20548_amd as soap
    import torch
    n = 700
    A = np.random.default_rng(9).standard_normal((n, n)).astype(np.float32)
    Qd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    Rd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    wsb = soap.soap_qr_workspace_bytes(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    soap.soap_qr_f32(n, dev(A), Qd, Rd, ws, wsb)
    Q, R = host(Qd), host(Rd)
    assert np.linalg.norm(Q @ R - A) / np.linalg.norm(A) <= 1e-5
    assert np.linalg.norm(Q.T @ Q - np.eye(n)) / np.sqrt(n) <= 1e-5


def test_qr_diagonal_input_gives_exact_identity():
    import paper_2607_20548_amd as soap
    import torch
    n = 300
    A = np.diag(np.linspace(0.5, 3.0, n)).astype(np.float32)
    Qd = torch.empty((n, n), dtype=torch.float32, device="cuda")
    wsb = soap.soap_qr_workspace_bytes(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    soap.soap_qr_f32(n, dev(A), Qd, None, ws, wsb)
    assert np.array_equal(host(Qd), np.eye(n))
