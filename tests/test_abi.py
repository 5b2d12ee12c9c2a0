"""C-ABI checks that need no GPU: the library loads, exports every entry
point soap.h declares, and its host-side validation returns the documented
status codes before anything is enqueued (only fake pointers are passed, and
only to calls that must fail validation)."""
import os
import re

import pytest

import paper_2607_20548_amd as soap

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    from paper_2607_20548_amd import build
    build.build(force=False)
    return soap.lib()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "soap.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(soap_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 10
    for name in names:
        assert hasattr(L, name), name
    assert sorted(names) == sorted(soap.EXPORTED)


BASE = 0x7f0000000000
MB = 1 << 24


def fake_args(m=8, n=12, ws=None, **over):
    p = {k: BASE + i * MB for i, k in enumerate(
        ["param", "grad", "L", "R", "Q_L", "Q_R", "M", "V", "workspace"])}
    args = dict(p, m=m, n=n, beta1=0.9, beta2=0.95, eps=1e-8, lr=1e-3, weight_decay=0.1, step=1,
                flags=0, workspace_bytes=soap.soap_workspace_bytes(1, m, n) if ws is None else ws)
    args.update(over)
    return args


def call_step(L, a):
    return L.soap_step(a["param"], a["grad"], a["L"], a["R"], a["Q_L"], a["Q_R"], a["M"], a["V"],
                       a["m"], a["n"], a["beta1"], a["beta2"], a["eps"], a["lr"],
                       a["weight_decay"], a["step"], a["flags"], a["workspace"],
                       a["workspace_bytes"], None)


@pytest.mark.parametrize("over,code", [
    (dict(param=None), soap.SOAP_ERR_NULL),
    (dict(V=None), soap.SOAP_ERR_NULL),
    (dict(m=0), soap.SOAP_ERR_SHAPE),
    (dict(n=soap.SOAP_MAX_DIM + 1), soap.SOAP_ERR_SHAPE),
    (dict(beta1=1.0), soap.SOAP_ERR_HPARAM),
    (dict(beta2=-0.1), soap.SOAP_ERR_HPARAM),
    (dict(eps=float("nan")), soap.SOAP_ERR_HPARAM),
    (dict(lr=float("inf")), soap.SOAP_ERR_HPARAM),
    (dict(weight_decay=-1.0), soap.SOAP_ERR_HPARAM),
    (dict(step=0), soap.SOAP_ERR_HPARAM),
    (dict(flags=8), soap.SOAP_ERR_HPARAM),
    (dict(grad=BASE + 1 * MB + 4), soap.SOAP_ERR_ALIGN),
    (dict(grad=BASE), soap.SOAP_ERR_ALIAS),                 # grad == param
    (dict(R=BASE + 2 * MB + 64), soap.SOAP_ERR_ALIAS),      # R inside L
])
def test_step_validation(L, over, code):
    assert call_step(L, fake_args(**over)) == code
    assert soap.soap_last_error() != ""


def test_workspace_too_small(L):
    need = soap.soap_workspace_bytes(1, 8, 12)
    assert need > 0
    assert call_step(L, fake_args(ws=need - 1)) == soap.SOAP_ERR_WORKSPACE
    assert "needed" in soap.soap_last_error()


def test_workspace_bytes_shapes(L):
    assert soap.soap_workspace_bytes(1, 0, 5) == 0
    assert soap.soap_workspace_bytes(0, 4, 5) == 0
    small = soap.soap_workspace_bytes(1, 256, 512)
    assert soap.soap_workspace_bytes(4, 256, 512) > 3 * small
    # the power products alone need (m^2 + n^2) floats
    assert soap.soap_workspace_bytes(1, 4096, 14336) > 4 * (4096 ** 2 + 14336 ** 2)


def test_batched_and_other_entry_points_validate(L):
    a = fake_args()
    rc = L.soap_step_batched(0, a["param"], a["grad"], a["L"], a["R"], a["Q_L"], a["Q_R"], a["M"],
                             a["V"], 8, 12, 0.9, 0.95, 1e-8, 1e-3, 0.1, 1, 0, a["workspace"],
                             a["workspace_bytes"], None)
    assert rc == soap.SOAP_ERR_SHAPE
    assert L.soap_qr_f32(0, BASE, BASE + MB, None, BASE + 2 * MB, 1 << 20, None) == soap.SOAP_ERR_SHAPE
    assert L.soap_qr_f32(64, BASE, BASE + MB, None, BASE + 2 * MB, 16, None) == soap.SOAP_ERR_WORKSPACE
    assert L.soap_init_state(1, 0, 4, None, None, None, None, None, None, None) == soap.SOAP_ERR_SHAPE
    assert L.soap_init_state(1, 4, 4, BASE + 8, None, None, None, None, None, None) == soap.SOAP_ERR_ALIGN
    assert L.soap_factor_ema_f32(0, 4, 4, BASE, BASE + MB, 1.5, None) == soap.SOAP_ERR_HPARAM
    assert L.soap_gemm_f32(0, 0, 0, 4, 4, 1.0, BASE, 4, BASE, 4, 0.0, BASE, 4, None) == soap.SOAP_ERR_SHAPE


def test_timing_api_without_gpu(L):
    n = soap.soap_timing_num_stages()
    names = [soap.soap_timing_stage_name(i) for i in range(n)]
    assert "qr_R" in names and "power_R" in names and len(set(names)) == n
    assert "qr_L_R" in names   # both square factors' QRs as one call
    soap.soap_timing_reset()
    assert soap.soap_timing_get(0) == (0.0, 0, 0.0)


def test_success_clears_error(L):
    call_step(L, fake_args(m=0))
    assert soap.soap_last_error() != ""
    soap.soap_timing_reset()   # a call that succeeds without touching the GPU
    assert L.soap_workspace_bytes(1, 4, 4) > 0


def call_kl_step(L, a, beta_kron=0.95, batch=None):
    args = (a["param"], a["grad"], a["L"], a["R"], a["Q_L"], a["Q_R"], a["M"], a["V"], a["m"],
            a["n"], a["beta1"], a["beta2"], beta_kron, a["eps"], a["lr"], a["weight_decay"],
            a["step"], a["flags"], a["workspace"], a["workspace_bytes"], None)
    if batch is None:
        return L.soap_kl_step(*args)
    return L.soap_kl_step_batched(batch, *args)


@pytest.mark.parametrize("over,beta_kron,code", [
    (dict(), 1.0, soap.SOAP_ERR_HPARAM),
    (dict(), -0.5, soap.SOAP_ERR_HPARAM),
    (dict(), float("nan"), soap.SOAP_ERR_HPARAM),
    (dict(L=None), 0.95, soap.SOAP_ERR_NULL),
    (dict(m=0), 0.95, soap.SOAP_ERR_SHAPE),
    (dict(beta1=1.0), 0.95, soap.SOAP_ERR_HPARAM),
    (dict(grad=BASE), 0.95, soap.SOAP_ERR_ALIAS),
])
def test_kl_step_validation(L, over, beta_kron, code):
    a = fake_args(ws=soap.soap_kl_workspace_bytes(1, 8, 12), **over)
    assert call_kl_step(L, a, beta_kron) == code
    assert soap.soap_last_error() != ""
    assert call_kl_step(L, a, beta_kron, batch=1) == code


def test_kl_workspace(L):
    m, n = 8, 12
    plain = soap.soap_workspace_bytes(1, m, n)
    kl = soap.soap_kl_workspace_bytes(1, m, n)
    assert kl > plain                       # one more m x n buffer and the estimates
    assert call_kl_step(L, fake_args(ws=plain)) == soap.SOAP_ERR_WORKSPACE
    assert soap.soap_kl_workspace_bytes(0, m, n) == 0
    assert soap.soap_kl_factors_workspace_bytes(m, 0) == 0
    big = soap.soap_kl_workspace_bytes(1, 4096, 14336)
    assert big > soap.soap_workspace_bytes(1, 4096, 14336) + 4 * 4096 * 14336


def test_kl_factors_validation(L):
    ws = soap.soap_kl_factors_workspace_bytes(8, 12)
    p = [BASE + i * MB for i in range(8)]
    # G, L, R, Q_L, Q_R, lam_L, lam_R, workspace
    assert L.soap_kl_factors_f32(8, 12, p[0], p[1], p[2], p[3], p[4], 1.0, 1e-8, None, None,
                                 p[7], ws, None) == soap.SOAP_ERR_HPARAM
    assert L.soap_kl_factors_f32(8, 12, p[0], p[1], p[2], p[3], p[4], 0.9, -1.0, None, None,
                                 p[7], ws, None) == soap.SOAP_ERR_HPARAM
    assert L.soap_kl_factors_f32(8, 12, None, p[1], p[2], p[3], p[4], 0.9, 1e-8, None, None,
                                 p[7], ws, None) == soap.SOAP_ERR_NULL
    assert L.soap_kl_factors_f32(8, 12, p[0], p[1], p[2], p[3], p[4], 0.9, 1e-8, None, None,
                                 p[7], ws - 1, None) == soap.SOAP_ERR_WORKSPACE
    assert L.soap_kl_factors_f32(8, 12, p[0], p[1], p[2], p[3], p[4], 0.9, 1e-8, p[1] + 64,
                                 None, p[7], ws, None) == soap.SOAP_ERR_ALIAS
    assert L.soap_kl_factors_f32(8, 12, p[0], p[1] + 4, p[2], p[3], p[4], 0.9, 1e-8, None, None,
                                 p[7], ws, None) == soap.SOAP_ERR_ALIGN


def test_muon_validation(L):
    import numpy as np
    m, n = 8, 12
    ws = soap.soap_muon_workspace_bytes(1, m, n)
    assert ws > 0 and soap.soap_muon_workspace_bytes(1, 0, n) == 0
    co = np.array([1.5, -0.5, 0.0] * 2, dtype=np.float32)
    cp = co.ctypes.data
    P, G, M, W = BASE, BASE + MB, BASE + 2 * MB, BASE + 3 * MB

    def call(**o):
        a = dict(param=P, grad=G, M=M, m=m, n=n, beta1=0.9, lr=1e-3, wd=0.1, eps=1e-7, co=cp,
                 it=2, flags=0, ws=W, wsb=ws)
        a.update(o)
        return L.soap_muon_step(a["param"], a["grad"], a["M"], a["m"], a["n"], a["beta1"],
                                a["lr"], a["wd"], a["eps"], a["co"], a["it"], a["flags"],
                                a["ws"], a["wsb"], None)
    assert call(m=0) == soap.SOAP_ERR_SHAPE
    assert call(M=None) == soap.SOAP_ERR_NULL
    assert call(co=None) == soap.SOAP_ERR_NULL
    assert call(beta1=1.0) == soap.SOAP_ERR_HPARAM
    assert call(eps=0.0) == soap.SOAP_ERR_HPARAM
    assert call(it=-1) == soap.SOAP_ERR_HPARAM
    assert call(it=2000) == soap.SOAP_ERR_HPARAM
    assert call(flags=2) == soap.SOAP_ERR_HPARAM
    assert call(flags=soap.SOAP_MUON_BF16) == soap.SOAP_ERR_SHAPE    # n = 12: not a multiple of 8
    assert call(wsb=ws - 1) == soap.SOAP_ERR_WORKSPACE
    assert call(grad=P + 16) == soap.SOAP_ERR_ALIAS
    assert call(M=M + 4) == soap.SOAP_ERR_ALIGN
    bad = np.array([1.5, float("nan"), 0.0], dtype=np.float32)
    assert call(co=bad.ctypes.data, it=1) == soap.SOAP_ERR_HPARAM
    assert L.soap_muon_step_batched(0, P, G, M, m, n, 0.9, 1e-3, 0.1, 1e-7, cp, 2, 0, W, ws,
                                    None) == soap.SOAP_ERR_SHAPE


def test_status_and_diagnostic_entry_points_validate(L):
    word = __import__("ctypes").c_uint32(7)
    assert L.soap_workspace_status(None, None, None) == soap.SOAP_ERR_NULL
    assert L.soap_test_force_qr_give_up(4) == soap.SOAP_ERR_HPARAM
    assert L.soap_test_force_qr_give_up(soap.SOAP_STATUS_QR_L | soap.SOAP_STATUS_QR_R) == soap.SOAP_OK
    assert L.soap_test_force_qr_give_up(0) == soap.SOAP_OK
    assert word.value == 7
    # N sits inside the step workspace, past the power products and both
    # rotation intermediates, and is the same for the KL layout
    for b, m, n in [(1, 8, 12), (3, 256, 512), (1, 4096, 14336)]:
        off = soap.soap_workspace_update_offset(b, m, n)
        assert off % 256 == 0
        assert off >= 4 * b * (m * m + n * n + 2 * m * n)
        assert off + 4 * b * m * n <= soap.soap_workspace_bytes(b, m, n)
        assert off + 4 * b * m * n <= soap.soap_kl_workspace_bytes(b, m, n)
    assert soap.soap_workspace_update_offset(1, 0, 4) == 0
    # the QR stage's workspace holds its status word, A^T and the QR buffers
    assert soap.soap_qr_workspace_bytes(64) > 4 * 64 * 64


def test_noalloc_step_validates_before_touching_the_device(L):
    a = fake_args()
    args = lambda **o: [dict(a, **o)[k] for k in ("param", "grad", "L", "R", "Q_L", "Q_R", "M", "V")]
    hp = (0.9, 0.95, 1e-8, 1e-3, 0.1)
    assert L.soap_step_noalloc(*args(), 0, 12, *hp, 1, 0, None) == soap.SOAP_ERR_SHAPE
    assert L.soap_step_noalloc(*args(), 4096, 4096, *hp, 1, 0, None) == soap.SOAP_ERR_WORKSPACE
    assert "soap_step with a workspace" in soap.soap_last_error()
    assert L.soap_step_noalloc(*args(param=None), 8, 12, *hp, 1, 0, None) == soap.SOAP_ERR_NULL
    assert L.soap_step_noalloc(*args(), 8, 12, 1.5, 0.95, 1e-8, 1e-3, 0.1, 1, 0, None) == soap.SOAP_ERR_HPARAM
    assert L.soap_step_noalloc(*args(), 8, 12, *hp, 0, 0, None) == soap.SOAP_ERR_HPARAM
    # every shape up to 2048 x 2048 fits the scratch
    assert soap.soap_workspace_bytes(1, 2048, 2048) <= soap.SOAP_NOALLOC_MAX_WORKSPACE_BYTES
