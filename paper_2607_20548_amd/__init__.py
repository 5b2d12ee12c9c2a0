"""Python binding of the MI355X SOAP optimizer-step library (libsoap_mi355x.so).

Argument marshalling only: every function forwards to the C entry point of the
same name in ``include/soap.h``; all arithmetic runs in the HIP kernels.
Matrix arguments may be torch tensors (fp32, contiguous, on the GPU) or raw
integer device pointers; ``None`` passes NULL.  The stream defaults to torch's
current stream.  A nonzero status raises ``SoapError`` carrying
``soap_last_error()``.  There is no fallback: if the library is not built,
``lib()`` raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsoap_mi355x.so")

SOAP_OK = 0
SOAP_ERR_NULL = -1
SOAP_ERR_SHAPE = -2
SOAP_ERR_HPARAM = -3
SOAP_ERR_WORKSPACE = -4
SOAP_ERR_ALIGN = -5
SOAP_ERR_ALIAS = -6
SOAP_ERR_HIP = -7
SOAP_ERR_QR_GAVE_UP = -8
SOAP_STATUS_QR_L = 1
SOAP_STATUS_QR_R = 2
SOAP_FLAG_NO_BIAS_CORRECTION = 1
SOAP_FLAG_SKIP_REFRESH = 2
SOAP_FLAG_STALE_REFRESH = 4
SOAP_MUON_BF16 = 1
SOAP_MAX_DIM = 16384

EXPORTED = [
    "soap_workspace_bytes", "soap_init_state", "soap_step", "soap_step_batched",
    "soap_last_error", "soap_qr_workspace_bytes", "soap_qr_f32", "soap_gemm_f32",
    "soap_factor_ema_f32", "soap_timing_enable", "soap_timing_num_stages",
    "soap_timing_stage_name", "soap_timing_collect", "soap_timing_reset", "soap_timing_get",
    "soap_kl_workspace_bytes", "soap_kl_step", "soap_kl_step_batched",
    "soap_kl_factors_workspace_bytes", "soap_kl_factors_f32", "soap_muon_workspace_bytes",
    "soap_muon_step", "soap_muon_step_batched", "soap_workspace_status",
    "soap_workspace_update_offset", "soap_test_force_qr_give_up", "soap_step_noalloc",
]


class SoapError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"soap status {status}: {message}")
        self.status = status


_lib = None

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_F = ctypes.c_float
_U32 = ctypes.c_uint32
_SZ = ctypes.c_size_t
_INT = ctypes.c_int


def lib() -> ctypes.CDLL:
    """Load the built library (build it with paper_2607_20548_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(LIB_PATH)
    sig = {
        "soap_workspace_bytes": (_SZ, [_I64, _I64, _I64]),
        "soap_init_state": (_INT, [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P]),
        "soap_step": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _F, _F, _F, _F, _F,
                             _I64, _U32, _P, _SZ, _P]),
        "soap_step_batched": (_INT, [_I64, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _F, _F,
                                     _F, _F, _F, _I64, _U32, _P, _SZ, _P]),
        "soap_step_noalloc": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _F, _F, _F, _F,
                                     _F, _I64, _U32, _P]),
        "soap_kl_workspace_bytes": (_SZ, [_I64, _I64, _I64]),
        "soap_kl_step": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _F, _F, _F, _F, _F,
                                _F, _I64, _U32, _P, _SZ, _P]),
        "soap_kl_step_batched": (_INT, [_I64, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _F,
                                        _F, _F, _F, _F, _F, _I64, _U32, _P, _SZ, _P]),
        "soap_kl_factors_workspace_bytes": (_SZ, [_I64, _I64]),
        "soap_kl_factors_f32": (_INT, [_I64, _I64, _P, _P, _P, _P, _P, _F, _F, _P, _P, _P, _SZ,
                                       _P]),
        "soap_muon_workspace_bytes": (_SZ, [_I64, _I64, _I64]),
        "soap_muon_step": (_INT, [_P, _P, _P, _I64, _I64, _F, _F, _F, _F, _P, _I64, _U32, _P,
                                  _SZ, _P]),
        "soap_muon_step_batched": (_INT, [_I64, _P, _P, _P, _I64, _I64, _F, _F, _F, _F, _P, _I64,
                                          _U32, _P, _SZ, _P]),
        "soap_last_error": (ctypes.c_char_p, []),
        "soap_workspace_status": (_INT, [_P, ctypes.POINTER(ctypes.c_uint32), _P]),
        "soap_workspace_update_offset": (_SZ, [_I64, _I64, _I64]),
        "soap_test_force_qr_give_up": (_INT, [_U32]),
        "soap_qr_workspace_bytes": (_SZ, [_I64]),
        "soap_qr_f32": (_INT, [_I64, _P, _P, _P, _P, _SZ, _P]),
        "soap_gemm_f32": (_INT, [_INT, _INT, _I64, _I64, _I64, _F, _P, _I64, _P, _I64, _F, _P,
                                 _I64, _P]),
        "soap_factor_ema_f32": (_INT, [_INT, _I64, _I64, _P, _P, _F, _P]),
        "soap_timing_enable": (_INT, [_INT]),
        "soap_timing_num_stages": (_INT, []),
        "soap_timing_stage_name": (ctypes.c_char_p, [_INT]),
        "soap_timing_collect": (_INT, []),
        "soap_timing_reset": (_INT, []),
        "soap_timing_get": (_INT, [_INT, ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(ctypes.c_int64),
                                   ctypes.POINTER(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    import torch
    if not isinstance(x, torch.Tensor):
        raise TypeError(f"expected a torch tensor or an int pointer, got {type(x)}")
    if x.dtype != torch.float32 and x.dtype != torch.uint8:
        raise TypeError(f"tensors must be float32 (workspaces may be uint8), got {x.dtype}")
    if not x.is_cuda:
        raise ValueError("tensors must live on the GPU")
    if not x.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        if not torch.cuda.is_available():
            return None
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int) -> None:
    if status != SOAP_OK:
        raise SoapError(status, soap_last_error())


def soap_last_error() -> str:
    return lib().soap_last_error().decode()


def soap_workspace_bytes(batch: int, m: int, n: int) -> int:
    return lib().soap_workspace_bytes(batch, m, n)


def soap_workspace_status(workspace, stream=None):
    """Waits for the stream and returns (status code, status word) of the last
    step or QR enqueued with `workspace`: (SOAP_OK, 0) or
    (SOAP_ERR_QR_GAVE_UP, SOAP_STATUS_QR_* bits).  Other codes raise."""
    word = ctypes.c_uint32(0)
    rc = lib().soap_workspace_status(_ptr(workspace), ctypes.byref(word), _stream(stream))
    if rc not in (SOAP_OK, SOAP_ERR_QR_GAVE_UP):
        _check(rc)
    return rc, word.value


def soap_workspace_update_offset(batch: int, m: int, n: int) -> int:
    return lib().soap_workspace_update_offset(batch, m, n)


def soap_test_force_qr_give_up(mask: int) -> None:
    _check(lib().soap_test_force_qr_give_up(mask))


def soap_qr_workspace_bytes(n: int) -> int:
    return lib().soap_qr_workspace_bytes(n)


def soap_init_state(batch, m, n, L, R, Q_L, Q_R, M, V, stream=None) -> None:
    _check(lib().soap_init_state(batch, m, n, _ptr(L), _ptr(R), _ptr(Q_L), _ptr(Q_R), _ptr(M),
                                 _ptr(V), _stream(stream)))


def soap_step(param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, eps, lr, weight_decay,
              step, flags, workspace, workspace_bytes, stream=None) -> None:
    _check(lib().soap_step(_ptr(param), _ptr(grad), _ptr(L), _ptr(R), _ptr(Q_L), _ptr(Q_R),
                           _ptr(M), _ptr(V), m, n, beta1, beta2, eps, lr, weight_decay, step,
                           flags, _ptr(workspace), workspace_bytes, _stream(stream)))


SOAP_NOALLOC_MAX_WORKSPACE_BYTES = 256 << 20


def soap_step_noalloc(param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, eps, lr,
                      weight_decay, step, flags, stream=None) -> None:
    _check(lib().soap_step_noalloc(_ptr(param), _ptr(grad), _ptr(L), _ptr(R), _ptr(Q_L),
                                   _ptr(Q_R), _ptr(M), _ptr(V), m, n, beta1, beta2, eps, lr,
                                   weight_decay, step, flags, _stream(stream)))


def soap_step_batched(batch, param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, eps, lr,
                      weight_decay, step, flags, workspace, workspace_bytes, stream=None) -> None:
    _check(lib().soap_step_batched(batch, _ptr(param), _ptr(grad), _ptr(L), _ptr(R), _ptr(Q_L),
                                   _ptr(Q_R), _ptr(M), _ptr(V), m, n, beta1, beta2, eps, lr,
                                   weight_decay, step, flags, _ptr(workspace), workspace_bytes,
                                   _stream(stream)))


def soap_kl_workspace_bytes(batch: int, m: int, n: int) -> int:
    return lib().soap_kl_workspace_bytes(batch, m, n)


def soap_kl_step(param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, beta_kron, eps, lr,
                 weight_decay, step, flags, workspace, workspace_bytes, stream=None) -> None:
    _check(lib().soap_kl_step(_ptr(param), _ptr(grad), _ptr(L), _ptr(R), _ptr(Q_L), _ptr(Q_R),
                              _ptr(M), _ptr(V), m, n, beta1, beta2, beta_kron, eps, lr,
                              weight_decay, step, flags, _ptr(workspace), workspace_bytes,
                              _stream(stream)))


def soap_kl_step_batched(batch, param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, beta_kron,
                         eps, lr, weight_decay, step, flags, workspace, workspace_bytes,
                         stream=None) -> None:
    _check(lib().soap_kl_step_batched(batch, _ptr(param), _ptr(grad), _ptr(L), _ptr(R),
                                      _ptr(Q_L), _ptr(Q_R), _ptr(M), _ptr(V), m, n, beta1, beta2,
                                      beta_kron, eps, lr, weight_decay, step, flags,
                                      _ptr(workspace), workspace_bytes, _stream(stream)))


def soap_kl_factors_workspace_bytes(m: int, n: int) -> int:
    return lib().soap_kl_factors_workspace_bytes(m, n)


def soap_kl_factors_f32(m, n, G, L, R, Q_L, Q_R, beta_kron, eps, lam_L, lam_R, workspace,
                        workspace_bytes, stream=None) -> None:
    _check(lib().soap_kl_factors_f32(m, n, _ptr(G), _ptr(L), _ptr(R), _ptr(Q_L), _ptr(Q_R),
                                     beta_kron, eps, _ptr(lam_L), _ptr(lam_R), _ptr(workspace),
                                     workspace_bytes, _stream(stream)))


def _host_floats(values):
    """A host float array for a C `const float *` argument (kept alive by the caller)."""
    import numpy as np
    arr = np.ascontiguousarray(np.asarray(values, dtype=np.float32).ravel())
    return arr, arr.ctypes.data_as(ctypes.c_void_p)


def soap_muon_workspace_bytes(batch: int, m: int, n: int) -> int:
    return lib().soap_muon_workspace_bytes(batch, m, n)


def soap_muon_step(param, grad, M, m, n, beta1, lr, weight_decay, eps, coeffs, n_iters, flags,
                   workspace, workspace_bytes, stream=None) -> None:
    """coeffs: the 3 * n_iters Newton-Schulz coefficients (a_1, b_1, c_1, ...) on the host."""
    arr, ptr = _host_floats(coeffs)
    if arr.size < 3 * n_iters:
        raise ValueError("coeffs needs 3 * n_iters values")
    _check(lib().soap_muon_step(_ptr(param), _ptr(grad), _ptr(M), m, n, beta1, lr, weight_decay,
                                eps, ptr, n_iters, flags, _ptr(workspace), workspace_bytes,
                                _stream(stream)))


def soap_muon_step_batched(batch, param, grad, M, m, n, beta1, lr, weight_decay, eps, coeffs,
                           n_iters, flags, workspace, workspace_bytes, stream=None) -> None:
    arr, ptr = _host_floats(coeffs)
    if arr.size < 3 * n_iters:
        raise ValueError("coeffs needs 3 * n_iters values")
    _check(lib().soap_muon_step_batched(batch, _ptr(param), _ptr(grad), _ptr(M), m, n, beta1, lr,
                                        weight_decay, eps, ptr, n_iters, flags, _ptr(workspace),
                                        workspace_bytes, _stream(stream)))


def soap_qr_f32(n, A, Q, Rf, workspace, workspace_bytes, stream=None) -> None:
    _check(lib().soap_qr_f32(n, _ptr(A), _ptr(Q), _ptr(Rf), _ptr(workspace), workspace_bytes,
                             _stream(stream)))


def soap_gemm_f32(trans_a, trans_b, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc,
                  stream=None) -> None:
    _check(lib().soap_gemm_f32(int(trans_a), int(trans_b), M, N, K, alpha, _ptr(A), lda, _ptr(B),
                               ldb, beta, _ptr(C), ldc, _stream(stream)))


def soap_factor_ema_f32(trans, m, n, G, F, beta, stream=None) -> None:
    _check(lib().soap_factor_ema_f32(int(trans), m, n, _ptr(G), _ptr(F), beta, _stream(stream)))


def soap_timing_enable(enable: bool) -> None:
    _check(lib().soap_timing_enable(int(bool(enable))))


def soap_timing_num_stages() -> int:
    return lib().soap_timing_num_stages()


def soap_timing_stage_name(stage: int) -> str:
    return lib().soap_timing_stage_name(stage).decode()


def soap_timing_collect() -> None:
    _check(lib().soap_timing_collect())


def soap_timing_reset() -> None:
    _check(lib().soap_timing_reset())


def soap_timing_get(stage: int):
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    fl = ctypes.c_double()
    _check(lib().soap_timing_get(stage, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl)))
    return ms.value, n.value, fl.value


# ---------------------------------------------------------------- helpers
class SoapState:
    """Device-resident SOAP state for `batch` m x n matrices (fp32, contiguous),
    allocated with torch and initialised by soap_init_state.  With ``kl`` the
    step is KL-SOAP (soap_kl_step), whose coefficient ``beta_kron`` step()
    then takes."""

    def __init__(self, m: int, n: int, batch: int = 1, device: str = "cuda", kl: bool = False):
        import torch
        self.m, self.n, self.batch = m, n, batch
        shp = (lambda r, c: (batch, r, c)) if batch > 1 else (lambda r, c: (r, c))
        kw = dict(dtype=torch.float32, device=device)
        self.L = torch.empty(shp(m, m), **kw)
        self.R = torch.empty(shp(n, n), **kw)
        self.Q_L = torch.empty(shp(m, m), **kw)
        self.Q_R = torch.empty(shp(n, n), **kw)
        self.M = torch.empty(shp(m, n), **kw)
        self.V = torch.empty(shp(m, n), **kw)
        self.kl = kl
        self.ws_bytes = (soap_kl_workspace_bytes if kl else soap_workspace_bytes)(batch, m, n)
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        soap_init_state(batch, m, n, self.L, self.R, self.Q_L, self.Q_R, self.M, self.V)

    def status(self, stream=None):
        """(status code, SOAP_STATUS_QR_* bits) of the last step (synchronises)."""
        return soap_workspace_status(self.workspace, stream)

    def update(self):
        """The eigenbasis update N of the last step, a view into the workspace
        ([batch,] m x n fp32; valid until the next step)."""
        import torch
        off = soap_workspace_update_offset(self.batch, self.m, self.n)
        count = self.batch * self.m * self.n
        view = self.workspace[off:off + 4 * count].view(torch.float32)
        return view.view((self.batch, self.m, self.n) if self.batch > 1 else (self.m, self.n))

    def step(self, param, grad, t: int, beta1=0.95, beta2=0.95, eps=1e-8, lr=1e-3,
             weight_decay=0.1, flags=0, stream=None, beta_kron=None, refresh_every=1,
             stale_refresh=False) -> None:
        """One step t (1-based).  refresh_every = F refreshes the eigenbases
        when t mod F = 0 (SOAP_FLAG_SKIP_REFRESH on the other steps);
        stale_refresh sets SOAP_FLAG_STALE_REFRESH."""
        if refresh_every < 1:
            raise ValueError("refresh_every must be >= 1")
        if t % refresh_every != 0:
            flags |= SOAP_FLAG_SKIP_REFRESH
        if stale_refresh:
            flags |= SOAP_FLAG_STALE_REFRESH
        if self.kl:
            if beta_kron is None:
                raise ValueError("a KL-SOAP state needs beta_kron")
            if self.batch == 1:
                soap_kl_step(param, grad, self.L, self.R, self.Q_L, self.Q_R, self.M, self.V,
                             self.m, self.n, beta1, beta2, beta_kron, eps, lr, weight_decay, t,
                             flags, self.workspace, self.ws_bytes, stream)
            else:
                soap_kl_step_batched(self.batch, param, grad, self.L, self.R, self.Q_L, self.Q_R,
                                     self.M, self.V, self.m, self.n, beta1, beta2, beta_kron, eps,
                                     lr, weight_decay, t, flags, self.workspace, self.ws_bytes,
                                     stream)
            return
        if beta_kron is not None:
            raise ValueError("beta_kron applies to KL-SOAP states only")
        if self.batch == 1:
            soap_step(param, grad, self.L, self.R, self.Q_L, self.Q_R, self.M, self.V, self.m,
                      self.n, beta1, beta2, eps, lr, weight_decay, t, flags, self.workspace,
                      self.ws_bytes, stream)
        else:
            soap_step_batched(self.batch, param, grad, self.L, self.R, self.Q_L, self.Q_R, self.M,
                              self.V, self.m, self.n, beta1, beta2, eps, lr, weight_decay, t,
                              flags, self.workspace, self.ws_bytes, stream)


class MuonState:
    """Device-resident Muon state (the momentum buffer) for `batch` m x n
    matrices, zero-initialised, with its workspace."""

    def __init__(self, m: int, n: int, batch: int = 1, device: str = "cuda"):
        import torch
        self.m, self.n, self.batch = m, n, batch
        shp = (batch, m, n) if batch > 1 else (m, n)
        self.M = torch.zeros(shp, dtype=torch.float32, device=device)
        self.ws_bytes = soap_muon_workspace_bytes(batch, m, n)
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)

    def step(self, param, grad, coeffs, beta1=0.9, lr=1e-3, weight_decay=0.1, eps=1e-7,
             bf16=False, stream=None) -> None:
        """coeffs: a sequence of (a, b, c) Newton-Schulz triples, one per iteration.
        bf16: Newton-Schulz in bfloat16 (SOAP_MUON_BF16)."""
        flat = [float(x) for abc in coeffs for x in abc]
        n_iters = len(flat) // 3
        flags = SOAP_MUON_BF16 if bf16 else 0
        if self.batch == 1:
            soap_muon_step(param, grad, self.M, self.m, self.n, beta1, lr, weight_decay, eps, flat,
                           n_iters, flags, self.workspace, self.ws_bytes, stream)
        else:
            soap_muon_step_batched(self.batch, param, grad, self.M, self.m, self.n, beta1, lr,
                                   weight_decay, eps, flat, n_iters, flags, self.workspace,
                                   self.ws_bytes, stream)
