"""soap_step_noalloc, the entry point for callers that cannot allocate: the
same step as soap_step, with the library's static per-GPU scratch in place of
a caller workspace.  Its output must equal soap_step's bit for bit (same
kernels and launches; only the workspace address differs), over consecutive
calls where a smaller problem follows a larger one in the same scratch."""
import numpy as np
import pytest

from tests.gpu_helpers import dev, recipe_grads, HP

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_20548_amd as soap
    soap.lib()


def _state(m, n):
    import torch
    import paper_2607_20548_amd as soap
    kw = dict(dtype=torch.float32, device="cuda")
    st = {k: torch.empty(shp, **kw) for k, shp in
          [("L", (m, m)), ("R", (n, n)), ("Q_L", (m, m)), ("Q_R", (n, n)), ("M", (m, n)),
           ("V", (m, n))]}
    soap.soap_init_state(1, m, n, st["L"], st["R"], st["Q_L"], st["Q_R"], st["M"], st["V"])
    return st


def test_noalloc_step_equals_soap_step_larger_then_smaller():
    import torch
    import paper_2607_20548_amd as soap
    hp = (HP["beta1"], HP["beta2"], HP["eps"], HP["lr"], HP["weight_decay"])
    for m, n, seed in [(300, 600, 1), (70, 37, 2)]:     # the second call is smaller
        grads = recipe_grads(m, n, 2, 40 + seed)
        W0 = (0.02 * np.random.default_rng(seed).standard_normal((m, n))).astype(np.float32)
        ref = soap.SoapState(m, n)
        W_ref = dev(W0)
        st = _state(m, n)
        W = dev(W0)
        for t, G in enumerate(grads, start=1):
            Gd = dev(G)
            ref.step(W_ref, Gd, t, **HP)
            soap.soap_step_noalloc(W, Gd, st["L"], st["R"], st["Q_L"], st["Q_R"], st["M"], st["V"],
                                   m, n, *hp, t, 0)
            torch.cuda.synchronize()
            assert torch.equal(W, W_ref), (m, n, t, "W")
            for k in ("L", "R", "Q_L", "Q_R", "M", "V"):
                assert torch.equal(st[k], getattr(ref, k)), (m, n, t, k)


def test_noalloc_rejects_shapes_beyond_its_scratch():
    import paper_2607_20548_amd as soap
    st = _state(8, 12)
    W = dev(np.zeros((4096, 4096), np.float32))
    with pytest.raises(soap.SoapError) as exc:
        soap.soap_step_noalloc(W, W, st["L"], st["R"], st["Q_L"], st["Q_R"], st["M"], st["V"],
                               4096, 4096, 0.95, 0.95, 1e-8, 1e-3, 0.1, 1, 0)
    assert exc.value.status == soap.SOAP_ERR_WORKSPACE
