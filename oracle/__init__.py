"""fp64 CPU oracle for the SOAP optimizer step (and the Muon step).

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow reference that the
HIP library is checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import it; the library itself never
does, and the two share no code.

Parity status of each function is stated in its docstring; every function here
is pinned by a ``-m "not gpu"`` test against something other than itself
(closed forms, LAPACK, brute force in 50-digit arithmetic, the paper's
reductions to AdamW and to the polar factor; for the KL-Shampoo accumulation,
the exact-inverse rule, the fixed point and condition number of Appendix A.3,
and the reduction to the plain factor EMA).
"""
from .soap_oracle import (  # noqa: F401
    OracleState, init_state, factor_ema, householder_qr, lapack_qr, refresh_qr, momentum_ema,
    rotate_in,
    adam_eigenbasis, rotate_out, weight_update, bias_corrections, soap_step,
    soap_step_batched, eigenvalue_estimates, kl_factor_update, kl_factors, kl_soap_step,
    kl_soap_step_batched, refresh_due,
)
from .muon_oracle import newton_schulz, muon_step, round_bf16  # noqa: F401
