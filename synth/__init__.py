"""Seeded synthetic workloads shared by the tests, the bench and the smoke check.

This package only draws numbers: low-rank-plus-noise gradients, initial weights
and the five workload definitions.  It holds none of the optimizer's arithmetic,
so both the fp64 oracle and the HIP path can consume its output without sharing
any code of the method.
"""
from .gradients import (  # noqa: F401
    CONFIGS, Workload, MatrixSpec, HParams, make_matrix_stream, initial_weight,
    workload, matrix_specs,
)
