"""Seeded low-rank-plus-noise gradient streams with the shapes of LLM weights.

The paper trains on real pretraining data (Nemotron-3 mixture) that is not
available here; these synthetic streams stand in for it.  Every gradient is

    G_t = scale * (S + E_t),   S = U diag(s) V^T,  s_i = 1/i,

with U (m x k) and V (n x k) orthonormal, drawn once per matrix, and E_t fresh
noise per step.  U and V come from numpy's LAPACK QR of a Gaussian matrix with
the R diagonal made positive (a draw from the Haar measure); this is input
generation only.  All arithmetic here is in fp64 and each G_t is rounded to
fp32 once, so every consumer sees identical fp32 bits.

Seeding (numpy PCG64 via ``default_rng``):
  * U, V:  default_rng([seed, cfg, matrix_id, 0])
  * E_t:   default_rng([seed, cfg, matrix_id, 1, t])      (t = 1-based step)
  * W_0:   default_rng([seed, cfg, matrix_id, 2])         W_0 ~ N(0, 0.02^2)
  * expert scales (cfg 3): default_rng([seed, cfg, 3])
"""
from __future__ import annotations

import dataclasses
from typing import Iterator, List, Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class HParams:
    """Optimizer hyperparameters handed to both sides (not used in this module)."""
    beta1: float = 0.95
    beta2: float = 0.95
    eps: float = 1e-8
    lr: float = 1e-3
    weight_decay: float = 0.1
    bias_correction: bool = True


@dataclasses.dataclass(frozen=True)
class MatrixSpec:
    """One weight matrix of a workload: its shape and its gradient recipe."""
    name: str
    m: int
    n: int
    rank: int
    noise: str            # "abs" (iid N(0, noise_level^2)) or "rel" (||E||_F = level*||S||_F)
    noise_level: float
    noise_dist: str = "normal"   # "normal" or "student_t3"
    matrix_id: int = 0


@dataclasses.dataclass(frozen=True)
class Workload:
    """A named workload: a list of matrix groups, each run for `steps` steps."""
    cfg: int
    name: str
    matrices: List[MatrixSpec]
    steps: int
    batched: bool          # True: all matrices share a shape and go through one batched call
    hparams: HParams = HParams()


def _cfg0() -> Workload:
    return Workload(0, "single 256x512 weight, rank-16 signal + N(0,1e-3) noise",
                    [MatrixSpec("W", 256, 512, 16, "abs", 1e-3)], 10, False)


def _cfg1() -> Workload:
    return Workload(1, "dense attention projection 4096x4096, rank 64, 10% noise",
                    [MatrixSpec("Wproj", 4096, 4096, 64, "rel", 0.10)], 20, False)


def _cfg2() -> Workload:
    return Workload(2, "MLP up-projection 4096x14336, rank 128, 10% noise",
                    [MatrixSpec("W_up", 4096, 14336, 128, "rel", 0.10)], 10, False)


def _cfg3() -> Workload:
    mats = [MatrixSpec(f"expert{e}", 2048, 768, 8, "rel", 0.10, matrix_id=e)
            for e in range(64)]
    return Workload(3, "MoE expert bank 64 x (2048x768), rank 8, log-uniform scales",
                    mats, 20, True)


def _cfg4() -> Workload:
    mats = []
    shapes = [("Wqkv", 2048, 6144), ("Wo", 2048, 2048), ("W1", 2048, 8192), ("W2", 8192, 2048)]
    mid = 0
    for layer in range(24):
        for nm, m, n in shapes:
            mats.append(MatrixSpec(f"layer{layer}.{nm}", m, n, 32, "rel", 0.05,
                                   noise_dist="student_t3", matrix_id=mid))
            mid += 1
    return Workload(4, "24-layer dense transformer (h 2048, FFN 8192), 96 matrices",
                    mats, 5, False)


CONFIGS = {0: _cfg0, 1: _cfg1, 2: _cfg2, 3: _cfg3, 4: _cfg4}


def workload(cfg: int) -> Workload:
    return CONFIGS[cfg]()


def matrix_specs(cfg: int) -> List[MatrixSpec]:
    return workload(cfg).matrices


def _orthonormal(rng: np.random.Generator, rows: int, k: int) -> np.ndarray:
    z = rng.standard_normal((rows, k))
    q, r = np.linalg.qr(z)
    d = np.sign(np.diag(r))
    d[d == 0] = 1.0
    return q * d


def expert_scales(seed: int, cfg: int, count: int) -> np.ndarray:
    """Per-expert gradient scale 10^U(-4,-2), mimicking uneven routing."""
    rng = np.random.default_rng([seed, cfg, 3])
    return 10.0 ** rng.uniform(-4.0, -2.0, size=count)


def make_matrix_stream(spec: MatrixSpec, cfg: int, steps: int, seed: int = 0,
                       scale: float = 1.0, start_step: int = 1) -> Iterator[np.ndarray]:
    """Yield fp32 gradients G_t for t = start_step .. start_step+steps-1."""
    rng = np.random.default_rng([seed, cfg, spec.matrix_id, 0])
    k = min(spec.rank, spec.m, spec.n)
    U = _orthonormal(rng, spec.m, k)
    V = _orthonormal(rng, spec.n, k)
    s = 1.0 / np.arange(1, k + 1, dtype=np.float64)
    S = (U * s) @ V.T
    s_norm = np.sqrt(np.sum(s * s))          # ||S||_F for orthonormal U, V
    for t in range(start_step, start_step + steps):
        erng = np.random.default_rng([seed, cfg, spec.matrix_id, 1, t])
        if spec.noise_dist == "student_t3":
            E = erng.standard_t(3.0, size=(spec.m, spec.n))
        else:
            E = erng.standard_normal((spec.m, spec.n))
        if spec.noise == "abs":
            E *= spec.noise_level
        else:
            E *= spec.noise_level * s_norm / np.sqrt(np.sum(E * E))
        G = S + E
        if scale != 1.0:
            G *= scale
        yield G.astype(np.float32)


def initial_weight(spec: MatrixSpec, cfg: int, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng([seed, cfg, spec.matrix_id, 2])
    return (0.02 * rng.standard_normal((spec.m, spec.n))).astype(np.float32)


def small_matrix(m: int, n: int, seed: int, kind: str = "normal") -> np.ndarray:
    """Plain seeded fp32 test matrices for stage tests (ragged shapes, edge cases)."""
    rng = np.random.default_rng([seed, m, n, 7])
    if kind == "normal":
        return rng.standard_normal((m, n)).astype(np.float32)
    if kind == "spd":
        X = rng.standard_normal((m, max(m, n)))
        return ((X @ X.T) / X.shape[1] + np.eye(m)).astype(np.float32)
    if kind == "orthogonal":
        return _orthonormal(rng, m, m).astype(np.float32)
    raise ValueError(kind)


def permutation_gradient(m: int, n: int, seed: int, t: int) -> np.ndarray:
    """A gradient with at most one nonzero per row and per column (a scaled partial
    permutation).  Its Kronecker factors G G^T and G^T G are diagonal."""
    rng = np.random.default_rng([seed, m, n, 11, t])
    k = min(m, n)
    rows = rng.permutation(m)[:k]
    cols = rng.permutation(n)[:k]
    G = np.zeros((m, n), dtype=np.float32)
    G[rows, cols] = rng.standard_normal(k).astype(np.float32)
    return G
