"""Seeded synthetic weight matrices with the shapes of the paper's models.

This module only draws random numbers: it holds none of the method's
arithmetic.  Both the GPU tests / benchmark and the CPU oracle consume the
exact arrays it returns (fp16 workloads are drawn in float64, rounded to fp16
once, and both sides read those fp16 values).

The paper quantises OPT, Llama-2 and Pythia checkpoints (Sec. 5); those weights
are not available here, so these matrices stand in for them with the same
layer shapes and heavy-tailed value distributions.  Each row of an (M, N)
matrix is one length-N vector (one output channel).

Workloads:
  ``gauss512``     256 x 512 fp32, N(0, 0.02^2), k = 20
  ``opt125m``      768x768 (x4), 3072x768, 768x3072 fp32, N(0, 0.02^2) with
                   0.1 % of columns scaled x20, k = 30
  ``llama7b``      4096x4096 (x4), 11008x4096 (x2), 4096x11008 fp16,
                   Student-t(4) scaled to std 0.02, k = 30
  ``pythia7b``     4096x4096 (x4), 16384x4096, 4096x16384 fp16,
                   N(0, 0.02^2) times a per-row LogNormal(0, 0.5) scale, k = 30
  ``llama7b_stack`` the llama7b layer x 32, Student-t(3) std 0.02 with 0.1 %
                   outlier columns x50, k = 40
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = ["MatrixSpec", "Workload", "WORKLOADS", "make_matrix", "sign_seed"]


@dataclass(frozen=True)
class MatrixSpec:
    name: str
    rows: int          # M: number of vectors
    n: int             # N: vector length
    dist: str          # "gauss" | "student_t" | "gauss_lognorm_rows"
    dof: float = 0.0   # Student-t degrees of freedom
    outlier_scale: float = 0.0  # 0 = no outlier columns
    dtype: str = "f32"  # "f32" | "f16"


@dataclass(frozen=True)
class Workload:
    key: str
    iters: int
    matrices: tuple = field(default_factory=tuple)
    layers: int = 1
    seed: int = 0


def _llama_layer(dist, dof, outlier):
    return (
        MatrixSpec("q_proj", 4096, 4096, dist, dof, outlier, "f16"),
        MatrixSpec("k_proj", 4096, 4096, dist, dof, outlier, "f16"),
        MatrixSpec("v_proj", 4096, 4096, dist, dof, outlier, "f16"),
        MatrixSpec("o_proj", 4096, 4096, dist, dof, outlier, "f16"),
        MatrixSpec("gate_proj", 11008, 4096, dist, dof, outlier, "f16"),
        MatrixSpec("up_proj", 11008, 4096, dist, dof, outlier, "f16"),
        MatrixSpec("down_proj", 4096, 11008, dist, dof, outlier, "f16"),
    )


WORKLOADS = {
    "gauss512": Workload("gauss512", 20, (MatrixSpec("w", 256, 512, "gauss", dtype="f32"),)),
    "opt125m": Workload("opt125m", 30, (
        MatrixSpec("q_proj", 768, 768, "gauss", 0, 20.0, "f32"),
        MatrixSpec("k_proj", 768, 768, "gauss", 0, 20.0, "f32"),
        MatrixSpec("v_proj", 768, 768, "gauss", 0, 20.0, "f32"),
        MatrixSpec("out_proj", 768, 768, "gauss", 0, 20.0, "f32"),
        MatrixSpec("fc1", 3072, 768, "gauss", 0, 20.0, "f32"),
        MatrixSpec("fc2", 768, 3072, "gauss", 0, 20.0, "f32"),
    )),
    "llama7b": Workload("llama7b", 30, _llama_layer("student_t", 4.0, 0.0)),
    "pythia7b": Workload("pythia7b", 30, (
        MatrixSpec("qkv_0", 4096, 4096, "gauss_lognorm_rows", 0, 0, "f16"),
        MatrixSpec("qkv_1", 4096, 4096, "gauss_lognorm_rows", 0, 0, "f16"),
        MatrixSpec("qkv_2", 4096, 4096, "gauss_lognorm_rows", 0, 0, "f16"),
        MatrixSpec("dense", 4096, 4096, "gauss_lognorm_rows", 0, 0, "f16"),
        MatrixSpec("fc_in", 16384, 4096, "gauss_lognorm_rows", 0, 0, "f16"),
        MatrixSpec("fc_out", 4096, 16384, "gauss_lognorm_rows", 0, 0, "f16"),
    )),
    "llama7b_stack": Workload("llama7b_stack", 40, _llama_layer("student_t", 3.0, 50.0), layers=32),
}

_STD = 0.02


def sign_seed(workload: Workload, layer: int, index: int) -> int:
    """Seed of the per-matrix sign mask: one mask per weight matrix (per layer)."""
    return workload.seed + 7 * layer + index


def make_matrix(workload: Workload, layer: int, index: int, rows=None) -> np.ndarray:
    """Draw matrix ``index`` of layer ``layer`` (rows x N), as float32 or float16.

    ``rows`` (a slice or an index array) draws the full matrix and returns only
    those rows, so a sampled row is identical to the same row of the full draw.
    """
    spec = workload.matrices[index]
    ss = np.random.SeedSequence([workload.seed, hash_key(workload.key), layer, index])
    g = np.random.Generator(np.random.PCG64(ss))
    m, n = spec.rows, spec.n
    if spec.dist == "gauss":
        w = g.standard_normal((m, n)) * _STD
    elif spec.dist == "student_t":
        dof = spec.dof
        w = g.standard_t(dof, size=(m, n)) * (_STD / np.sqrt(dof / (dof - 2.0)))
    elif spec.dist == "gauss_lognorm_rows":
        w = g.standard_normal((m, n)) * _STD
        w *= g.lognormal(0.0, 0.5, size=(m, 1))
    else:
        raise ValueError(spec.dist)
    if spec.outlier_scale:
        n_out = max(1, int(round(0.001 * n)))
        cols = g.choice(n, size=n_out, replace=False)
        w[:, cols] *= spec.outlier_scale
    dt = np.float16 if spec.dtype == "f16" else np.float32
    w = w.astype(dt)
    if rows is not None:
        w = np.ascontiguousarray(w[rows])
    return w


def hash_key(key: str) -> int:
    """Stable small integer from a workload name (Python's hash() is salted per process)."""
    h = 0
    for ch in key.encode():
        h = (h * 131 + ch) % (1 << 31)
    return h
