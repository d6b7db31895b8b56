"""Seeded synthetic inputs, shared by the tests, the smoke check and the bench.

numpy only.  This module holds none of the method's arithmetic: it draws the
operand values, rounds them to fp16 and lays them out in memory.  Both the
HIP path and the CPU oracle consume what it produces.

Value recipe: values are drawn in float64 from ``numpy.random.default_rng``
and rounded to the nearest fp16 (ties to even) by ``astype(float16)``.  Seeds
for workload number c are 100*c + 1 (A), 100*c + 2 (B) and 100*c + 3 (bias).
The paper measured on random problem sizes only (Experimental Evaluation
section), so these synthetic operands are the whole workload.
"""
from dataclasses import dataclass, field
from typing import Tuple

import numpy as np

ROW, COL = 0, 1
LAYOUT_NAMES = {"RR": (ROW, ROW), "RC": (ROW, COL), "CR": (COL, ROW), "CC": (COL, COL)}


def uniform_f16(seed: int, shape: Tuple[int, ...], lo: float = -1.0, hi: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.uniform(lo, hi, size=shape).astype(np.float16)


def normal_f16(seed: int, shape: Tuple[int, ...], std: float) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.normal(0.0, std, size=shape).astype(np.float16)


def integer_f16(seed: int, shape: Tuple[int, ...], lo: int, hi: int) -> np.ndarray:
    """Integers in [lo, hi] stored as fp16 (exact for |v| <= 2048)."""
    rng = np.random.default_rng(seed)
    return rng.integers(lo, hi + 1, size=shape).astype(np.float16)


def store(logical: np.ndarray, layout: int, ld: int = None) -> np.ndarray:
    """Lay a logical rows x cols matrix out in memory as a 2-D array.

    Row-major: shape (rows, ld), element (r, c) at [r, c].
    Column-major: shape (cols, ld), element (r, c) at [c, r].
    Padding columns (beyond the extent) are filled with NaN bit patterns so a
    reader that strays into them is caught.
    """
    rows, cols = logical.shape
    if layout == ROW:
        ext, data = cols, logical
    else:
        ext, data = rows, logical.T
    ld = ext if ld is None else ld
    if ld < ext:
        raise ValueError("leading dimension smaller than the extent")
    out = np.full((data.shape[0], ld), np.float16(np.nan), dtype=np.float16)
    out[:, :ext] = data
    return out


@dataclass
class Workload:
    name: str
    M: int
    N: int
    K: int
    layouts: Tuple[str, ...] = ("RC",)
    dist: str = "uniform"          # "uniform" U[-1,1] or "mlp" N(0, 1/sqrt(K)), bias N(0, 0.1)
    accum: Tuple[str, ...] = ("f32",)
    seed_base: int = 0
    extra: dict = field(default_factory=dict)


# The five workload families: a 128^3 check, 1024^3 in all four layouts,
# 4096^3 (plain, fused and unfused), two MLP-layer shapes, and small-M
# inference shapes plus a ragged 1000^3.
WORKLOADS = {
    "cube128_RC": Workload("cube128_RC", 128, 128, 128, ("RC",), "uniform", ("f32",), 100),
    "cube1024_all_layouts": Workload("cube1024_all_layouts", 1024, 1024, 1024,
                                     ("RR", "RC", "CR", "CC"), "uniform", ("f32",), 200),
    "cube4096_RC": Workload("cube4096_RC", 4096, 4096, 4096, ("RC",), "uniform", ("f32",), 300),
    "mlp_up_8192x4096x1024": Workload("mlp_up_8192x4096x1024", 8192, 4096, 1024, ("RC",), "mlp",
                                      ("f32",), 400),
    "mlp_down_8192x1024x4096": Workload("mlp_down_8192x1024x4096", 8192, 1024, 4096, ("RC",), "mlp",
                                        ("f32",), 410),
    "infer_m32_n4096_k1024": Workload("infer_m32_n4096_k1024", 32, 4096, 1024, ("RC",), "uniform",
                                      ("f32", "f16"), 500),
    "infer_m128_n4096_k1024": Workload("infer_m128_n4096_k1024", 128, 4096, 1024, ("RC",), "uniform",
                                       ("f32", "f16"), 510),
    "infer_m256_n4096_k1024": Workload("infer_m256_n4096_k1024", 256, 4096, 1024, ("RC",), "uniform",
                                       ("f32", "f16"), 520),
    "ragged1000": Workload("ragged1000", 1000, 1000, 1000, ("RR", "RC", "CR", "CC"), "uniform",
                           ("f32", "f16"), 530),
    # the other idioms at the headline shape: relu(A).B + bias -> ReLU
    # (prologue), and A.B + P.Q + bias -> ReLU with K2 = K (sum of matmuls)
    "prologue4096_RC": Workload("prologue4096_RC", 4096, 4096, 4096, ("RC",), "uniform", ("f32",),
                                600, {"prologue": "relu"}),
    "sum4096_RC": Workload("sum4096_RC", 4096, 4096, 4096, ("RC",), "uniform", ("f32",), 610,
                           {"second": "add", "K2": 4096}),
}


def second_inputs(w: Workload):
    """Logical P (M x K2) and Q (K2 x N) of a sum-of-matmuls workload,
    drawn like A and B."""
    K2 = w.extra["K2"]
    s = w.seed_base + 10
    if w.dist == "uniform":
        return uniform_f16(s + 1, (w.M, K2)), uniform_f16(s + 2, (K2, w.N))
    std = 1.0 / np.sqrt(K2)
    return normal_f16(s + 1, (w.M, K2), std), normal_f16(s + 2, (K2, w.N), std)


def logical_inputs(w: Workload):
    """Logical fp16 A (M x K), B (K x N) and bias (N,) for a workload."""
    s = w.seed_base
    if w.dist == "uniform":
        A = uniform_f16(s + 1, (w.M, w.K))
        B = uniform_f16(s + 2, (w.K, w.N))
        bias = uniform_f16(s + 3, (w.N,))
    elif w.dist == "mlp":
        std = 1.0 / np.sqrt(w.K)
        A = normal_f16(s + 1, (w.M, w.K), std)
        B = normal_f16(s + 2, (w.K, w.N), std)
        bias = normal_f16(s + 3, (w.N,), 0.1)
    else:
        raise ValueError(w.dist)
    return A, B, bias


def random_problem(seed: int, M: int, N: int, K: int, dist: str = "uniform"):
    """Logical A, B, bias for an arbitrary shape: uniform[-1,1], integer
    ({-1,0,1} operands, bias in -8..8) or mlp (N(0, 1/sqrt(K)), bias
    N(0, 0.1)) data."""
    if dist == "mlp":
        std = 1.0 / np.sqrt(max(K, 1))
        return (normal_f16(seed + 1, (M, K), std), normal_f16(seed + 2, (K, N), std),
                normal_f16(seed + 3, (N,), 0.1))
    if dist == "uniform":
        return (uniform_f16(seed + 1, (M, K)), uniform_f16(seed + 2, (K, N)),
                uniform_f16(seed + 3, (N,)))
    if dist == "int":
        return (integer_f16(seed + 1, (M, K), -1, 1), integer_f16(seed + 2, (K, N), -1, 1),
                integer_f16(seed + 3, (N,), -8, 8))
    raise ValueError(dist)


def sweep_shapes(seed: int = 2006, count: int = 100, step: int = 128, top: int = 4096):
    """Random problem sizes, each a multiple of ``step`` up to ``top``.

    Mirrors the evaluation protocol of random sizes that are multiples of the
    largest tile (Experimental Evaluation section).
    """
    rng = np.random.default_rng(seed)
    return [tuple(int(v) for v in rng.integers(1, top // step + 1, size=3) * step)
            for _ in range(count)]
