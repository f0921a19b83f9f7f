"""Seeded synthetic inputs for batched HDC inference.

This module only draws random numbers and rounds them to the storage format;
it holds none of the inference arithmetic. It is the one piece of code that
both the CPU oracle's tests and the GPU path's tests/bench import, so that
the two sides see bit-identical inputs.

Shapes follow the paper's problem statement (Alg. 1): X[N, F] raw features,
B[F, D] base hypervectors, C[K, D] class hypervectors (the paper's M). B is
Gaussian as at initialisation of the nonlinear encoding (Sec. II-B). The
paper's datasets (Table I) are not available; the workloads below are
synthetic stand-ins with the (F, K) shapes of those datasets.

Seeding: one ``numpy.random.SeedSequence(seed)`` is spawned into three
independent generators (X, B, C), so B and C stay identical across a sweep
over N for a fixed (F, D, K, seed).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "make_model",
    "make_x",
    "make_inputs",
    "make_integer_inputs",
    "round_bf16",
    "bf16_bits",
]


@dataclass(frozen=True)
class Workload:
    """A named synthetic workload: sizes plus the distribution of X."""

    name: str
    N: int
    F: int
    D: int
    K: int
    x_dist: str  # "uniform_pm1" | "uniform01" | "uniform01_zero20" | "normal"
    dtypes: tuple = ("f32",)
    note: str = ""


# Activity-recognition-shaped (F=561 echoes SA12's feature count), image-shaped
# (F=784, K=10 echoes MNIST), speech-letter-shaped (F=617, K=26 echoes
# ISOLET), colour-image-shaped (F=3072, K=10/100). D=10240 throughout except
# the tiny case; the paper itself uses D=10000 (Sec. IV-A), which the tests
# keep as a boundary shape.
WORKLOADS = {
    "tiny": Workload("tiny", 64, 561, 2048, 6, "uniform_pm1", ("f32", "bf16"),
                     "tiny HDC inference, oracle well under a second"),
    "activity_n1": Workload("activity_n1", 1, 561, 10240, 6, "uniform_pm1", ("f32",),
                            "activity-recognition-shaped, single sample"),
    "activity_n32": Workload("activity_n32", 32, 561, 10240, 6, "uniform_pm1", ("f32",),
                             "activity-recognition-shaped, small batch"),
    "image": Workload("image", 4096, 784, 10240, 10, "uniform01_zero20", ("f32", "bf16"),
                      "28x28 grayscale-shaped, 20% exact zeros"),
    "speech": Workload("speech", 65536, 617, 10240, 26, "normal", ("bf16",),
                       "speech-letter-shaped large batch"),
    "colour_k10": Workload("colour_k10", 16384, 3072, 10240, 10, "uniform01", ("bf16", "f32"),
                           "colour-image-shaped, wide features"),
    "colour_k100": Workload("colour_k100", 16384, 3072, 10240, 100, "uniform01", ("bf16", "f32"),
                            "colour-image-shaped, 100 classes"),
    "colour_n1": Workload("colour_n1", 1, 3072, 10240, 10, "uniform01", ("f32", "bf16"),
                          "colour-image-shaped single sample; base of the D sweep 2048..20480"),
}

# D values of the single-sample bandwidth sweep (bench.py --sweep-d)
D_SWEEP = (2048, 4096, 8192, 10240, 16384, 20480)

# batch sizes of the samples/s curve at D = 10240 (bench.py --sweep-n, activity shape)
N_SWEEP = (1, 2, 4, 8, 16, 32, 64, 65, 128, 256, 1024, 4096, 16384, 65536)


def _generators(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.default_rng(s) for s in ss.spawn(3)]


def make_x(N: int, F: int, dist: str, seed: int = 0) -> np.ndarray:
    """Draw X[N, F] as float32 from the X generator of ``seed``."""
    gX, _, _ = _generators(seed)
    if dist == "uniform_pm1":
        X = gX.uniform(-1.0, 1.0, (N, F)).astype(np.float32)
    elif dist == "uniform01":
        X = gX.random((N, F), dtype=np.float32)
    elif dist == "uniform01_zero20":
        X = gX.random((N, F), dtype=np.float32)
        mask = gX.random((N, F)) < 0.2
        X[mask] = 0.0
    elif dist == "normal":
        X = gX.standard_normal((N, F), dtype=np.float32)
    else:
        raise ValueError(f"unknown X distribution {dist!r}")
    return np.ascontiguousarray(X)


def make_model(F: int, D: int, K: int, seed: int = 0):
    """Draw B[F, D] and C[K, D] as float32 standard normals."""
    _, gB, gC = _generators(seed)
    B = gB.standard_normal((F, D), dtype=np.float32)
    C = gC.standard_normal((K, D), dtype=np.float32)
    return np.ascontiguousarray(B), np.ascontiguousarray(C)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even).

    Returns the raw 16-bit patterns as uint16. NaN stays NaN (quiet).
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        rounded[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return rounded


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Float32 array holding the bfloat16-rounded values of ``a`` (exact)."""
    bits = bf16_bits(a).astype(np.uint32) << 16
    return bits.view(np.float32)


def make_inputs(N: int, F: int, D: int, K: int, x_dist: str = "uniform_pm1",
                seed: int = 0, dtype: str = "f32"):
    """Return (X, B, C) float32 arrays; for dtype "bf16" the values are the
    bfloat16-rounded ones (still stored as float32 so both sides can widen
    them exactly)."""
    X = make_x(N, F, x_dist, seed)
    B, C = make_model(F, D, K, seed)
    if dtype == "bf16":
        X, B, C = round_bf16(X), round_bf16(B), round_bf16(C)
    elif dtype != "f32":
        raise ValueError(dtype)
    return X, B, C


def make_integer_inputs(N: int, F: int, D: int, K: int, seed: int = 0,
                        x_range: int = 4, b_range: int = 8, c_range: int = 8):
    """Small-integer inputs (exact in bf16 and fp32).

    X ~ U{-x_range..x_range}, B ~ U{-b_range..b_range}, C ~ U{-c_range..c_range}.
    With |X|<=4, |B|<=8, F<=3072 every partial sum of the encoding stays below
    2^24 and every partial similarity below 2^24 for D<=20480, so any
    summation order is exact in fp32.
    """
    gX, gB, gC = _generators(seed)
    X = gX.integers(-x_range, x_range + 1, (N, F)).astype(np.float32)
    B = gB.integers(-b_range, b_range + 1, (F, D)).astype(np.float32)
    C = gC.integers(-c_range, c_range + 1, (K, D)).astype(np.float32)
    return np.ascontiguousarray(X), np.ascontiguousarray(B), np.ascontiguousarray(C)


def make_int8_inputs(N: int, F: int, D: int, K: int, seed: int = 0, lo: int = -128,
                     hi: int = 127):
    """int8 inputs X[N, F], B[F, D], C[K, D] ~ U{lo..hi} (the int8 model
    variant); returned as int8 arrays."""
    gX, gB, gC = _generators(seed)
    X = gX.integers(lo, hi + 1, (N, F)).astype(np.int8)
    B = gB.integers(lo, hi + 1, (F, D)).astype(np.int8)
    C = gC.integers(lo, hi + 1, (K, D)).astype(np.int8)
    return np.ascontiguousarray(X), np.ascontiguousarray(B), np.ascontiguousarray(C)
