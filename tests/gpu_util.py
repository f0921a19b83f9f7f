"""Helpers for the GPU parity tests: device upload of the seeded inputs and
comparison with the oracle under the rules of tolerance.py."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import hd_inputs
import oracle
from tolerance import compare

RTOL = 1e-4          # fp32 and bf16-vs-bf16-rounded-oracle score tolerance (of ||c_k||_1)
BF16_DRIFT = 3e-2    # bf16 path against the fp32-input oracle


def torch_or_skip():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def dev(a: np.ndarray, dtype: str):
    torch = torch_or_skip()
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    bits = hd_inputs.bf16_bits(a).view(np.int16)
    return torch.from_numpy(bits).cuda().view(torch.bfloat16)


def announce(msg: str):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def check_against_oracle(X, B, C, y_gpu, S_gpu, act="hardsign", rows=None, rtol=RTOL):
    """Oracle on the same (already dtype-rounded) values, then the rule."""
    ref = oracle.infer(X, B, C, act=act, rows=rows, want_va=True)
    if rows is not None:
        y_gpu = np.asarray(y_gpu)[rows]
        S_gpu = None if S_gpu is None else np.asarray(S_gpu)[rows]
    rep = compare(S_gpu, y_gpu, ref, C, X.shape[1], rtol, act=act)
    return rep, ref
