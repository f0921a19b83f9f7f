"""Helpers for the GPU parity tests: device upload of the seeded inputs and
comparison with the oracle under the rules of tolerance.py."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import hd_inputs
import oracle
from tolerance import compare, drift_scale, score_scale
from tolerance import score_allowance as tolerance_allowance

RTOL = 1e-4          # fp32 and bf16-vs-bf16-rounded-oracle score tolerance (of ||c_k||_2)
BF16_DRIFT = 3e-2    # bf16 path against the fp32-input oracle (of ||c_k||_1)


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


def check_all_rows(X, B, C, y_gpu, S_gpu, chunk=4096, rtol=RTOL):
    """Every row of a large batch against the oracle, in row chunks.

    Each chunk is first checked with the oracle's labels and scores alone and
    the rule without its fragile-set term (half the oracle's work, and never
    looser than the full rule); the rows that this flags are checked again
    under the full rule, with v and a from the oracle. Returns a summary
    report whose ``ok`` is the verdict over all rows."""
    N = X.shape[0]
    total = {"n": N, "rechecked": 0, "label_mismatch": 0, "label_unjustified": 0,
             "score_bad": 0, "max_rel_c2": 0.0, "ok": True}
    S_gpu = None if S_gpu is None else np.asarray(S_gpu, dtype=np.float64)
    y_gpu = np.asarray(y_gpu)
    for r0 in range(0, N, chunk):
        print(f"[rows] {r0}..{min(N, r0 + chunk)} of {N}", flush=True)
        rows = np.arange(r0, min(N, r0 + chunk))
        ref = oracle.infer(X, B, C, rows=rows)
        Sg = None if S_gpu is None else S_gpu[rows]
        yg = y_gpu[rows]
        allow, _ = tolerance_allowance(ref, C, X.shape[1], rtol)
        bad = np.zeros(len(rows), dtype=bool)
        if Sg is not None:
            err = np.abs(Sg - ref["S"])
            bad |= (err > allow).any(axis=1)
            total["max_rel_c2"] = max(total["max_rel_c2"], float(
                (err / score_scale(C)[None, :]).max()))
        bad |= yg.astype(np.int64) != ref["y"]
        if bad.any():
            sub = rows[bad]
            total["rechecked"] += int(len(sub))
            rep, _ = check_against_oracle(X, B, C, y_gpu, S_gpu, rows=sub, rtol=rtol)
            for k in ("label_mismatch", "label_unjustified", "score_bad"):
                total[k] += int(rep.get(k, 0))
            total["ok"] = total["ok"] and rep["ok"]
    return total
