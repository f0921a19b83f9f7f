"""Comparison rules between a GPU result and the oracle.

Scores are compared relative to ||c_k||_1 = sum_d |c_kd|, the natural scale of
a similarity with a bipolar hypervector (|h_d| = 1, Eq. 5). HardSign (Eq. 1)
turns any difference in the fp32 summation order of the encoding sum into a
+-1 flip when v is within rounding distance of zero; such "fragile"
dimensions are identified from the oracle's float64 v and the scale
a = sum_f |x_f||b_fd|, and each flip may move a score by 2|c_kd|.

Fragile set:   Fr_n = { d : |v_nd| <= gamma_F * a_nd },
               gamma_F = F u / (1 - F u), u = 2^-23
(Higham's bound for an F-term dot product, with the unit roundoff doubled
because the GPU accumulation order and the matrix-core internal rounding are
unspecified).
Score allowance: A_nk = rtol * ||c_k||_1 + 2 * sum_{d in Fr_n} |c_kd|.
Labels: equal, or the oracle's margin between the two labels lies within the
two allowances (exact ties resolve to the lowest index and must match).
"""
from __future__ import annotations

import numpy as np

U_FP32_DOUBLED = 2.0 ** -23


def gamma(F: int, u: float = U_FP32_DOUBLED) -> float:
    return F * u / (1.0 - F * u)


def score_allowance(ref, C, F: int, rtol: float, act: str = "hardsign"):
    """Per-(n, k) allowance for |S_gpu - S_oracle|."""
    C = np.asarray(C, dtype=np.float64)
    absC = np.abs(C)
    if act == "hardsign":
        fragile = np.abs(ref["V"]) <= gamma(F) * ref["A"]
        fr_mass = fragile.astype(np.float64) @ absC.T
        c1 = absC.sum(axis=1)
        return rtol * c1[None, :] + 2.0 * fr_mass, fragile
    # identity: S = V C^T; a perturbation of V bounded by gamma_F*A moves
    # s_nk by at most gamma_F * sum_d A_nd |c_kd|; the second stage adds a
    # relative rtol of sum_d |v_nd||c_kd|.
    prop = gamma(F) * (ref["A"] @ absC.T)
    scale = np.abs(ref["V"]) @ absC.T
    return prop + rtol * scale, None


def compare(S_gpu, y_gpu, ref, C, F: int, rtol: float, act: str = "hardsign",
            S_ref=None):
    """Check GPU scores/labels against oracle output ``ref`` (dict with
    y, S, V, A in float64). Returns a report dict; ``ok`` is the verdict."""
    allow, fragile = score_allowance(ref, C, F, rtol, act)
    S_or = ref["S"] if S_ref is None else S_ref
    y_or = ref["y"]
    rep = {"n": int(len(y_or))}
    if S_gpu is not None:
        S_gpu = np.asarray(S_gpu, dtype=np.float64)
        err = np.abs(S_gpu - S_or)
        rep["score_ok"] = bool(np.all(err <= allow))
        rep["score_bad"] = int(np.sum(err > allow))
        if act == "hardsign":
            c1 = np.abs(np.asarray(C, dtype=np.float64)).sum(axis=1)
            rel = err / c1[None, :]
            rep["max_rel_c1"] = float(rel.max()) if rel.size else 0.0
            rep["literal_violations"] = int(np.sum(rel > rtol))
    else:
        rep["score_ok"] = True
    y_gpu = np.asarray(y_gpu).astype(np.int64)
    idx = np.arange(len(y_or))
    in_range = (y_gpu >= 0) & (y_gpu < np.asarray(C).shape[0])
    rep["labels_in_range"] = bool(np.all(in_range))
    yg = np.clip(y_gpu, 0, np.asarray(C).shape[0] - 1)
    mism = yg != y_or
    just = S_or[idx, yg] >= S_or[idx, y_or] - (allow[idx, yg] + allow[idx, y_or])
    rep["label_mismatch"] = int(mism.sum())
    rep["label_unjustified"] = int(np.sum(mism & ~just))
    if fragile is not None:
        rep["fragile_dims"] = int(fragile.sum())
    rep["ok"] = bool(rep["score_ok"] and rep["labels_in_range"] and rep["label_unjustified"] == 0)
    return rep


def encode_allowed_mismatch(H_gpu, ref, F: int, act: str = "hardsign"):
    """For Stage I alone: positions where GPU H may differ from the oracle.

    HardSign: H must match exactly outside the fragile set. Identity: |H-V|
    must lie within gamma_F * A. Returns (ok, n_outside, n_fragile_flips)."""
    H_gpu = np.asarray(H_gpu, dtype=np.float64)
    if act == "hardsign":
        fragile = np.abs(ref["V"]) <= gamma(F) * ref["A"]
        Hor = np.where(ref["V"] >= 0, 1.0, -1.0)
        diff = H_gpu != Hor
        bad = diff & ~fragile
        return (not bad.any()), int(bad.sum()), int((diff & fragile).sum())
    err = np.abs(H_gpu - ref["V"])
    bad = err > gamma(F) * ref["A"] + 1e-30
    return (not bad.any()), int(bad.sum()), 0
