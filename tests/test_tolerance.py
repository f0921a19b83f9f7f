"""CPU checks of the comparison rule itself (tolerance.py): it must accept
the oracle's own result and the HardSign flips that rounding can cause, and
reject the plausible kernel mistakes it exists to catch (one hypervector
dimension dropped or counted twice, one flip outside the fragile set, a wrong
label)."""
import numpy as np

import hd_inputs
import oracle
from tolerance import compare, drift_scale, gamma, score_scale

RTOL = 1e-4


def _case(N=24, F=561, D=10240, K=6, seed=0):
    X, B, C = hd_inputs.make_inputs(N, F, D, K, "uniform_pm1", seed=seed)
    ref = oracle.infer(X, B, C, want_va=True)
    H = np.where(ref["V"] >= 0, 1.0, -1.0)
    return X, B, C.astype(np.float64), ref, H


def test_oracle_against_itself_passes():
    X, B, C, ref, _ = _case()
    rep = compare(ref["S"], ref["y"], ref, C, X.shape[1], RTOL)
    assert rep["ok"] and rep["literal_violations"] == 0


def test_dropped_or_doubled_dimension_fails():
    """S computed with one dimension d left out (or added twice) must fail for
    most choices of d: the rule's scale is ||c_k||_2, not ||c_k||_1."""
    X, B, C, ref, H = _case()
    rng = np.random.default_rng(1)
    caught = 0
    trials = 40
    for _ in range(trials):
        d = int(rng.integers(0, C.shape[1]))
        sign = rng.choice([-1.0, 1.0])  # -1 drops the term, +1 counts it twice
        S = ref["S"] + sign * np.outer(H[:, d], C[:, d])
        rep = compare(S, ref["y"], ref, C, X.shape[1], RTOL)
        caught += not rep["ok"]
    # only a term with every |c_kd| below rtol * ||c_k||_2 (about 0.01) escapes
    assert caught >= trials - 1, caught


def test_flip_outside_fragile_set_fails_inside_passes():
    X, B, C, ref, H = _case()
    F = X.shape[1]
    fragile = np.abs(ref["V"]) <= gamma(F) * ref["A"]
    n = 3
    solid = np.flatnonzero(~fragile[n])
    d = int(solid[np.argmax(np.abs(C[:, solid]).min(axis=0))])
    S = ref["S"].copy()
    S[n] -= 2.0 * H[n, d] * C[:, d]
    assert not compare(S, ref["y"], ref, C, F, RTOL)["ok"]
    # the same flip on a dimension whose v lies within rounding distance of
    # zero (same sign, so the oracle's H and S are unchanged) is explained
    ref2 = {k: v.copy() for k, v in ref.items()}
    ref2["V"][n, d] = np.copysign(1e-12, ref["V"][n, d])
    rep = compare(S, ref["y"], ref2, C, F, RTOL)
    assert rep["ok"] and rep["flips"] == 1, rep


def test_two_fragile_flips_explained_not_a_wrong_move():
    X, B, C, ref, H = _case()
    F = X.shape[1]
    n = 5
    ref2 = {k: v.copy() for k, v in ref.items()}
    ds = [100, 2000]
    for d in ds:
        ref2["V"][n, d] = np.copysign(1e-12, ref["V"][n, d])
    S = ref["S"].copy()
    for d in ds:
        S[n] -= 2.0 * H[n, d] * C[:, d]
    rep = compare(S, ref["y"], ref2, C, F, RTOL)
    assert rep["ok"] and rep["flips"] == 2, rep
    # the flips' moves with the wrong sign are not flips of those dimensions
    S = ref["S"].copy()
    for d in ds:
        S[n] += 2.0 * H[n, d] * C[:, d]
    assert not compare(S, ref["y"], ref2, C, F, RTOL)["ok"]
    # one class off by three tolerances, the others exact
    S = ref["S"].copy()
    S[n, 2] += 3 * RTOL * np.sqrt((C[2] ** 2).sum())
    assert not compare(S, ref["y"], ref2, C, F, RTOL)["ok"]


def test_wrong_label_fails_unless_margin_inside_allowance():
    X, B, C, ref, _ = _case()
    y = ref["y"].copy()
    S = ref["S"]
    order = np.argsort(S, axis=1)
    margin = S[np.arange(len(y)), order[:, -1]] - S[np.arange(len(y)), order[:, -2]]
    n = int(np.argmax(margin))
    y[n] = order[n, -2]
    assert not compare(S, y, ref, C, X.shape[1], RTOL)["ok"]


def test_rule_without_fragile_term_is_never_looser():
    X, B, C, ref, H = _case(N=8)
    no_va = {"S": ref["S"], "y": ref["y"]}
    rng = np.random.default_rng(2)
    for _ in range(20):
        S = ref["S"] + rng.normal(0, 2e-3, ref["S"].shape)
        if compare(S, ref["y"], no_va, C, X.shape[1], RTOL)["ok"]:
            assert compare(S, ref["y"], ref, C, X.shape[1], RTOL)["ok"]


def test_scales():
    C = np.array([[3.0, -4.0], [1.0, 1.0]])
    assert np.allclose(score_scale(C), [5.0, np.sqrt(2.0)])
    assert np.allclose(drift_scale(C), [7.0, 2.0])


def test_bf16_drift_scale_is_attainable():
    """The exact result on bf16-rounded inputs meets the 3e-2 drift bound on
    the ||c_k||_1 scale (and not on ||c_k||_2: the reason for the scale)."""
    w = hd_inputs.WORKLOADS["speech"]
    X32, B32, C32 = hd_inputs.make_inputs(64, w.F, w.D, w.K, w.x_dist, seed=0)
    Xb, Bb, Cb = hd_inputs.make_inputs(64, w.F, w.D, w.K, w.x_dist, seed=0, dtype="bf16")
    d = np.abs(oracle.infer(Xb, Bb, Cb)["S"] - oracle.infer(X32, B32, C32)["S"])
    assert (d / drift_scale(C32)[None, :]).max() <= 3e-2
    assert (d / score_scale(C32)[None, :]).max() > 3e-2
