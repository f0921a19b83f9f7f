"""Pins for the oracle: checks against facts the paper and mathematics fix.

Each pin takes an ``oracle.Oracle`` instance and raises AssertionError on a
mismatch. ``test_oracle_pins.py`` runs them on the real oracle;
``test_oracle_mutants.py`` plants plausible mistakes in copies of the
oracle's C source and checks that each one trips at least one pin.

Sources of truth used here, none of which is the oracle itself:
  - a hand-worked example of Eq. 1 and Eq. 7-9 (tests/golden/hand_worked.json);
  - exact rational brute force (brute.py) on tiny inputs;
  - closed forms: a zero sample, F = 1, K = 1, a planted class;
  - library routines where the method reduces to one (numpy matmul in the
    identity-activation mode, and on small-integer inputs where float64 is
    exact);
  - invariances of Alg. 1: positive scaling of X, a joint permutation of the
    hypervector dimensions, scaling one class row, negating X;
  - the paper's own blocked decomposition (Alg. 2-4), simulated in blocked.py.
"""
from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np

import hd_inputs
from blocked import stage1, stage2_large, stage2_small
from brute import brute_infer

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _int_inputs(N, F, D, K, seed, xr=4, br=8, cr=8):
    return hd_inputs.make_integer_inputs(N, F, D, K, seed=seed, x_range=xr, b_range=br,
                                         c_range=cr)


def pin_hand_worked(orc):
    g = json.load(open(os.path.join(GOLDEN, "hand_worked.json")))
    X, B, C = (np.array(g[k], dtype=np.float64) for k in ("X", "B", "C"))
    r = orc.infer(X, B, C, want_va=True)
    assert np.array_equal(r["V"], np.array(g["V"], float)), r["V"]
    assert np.array_equal(r["S"], np.array(g["S"], float)), r["S"]
    assert np.array_equal(r["y"], np.array(g["y"])), r["y"]
    e = orc.encode(X, B)
    assert np.array_equal(e["H"], np.array(g["H"], float)), e["H"]
    ri = orc.infer(X, B, C, act="identity")
    assert np.array_equal(ri["S"], np.array(g["S_identity"], float)), ri["S"]
    assert np.array_equal(ri["y"], np.array(g["y_identity"])), ri["y"]


def pin_bruteforce_float(orc):
    """Random fp32 and bf16 values on tiny shapes against exact rationals."""
    for seed in range(12):
        rng = np.random.default_rng(100 + seed)
        N, F, D, K = (int(v) for v in rng.integers(1, [5, 9, 17, 5], endpoint=True))
        X, B, C = hd_inputs.make_inputs(N, F, D, K, "normal", seed=seed,
                                        dtype="bf16" if seed % 2 else "f32")
        ex = brute_infer(X, B, C)
        r = orc.infer(X, B, C, want_va=True)
        for n in range(N):
            for d in range(D):
                v, a = ex["V"][n][d], ex["A"][n][d]
                # float64 sums of <= 8 exact products: error <= 8 * 2^-53 * a
                assert abs(Fraction(r["V"][n, d]) - v) <= Fraction(2) ** -49 * a + Fraction(0)
                assert Fraction(r["A"][n, d]) == a or abs(Fraction(r["A"][n, d]) - a) <= Fraction(2) ** -49 * a
            for k in range(K):
                s = ex["S"][n][k]
                c1 = sum(abs(Fraction(float(c))) for c in C[k])
                assert abs(Fraction(r["S"][n, k]) - s) <= Fraction(2) ** -40 * c1, (n, k)
        srt = [sorted(s, reverse=True) for s in ex["S"]]
        for n in range(N):
            if K == 1 or srt[n][0] - srt[n][1] > 0:
                assert r["y"][n] == ex["y"][n], (seed, n)


def pin_bruteforce_ties(orc):
    """Inputs in {-1, 0, 1}: many encoding sums are exactly 0 (HardSign tie)
    and many scores tie (argmax tie). Everything is exact in float64."""
    for seed in range(10):
        rng = np.random.default_rng(200 + seed)
        N, F, D, K = (int(v) for v in rng.integers(1, [6, 7, 20, 6], endpoint=True))
        X, B, C = _int_inputs(N, F, D, K, seed, 1, 1, 1)
        ex = brute_infer(X, B, C)
        r = orc.infer(X, B, C, want_va=True)
        assert np.array_equal(r["V"], np.array(ex["V"], dtype=float))
        assert np.array_equal(r["S"], np.array(ex["S"], dtype=float)), seed
        assert np.array_equal(r["y"], np.array(ex["y"])), seed
        e = orc.encode(X, B)
        assert np.array_equal(e["H"], np.array(ex["H"], dtype=float))


def pin_zero_sample(orc):
    """x = 0 gives v = 0, so HardSign makes h all +1 and s_k = sum_d c_kd."""
    X, B, C = hd_inputs.make_inputs(3, 37, 129, 7, seed=5)
    X[1] = 0.0
    Ci = np.round(C * 8)  # integers: the row sums are exact
    r = orc.infer(X, B, Ci)
    assert np.array_equal(r["S"][1], Ci.sum(axis=1))
    assert r["y"][1] == int(np.argmax(Ci.sum(axis=1)))


def pin_single_feature(orc):
    """F = 1: h_d = HardSign(x b_d). For x > 0 that is HardSign(b_d) for
    every x, so all positive samples share one score vector and label."""
    B = np.array([[0.5, -1.0, 0.0, 2.0, -0.25, 3.0]])
    C = np.array([[1.0, 2.0, -1.0, 0.5, 4.0, -2.0],
                  [-1.0, 1.0, 3.0, 1.0, -2.0, 1.0]])
    X = np.array([[0.1], [7.0], [1e-3], [-2.0]])
    r = orc.infer(X, B, C)
    hpos = np.where(B[0] >= 0, 1.0, -1.0)
    spos = C @ hpos
    for n in range(3):
        assert np.array_equal(r["S"][n], spos)
        assert r["y"][n] == int(np.argmax(spos))
    # x < 0: x*b_d >= 0 exactly when b_d <= 0
    hneg = np.where(B[0] <= 0, 1.0, -1.0)
    assert np.array_equal(r["S"][3], C @ hneg)


def pin_single_class(orc):
    X, B, C = hd_inputs.make_inputs(9, 13, 64, 1, seed=3)
    assert np.all(orc.infer(X, B, C)["y"] == 0)


def pin_planted_class(orc):
    """If C[k*] equals the encoded sample (bipolar), s_nk* = D, the largest
    value any bipolar or bounded row can reach; other rows are bipolar and
    differ from it, so k* is the strict argmax."""
    N, F, D, K = 4, 31, 257, 5
    X, B, _ = _int_inputs(N, F, D, K, seed=11)
    V = X.astype(np.float64) @ B.astype(np.float64)  # exact on small integers
    H = np.where(V >= 0, 1.0, -1.0)
    rng = np.random.default_rng(7)
    for n in range(N):
        C = rng.choice([-1.0, 1.0], size=(K, D))
        ks = int(rng.integers(0, K))
        C[ks] = H[n]
        for k in range(K):
            if k != ks and np.array_equal(C[k], H[n]):
                C[k, 0] = -C[k, 0]
        r = orc.infer(X, B, C)
        assert r["S"][n, ks] == D
        assert r["y"][n] == ks
        assert np.all(np.delete(r["S"][n], ks) < D)


def pin_identity_matmul(orc):
    """Without HardSign, Alg. 1 is S = X B C^T; compare with numpy's matmul
    in the other association, X (B C^T)."""
    X, B, C = hd_inputs.make_inputs(6, 45, 300, 4, "normal", seed=9)
    r = orc.infer(X, B, C, act="identity")
    Xd, Bd, Cd = (a.astype(np.float64) for a in (X, B, C))
    S_ref = Xd @ (Bd @ Cd.T)
    scale = np.abs(Xd) @ (np.abs(Bd) @ np.abs(Cd).T)
    assert np.all(np.abs(r["S"] - S_ref) <= 1e-12 * scale)
    assert np.array_equal(r["y"], np.argmax(S_ref, axis=1))
    Xi, Bi, Ci = _int_inputs(5, 23, 99, 3, seed=4)
    ri = orc.infer(Xi, Bi, Ci, act="identity")
    assert np.array_equal(ri["S"], Xi.astype(float) @ (Bi.astype(float) @ Ci.astype(float).T))


def pin_encoding_scale(orc):
    """Eq. 2 summed and A = |X||B|: exact against numpy on small integers."""
    X, B, C = _int_inputs(7, 40, 90, 3, seed=2)
    r = orc.infer(X, B, C, want_va=True)
    assert np.array_equal(r["V"], X.astype(float) @ B.astype(float))
    assert np.array_equal(r["A"], np.abs(X).astype(float) @ np.abs(B).astype(float))


def pin_positive_scaling(orc):
    """HardSign(alpha v) = HardSign(v) for alpha > 0: scaling X changes no
    score or label (exact for integer inputs and for powers of two)."""
    X, B, C = _int_inputs(8, 33, 140, 5, seed=6)
    r0 = orc.infer(X, B, C)
    for alpha in (3.0, 0.5, 1024.0):
        r1 = orc.infer(alpha * X, B, C)
        assert np.array_equal(r0["S"], r1["S"]) and np.array_equal(r0["y"], r1["y"])
    Xf, Bf, Cf = hd_inputs.make_inputs(5, 61, 200, 6, seed=8)
    a0 = orc.infer(Xf, Bf, Cf)
    a1 = orc.infer(Xf * 0.25, Bf, Cf)
    assert np.array_equal(a0["S"], a1["S"]) and np.array_equal(a0["y"], a1["y"])


def pin_dimension_permutation(orc):
    """Permuting the D hypervector dimensions of B and C together leaves
    every score unchanged (Eq. 8 sums over d)."""
    X, B, C = _int_inputs(6, 29, 173, 4, seed=12)
    perm = np.random.default_rng(3).permutation(B.shape[1])
    r0 = orc.infer(X, B, C)
    r1 = orc.infer(X, B[:, perm], C[:, perm])
    assert np.array_equal(r0["S"], r1["S"]) and np.array_equal(r0["y"], r1["y"])


def pin_negation(orc):
    """Negating X negates v; HardSign then flips h except where v = 0, which
    stays +1. So S(-X) = -S(X) + 2 sum_{d: v_d = 0} c_kd (exact on integers)."""
    X, B, C = _int_inputs(6, 9, 300, 4, seed=13, xr=1, br=1)
    V = X.astype(float) @ B.astype(float)
    zero_mass = (V == 0).astype(float) @ C.astype(float).T
    assert zero_mass.any(), "fixture should contain v = 0 dimensions"
    r0 = orc.infer(X, B, C)
    r1 = orc.infer(-X, B, C)
    assert np.array_equal(r1["S"], -r0["S"] + 2.0 * zero_mass)


def pin_class_row_scaling(orc):
    X, B, C = _int_inputs(5, 17, 64, 4, seed=14)
    r0 = orc.infer(X, B, C)
    C2 = C.astype(float).copy()
    C2[2] *= 4.0
    r1 = orc.infer(X, B, C2)
    assert np.array_equal(r1["S"][:, 2], 4.0 * r0["S"][:, 2])
    assert np.array_equal(np.delete(r1["S"], 2, axis=1), np.delete(r0["S"], 2, axis=1))


def pin_duplicate_class(orc):
    """Equal class rows give equal scores; the label is the lower index."""
    X, B, C = hd_inputs.make_inputs(16, 20, 128, 4, seed=15)
    best = orc.infer(X, B, C)["y"]
    for n in range(16):
        k = int(best[n])
        Cdup = np.vstack([C[:k], C[k:k + 1], C[k:]])  # a copy of row k inserted before it
        r1 = orc.infer(X[n:n + 1], B, Cdup)
        assert r1["y"][0] == k
        assert r1["S"][0, k] == r1["S"][0, k + 1]


def pin_blocked_equivalence(orc):
    """The paper's blocked Stage I (Alg. 2) and both Stage II variants
    (Alg. 3, Alg. 4) give exactly the plain definition on exact inputs."""
    rng = np.random.default_rng(21)
    for trial in range(6):
        N, F, D, K = (int(v) for v in rng.integers([1, 1, 1, 1], [40, 50, 90, 12]))
        X, B, C = _int_inputs(N, F, D, K, seed=30 + trial, xr=2, br=3, cr=5)
        n, f, d, k = (int(v) for v in rng.integers(1, 9, size=4))
        R, T = int(rng.integers(1, 5)), int(rng.integers(1, 6))
        H = stage1(X.astype(float), B.astype(float), n, f, d, R, T)
        J = C.astype(float).T
        r = orc.infer(X, B, C)
        S_s, y_s = stage2_small(H, J, n, d, k, T)
        S_l, y_l = stage2_large(H, J, n, d, k, T)
        assert np.array_equal(r["S"], S_s) and np.array_equal(r["y"], y_s), trial
        assert np.array_equal(r["S"], S_l) and np.array_equal(r["y"], y_l), trial


def pin_row_subset(orc):
    X, B, C = hd_inputs.make_inputs(20, 30, 100, 5, seed=16)
    full = orc.infer(X, B, C, want_va=True)
    rows = [19, 0, 7, 7, 3]
    sub = orc.infer(X, B, C, rows=rows, want_va=True)
    assert np.array_equal(sub["S"], full["S"][rows])
    assert np.array_equal(sub["y"], full["y"][rows])
    assert np.array_equal(sub["V"], full["V"][rows])


def pin_stages_compose(orc):
    """Stage I then Stage II alone equal Alg. 1 end to end."""
    X, B, C = hd_inputs.make_inputs(11, 25, 77, 6, seed=17)
    for act in ("hardsign", "identity"):
        full = orc.infer(X, B, C, act=act)
        H = orc.encode(X, B, act=act)["H"]
        s2 = orc.similarity(H, C)
        assert np.array_equal(s2["S"], full["S"]) and np.array_equal(s2["y"], full["y"])


PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
