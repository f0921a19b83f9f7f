"""Pins for the oracle's single-pass training (Sec. II-C): the codebook row
of class k is HardSign of the sum of the encoded hypervectors of the samples
labelled k (normalised bundling, Sec. II-A; ties to +1, Eq. 1).

Sources of truth, none of which is the oracle's own arithmetic:
  - exact rational brute force (brute.py) of the encoding, on tiny inputs;
  - closed forms: a class with a single sample reproduces that sample's
    encoding, which then scores D against it (the planted-class round trip
    through inference); an empty class is all +1; identical samples;
  - invariants: relabelling the classes permutes the rows, the class sums
    add up to the column sums of the encodings, labels outside [0, K) are
    ignored.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

import hd_inputs
from brute import brute_infer


def _tiny(seed, N, F, D, K, ints=False):
    if ints:
        X, B, _ = hd_inputs.make_integer_inputs(N, F, D, 1, seed=seed, x_range=1, b_range=1)
    else:
        X, B, _ = hd_inputs.make_inputs(N, F, D, 1, "normal", seed=seed)
    y = np.random.default_rng(seed + 1).integers(0, K, N).astype(np.int32)
    return X, B, y


def _brute_counts(X, B, y, K):
    H = brute_infer(X, B, np.zeros((1, B.shape[1]), np.float32))["H"]
    D = B.shape[1]
    counts = [[0] * D for _ in range(K)]
    for n, k in enumerate(y):
        if 0 <= k < K:
            for d in range(D):
                counts[k][d] += int(H[n][d])
    return counts, H


def pin_train_bruteforce(orc):
    """Random fp32 and {-1, 0, 1} inputs (many encoding sums exactly 0, many
    tied class sums) against exact rationals, including an empty class."""
    for seed in range(8):
        ints = seed % 2 == 1
        X, B, y = _tiny(seed, 7, 4, 11, 4, ints=ints)
        y[y == 3] = 2  # class 3 stays empty
        r = orc.bundle(X, B, y, 4)
        counts, _ = _brute_counts(X, B, y, 4)
        assert np.array_equal(r["counts"], np.array(counts)), seed
        M = [[1.0 if Fraction(c) >= 0 else -1.0 for c in row] for row in counts]
        assert np.array_equal(r["M"], np.array(M)), seed
        assert np.all(r["M"][3] == 1.0) and np.all(r["counts"][3] == 0)


def pin_train_single_sample_class_round_trip(orc):
    """A class with one sample gets that sample's encoding as its codebook
    row (HardSign of a bipolar vector is itself), so inference with the
    trained codebook scores that sample D on its class: the largest score a
    bipolar row can reach."""
    N, F, D = 6, 23, 301
    X, B, _ = hd_inputs.make_inputs(N, F, D, 1, "normal", seed=31)
    y = np.arange(N, dtype=np.int32)  # one sample per class
    r = orc.bundle(X, B, y, N)
    ex = brute_infer(X, B, np.zeros((1, D), np.float32))
    assert np.array_equal(r["M"], np.array(ex["H"], dtype=float))
    assert np.array_equal(np.abs(r["counts"]), np.ones((N, D), np.int64))
    inf = orc.infer(X, B, r["M"])
    assert np.all(inf["y"] == y)
    assert np.all(inf["S"][np.arange(N), y] == D)


def pin_train_identical_samples(orc):
    """n identical samples of a class sum to n times their encoding."""
    X, B, _ = hd_inputs.make_inputs(1, 19, 97, 1, "normal", seed=33)
    Xr = np.repeat(X, 5, axis=0)
    y = np.array([0, 0, 0, 1, 0], np.int32)
    r = orc.bundle(Xr, B, y, 2)
    h = np.array(brute_infer(X, B, np.zeros((1, 97), np.float32))["H"][0], dtype=float)
    assert np.array_equal(r["counts"][0], (4 * h).astype(np.int64))
    assert np.array_equal(r["counts"][1], h.astype(np.int64))
    assert np.array_equal(r["M"][0], h) and np.array_equal(r["M"][1], h)


def pin_train_relabel_and_totals(orc):
    """Relabelling classes by a permutation permutes the codebook rows; the
    class sums over all labels equal the column sums of the encodings;
    labels outside [0, K) change nothing."""
    X, B, y = _tiny(41, 9, 5, 13, 5)
    r = orc.bundle(X, B, y, 5)
    perm = np.array([3, 0, 4, 1, 2])
    rp = orc.bundle(X, B, perm[y].astype(np.int32), 5)
    assert np.array_equal(rp["counts"][perm], r["counts"])
    _, H = _brute_counts(X, B, y, 5)
    colsum = [sum(int(H[n][d]) for n in range(9)) for d in range(13)]
    assert np.array_equal(r["counts"].sum(axis=0), np.array(colsum))
    Xo = np.vstack([X, X[:2]])
    yo = np.concatenate([y, np.array([-1, 5], np.int32)])
    ro = orc.bundle(Xo, B, yo, 5)
    assert np.array_equal(ro["counts"], r["counts"])


TRAIN_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_train_")]
