"""Exact rational brute force of Alg. 1 for tiny inputs.

Every fp32/bf16 value is a dyadic rational, so ``fractions.Fraction`` holds it
exactly and all sums below are exact: no rounding anywhere. This pins the
oracle's encoding signs, scores and labels independently of any floating-point
summation order.
"""
from __future__ import annotations

from fractions import Fraction


def brute_infer(X, B, C, act: str = "hardsign"):
    N = len(X)
    F = len(B)
    D = len(B[0]) if F else 0
    K = len(C)
    Xq = [[Fraction(float(v)) for v in row] for row in X]
    Bq = [[Fraction(float(v)) for v in row] for row in B]
    Cq = [[Fraction(float(v)) for v in row] for row in C]
    V, A, H, S, y = [], [], [], [], []
    for n in range(N):
        v = [sum((Xq[n][f] * Bq[f][d] for f in range(F)), Fraction(0)) for d in range(D)]
        a = [sum((abs(Xq[n][f]) * abs(Bq[f][d]) for f in range(F)), Fraction(0)) for d in range(D)]
        if act == "hardsign":
            h = [Fraction(1) if vd >= 0 else Fraction(-1) for vd in v]
        else:
            h = list(v)
        s = [sum((h[d] * Cq[k][d] for d in range(D)), Fraction(0)) for k in range(K)]
        best = max(s)
        y.append(min(k for k in range(K) if s[k] == best))
        V.append(v)
        A.append(a)
        H.append(h)
        S.append(s)
    return {"V": V, "A": A, "H": H, "S": S, "y": y}
