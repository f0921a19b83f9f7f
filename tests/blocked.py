"""Sequential simulation of the paper's blocked two-stage decomposition.

Stage I (Sec. III-B, Alg. 2): worker t owns the column blocks j of H with
j mod T = t; for each it accumulates, round by round, the products of R
blocks of a row block of X with the matching R blocks of column block j of B,
then applies HardSign to the finished column block.
Stage II, small-batch variant (Sec. III-C, Alg. 3): each worker multiplies the
column blocks it received with the matching row blocks of J = M^T into a
private S_local; the locals are summed, then a row argmax.
Stage II, large-batch variant (Sec. III-C, Alg. 4): worker t' owns a band of
about N/T rows and accumulates those rows of S over all column blocks.

Used only to check, on inputs where every order of summation is exact, that
these decompositions compute exactly the plain definition the oracle follows
(the paper states it makes no change to the HDC algorithm).
"""
from __future__ import annotations

import numpy as np


def _cdiv(a, b):
    return -(-a // b)


def stage1(X, B, n, f, d, R, T, act="hardsign"):
    N, F = X.shape
    D = B.shape[1]
    H = np.zeros((N, D), dtype=np.float64)
    nf = _cdiv(F, f)
    for t in range(T):
        for j in range(t, _cdiv(D, d), T):
            c0, c1 = j * d, min((j + 1) * d, D)
            buf = np.zeros((N, c1 - c0))
            for r in range(0, nf, R):
                r_end = min(r + R - 1, nf - 1)
                for i in range(_cdiv(N, n)):
                    r0, r1 = i * n, min((i + 1) * n, N)
                    local = np.zeros((r1 - r0, c1 - c0))
                    for kb in range(r, r_end + 1):
                        k0, k1 = kb * f, min((kb + 1) * f, F)
                        local += X[r0:r1, k0:k1] @ B[k0:k1, c0:c1]
                    buf[r0:r1] += local
            H[:, c0:c1] = np.where(buf >= 0, 1.0, -1.0) if act == "hardsign" else buf
    return H


def stage2_small(H, J, n, d, k, T):
    N, D = H.shape
    K = J.shape[1]
    S = np.zeros((N, K))
    for t in range(T):
        S_local = np.zeros((N, K))
        for j in range(t, _cdiv(D, d), T):
            c0, c1 = j * d, min((j + 1) * d, D)
            for i in range(_cdiv(N, n)):
                r0, r1 = i * n, min((i + 1) * n, N)
                for kb in range(_cdiv(K, k)):
                    q0, q1 = kb * k, min((kb + 1) * k, K)
                    S_local[r0:r1, q0:q1] += H[r0:r1, c0:c1] @ J[c0:c1, q0:q1]
        S += S_local
    return S, np.argmax(S, axis=1)


def stage2_large(H, J, n, d, k, T):
    N, D = H.shape
    K = J.shape[1]
    S = np.zeros((N, K))
    band = _cdiv(N, T)
    for t in range(T):
        b0, b1 = t * band, min((t + 1) * band, N)
        if b0 >= b1:
            continue
        St = np.zeros((b1 - b0, K))
        for j in range(_cdiv(D, d)):
            c0, c1 = j * d, min((j + 1) * d, D)
            Hc = H[b0:b1, c0:c1]
            for i in range(_cdiv(b1 - b0, n)):
                r0, r1 = i * n, min((i + 1) * n, b1 - b0)
                for kb in range(_cdiv(K, k)):
                    q0, q1 = kb * k, min((kb + 1) * k, K)
                    St[r0:r1, q0:q1] += Hc[r0:r1] @ J[c0:c1, q0:q1]
        S[b0:b1] = St
    return S, np.argmax(S, axis=1)
