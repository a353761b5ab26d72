"""A second, deliberately naive evaluation of the same definition, with pure
Python loops and math.fsum, for tiny inputs (N, d up to about 16).
TEST INFRASTRUCTURE ONLY (see the package docstring).

It shares no code with attention.py: the softmax is formed without a running
max (the tiny test inputs cannot overflow), LSE is log of the fsum of
exponentials, and D is taken from its second form, sum_j P_ij dP_ij, rather
than from rowsum(dO o O).
"""
from __future__ import annotations

import math


def attention_head(Q, K, V, s, dO=None):
    """Q, K, V, dO: lists of N rows of d floats; s: scale. Returns a dict of
    nested lists: o, lse and, with dO, dq, dk, dv, D."""
    N = len(Q)
    d = len(Q[0])
    S = [[s * math.fsum(Q[i][c] * K[j][c] for c in range(d)) for j in range(N)] for i in range(N)]
    E = [[math.exp(S[i][j]) for j in range(N)] for i in range(N)]
    Z = [math.fsum(E[i]) for i in range(N)]
    P = [[E[i][j] / Z[i] for j in range(N)] for i in range(N)]
    O = [[math.fsum(P[i][j] * V[j][c] for j in range(N)) for c in range(d)] for i in range(N)]
    out = {"o": O, "lse": [math.log(Z[i]) for i in range(N)]}
    if dO is None:
        return out
    dP = [[math.fsum(dO[i][c] * V[j][c] for c in range(d)) for j in range(N)] for i in range(N)]
    D = [math.fsum(P[i][j] * dP[i][j] for j in range(N)) for i in range(N)]
    dS = [[P[i][j] * (dP[i][j] - D[i]) for j in range(N)] for i in range(N)]
    out["D"] = D
    out["dq"] = [[s * math.fsum(dS[i][j] * K[j][c] for j in range(N)) for c in range(d)] for i in range(N)]
    out["dk"] = [[s * math.fsum(dS[i][j] * Q[i][c] for i in range(N)) for c in range(d)] for j in range(N)]
    out["dv"] = [[math.fsum(P[i][j] * dO[i][c] for i in range(N)) for c in range(d)] for j in range(N)]
    return out
