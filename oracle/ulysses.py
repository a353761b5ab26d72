"""The data layouts around DeepSpeed-Ulysses' all-to-all, in plain numpy.
TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's best sequence-parallel scheme, DeepSpeed-Ulysses (Sec. II,
"Sequence Parallel"; two all-to-all calls per attention in the forward and
in the backward pass, Sec. V), keeps activations sharded by sequence (rank r
holds tokens r*Nl .. (r+1)*Nl - 1 of every head) and hands attention the
full sequence of H/P heads per rank. Written as definitions with P ranks,
H heads, Hl = H/P heads per rank, Nl tokens per rank and rows of any width:

  pack       x[b, i, h]           -> send[p, b, j, i]   = x[b, i, p*Hl + j]
  all-to-all send_r[p] (rank r)   -> recv_p[r]
  unpack     recv[r, b, j, i]     -> y[b, j, r*Nl + i]  (the attention layout)
  pack_out   y[b, j, r*Nl + i]    -> send[r, b, j, i]   (inverse of unpack)
  unpack_out recv[p, b, j, i]     -> x[b, i, p*Hl + j]  (inverse of pack)

so that y on rank p is head group p of the global tensor X[b, n, h] (the
concatenation of the ranks' x along the sequence), transposed to [b, j, n].
"""
from __future__ import annotations

import numpy as np


def pack(x, P):
    """x (B, Nl, H, ...) -> send (P, B, H/P, Nl, ...)."""
    B, Nl, H = x.shape[:3]
    Hl = H // P
    out = np.empty((P, B, Hl, Nl) + x.shape[3:], dtype=x.dtype)
    for p in range(P):
        for j in range(Hl):
            out[p, :, j] = x[:, :, p * Hl + j]
    return out


def unpack(recv):
    """recv (P, B, Hl, Nl, ...) -> y (B, Hl, P*Nl, ...)."""
    P, B, Hl, Nl = recv.shape[:4]
    out = np.empty((B, Hl, P * Nl) + recv.shape[4:], dtype=recv.dtype)
    for r in range(P):
        out[:, :, r * Nl:(r + 1) * Nl] = recv[r]
    return out


def pack_out(y, P):
    """y (B, Hl, P*Nl, ...) -> send (P, B, Hl, Nl, ...)."""
    B, Hl, N = y.shape[:3]
    Nl = N // P
    out = np.empty((P, B, Hl, Nl) + y.shape[3:], dtype=y.dtype)
    for r in range(P):
        out[r] = y[:, :, r * Nl:(r + 1) * Nl]
    return out


def unpack_out(recv):
    """recv (P, B, Hl, Nl, ...) -> x (B, Nl, P*Hl, ...)."""
    P, B, Hl, Nl = recv.shape[:4]
    out = np.empty((B, Nl, P * Hl) + recv.shape[4:], dtype=recv.dtype)
    for p in range(P):
        for j in range(Hl):
            out[:, :, p * Hl + j] = recv[p, :, j]
    return out


def all_to_all(sends):
    """Simulated all-to-all among len(sends) ranks: recv_p[r] = send_r[p]."""
    P = len(sends)
    return [np.stack([sends[r][p] for r in range(P)]) for p in range(P)]
