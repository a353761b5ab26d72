"""Attention over key segments and the merge of the partial results, in fp64.
TEST INFRASTRUCTURE ONLY (see the package docstring).

Sequence parallelism over contiguous segments of the sequence (Long Sequence
Segmentation, which the paper builds on in Sec. I and describes in Sec. II,
"Sequence Parallel"; one segment per worker) leaves a worker with the
attention of its queries over one segment of the keys at a time. Written
from the definition of softmax over a union of key sets (LSE is the natural
log of the summed exponentials of the scaled logits, as in the forward):

    exp(LSE_i) = sum_j exp(S_ij) = sum_s sum_{j in s} exp(S_ij) = sum_s exp(LSE_s,i)
    O_i        = sum_j exp(S_ij - LSE_i) V_j = sum_s exp(LSE_s,i - LSE_i) O_s,i

so a segment's (O_s, LSE_s), i.e. plain attention restricted to its keys,
carries everything the merge needs. In the backward pass the global LSE and
D = rowsum(dO o O) of the merged output make every probability of a segment
exact, so that segment's dK and dV rows are complete and its dQ is the
segment's share of the sum over all keys:

    P_ij  = exp(s q_i.k_j - LSE_i)                   j in the segment
    dS_ij = P_ij (dO_i.v_j - D_i)
    dQ_i  = s sum_{j in seg} dS_ij k_j   (summed over segments gives dQ)
    dK_j  = s sum_i dS_ij q_i,   dV_j = sum_i P_ij dO_i
"""
from __future__ import annotations

import numpy as np

from .attention import _as_f64, fp32_scale


def merge(o_parts, lse_parts):
    """Merge P partial results. o_parts (P, ..., N, d) and lse_parts (P, ..., N)
    -> o (..., N, d), lse (..., N), as written in the module docstring (the
    largest partial LSE is subtracted before exponentiating, which changes
    nothing in exact arithmetic)."""
    o_parts = np.asarray(o_parts, dtype=np.float64)
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    m = lse_parts.max(axis=0)
    w = np.exp(lse_parts - m[None])
    tot = w.sum(axis=0)
    lse = m + np.log(tot)
    o = (w[..., None] * o_parts).sum(axis=0) / tot[..., None]
    return o, lse


def segment_backward(q, k, v, dout, o, lse, scale):
    """dQ share and the complete dK, dV of the keys in k, v (one segment),
    given the merged o and lse of all keys. q, dout, o: (B, H, Nq, d);
    k, v: (B, H, Nk, d); lse: (B, H, Nq). Returns dq_part (B, H, Nq, d),
    dk, dv (B, H, Nk, d)."""
    q, k, v, dout = _as_f64(q), _as_f64(k), _as_f64(v), _as_f64(dout)
    o, lse = np.asarray(o, dtype=np.float64), np.asarray(lse, dtype=np.float64)
    s = fp32_scale(scale)
    B, H, Nq, d = q.shape
    Nk = k.shape[2]
    dq = np.empty((B, H, Nq, d))
    dk = np.empty((B, H, Nk, d))
    dv = np.empty((B, H, Nk, d))
    for b in range(B):
        for h in range(H):
            Q, K, V, dO = q[b, h], k[b, h], v[b, h], dout[b, h]
            D = np.einsum("ic,ic->i", dO, o[b, h])
            P = np.exp(s * (Q @ K.T) - lse[b, h][:, None])
            dS = P * (dO @ V.T - D[:, None])
            dq[b, h] = s * (dS @ K)
            dk[b, h] = s * (dS.T @ Q)
            dv[b, h] = P.T @ dO
    return dq, dk, dv
