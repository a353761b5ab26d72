"""Plain fp64 evaluation of exact (dense, non-causal) multi-head attention and
its gradients. TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed, per batch element b and head h (Sec. I and III of the paper
ask for dense attention in which every patch token attends to every other;
Sec. II-E gives one GPU the full sequence for a subset of heads; Sec. II-F
cites FlashAttention-2, whose saved per-row logsumexp and backward identities
are used here):

    S   = s Q K^T                          s = the fp32 softmax scale
    LSE = log sum_j exp(S_ij)              natural log, of the scaled logits
    P   = exp(S - LSE 1^T)                 rows sum to one
    O   = P V
    dP  = dO V^T
    D_i = sum_c dO_ic O_ic                 (= sum_j P_ij dP_ij)
    dS  = P o (dP - D 1^T)
    dQ  = s dS K,   dK = s dS^T Q,   dV = P^T dO

There is no mask, no bias and no dropout. Inputs are the same bfloat16 bit
patterns the GPU receives, widened exactly to fp64; every sum is in fp64.

Query rows are processed in independent blocks only to bound the N x N
working set; each block is the definition above restricted to its rows.
"""
from __future__ import annotations

import numpy as np

QUERY_BLOCK = 512


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> exactly equal float64 values."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def fp32_scale(scale: float) -> float:
    """The softmax scale as the kernels receive it: rounded to fp32."""
    return float(np.float32(scale))


def _as_f64(x):
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return decode_bf16(x)
    return x.astype(np.float64, copy=False)


def _block_forward(qb, K, V, s):
    """Rows of S, LSE, P and O for a block of query rows of one head."""
    S = s * (qb @ K.T)
    m = S.max(axis=1)
    E = np.exp(S - m[:, None])
    l = E.sum(axis=1)
    lse = m + np.log(l)
    P = E / l[:, None]
    return S, lse, P, P @ V


def forward(q, k, v, scale, block=QUERY_BLOCK):
    """O (B,H,N,d) and LSE (B,H,N) in fp64."""
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    s = fp32_scale(scale)
    B, H, N, d = q.shape
    o = np.empty((B, H, N, v.shape[-1]))
    lse = np.empty((B, H, N))
    for b in range(B):
        for h in range(H):
            K, V = k[b, h], v[b, h]
            for r0 in range(0, N, block):
                r1 = min(N, r0 + block)
                _, lse[b, h, r0:r1], _, o[b, h, r0:r1] = _block_forward(q[b, h, r0:r1], K, V, s)
    return o, lse


def _block_backward(qb, K, V, dOb, s):
    """Forward and backward quantities of a block of query rows of one head;
    dK and dV are this block's contributions (sums over its rows)."""
    _, lse, P, O = _block_forward(qb, K, V, s)
    dP = dOb @ V.T
    D = np.einsum("ic,ic->i", dOb, O)
    dS = P * (dP - D[:, None])
    return {
        "o": O,
        "lse": lse,
        "D": D,
        "dq": s * (dS @ K),
        "dk_part": s * (dS.T @ qb),
        "dv_part": P.T @ dOb,
    }


def forward_backward(q, k, v, dout, scale, block=QUERY_BLOCK, heads=None):
    """Full fp64 forward and backward. Returns a dict with o, lse, D, dq (one
    row per query) and dk, dv (one row per key; the key count may differ
    from the query count) over all (b, h), or only over the (b, h) pairs
    listed in `heads` (other entries are left as NaN)."""
    q, k, v, dout = _as_f64(q), _as_f64(k), _as_f64(v), _as_f64(dout)
    s = fp32_scale(scale)
    B, H, N, d = q.shape
    Nk = k.shape[2]
    out = {
        "o": np.full((B, H, N, d), np.nan),
        "lse": np.full((B, H, N), np.nan),
        "D": np.full((B, H, N), np.nan),
        "dq": np.full((B, H, N, d), np.nan),
        "dk": np.full((B, H, Nk, d), np.nan),
        "dv": np.full((B, H, Nk, d), np.nan),
    }
    pairs = heads if heads is not None else [(b, h) for b in range(B) for h in range(H)]
    for b, h in pairs:
        K, V = k[b, h], v[b, h]
        dk = np.zeros((Nk, d))
        dv = np.zeros((Nk, d))
        for r0 in range(0, N, block):
            r1 = min(N, r0 + block)
            r = _block_backward(q[b, h, r0:r1], K, V, dout[b, h, r0:r1], s)
            for name in ("o", "lse", "D", "dq"):
                out[name][b, h, r0:r1] = r[name]
            dk += r["dk_part"]
            dv += r["dv_part"]
        out["dk"][b, h] = dk
        out["dv"][b, h] = dv
    return out


def forward_backward_rows(q, k, v, dout, scale, b, h, r0, r1):
    """The forward and backward work of query rows r0..r1-1 of head (b, h)
    against all keys: their o, lse, D and dq, plus their contributions
    dk_part and dv_part to dK and dV (summing these over all row ranges gives
    dK and dV). Used to time the oracle on a bounded slice of a workload."""
    s = fp32_scale(scale)
    return _block_backward(_as_f64(q[b, h, r0:r1]), _as_f64(k[b, h]), _as_f64(v[b, h]), _as_f64(dout[b, h, r0:r1]),
                           s)


def query_rows(q, k, v, scale, rows, dout=None):
    """Per-row outputs for sampled query rows.

    rows: int array (R, 3) of (b, h, i). Each row needs only its own query
    against all keys of its head, so this costs O(N d) per row. Returns o
    (R, d) and lse (R,), plus D (R,) and dq (R, d) when dout is given."""
    s = fp32_scale(scale)
    rows = np.asarray(rows, dtype=np.int64)
    R = rows.shape[0]
    d = q.shape[-1]
    res = {"o": np.empty((R, d)), "lse": np.empty(R)}
    if dout is not None:
        res["D"] = np.empty(R)
        res["dq"] = np.empty((R, d))
    # group rows by head so that each head's K and V are widened once
    for b, h in sorted({(int(b), int(h)) for b, h, _ in rows}):
        sel = np.nonzero((rows[:, 0] == b) & (rows[:, 1] == h))[0]
        idx = rows[sel, 2]
        K, V = _as_f64(k[b, h]), _as_f64(v[b, h])
        qb = _as_f64(q[b, h][idx])
        if dout is None:
            _, lse, _, O = _block_forward(qb, K, V, s)
            res["o"][sel], res["lse"][sel] = O, lse
        else:
            r = _block_backward(qb, K, V, _as_f64(dout[b, h][idx]), s)
            for name in ("o", "lse", "D", "dq"):
                res[name][sel] = r[name]
    return res


def row_statistics(q, k, v, dout, scale, b, h, block=QUERY_BLOCK):
    """LSE_i and D_i for every query row i of head (b, h): one full fp64
    forward pass of that head. These are what a key row's dK and dV need."""
    s = fp32_scale(scale)
    K, V = _as_f64(k[b, h]), _as_f64(v[b, h])
    N = q.shape[2]  # query rows (the keys may be a different number)
    lse = np.empty(N)
    D = np.empty(N)
    for r0 in range(0, N, block):
        r1 = min(N, r0 + block)
        _, lse[r0:r1], _, O = _block_forward(_as_f64(q[b, h, r0:r1]), K, V, s)
        D[r0:r1] = np.einsum("ic,ic->i", _as_f64(dout[b, h, r0:r1]), O)
    return lse, D


def key_rows(q, k, v, dout, scale, b, h, keys, lse, D, block=4096):
    """dK and dV rows of head (b, h) at key indices `keys`, given that head's
    full LSE and D (from row_statistics):

        P_ij  = exp(s q_i.k_j - LSE_i)
        dS_ij = P_ij (dO_i.v_j - D_i)
        dK_j  = s sum_i dS_ij q_i,     dV_j = sum_i P_ij dO_i
    """
    s = fp32_scale(scale)
    keys = np.asarray(keys, dtype=np.int64)
    Kj, Vj = _as_f64(k[b, h][keys]), _as_f64(v[b, h][keys])
    N = q.shape[2]
    d = q.shape[-1]
    dk = np.zeros((len(keys), d))
    dv = np.zeros((len(keys), d))
    for r0 in range(0, N, block):
        r1 = min(N, r0 + block)
        Q, dO = _as_f64(q[b, h, r0:r1]), _as_f64(dout[b, h, r0:r1])
        P = np.exp(s * (Q @ Kj.T) - lse[r0:r1, None])
        dS = P * (dO @ Vj.T - D[r0:r1, None])
        dk += s * (dS.T @ Q)
        dv += P.T @ dO
    return dk, dv
