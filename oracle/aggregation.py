"""Channel aggregation by attention with a learnable query, in fp64.
TEST INFRASTRUCTURE ONLY (see the package docstring).

The Agg-Ch-ViT variant the paper describes (Sec. II, "Patch Embedding and
Sequence Length") folds the channel tokens of each patch into one token with
a multi-head attention layer whose query is a learnable vector, so that the
number of channels does not lengthen the sequence. For M patch positions
(batch x patches), H heads of width d and C channel tokens per patch, with
the projected keys and values K, V of shape [M][H][C][d] and one learnable
query q_h per head (shared by every patch):

    s_mhc = scale q_h . k_mhc,   LSE_mh = log sum_c exp(s_mhc),
    p_mhc = exp(s_mhc - LSE_mh), o_mh = sum_c p_mhc v_mhc

and, for the upstream gradient do_mh,

    dp_mhc = do_mh . v_mhc,  D_mh = do_mh . o_mh,  ds_mhc = p_mhc (dp_mhc - D_mh)
    dk_mhc = scale ds_mhc q_h,  dv_mhc = p_mhc do_mh,
    dq_h   = scale sum_m sum_c ds_mhc k_mhc        (q is shared: summed over m)
"""
from __future__ import annotations

import numpy as np

from .attention import _as_f64, fp32_scale


def forward(q, k, v, scale):
    """q (H, d), k and v (M, H, C, d) -> o (M, H, d), lse (M, H)."""
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    s = fp32_scale(scale) * np.einsum("hd,mhcd->mhc", q, k)
    m = s.max(axis=2)
    e = np.exp(s - m[..., None])
    tot = e.sum(axis=2)
    p = e / tot[..., None]
    return np.einsum("mhc,mhcd->mhd", p, v), m + np.log(tot)


def backward(q, k, v, dout, scale):
    """The gradients dq (H, d), dk and dv (M, H, C, d), plus o and lse."""
    q, k, v, dout = _as_f64(q), _as_f64(k), _as_f64(v), _as_f64(dout)
    sc = fp32_scale(scale)
    o, lse = forward(q, k, v, scale)
    p = np.exp(sc * np.einsum("hd,mhcd->mhc", q, k) - lse[..., None])
    dp = np.einsum("mhd,mhcd->mhc", dout, v)
    D = np.einsum("mhd,mhd->mh", dout, o)
    ds = p * (dp - D[..., None])
    return {
        "o": o,
        "lse": lse,
        "dq": sc * np.einsum("mhc,mhcd->hd", ds, k),
        "dk": sc * ds[..., None] * q[None, :, None, :],
        "dv": p[..., None] * dout[:, :, None, :],
    }
