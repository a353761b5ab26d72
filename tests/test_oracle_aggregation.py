"""Pins of the oracle's channel aggregation (CPU only).

Against what the definition fixes, through code paths other than its own:
each patch and head is an attention with one query over C keys, so the
forward equals the general attention oracle with Nq = 1 (query broadcast);
dk and dv equal that oracle's per-instance gradients; dq of the shared query
is the sum over patches of the per-instance dq; central finite differences
of a scalar loss confirm dq; and identical channel keys give the mean of V.
"""
import numpy as np
import pytest

import oracle
from oracle import aggregation as agg


def _inputs(M, H, C, d, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((H, d)), rng.standard_normal((M, H, C, d)), rng.standard_normal((M, H, C, d)),
            rng.standard_normal((M, H, d)))


def _as_instances(q, k, v, dout):
    """The same problem as B = M batches of ordinary attention, Nq = 1."""
    M, H = k.shape[:2]
    qb = np.broadcast_to(q[None, :, None, :], (M, H, 1, q.shape[1])).copy()
    return qb, k, v, dout[:, :, None, :]


@pytest.mark.parametrize("M,H,C,d", [(3, 2, 92, 8), (1, 1, 1, 4), (5, 3, 7, 16)])
def test_forward_equals_general_attention_with_one_query(M, H, C, d):
    q, k, v, _ = _inputs(M, H, C, d, seed=M * 100 + C)
    o, lse = agg.forward(q, k, v, 0.25)
    qb, _, _, _ = _as_instances(q, k, v, np.zeros((M, H, d)))
    o_ref, lse_ref = oracle.forward(qb, k, v, 0.25)
    np.testing.assert_allclose(o, o_ref[:, :, 0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lse_ref[:, :, 0], rtol=0, atol=1e-12)


@pytest.mark.parametrize("M,H,C,d", [(3, 2, 92, 8), (4, 1, 5, 4)])
def test_backward_equals_per_instance_gradients_summed_over_patches(M, H, C, d):
    q, k, v, dout = _inputs(M, H, C, d, seed=7 + C)
    g = agg.backward(q, k, v, dout, 0.5)
    qb, _, _, db = _as_instances(q, k, v, dout)
    # per-instance gradients from the general oracle (one query, C keys)
    dq_sum = np.zeros((H, d))
    for m in range(M):
        for h in range(H):
            Q = qb[m:m + 1, h:h + 1]
            K = k[m:m + 1, h:h + 1]
            V = v[m:m + 1, h:h + 1]
            dO = db[m:m + 1, h:h + 1]
            o1, lse1 = oracle.forward(Q, K, V, 0.5)
            dq1, dk1, dv1 = oracle.segment_backward(Q, K, V, dO, o1, lse1, 0.5)
            np.testing.assert_allclose(g["dk"][m, h], dk1[0, 0], rtol=0, atol=1e-12)
            np.testing.assert_allclose(g["dv"][m, h], dv1[0, 0], rtol=0, atol=1e-12)
            dq_sum[h] += dq1[0, 0, 0]
    np.testing.assert_allclose(g["dq"], dq_sum, rtol=0, atol=1e-11)


def test_dq_matches_finite_differences():
    M, H, C, d = 3, 2, 6, 4
    q, k, v, dout = _inputs(M, H, C, d, seed=31)
    g = agg.backward(q, k, v, dout, 0.5)
    loss = lambda qq: float((agg.forward(qq, k, v, 0.5)[0] * dout).sum())
    eps = 1e-6
    for h in range(H):
        for e in range(d):
            qp, qm = q.copy(), q.copy()
            qp[h, e] += eps
            qm[h, e] -= eps
            fd = (loss(qp) - loss(qm)) / (2 * eps)
            assert abs(fd - g["dq"][h, e]) < 1e-6 * max(1.0, abs(fd))


def test_identical_channel_keys_give_mean_of_values():
    M, H, C, d = 2, 1, 9, 3
    q, k, v, _ = _inputs(M, H, C, d, seed=5)
    k[:] = k[:, :, :1]
    o, lse = agg.forward(q, k, v, 1.0)
    np.testing.assert_allclose(o, v.mean(axis=2), rtol=0, atol=1e-13)
    s = np.einsum("hd,mhd->mh", q, k[:, :, 0])
    np.testing.assert_allclose(lse, s + np.log(C), rtol=0, atol=1e-12)
