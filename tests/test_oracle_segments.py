"""Pins of the oracle's key-segment attention and merge (CPU only).

Checked against what the definition fixes: merging the attention over any
split of the keys equals the attention over all keys (computed by the
oracle's full forward, a different code path); a single segment merges to
itself; a segment duplicated twice adds exactly log 2 to LSE and leaves O
unchanged; and the per-segment backward with the merged statistics sums to
the full backward (dQ) and reproduces its dK, dV rows.
"""
import math

import numpy as np
import pytest

import oracle
from workloads import make_small_inputs


def _split(n, cuts):
    edges = [0] + list(cuts) + [n]
    return [(a, b) for a, b in zip(edges[:-1], edges[1:])]


def _segment_forwards(x, segs, scale):
    parts = [oracle.forward(x["q"], x["k"][:, :, a:b], x["v"][:, :, a:b], scale) for a, b in segs]
    return np.stack([p[0] for p in parts]), np.stack([p[1] for p in parts])


@pytest.mark.parametrize("cuts", [(1,), (17, 40), (5, 6, 7, 63)])
def test_merge_of_segments_equals_full_attention(cuts):
    x = make_small_inputs(2, 2, 70, 16, seed=11, with_dout=False)
    scale = 0.25
    o_full, lse_full = oracle.forward(x["q"], x["k"], x["v"], scale)
    o_p, l_p = _segment_forwards(x, _split(70, cuts), scale)
    o, lse = oracle.merge(o_p, l_p)
    np.testing.assert_allclose(lse, lse_full, rtol=0, atol=1e-12)
    np.testing.assert_allclose(o, o_full, rtol=0, atol=1e-12)


def test_merge_single_segment_is_identity():
    rng = np.random.default_rng(3)
    o = rng.standard_normal((1, 2, 9, 4))
    lse = rng.standard_normal((1, 2, 9))
    om, lm = oracle.merge(o[None], lse[None])
    np.testing.assert_allclose(om, o, rtol=0, atol=1e-15)
    np.testing.assert_allclose(lm, lse, rtol=0, atol=1e-15)


def test_merge_duplicate_segment_adds_log2():
    rng = np.random.default_rng(4)
    o = rng.standard_normal((2, 1, 5, 8))
    lse = 3.0 * rng.standard_normal((2, 1, 5))
    om, lm = oracle.merge(np.stack([o, o]), np.stack([lse, lse]))
    np.testing.assert_allclose(lm, lse + math.log(2.0), rtol=0, atol=1e-14)
    np.testing.assert_allclose(om, o, rtol=0, atol=1e-14)


def test_merge_weights_follow_lse():
    # two partials whose LSEs differ by log 3: weights 3/4 and 1/4
    o = np.stack([np.full((1, 1, 1, 2), 1.0), np.full((1, 1, 1, 2), 5.0)])
    lse = np.stack([np.full((1, 1, 1), math.log(3.0)), np.zeros((1, 1, 1))])
    om, lm = oracle.merge(o, lse)
    np.testing.assert_allclose(om, np.full((1, 1, 1, 2), 0.75 * 1.0 + 0.25 * 5.0), rtol=0, atol=1e-15)
    np.testing.assert_allclose(lm, np.full((1, 1, 1), math.log(4.0)), rtol=0, atol=1e-15)


@pytest.mark.parametrize("cuts", [(33,), (8, 50, 51)])
def test_segment_backward_sums_to_full_backward(cuts):
    x = make_small_inputs(1, 2, 64, 16, seed=12, with_dout=True)
    scale = 0.25
    full = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    dq = np.zeros_like(full["dq"])
    for a, b in _split(64, cuts):
        dq_p, dk, dv = oracle.segment_backward(x["q"], x["k"][:, :, a:b], x["v"][:, :, a:b], x["dout"], full["o"],
                                               full["lse"], scale)
        np.testing.assert_allclose(dk, full["dk"][:, :, a:b], rtol=0, atol=1e-12)
        np.testing.assert_allclose(dv, full["dv"][:, :, a:b], rtol=0, atol=1e-12)
        dq += dq_p
    np.testing.assert_allclose(dq, full["dq"], rtol=0, atol=1e-12)


def test_segment_backward_with_cross_lengths():
    # queries and keys of different lengths (a segment), against a direct
    # evaluation through the oracle's key-row function on a concatenation
    x = make_small_inputs(1, 1, 40, 8, seed=13, with_dout=True)
    scale = 0.5
    full = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    keys = np.arange(10, 23)
    dk_ref, dv_ref = oracle.key_rows(x["q"], x["k"], x["v"], x["dout"], scale, 0, 0, keys, full["lse"][0, 0],
                                     full["D"][0, 0])
    _, dk, dv = oracle.segment_backward(x["q"], x["k"][:, :, 10:23], x["v"][:, :, 10:23], x["dout"], full["o"],
                                        full["lse"], scale)
    np.testing.assert_allclose(dk[0, 0], dk_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dv[0, 0], dv_ref, rtol=0, atol=1e-12)


def test_planted_merge_mistake_is_caught():
    # a merge that forgets the weights (plain average) must fail the identity
    x = make_small_inputs(1, 1, 30, 8, seed=14, with_dout=False)
    scale = 1.0
    o_full, _ = oracle.forward(x["q"], x["k"], x["v"], scale)
    o_p, _ = _segment_forwards(x, _split(30, (7,)), scale)
    assert np.max(np.abs(o_p.mean(axis=0) - o_full)) > 1e-3
