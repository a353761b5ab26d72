"""Pins of the oracle's Ulysses layouts (CPU only): the pack / all-to-all /
unpack pipeline must hand rank p exactly head group p of the global tensor
in the attention layout (checked against a direct slice-and-transpose of the
concatenated input), and the return trip must restore every rank's input."""
import numpy as np
import pytest

from oracle import ulysses


def _ranks(B, Nl, H, P, d, seed):
    rng = np.random.default_rng(seed)
    return [rng.integers(0, 2 ** 16, size=(B, Nl, H, d), dtype=np.uint16) for _ in range(P)]


@pytest.mark.parametrize("B,Nl,H,P,d", [(1, 5, 4, 2, 3), (2, 3, 8, 4, 8), (1, 1, 3, 3, 1), (2, 7, 6, 1, 4)])
def test_pipeline_gives_each_rank_its_head_group(B, Nl, H, P, d):
    xs = _ranks(B, Nl, H, P, d, seed=B * 100 + Nl * 10 + H + P)
    X = np.concatenate(xs, axis=1)  # global [B, N, H, d]
    recvs = ulysses.all_to_all([ulysses.pack(x, P) for x in xs])
    Hl = H // P
    for p in range(P):
        y = ulysses.unpack(recvs[p])
        ref = X[:, :, p * Hl:(p + 1) * Hl].transpose(0, 2, 1, 3)
        assert np.array_equal(y, ref)


@pytest.mark.parametrize("B,Nl,H,P,d", [(1, 5, 4, 2, 3), (2, 3, 8, 4, 8)])
def test_return_trip_restores_inputs(B, Nl, H, P, d):
    xs = _ranks(B, Nl, H, P, d, seed=7)
    ys = [ulysses.unpack(r) for r in ulysses.all_to_all([ulysses.pack(x, P) for x in xs])]
    back = [ulysses.unpack_out(r) for r in ulysses.all_to_all([ulysses.pack_out(y, P) for y in ys])]
    for x, b in zip(xs, back):
        assert np.array_equal(x, b)


def test_pack_index_map():
    x = np.arange(1 * 2 * 4).reshape(1, 2, 4)  # rows labelled b*8 + i*4 + h
    send = ulysses.pack(x, 2)
    # send[p, b, j, i] = x[b, i, p*2 + j]
    assert send[1, 0, 0, 1] == x[0, 1, 2] and send[0, 0, 1, 0] == x[0, 0, 1]


def test_planted_transpose_mistake_is_caught():
    xs = _ranks(1, 4, 4, 2, 2, seed=9)
    X = np.concatenate(xs, axis=1)
    y = ulysses.unpack(ulysses.all_to_all([ulysses.pack(x, 2) for x in xs])[1])
    wrong = X[:, :, 0:2].transpose(0, 2, 1, 3)  # rank 1 must not hold head group 0
    assert not np.array_equal(y, wrong)
