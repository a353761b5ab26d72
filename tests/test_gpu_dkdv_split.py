"""GPU parity of the dK/dV kernel's grid balance: when the last round of
key-block workgroups is at most half full, those key blocks are split into
two workgroups over the two halves of the query tiles, which add dK and dV
into zeroed rows, while whole key blocks form the same two partial sums
(the first stored at the midpoint), so the bits do not depend on the
split. The shapes below put whole and split key blocks in one
launch on a 256-CU part with one dK/dV workgroup per CU (B*H*ceil(N/BK)
work items, BK = 128 keys, or in the recompute mode 256 at head dims up to
64 and 192 at 65-80: 257 -> 256 whole + 1 split, 600 -> 512 + 88, 280 ->
256 + 24, 260 -> 256 + 4 with 130 query tiles per half, the last one
ragged, and in the last work item a wave whose first 32-key block holds 24
keys and whose second lies past the end; at d = 72, 270 -> 256 + 14 twelve-
wave work items in the recompute mode and 360 -> 256 + 104 in the dS mode),
including an odd tile count (the second half one tile longer). Both
backward modes, against the fp64 oracle; on any other device the same
comparisons hold whatever the split."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_close, run_hip, torch

pytestmark = pytest.mark.gpu

CASES = [(1, 257, 256, 64), (1, 300, 130, 128), (2, 70, 200, 160), (1, 4, 16600, 64), (1, 33, 1000, 96),
         (1, 45, 1000, 72)]


def np64(t):
    return t.detach().double().cpu().numpy()


@pytest.mark.parametrize("store_ds", [False, True], ids=["recompute", "stored-ds"])
@pytest.mark.parametrize("B,H,N,d", CASES)
def test_split_key_blocks_match_oracle(B, H, N, d, store_ds):
    print(f"case dkdv split B={B} H={H} N={N} d={d} store_ds={store_ds}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=7700 + H + N + d)
    scale = 1.0 / np.sqrt(d)
    got = {n: np64(t) for n, t in run_hip(x, scale, store_ds=store_ds).items()}
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    assert_close(got, ref, label=f"dkdv split {B},{H},{N},{d} store_ds={store_ds}")


def test_split_key_blocks_are_deterministic():
    # two fp32 adds onto zero commute exactly, so the split blocks' atomics
    # give the same bits on every run
    t = torch()
    B, H, N, d = 1, 300, 130, 128
    print(f"case dkdv split determinism B={B} H={H} N={N} d={d}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=7799)
    runs = [run_hip(x, 1.0 / np.sqrt(d), store_ds=s) for s in (False, False, True, True)]
    for a, b in ((runs[0], runs[1]), (runs[2], runs[3])):
        for name in ("dq", "dk", "dv"):
            assert t.equal(a[name], b[name]), name


@pytest.mark.parametrize("store_ds", [False, True], ids=["recompute", "stored-ds"])
def test_head_alone_and_among_others(store_ds):
    # N = 25,600 at d = 64 gives 100 key blocks of 256 per head: a head alone
    # is 100 work items (all split on a 256-CU part), three heads are 300
    # (the last 44, all of head 2, split; head 2's first 56 whole). Every key block sums its query tiles as the same two
    # rounded partials whether it is split or whole, so all five outputs of
    # head 2 are bitwise equal (the check of Sec. VI-A that every process
    # computes the same matrices, here across call shapes).
    t = torch()
    B, H, N, d = 1, 3, 25600, 64
    print(f"case head alone vs among others store_ds={store_ds}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=7801)
    scale = 1.0 / np.sqrt(d)
    full = run_hip(x, scale, store_ds=store_ds)
    alone = run_hip({n: np.ascontiguousarray(a[:, 2:3]) for n, a in x.items()}, scale, store_ds=store_ds)
    for name in ("o", "lse", "dq", "dk", "dv"):
        assert t.equal(full[name][:, 2:3], alone[name]), name


@pytest.mark.parametrize("B,H,N,d", [(1, 300, 130, 128), (1, 4, 16600, 64), (1, 33, 1000, 96), (2, 70, 200, 160),
                                     (1, 45, 1000, 72)])
def test_split_blocks_bitwise_equal_to_single_head_calls(B, H, N, d):
    # every head of a launch whose last round splits (see CASES) against the
    # same head in a call of its own, where the grid is far from a whole
    # round and no block splits
    t = torch()
    print(f"case split vs single-head calls B={B} H={H} N={N} d={d}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=7900 + H + N + d)
    scale = 1.0 / np.sqrt(d)
    full = run_hip(x, scale)
    for h in sorted({0, H // 2, H - 1}):
        for b in range(B):
            one = run_hip({n: np.ascontiguousarray(a[b:b + 1, h:h + 1]) for n, a in x.items()}, scale)
            for name in ("o", "lse", "dq", "dk", "dv"):
                assert t.equal(full[name][b:b + 1, h:h + 1], one[name]), (name, b, h)
