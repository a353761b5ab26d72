"""GPU parity of the dK/dV kernel's grid balance: when the last round of
key-block workgroups is at most half full, those key blocks are split into
two workgroups over the two halves of the query tiles, which add dK and dV
into zeroed rows. The shapes below put whole and split key blocks in one
launch on a 256-CU part with one dK/dV workgroup per CU (B*H*ceil(N/128)
work items: 257 -> 256 whole + 1 split, 600 -> 512 + 88, 280 -> 256 + 24,
260 -> 256 + 4 with 65 query tiles per half), including an odd tile count
(the second half one tile longer) and a ragged last tile. Both backward
modes, against the fp64 oracle; on any other device the same comparisons
hold whatever the split."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_close, run_hip, torch

pytestmark = pytest.mark.gpu

CASES = [(1, 257, 256, 64), (1, 300, 130, 128), (2, 70, 200, 160), (1, 4, 8320, 64), (1, 33, 1000, 96)]


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
    # N = 25,600 gives 200 key blocks per head: a head alone is 200 work items
    # (no split on a 256-CU part), three heads are 600 (the last 88, all of
    # head 2, split). O, LSE and dQ do not depend on the split and stay
    # bitwise equal; dK and dV of head 2 sum its query tiles in another order,
    # so they agree to fp32 rounding.
    t = torch()
    B, H, N, d = 1, 3, 25600, 64
    print(f"case head alone vs among others store_ds={store_ds}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=7801)
    scale = 1.0 / np.sqrt(d)
    full = run_hip(x, scale, store_ds=store_ds)
    alone = run_hip({n: np.ascontiguousarray(a[:, 2:3]) for n, a in x.items()}, scale, store_ds=store_ds)
    for name in ("o", "lse", "dq"):
        assert t.equal(full[name][:, 2:3], alone[name]), name
    for name in ("dk", "dv"):
        a, b = full[name][:, 2:3].double(), alone[name].double()
        rel = ((a - b).norm() / b.norm()).item()
        print(f"{name}: rel L2 {rel:.2e}", flush=True)
        assert rel < 1e-5, (name, rel)
