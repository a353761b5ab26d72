"""At the narrowest tile (head dims up to 64) the forward and dQ kernels
choose between 8- and 12-wave workgroups from the grid size, and each dK/dV
wave holds two 32-key blocks (256 keys per workgroup); in the 96-wide tile
with d <= 80 the dQ kernel makes the same choice and dK/dV runs six pairs of
waves (192 keys). B=1, H=6, N=22,001 makes the six-head call take the
12-wave dQ (and at d <= 64 forward) on a 256-CU part (two rounds of
384-query workgroups instead of three of 256) while each single-head call
takes the 8-wave ones; dK/dV splits 4 of its 516 key blocks at d <= 64 (none
of 690 at d = 72) where a single-head call splits all 86 (115). Every
output must be bitwise equal between the two, and sampled query and key
rows must match the fp64 oracle."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_close, run_hip, torch

pytestmark = pytest.mark.gpu


def np64(t):
    return t.detach().double().cpu().numpy()


@pytest.mark.parametrize("d", [56, 64, 72])
def test_twelve_wave_grid_matches_single_heads_and_oracle(d):
    t = torch()
    B, H, N = 1, 6, 22001
    print(f"case wave variants B={B} H={H} N={N} d={d}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=9900 + d)
    scale = 1.0 / np.sqrt(d)
    full = run_hip(x, scale)
    for h in range(H):
        one = run_hip({n: np.ascontiguousarray(a[:, h:h + 1]) for n, a in x.items()}, scale)
        for name in ("o", "lse", "dq", "dk", "dv"):
            assert t.equal(full[name][:, h:h + 1], one[name]), (name, h)
    rng = np.random.default_rng(d)
    rows = np.stack([np.zeros(64, np.int64), rng.integers(0, H, 64), rng.choice(N, 64, replace=False)], axis=1)
    rows = rows[np.lexsort((rows[:, 2], rows[:, 1]))]
    ref = oracle.query_rows(x["q"], x["k"], x["v"], scale, rows, dout=x["dout"])
    sel = tuple(t.from_numpy(rows[:, i]).cuda() for i in range(3))
    got = {n: np64(full[n][sel]) for n in ("o", "lse", "dq")}
    assert_close(got, ref, names=("o", "lse", "dq"), label=f"wave variants d={d} sampled query rows")
    h = 4
    lse, D = oracle.row_statistics(x["q"], x["k"], x["v"], x["dout"], scale, 0, h)
    keys = np.sort(rng.choice(N, 64, replace=False))
    dk, dv = oracle.key_rows(x["q"], x["k"], x["v"], x["dout"], scale, 0, h, keys, lse, D)
    kk = t.from_numpy(keys).cuda()
    assert_close({"dk": np64(full["dk"][0, h][kk]), "dv": np64(full["dv"][0, h][kk])}, {"dk": dk, "dv": dv},
                 names=("dk", "dv"), label=f"wave variants d={d} sampled key rows")


def test_twelve_wave_grid_in_the_sequence_major_layout():
    # the same grid through the strided entry points ([B, N, H, d] operands
    # and outputs, as an all-to-all hands them over): bitwise equal to the
    # dense call, which takes the same kernel variants
    import paper_2405_15780_amd as va

    t = torch()
    B, H, N, d = 1, 6, 22001, 64
    print(f"case wave variants sequence-major B={B} H={H} N={N} d={d}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=9990)
    scale = 1.0 / np.sqrt(d)
    dense = run_hip(x, scale)

    def bnhd(bits):  # stored [B, N, H, d], viewed as [B, H, N, d]
        a = t.from_numpy(np.ascontiguousarray(bits.transpose(0, 2, 1, 3)).view(np.int16)).view(t.bfloat16).cuda()
        return a.transpose(1, 2)

    dev = {n: bnhd(a) for n, a in x.items()}
    f32 = dict(dtype=t.float32, device="cuda")
    outs = [t.empty((B, N, H, d), **f32).transpose(1, 2) for _ in range(4)]
    o, dq, dk, dv = outs
    lse = t.empty((B, H, N), **f32)
    va.fwd(dev["q"], dev["k"], dev["v"], scale, out=(o, lse))
    va.bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], scale, out=(dq, dk, dv))
    t.cuda.synchronize()
    for name, a in (("o", o), ("lse", lse), ("dq", dq), ("dk", dk), ("dv", dv)):
        assert t.equal(a, dense[name]), name
