"""Seeded random sweep of valid attention calls: batch, heads, query and key
counts (Nq != Nk), every head dim up to 160, softmax scales of 1/2, 1 and 2
times 1/sqrt(d), dense / sequence-major / padded operand layouts and both
backward modes, each compared element by element
with the oracle (forward, and the backward of one key segment holding all
keys)."""
import numpy as np
import pytest

import oracle
from oracle.segments import segment_backward
import workloads
from gpu_util import assert_close, to_device, torch

pytestmark = pytest.mark.gpu


def np64(t):
    return t.detach().double().cpu().numpy()


def draw_case(rng):
    return dict(B=int(rng.choice([1, 2, 3])), H=int(rng.choice([1, 2, 3, 5])), Nq=int(rng.integers(1, 600)),
                Nk=int(rng.integers(1, 600)), d=int(rng.choice(np.arange(8, 161, 8))),
                layout=str(rng.choice(["dense", "bnhd", "padded"])), store_ds=bool(rng.integers(0, 2)),
                pad=8 * int(rng.integers(1, 5)), scale_x=float(rng.choice([0.5, 1.0, 2.0])))


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_random_valid_calls_match_the_oracle(seed):
    import paper_2405_15780_amd as va

    t = torch()
    rng = np.random.default_rng(seed)
    for case in range(40):
        c = draw_case(rng)
        B, H, Nq, Nk, d, layout = c["B"], c["H"], c["Nq"], c["Nk"], c["d"], c["layout"]
        label = f"seed {seed} case {case}: {c}"
        print(label, flush=True)
        xq = workloads.make_small_inputs(B, H, Nq, d, seed=100000 * seed + 2 * case)
        xk = workloads.make_small_inputs(B, H, Nk, d, seed=100000 * seed + 2 * case + 1, with_dout=False)
        scale = c["scale_x"] / np.sqrt(d)

        def put(bits):
            if layout == "dense":
                return to_device(bits)
            if layout == "bnhd":
                return to_device(np.ascontiguousarray(bits.transpose(0, 2, 1, 3))).transpose(1, 2)
            buf = t.zeros(bits.shape[:3] + (d + c["pad"],), dtype=t.bfloat16, device="cuda")
            buf[..., :d] = to_device(bits)
            return buf[..., :d]

        def out(n):
            if layout == "bnhd":
                return t.empty((B, n, H, d), dtype=t.float32, device="cuda").transpose(1, 2)
            return t.empty((B, H, n, d), dtype=t.float32, device="cuda")

        q, k, v, g = put(xq["q"]), put(xk["k"]), put(xk["v"]), put(xq["dout"])
        lse = t.empty((B, H, Nq), dtype=t.float32, device="cuda")
        o, lse = va.fwd(q, k, v, scale, out=(out(Nq), lse))
        dq, dk, dv = va.bwd(q, k, v, o, lse, g, scale, out=(out(Nq), out(Nk), out(Nk)), store_ds=c["store_ds"])
        t.cuda.synchronize()
        ref_o, ref_lse = oracle.forward(xq["q"], xk["k"], xk["v"], scale)
        ref_dq, ref_dk, ref_dv = segment_backward(xq["q"], xk["k"], xk["v"], xq["dout"], ref_o, ref_lse, scale)
        assert_close({"o": np64(o), "lse": np64(lse), "dq": np64(dq), "dk": np64(dk), "dv": np64(dv)},
                     {"o": ref_o, "lse": ref_lse, "dq": ref_dq, "dk": ref_dk, "dv": ref_dv}, label=label)
