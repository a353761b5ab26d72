"""GPU parity of the channel aggregation (one learnable query per head over
each patch's channel tokens): forward and backward against the oracle,
element by element, over channel counts below, at and above one 64-key
chunk (the paper's 92 included), more patches than the backward's block
count (several patches per block in the dq reduction), and determinism."""
import numpy as np
import pytest

from oracle import aggregation as agg
import workloads
from gpu_util import TOL_GRAD_REL, TOL_LSE_MAX, TOL_O_MAX, TOL_O_REL, rel_l2, to_device, torch

pytestmark = pytest.mark.gpu

SHAPES = [(3, 2, 92, 64), (5, 4, 92, 128), (1, 1, 1, 64), (7, 3, 200, 128), (2, 2, 64, 64), (2100, 2, 92, 64),
          (4, 12, 92, 64)]


def np64(t):
    return t.detach().double().cpu().numpy()


def run(M, H, C, d, seed):
    import paper_2405_15780_amd as va

    x = workloads.make_aggregation_inputs(M, H, C, d, seed=seed)
    dev = {n: to_device(a) for n, a in x.items()}
    scale = 1.0 / np.sqrt(d)
    o, lse = va.agg_fwd(dev["q"], dev["k"], dev["v"], scale)
    dq, dk, dv = va.agg_bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], scale)
    torch().cuda.synchronize()
    return x, scale, {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


@pytest.mark.parametrize("M,H,C,d", SHAPES)
def test_aggregation_forward_backward_against_oracle(M, H, C, d):
    print(f"case M={M} H={H} C={C} d={d}", flush=True)
    x, scale, got = run(M, H, C, d, seed=800 + M + C + d)
    ref = agg.backward(x["q"], x["k"], x["v"], x["dout"], scale)
    g = {n: np64(t) for n, t in got.items()}
    rep = {"o_max": float(np.abs(g["o"] - ref["o"]).max()), "o_rel": rel_l2(g["o"], ref["o"]),
           "lse_max": float(np.abs(g["lse"] - ref["lse"]).max())}
    for n in ("dq", "dk", "dv"):
        if np.linalg.norm(ref[n]) == 0.0:  # e.g. C = 1: p = 1 and ds = 0 exactly
            rep[n + "_abs"] = float(np.abs(g[n]).max())
        else:
            rep[n + "_rel"] = rel_l2(g[n], ref[n])
    print(f"aggregation M={M} H={H} C={C} d={d}", rep, flush=True)
    assert rep["o_max"] <= TOL_O_MAX and rep["o_rel"] <= TOL_O_REL and rep["lse_max"] <= TOL_LSE_MAX, rep
    for n in ("dq", "dk", "dv"):
        assert rep.get(n + "_rel", 0.0) <= TOL_GRAD_REL and rep.get(n + "_abs", 0.0) <= 1e-5, rep


def test_aggregation_is_deterministic():
    _, _, a = run(1500, 2, 92, 128, seed=881)
    _, _, b = run(1500, 2, 92, 128, seed=881)
    for n in a:
        assert torch().equal(a[n], b[n]), n
