"""attention() as a torch.autograd op: its gradients are the library's
backward on the bf16-rounded upstream gradient (bitwise), in both backward
modes and for a sequence-major operand layout, and they match the oracle."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_close, to_device, torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("store_ds", [False, True], ids=["recompute", "stored-ds"])
@pytest.mark.parametrize("layout", ["dense", "bnhd"])
def test_autograd_gradients_are_the_library_backward(store_ds, layout):
    import paper_2405_15780_amd as va

    t = torch()
    B, H, N, d = 1, 2, 333, 64
    print(f"case autograd store_ds={store_ds} layout={layout}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=7100)
    scale = 1.0 / np.sqrt(d)

    def put(bits):
        if layout == "bnhd":
            return to_device(np.ascontiguousarray(bits.transpose(0, 2, 1, 3))).transpose(1, 2)
        return to_device(bits)

    q, k, v = (put(x[n]).detach().requires_grad_(True) for n in ("q", "k", "v"))
    dout_bf16 = put(x["dout"])
    g = dout_bf16.float()  # exactly representable in bf16, so the op's rounding is exact
    o = va.attention(q, k, v, store_ds=store_ds)
    (o * g).sum().backward()
    t.cuda.synchronize()
    o_ref, lse = va.fwd(q.detach(), k.detach(), v.detach(), scale)
    dq, dk, dv = va.bwd(q.detach(), k.detach(), v.detach(), o_ref, lse, dout_bf16, scale, store_ds=store_ds)
    t.cuda.synchronize()
    assert t.equal(o, o_ref)
    for name, a, b in (("dq", q.grad, dq), ("dk", k.grad, dk), ("dv", v.grad, dv)):
        assert a.dtype == t.bfloat16 and t.equal(a, b.to(t.bfloat16)), name
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    got = {"o": o.detach().double().cpu().numpy(), "dq": dq.double().cpu().numpy(),
           "dk": dk.double().cpu().numpy(), "dv": dv.double().cpu().numpy()}
    assert_close(got, ref, names=("o", "dq", "dk", "dv"), label=f"autograd {layout} store_ds={store_ds}")
