"""The allocation-free backward (vitattn_bwd_noalloc, the library's static
scratch in place of a workspace) against vitattn_bwd, through the C ABI:
bitwise equal outputs on two calls in a row, the second on a smaller input
(the scratch keeps the first call's contents), both also within the
oracle's tolerances."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_close, to_device, torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("first,second", [((2, 3, 1000, 128), (1, 2, 300, 64)), ((1, 2, 4097, 72), (1, 1, 17, 128))])
def test_noalloc_backward_matches_workspace_backward(first, second):
    import paper_2405_15780_amd as va

    t = torch()
    for B, H, N, d in (first, second):
        print(f"case noalloc B={B} H={H} N={N} d={d}", flush=True)
        x = workloads.make_small_inputs(B, H, N, d, seed=8800 + N + d)
        dev = {n: to_device(a) for n, a in x.items()}
        scale = 1.0 / np.sqrt(d)
        o, lse = va.fwd(dev["q"], dev["k"], dev["v"], scale)
        ref = va.bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], scale)
        got = va.bwd_noalloc(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], scale)
        t.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv"), got, ref):
            assert t.equal(a, b), (name, B, H, N, d)
        want = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
        assert_close({n: a.double().cpu().numpy() for n, a in zip(("dq", "dk", "dv"), got)}, want,
                     names=("dq", "dk", "dv"), label=f"noalloc {B},{H},{N},{d}")
