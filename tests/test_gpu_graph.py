"""The library's calls only launch kernels on the caller's stream (no
allocation, synchronisation or memset), so a forward + backward step can be
captured in a HIP graph and replayed. Each replay is checked bitwise against
the eager call on the same inputs, with eager work and synchronisations
between replays, and after the inputs change in place."""
import numpy as np
import pytest

import workloads
from gpu_util import to_device, torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("store_ds", [False, True], ids=["recompute", "stored-ds"])
def test_captured_step_replays_match_eager(store_ds):
    import paper_2405_15780_amd as va

    t = torch()
    B, H, N, d = 1, 2, 1000, 128
    print(f"case graph replay store_ds={store_ds}", flush=True)
    scale = 1.0 / np.sqrt(d)
    flags = va.VITATTN_BWD_STORE_DS if store_ds else 0

    def inputs(seed):
        x = workloads.make_small_inputs(B, H, N, d, seed=seed)
        return {n: to_device(a) for n, a in x.items()}

    static = inputs(6100)
    f32 = dict(dtype=t.float32, device="cuda")
    o, lse = t.empty((B, H, N, d), **f32), t.empty((B, H, N), **f32)
    dq, dk, dv = (t.empty((B, H, N, d), **f32) for _ in range(3))
    ws = t.empty(va.workspace_bytes_kv(B, H, N, N, d, flags) // 4 + 64, **f32)

    def step(x, outs):
        o_, lse_, dq_, dk_, dv_ = outs
        va.fwd(x["q"], x["k"], x["v"], scale, out=(o_, lse_))
        va.bwd(x["q"], x["k"], x["v"], o_, lse_, x["dout"], scale, workspace=ws, out=(dq_, dk_, dv_),
               store_ds=store_ds)

    def eager(x):
        outs = (t.empty_like(o), t.empty_like(lse), t.empty_like(dq), t.empty_like(dk), t.empty_like(dv))
        step(x, outs)
        t.cuda.synchronize()
        return outs

    side = t.cuda.Stream()
    side.wait_stream(t.cuda.current_stream())
    with t.cuda.stream(side):  # warm-up off the default stream, as torch asks before capture
        step(static, (o, lse, dq, dk, dv))
    t.cuda.current_stream().wait_stream(side)
    t.cuda.synchronize()

    g = t.cuda.CUDAGraph()
    with t.cuda.graph(g):
        step(static, (o, lse, dq, dk, dv))
    t.cuda.synchronize()

    ref = eager(static)
    for rep in range(3):
        g.replay()
        t.cuda.synchronize()
        for name, a, b in zip(("o", "lse", "dq", "dk", "dv"), (o, lse, dq, dk, dv), ref):
            assert t.equal(a, b), f"replay {rep}: {name} differs from the eager call"
        eager(inputs(6200 + rep))  # unrelated eager work between replays

    new = inputs(6300)
    for n in static:
        static[n].copy_(new[n])
    ref = eager(static)
    g.replay()
    t.cuda.synchronize()
    for name, a, b in zip(("o", "lse", "dq", "dk", "dv"), (o, lse, dq, dk, dv), ref):
        assert t.equal(a, b), f"replay on new inputs: {name} differs from the eager call"


_FIRST_CALL_CAPTURED = r"""
import sys
import numpy as np
import torch
sys.path.insert(0, sys.argv[1])
sys.path.insert(0, sys.argv[1] + "/tests")
import paper_2405_15780_amd as va
import workloads
from gpu_util import to_device
B, H, N, d = 1, 3, 700, 96
x = {n: to_device(a) for n, a in workloads.make_small_inputs(B, H, N, d, seed=6400).items()}
f32 = dict(dtype=torch.float32, device="cuda")
o, lse = torch.empty((B, H, N, d), **f32), torch.empty((B, H, N), **f32)
grads = tuple(torch.empty((B, H, N, d), **f32) for _ in range(3))
ws = torch.empty(va.workspace_bytes_kv(B, H, N, N, d, va.VITATTN_BWD_STORE_DS) // 4 + 64, **f32)
va.fwd(x["q"], x["k"], x["v"], out=(o, lse))
torch.cuda.synchronize()
g = torch.cuda.CUDAGraph()
with torch.cuda.graph(g):  # the process's first backward call
    va.bwd(x["q"], x["k"], x["v"], o, lse, x["dout"], workspace=ws, out=grads, store_ds=True)
for rep in range(2):
    g.replay()
    torch.cuda.synchronize()
    ref = va.bwd(x["q"], x["k"], x["v"], o, lse, x["dout"], store_ds=True)
    torch.cuda.synchronize()
    for name, a, b in zip(("dq", "dk", "dv"), grads, ref):
        assert torch.equal(a, b), (rep, name)
print("first captured call ok", flush=True)
"""


def test_first_backward_call_inside_capture():
    # The backward's launch looks up, once per device, how many dK/dV
    # workgroups are resident at once (no stream work). In a fresh process the
    # first call, and with it that lookup, happens during capture.
    import os
    import subprocess
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    print("case first backward call inside capture (child process)", flush=True)
    r = subprocess.run([sys.executable, "-c", _FIRST_CALL_CAPTURED, root], capture_output=True, text=True,
                       timeout=300)
    print(r.stdout[-2000:], r.stderr[-2000:], flush=True)
    assert r.returncode == 0 and "first captured call ok" in r.stdout


_NOALLOC_CAPTURED = r"""
import sys
import numpy as np
import torch
sys.path.insert(0, sys.argv[1])
sys.path.insert(0, sys.argv[1] + "/tests")
import paper_2405_15780_amd as va
import workloads
from gpu_util import to_device
B, H, N, d = 1, 6, 2300, 64
x = {n: to_device(a) for n, a in workloads.make_small_inputs(B, H, N, d, seed=6500).items()}
f32 = dict(dtype=torch.float32, device="cuda")
o, lse = torch.empty((B, H, N, d), **f32), torch.empty((B, H, N), **f32)
grads = tuple(torch.empty((B, H, N, d), **f32) for _ in range(3))
torch.cuda.synchronize()
g = torch.cuda.CUDAGraph()
with torch.cuda.graph(g):  # the process's first forward and backward calls, without a workspace
    va.fwd(x["q"], x["k"], x["v"], out=(o, lse))
    va.bwd_noalloc(x["q"], x["k"], x["v"], o, lse, x["dout"], out=grads)
for rep in range(3):
    g.replay()
    torch.cuda.synchronize()
    o2, lse2 = va.fwd(x["q"], x["k"], x["v"])
    ref = va.bwd(x["q"], x["k"], x["v"], o2, lse2, x["dout"])
    torch.cuda.synchronize()
    for name, a, b in zip(("o", "lse", "dq", "dk", "dv"), (o, lse) + grads, (o2, lse2) + ref):
        assert torch.equal(a, b), (rep, name)
print("captured noalloc step ok", flush=True)
"""


def test_first_calls_captured_with_the_allocation_free_backward():
    # A fresh process whose first forward and backward calls are captured:
    # the once-per-device lookups (resident workgroups of the d <= 64 kernel
    # variants, the static scratch's device address) happen during capture,
    # and the allocation-free backward needs no workspace there.
    import os
    import subprocess
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    print("case first calls inside capture with bwd_noalloc (child process)", flush=True)
    r = subprocess.run([sys.executable, "-c", _NOALLOC_CAPTURED, root], capture_output=True, text=True, timeout=300)
    print(r.stdout[-2000:], r.stderr[-2000:], flush=True)
    assert r.returncode == 0 and "captured noalloc step ok" in r.stdout
