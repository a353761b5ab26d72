"""Run-to-run bitwise determinism of every entry point that has no fixed
summation order elsewhere: the dS-mode backward (dK/dV kernel with its dS
stores, dQ from the stored blocks), dQ accumulated over key segments, the
merge, and the channel aggregation with its dq partials. The only atomics
are the dK/dV kernel's split key blocks (all of this shape's key blocks: two
fp32 adds onto zero per element, which commute exactly), so two runs on the
same inputs must agree bit for bit. Calls made at the same time from two
host threads on two streams give the bits of the same calls made alone."""
import numpy as np
import pytest

import workloads
from gpu_util import to_device, torch

pytestmark = pytest.mark.gpu


def _run_all():
    import paper_2405_15780_amd as va

    t = torch()
    out = {}
    B, H, N, d = 2, 3, 1000, 128
    x = workloads.make_small_inputs(B, H, N, d, seed=9600)
    dev = {n: to_device(a) for n, a in x.items()}
    o, lse = va.fwd(dev["q"], dev["k"], dev["v"])
    out["ds-mode"] = va.bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], store_ds=True)
    dq = t.zeros((B, H, N, d), dtype=t.float32, device="cuda")
    for a, b in ((0, 311), (311, 1000)):
        va.bwd(dev["q"], dev["k"][:, :, a:b].contiguous(), dev["v"][:, :, a:b].contiguous(), o, lse, dev["dout"],
               out=(dq, t.empty((B, H, b - a, d), device="cuda"), t.empty((B, H, b - a, d), device="cuda")),
               accumulate_dq=True)
    out["segments dq"] = (dq,)
    rng = np.random.default_rng(1)
    parts = t.from_numpy(rng.standard_normal((5, B, H, N, 72)).astype(np.float32)).cuda()
    lparts = t.from_numpy(rng.standard_normal((5, B, H, N)).astype(np.float32)).cuda()
    out["merge"] = va.merge(parts, lparts)
    xa = workloads.make_aggregation_inputs(2100, 4, 92, 64, seed=9601)
    da = {n: to_device(a) for n, a in xa.items()}
    oa, la = va.agg_fwd(da["q"], da["k"], da["v"])
    out["agg"] = (oa, la) + tuple(va.agg_bwd(da["q"], da["k"], da["v"], oa, la, da["dout"]))
    t.cuda.synchronize()
    return out


def test_repeated_runs_are_bitwise_equal():
    t = torch()
    print("case determinism", flush=True)
    first, second = _run_all(), _run_all()
    for name, tensors in first.items():
        for i, (a, b) in enumerate(zip(tensors, second[name])):
            assert t.equal(a, b), f"{name} output {i} differs between two runs"


def test_concurrent_calls_on_two_streams_from_two_threads():
    """Two host threads, each on a stream of its own (default priority), run
    forward and backward passes of different shapes and head dims at the same
    time, three times each, on the first calls of their kernel variants in
    this process where the test runs alone: every output is bitwise equal to
    that of the same call made on its own. The calls share nothing but the
    per-device kernel lookups (atomics), so they must not interfere."""
    import threading

    import paper_2405_15780_amd as va

    t = torch()
    cases = [(1, 3, 3001, 56), (2, 1, 2500, 136)]
    print(f"case concurrent streams {cases}", flush=True)
    inputs = [{n: to_device(a) for n, a in workloads.make_small_inputs(*c, seed=9700 + i).items()}
              for i, c in enumerate(cases)]
    t.cuda.synchronize()

    def call(x):
        o, lse = va.fwd(x["q"], x["k"], x["v"])
        return (o, lse) + tuple(va.bwd(x["q"], x["k"], x["v"], o, lse, x["dout"]))

    results = [[None] * 3 for _ in cases]
    errors = []

    def worker(i):
        try:
            s = t.cuda.Stream()
            with t.cuda.stream(s):
                for rep in range(3):
                    results[i][rep] = call(inputs[i])
            s.synchronize()
        except Exception as e:  # reported on the main thread
            errors.append((i, e))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(cases))]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors
    alone = [call(x) for x in inputs]
    t.cuda.synchronize()
    for i, c in enumerate(cases):
        for rep in range(3):
            for n, a, b in zip(("o", "lse", "dq", "dk", "dv"), results[i][rep], alone[i]):
                assert t.equal(a, b), f"{c} repeat {rep}: {n} differs from the call made alone"
