"""The LDS-poison debug build (-DVITATTN_DEBUG_LDS_POISON): every kernel first
fills its LDS with all-ones bytes, NaN as bf16 and as fp32, so a read of LDS
that nothing wrote would turn outputs into NaN. Each case runs through the
normal library and then through the poisoned one (swapped in for the
package's library), and every output must be equal bitwise: forward and both
backward modes over ragged tails, Nq != Nk, every tile width and a
sequence-major layout, the merge and the channel aggregation."""
import os

import numpy as np
import pytest

import workloads
from gpu_util import to_device, torch

pytestmark = pytest.mark.gpu


def _outputs():
    import paper_2405_15780_amd as va

    t = torch()
    res = {}
    cases = [(1, 2, 300, 300, 64), (2, 1, 129, 77, 128), (1, 1, 1, 1, 8), (1, 2, 200, 450, 72), (1, 1, 257, 130, 160),
             (2, 3, 70, 600, 96)]
    for ci, (B, H, Nq, Nk, d) in enumerate(cases):
        xq = workloads.make_small_inputs(B, H, Nq, d, seed=9000 + ci)
        xk = workloads.make_small_inputs(B, H, Nk, d, seed=9100 + ci, with_dout=False)
        scale = 1.0 / np.sqrt(d)
        bnhd = ci % 2 == 1

        def put(bits):
            if bnhd:
                return to_device(np.ascontiguousarray(bits.transpose(0, 2, 1, 3))).transpose(1, 2)
            return to_device(bits)

        q, k, v, g = put(xq["q"]), put(xk["k"]), put(xk["v"]), put(xq["dout"])
        o, lse = va.fwd(q, k, v, scale)
        res[f"case {ci} o"], res[f"case {ci} lse"] = o, lse
        for store_ds in (False, True):
            dq, dk, dv = va.bwd(q, k, v, o, lse, g, scale, store_ds=store_ds)
            for n, x in (("dq", dq), ("dk", dk), ("dv", dv)):
                res[f"case {ci} {n} store_ds={store_ds}"] = x
    rng = np.random.default_rng(5)
    parts = t.from_numpy(rng.standard_normal((3, 1, 2, 77, 72)).astype(np.float32)).cuda()
    lparts = t.from_numpy(rng.standard_normal((3, 1, 2, 77)).astype(np.float32)).cuda()
    res["merge o"], res["merge lse"] = va.merge(parts, lparts)
    for M, H, C, d in ((3, 2, 92, 64), (5, 3, 200, 128), (1, 1, 1, 64)):
        x = workloads.make_aggregation_inputs(M, H, C, d, seed=9200 + C)
        dev = {n: to_device(a) for n, a in x.items()}
        o, lse = va.agg_fwd(dev["q"], dev["k"], dev["v"])
        dq, dk, dv = va.agg_bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"])
        for n, y in (("o", o), ("lse", lse), ("dq", dq), ("dk", dk), ("dv", dv)):
            res[f"agg {M},{H},{C},{d} {n}"] = y
    t.cuda.synchronize()
    return res


def test_poisoned_lds_changes_no_output():
    import paper_2405_15780_amd.binding as b
    from paper_2405_15780_amd._build import LDS_POISON_LIB_PATH

    t = torch()
    print("case LDS poison build", flush=True)
    assert os.path.exists(LDS_POISON_LIB_PATH), "build() compiles the LDS-poison variant beside the library"
    normal = b.library()
    ref = _outputs()
    b._lib = b.open_library(LDS_POISON_LIB_PATH)
    try:
        got = _outputs()
    finally:
        b._lib = normal
    for name, x in ref.items():
        y = got[name]
        assert bool(t.isfinite(y).all()) == bool(t.isfinite(x).all()), f"{name}: non-finite values with poisoned LDS"
        assert t.equal(x, y), f"{name} differs when the kernels' LDS starts as NaN"
