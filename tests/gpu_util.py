"""Helpers for the GPU parity tests: move seeded bf16 inputs to the device,
run the HIP path through the binding, and compare with the oracle."""
import numpy as np

# Tolerances: bf16 inputs, fp32 accumulation. O and the gradients use the
# stated bounds; the LSE bound is derived from fp32 rounding of logits that
# reach a few hundred nats in the stress head (ulp(300) ~ 3e-5) plus the
# bf16 rounding of nothing (LSE uses fp32 P only).
TOL_O_MAX = 1e-2
TOL_O_REL = 5e-3
TOL_GRAD_REL = 1e-2
TOL_LSE_MAX = 2e-3


def torch():
    import torch as t

    return t


def to_device(bits):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(t.bfloat16).cuda()


def run_hip(x, scale, backward=True, store_ds=False):
    """Forward (and backward) through the binding; store_ds selects the
    backward's dS mode (dQ from stored dS), whose workspace is freed again."""
    import paper_2405_15780_amd as va

    t = torch()
    dev = {n: to_device(a) for n, a in x.items()}
    o, lse = va.fwd(dev["q"], dev["k"], dev["v"], scale)
    res = {"o": o, "lse": lse}
    if backward:
        dq, dk, dv = va.bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], scale, store_ds=store_ds)
        res.update(dq=dq, dk=dk, dv=dv)
    t.cuda.synchronize()
    if store_ds:
        t.cuda.empty_cache()
    return res


def oracle_all_heads(x, scale):
    """oracle.forward_backward over every (b, h) of x, one head per task on a
    thread pool (numpy releases the GIL in its array loops; BLAS is held to
    one thread per task). The arithmetic is the oracle's own; only the heads
    are evaluated concurrently, which keeps a 32-head 16,384-token workload
    to well under a minute on the host's cores."""
    import os
    from concurrent.futures import ThreadPoolExecutor

    from threadpoolctl import threadpool_limits

    import oracle

    B, H = x["q"].shape[:2]
    out = {}

    def one(bh):
        b, h = bh
        sl = {n: a[b:b + 1, h:h + 1] for n, a in x.items()}
        return bh, oracle.forward_backward(sl["q"], sl["k"], sl["v"], sl["dout"], scale)

    workers = max(1, min(16, len(os.sched_getaffinity(0))))
    with threadpool_limits(1), ThreadPoolExecutor(workers) as ex:
        for (b, h), r in ex.map(one, [(b, h) for b in range(B) for h in range(H)]):
            for n, a in r.items():
                if n not in out:
                    out[n] = np.empty((B, H) + a.shape[2:])
                out[n][b, h] = a[0, 0]
    return out


def oracle_one_head(x, scale, b, h, block=256):
    """All outputs of head (b, h) from the oracle, its query blocks evaluated
    concurrently (oracle.forward_backward_rows on a thread pool, BLAS held to
    one thread per task) and the blocks' dK, dV contributions summed in block
    order: the oracle's arithmetic, with a head too long for one core done in
    parallel."""
    import os
    from concurrent.futures import ThreadPoolExecutor

    from threadpoolctl import threadpool_limits

    import oracle

    N = x["q"].shape[2]
    starts = list(range(0, N, block))

    def one(r0):
        return oracle.forward_backward_rows(x["q"], x["k"], x["v"], x["dout"], scale, b, h, r0, min(N, r0 + block))

    workers = max(1, min(16, len(os.sched_getaffinity(0))))
    d = x["q"].shape[3]
    out = {"o": np.empty((N, d)), "lse": np.empty(N), "dq": np.empty((N, d)), "dk": np.zeros((N, d)),
           "dv": np.zeros((N, d))}
    with threadpool_limits(1), ThreadPoolExecutor(workers) as ex:
        for r0, r in zip(starts, ex.map(one, starts)):
            r1 = min(N, r0 + block)
            out["o"][r0:r1], out["lse"][r0:r1], out["dq"][r0:r1] = r["o"], r["lse"], r["dq"]
            out["dk"] += r["dk_part"]
            out["dv"] += r["dv_part"]
    return out


def rel_l2(got, ref):
    return float(np.linalg.norm(got - ref) / np.linalg.norm(ref))


def assert_close(got: dict, ref: dict, names=("o", "lse", "dq", "dk", "dv"), label=""):
    """got: numpy fp64 arrays from the GPU; ref: oracle arrays (same shapes)."""
    report = {}
    for n in names:
        if n not in got:
            continue
        g, r = got[n], ref[n]
        assert g.shape == r.shape, (n, g.shape, r.shape)
        assert np.isfinite(g).all(), f"{label} {n}: non-finite values"
        if n == "o":
            report["o_max"] = float(np.abs(g - r).max())
            report["o_rel"] = rel_l2(g, r)
        elif n == "lse":
            report["lse_max"] = float(np.abs(g - r).max())
        elif np.linalg.norm(r) == 0.0:
            # exact gradient is zero (e.g. N = 1): bound the absolute error
            report[n + "_abs"] = float(np.abs(g).max())
        else:
            report[n + "_rel"] = rel_l2(g, r)
    print(label, report, flush=True)
    if "o_max" in report:
        assert report["o_max"] <= TOL_O_MAX, (label, report)
        assert report["o_rel"] <= TOL_O_REL, (label, report)
    if "lse_max" in report:
        assert report["lse_max"] <= TOL_LSE_MAX, (label, report)
    for n in ("dq", "dk", "dv"):
        if n + "_rel" in report:
            assert report[n + "_rel"] <= TOL_GRAD_REL, (label, report)
        if n + "_abs" in report:
            assert report[n + "_abs"] <= 1e-5, (label, report)
    return report
