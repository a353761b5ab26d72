"""Write the stored expected dK/dV rows for the long-sequence workloads.

A key row's dK and dV depend on LSE_i and D_i of every query row i of its
head, i.e. on one full fp64 forward pass per head, which takes minutes on a
CPU. This script runs that pass with the oracle once, for the 256 seeded
sampled key rows of each workload, and stores the results as
sampled_grads_c<id>.npz next to itself, together with content hashes of the
seeded inputs so a reader can detect generator drift.

Only the oracle and the seeded input generator are called.
Usage: python tests/golden/make_sampled_grads.py [workload ids...]  (default 3 4)
"""
import os
import sys

os.environ.setdefault("OPENBLAS_NUM_THREADS", "1")
os.environ.setdefault("OMP_NUM_THREADS", "1")

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import multiprocessing as mp  # noqa: E402
import time  # noqa: E402

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import workloads  # noqa: E402

_inputs = {}


def _task(args):
    cid, b, h, keys = args
    w = workloads.WORKLOADS[cid]
    x = _inputs[cid]
    t0 = time.time()
    lse, D = oracle.row_statistics(x["q"], x["k"], x["v"], x["dout"], w.scale, b, h)
    dk, dv = oracle.key_rows(x["q"], x["k"], x["v"], x["dout"], w.scale, b, h, keys, lse, D)
    print(f"{w.name} head ({b},{h}): {len(keys)} key rows in {time.time() - t0:.0f}s", flush=True)
    return cid, b, h, keys, dk, dv


def main(cids):
    for cid in cids:
        _inputs[cid] = workloads.make_inputs(workloads.WORKLOADS[cid])
    tasks = []
    for cid in cids:
        rows = workloads.sampled_key_rows(workloads.WORKLOADS[cid])
        for b, h in sorted({(int(r[0]), int(r[1])) for r in rows}):
            sel = (rows[:, 0] == b) & (rows[:, 1] == h)
            tasks.append((cid, b, h, rows[sel, 2]))
    procs = min(len(tasks), max(1, (os.cpu_count() or 2) - 1))
    with mp.get_context("fork").Pool(procs) as pool:
        results = pool.map(_task, tasks, chunksize=1)
    for cid in cids:
        w = workloads.WORKLOADS[cid]
        rows = workloads.sampled_key_rows(w)
        dk = np.full((len(rows), w.d), np.nan)
        dv = np.full((len(rows), w.d), np.nan)
        for rc, b, h, keys, rdk, rdv in results:
            if rc != cid:
                continue
            for j, key in enumerate(keys):
                idx = np.nonzero((rows[:, 0] == b) & (rows[:, 1] == h) & (rows[:, 2] == key))[0][0]
                dk[idx], dv[idx] = rdk[j], rdv[j]
        assert np.isfinite(dk).all() and np.isfinite(dv).all()
        x = _inputs[cid]
        out = os.path.join(HERE, f"sampled_grads_c{cid}.npz")
        np.savez_compressed(
            out, key_rows=rows, dk=dk.astype(np.float32), dv=dv.astype(np.float32),
            fingerprints=np.array([workloads.fingerprint(x[n]) for n in ("q", "k", "v", "dout")]),
            workload=np.array(w.name))
        print("wrote", out, flush=True)


if __name__ == "__main__":
    main([int(a) for a in sys.argv[1:]] or [3, 4])
