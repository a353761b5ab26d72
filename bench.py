"""Benchmark: exact non-causal attention forward + backward on one MI355X.

One step = the whole hot path over one batch: vitattn_fwd, then the three
backward stages (rowdot preprocess, dK/dV, dQ), on inputs already resident in
HBM. The default workload is the paper-scale shard B=1, H=2, N=188,416
(368 x 512 patches = 92 channels x 2,048), d=128, bf16 inputs with fp32
accumulation and outputs.

value = counted FLOPs / step time, FlashAttention convention: forward
4 B H N^2 d, backward 10 B H N^2 d (P's recomputation is not counted).

Prints one JSON line. `roofline` describes the kernel with the largest share
of the step time, timed with HIP events on the stream it is launched on
(PyTorch's current stream, which the binding passes to the library).
`cpu_baseline` times the fp64 oracle on a bounded slice of the same workload
(a block of query rows of head 0, forward plus that block's backward work)
and extrapolates it, labelled as such, to the whole workload. `clock` holds
the graphics clock and socket power amd-smi read during the timed steps and
the percentage of the dense bf16 peak at that clock (the chip holds well
below its 2.4 GHz peak clock under this load).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # MI355X dense bf16 MFMA (256 CU x 4096 flop/clk x 2.4 GHz)
PEAK_HBM_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", type=int, default=4,
                   help="attention workload id of workloads.WORKLOADS (4 = B1 H2 N188416 d128, the metric's)")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle time budget for cpu_baseline")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain 512 MiB device copy (to scale rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    p.add_argument("--bwd-mode", choices=["recompute", "stored-ds"], default="recompute",
                   help="backward pass: recompute (the default: dQ recomputes S and dP, O(N d) memory), or "
                        "stored-ds (opt-in: dQ from the dS blocks the dK/dV kernel stores, a B*H*N^2*2-byte "
                        "workspace, 142 GB at the 188,416-token workload)")
    p.add_argument("--hbm-reference", action="store_true",
                   help="only measure the streaming rates of plain elementwise kernels (read+write, "
                        "read 1 : write 2, write only)")
    p.add_argument("--mfma-reference", action="store_true",
                   help="only measure the library bf16 GEMM (torch.matmul, 16384^3) on random normal and on "
                        "zero operands, with the clock and power it runs at")
    p.add_argument("--no-compare", action="store_true",
                   help="skip timing the other backward mode after the timed region (for profiler runs)")
    p.add_argument("--row", choices=["attention", "merge", "ulysses", "agg", "d64", "m1", "d72", "d160", "bnhd"],
                   default="attention",
                   help="which workload to time (default: the attention forward+backward hot path at "
                        "N=188,416, d=128; d64: the paper's own 188K shard, ViT-Base heads at d=64, B=4, "
                        "same flops; m1: ViT-Base at 1M tokens, one head; d72 / d160: the paper's other head dims; bnhd: the default workload "
                        "with sequence-major operands)")
    return p.parse_args()


COPY_BYTES = 512 * 1024 * 1024
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_N188416_d128.json")
ROW_TRAFFIC = {r: os.path.join(ROOT, "profiles", f"hbm_traffic_{r}.json")
               for r in ("merge", "ulysses", "agg", "d64", "m1", "d72", "d160", "bnhd")}


KERNEL_FILES = {
    "attention": ("vitattn_fwd.hip", "vitattn_bwd.hip"),
    "merge": ("vitattn_merge.hip",),
    "ulysses": ("vitattn_ulysses.hip",),
    "agg": ("vitattn_agg.hip",),
    "d64": ("vitattn_fwd.hip", "vitattn_bwd.hip"),
    "m1": ("vitattn_fwd.hip", "vitattn_bwd.hip"),
    "d72": ("vitattn_fwd.hip", "vitattn_bwd.hip"),
    "d160": ("vitattn_fwd.hip", "vitattn_bwd.hip"),
    "bnhd": ("vitattn_fwd.hip", "vitattn_bwd.hip"),
}


def strip_comments(src):
    """C++ source without its comments and blank lines (string and character
    literals kept as they are), so that editing a comment leaves the digest
    below unchanged."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        else:
            out.append(c)
            i += 1
    return "\n".join(line.rstrip() for line in "".join(out).splitlines() if line.strip())


def kernel_sources_digest(row="attention", csrc=None):
    """Hash of the code (comments stripped) of the HIP sources that define one
    kernel family, plus the shared headers, to tell whether stored counter
    readings still describe the kernels being timed."""
    import hashlib

    csrc = csrc or os.path.join(ROOT, "paper_2405_15780_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(KERNEL_FILES[row] + ("vitattn_common.h", "vitattn_launch.h")):
        with open(os.path.join(csrc, name), encoding="utf-8") as f:
            h.update(name.encode() + b"\0" + strip_comments(f.read()).encode())
    return h.hexdigest()[:16]


def stored_traffic(kernel, config_name, row="attention"):
    """HBM bytes per launch of `kernel` from the committed counter summary,
    or None if it is missing or was taken on different kernel sources."""
    path = TRAFFIC_FILE if row == "attention" else ROW_TRAFFIC[row]
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("sources") != kernel_sources_digest(row) or rec.get("workload") != config_name:
        return None
    roof = rec.get("roofline")
    if roof is not None and roof.get("kernel") == kernel:
        return roof.get("hbm_bytes")
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("hbm_bytes_per_launch")


def copy_calibration():
    import torch

    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "launches": 3}), flush=True)


def hbm_reference():
    """Practical HBM streaming rates on this GPU: elementwise torch kernels
    over GiB-sized arrays, the ceilings that the HBM-bound kernels here are
    compared with besides the 8 TB/s datasheet peak. Three mixes: read and
    write equal bytes (fp32 add over 8 GiB), write twice what is read (a
    bf16 -> fp32 conversion copy, 3 GiB in, 6 GiB out: the aggregation
    backward's mix) and write only (fp32 fill over 6 GiB)."""
    import torch

    def timed(fn, reps=10):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    out = {"hbm_reference": "plain torch elementwise kernels", "peak_GB_s": PEAK_HBM_GBS}
    n = (8 << 30) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    ms = timed(lambda: torch.add(a, 1.0, out=b))
    out["add_fp32_read1_write1"] = {"bytes": 2 * n * 4, "ms": ms, "GB_s": 2 * n * 4 / ms / 1e6}
    del a, b
    n = 1536 << 20
    a = torch.ones(n, dtype=torch.bfloat16, device="cuda:0")
    b = torch.empty(n, dtype=torch.float32, device="cuda:0")
    ms = timed(lambda: b.copy_(a))
    out["convert_bf16_to_fp32_read1_write2"] = {"bytes": 6 * n, "ms": ms, "GB_s": 6 * n / ms / 1e6}
    ms = timed(lambda: b.fill_(1.0))
    out["fill_fp32_write_only"] = {"bytes": 4 * n, "ms": ms, "GB_s": 4 * n / ms / 1e6}
    for v in out.values():
        if isinstance(v, dict):
            v["frac_of_8TBs"] = v["GB_s"] / PEAK_HBM_GBS
    print(json.dumps(out), flush=True)


def vendor_gemm_tflops(x, y, reps):
    """Mean rate of torch.matmul (hipBLASLt) on two square bf16 operands."""
    import torch

    n = x.shape[0]
    c = x @ y
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        c = x @ y
    e1.record()
    torch.cuda.synchronize()
    del c
    ms = e0.elapsed_time(e1) / reps
    return ms, 2 * n**3 / ms / 1e9


def mfma_reference():
    """Practical bf16 matrix-core rate on this GPU: the vendor GEMM
    (torch.matmul, which calls hipBLASLt) on 16384^3 bf16 operands, first
    random normal (the bit activity of real activations), then all zeros. The
    dense 2.5 PF/s peak assumes the 2.4 GHz peak clock; under a sustained MFMA
    load the board power limit lowers the clock, and more so the more operand
    bits toggle, so the random-operand rate is the ceiling that the attention
    kernels are compared with besides the datasheet peak."""
    import torch

    n = 16384
    out = {"mfma_reference": "torch.matmul bf16 16384^3", "peak_tflops": PEAK_BF16_TFLOPS}
    a = torch.randn(n, n, device="cuda:0").to(torch.bfloat16)
    b = torch.randn(n, n, device="cuda:0").to(torch.bfloat16)
    z = torch.zeros_like(a)
    for name, x, y in (("random_normal", a, b), ("zeros", z, z)):
        with SmiSampler() as smi:
            ms, tf = vendor_gemm_tflops(x, y, 300)
        out[name] = {"ms": ms, "tflops": tf, "frac_of_peak": tf / PEAK_BF16_TFLOPS, "smi": smi.summary()}
    print(json.dumps(out), flush=True)


class SmiSampler:
    """Samples socket power and the graphics clock with `amd-smi metric -p -c`
    in a background thread (about every 0.25 s) while the timed loop runs.
    Reports nothing if amd-smi is missing or prints something unexpected."""

    def __init__(self):
        import shutil
        import threading

        self.exe = shutil.which("amd-smi")
        # Under a profiler its preloaded library would start in the amd-smi
        # child too and bring up the GPU there before that launcher replaces
        # itself with python: never sample while profiled.
        if "rocprof" in os.environ.get("LD_PRELOAD", "") or any(k.startswith("ROCPROF") for k in os.environ):
            self.exe = None
        self.samples = []
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        import re
        import subprocess

        while not self._stop.is_set():
            try:
                out = subprocess.run([self.exe, "metric", "-p", "-c"], capture_output=True, text=True,
                                     timeout=5).stdout
            except Exception:  # sampling is best effort
                return
            pw = re.search(r"SOCKET_POWER:\s*([0-9.]+)\s*W", out)
            clk = re.search(r"GFX_0:\s*\n\s*CLK:\s*([0-9.]+)\s*MHz", out)
            if pw and clk:
                self.samples.append((float(pw.group(1)), float(clk.group(1))))
            self._stop.wait(0.25)

    def __enter__(self):
        if self.exe:
            self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self.exe and self._thread.is_alive():
            self._thread.join(timeout=10)

    def summary(self):
        if not self.samples:
            return None
        import statistics

        # drop readings taken while the GPU was still idle or ramping; a timed
        # region shorter than amd-smi's sampling interval may have none left,
        # and then nothing is reported
        busy = [(p, c) for p, c in self.samples if c >= 500.0]
        if not busy:
            return None
        pw = [p for p, _ in busy]
        clk = [c for _, c in busy]
        return {"samples": len(busy), "power_w_median": statistics.median(pw),
                "sclk_mhz_median": statistics.median(clk), "sclk_mhz_min": min(clk), "sclk_mhz_max": max(clk)}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w, x, budget_s):
    import numpy as np

    import oracle

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # threadpoolctl missing: report the BLAS default
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    # blocks of up to 512 query rows in workload order (b, h, rows), each
    # against all N keys of its head; a workload smaller than the budget is
    # gone through again from the start
    rows_per_block = 512
    blocks = [(b, h, r0) for b in range(w.B) for h in range(w.H) for r0 in range(0, w.N, rows_per_block)]
    done = n_blocks = 0
    t0 = time.perf_counter()
    while n_blocks == 0 or time.perf_counter() - t0 < budget_s:
        b, h, r0 = blocks[n_blocks % len(blocks)]
        r1 = min(w.N, r0 + rows_per_block)
        if w.backward:
            oracle.forward_backward_rows(x["q"], x["k"], x["v"], x["dout"], w.scale, b, h, r0, r1)
        else:
            rows = np.stack([np.full(r1 - r0, b, np.int64), np.full(r1 - r0, h, np.int64),
                             np.arange(r0, r1, dtype=np.int64)], axis=1)
            oracle.query_rows(x["q"], x["k"], x["v"], w.scale, rows)
        done += r1 - r0
        n_blocks += 1
    dt = time.perf_counter() - t0
    flops = 14.0 * done * w.N * w.d if w.backward else 4.0 * done * w.N * w.d
    rows_total = w.B * w.H * w.N
    passes = "forward+backward" if w.backward else "forward"
    covered = (f"the first {done} of the workload's {rows_total} query rows" if n_blocks <= len(blocks) else
               f"all {rows_total} query rows of the workload, {done / rows_total:.1f} times over")
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"fp64 {passes} of {covered} (blocks of {rows_per_block} rows in (b, h, row) order), each "
                  f"against all {w.N} keys of its head, {dt:.1f} s",
        "seconds": dt,
        "extrapolated_full_seconds": dt * rows_total / done,
        "extrapolated": "per-row time of the sample times all B*H*N query rows (labelled extrapolated, not run)",
        "host_cpus": len(os.sched_getaffinity(0)),
        "cpu_model": cpu_model(),
        "blas_threads": int(threads),
    }


ROW_DOC = {
    "merge": "merge of 8 key-segment partials (O fp32, LSE) at B=1, H=2, N=188,416, d=128",
    "ulysses": ("Ulysses layouts around both all-to-alls of one attention, 8 ranks, ViT-Base heads "
                "(H=16, d=64) at N=188,416 (23,552 tokens per rank): pack + unpack of bf16 Q, K, V, "
                "pack_out + unpack_out of fp32 O"),
    "agg": ("channel aggregation fwd+bwd, Agg-Ch-ViT on ViT-Base heads: M=8,192 patch positions "
            "(batch 4 x 2,048), H=16, C=92 channels, d=64"),
}


def time_events(fn, reps):
    """Mean milliseconds of fn() over `reps` back-to-back calls (HIP events on
    the current stream), after two warm-up calls."""
    import torch

    for _ in range(2):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def timed_cpu(fn, budget_s):
    """Run fn() repeatedly for about budget_s seconds; returns (calls, seconds)."""
    n, t0 = 0, time.perf_counter()
    while n == 0 or time.perf_counter() - t0 < budget_s:
        fn()
        n += 1
    return n, time.perf_counter() - t0


def bench_row(args):
    """Time one of the HBM-bound kernel families beside the attention (key-segment
    merge, Ulysses layouts, channel aggregation) against the HBM roofline, with
    the oracle timed beside it on a bounded sample. Algorithmic bytes are the
    minimal ones: every input read once, every output written once."""
    import numpy as np
    import torch

    import oracle
    import paper_2405_15780_amd as va
    import workloads

    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(0)
    budget = min(args.cpu_seconds, 10.0)
    per_kernel = {}
    if args.row == "merge":
        P, BH, N, d = 8, 2, 188416, 128
        o_parts = torch.randn((P, 1, BH, N, d), device=dev, generator=g)
        lse_parts = 3.0 * torch.randn((P, 1, BH, N), device=dev, generator=g)
        outs = (torch.empty((1, BH, N, d), device=dev), torch.empty((1, BH, N), device=dev))
        ms = time_events(lambda: va.merge(o_parts, lse_parts, out=outs), args.steps)
        nbytes = (P + 1) * BH * N * (d + 1) * 4
        dom, dom_ms, dom_bytes = "attn_merge_kernel", ms, nbytes
        rows = 4096
        op = o_parts[:, :, 0, :rows].double().cpu().numpy()
        lp = lse_parts[:, :, 0, :rows].double().cpu().numpy()
        cpu_fn, cpu_bytes = (lambda: oracle.merge(op, lp)), (P + 1) * rows * (d + 1) * 4
        sample = f"fp64 merge of {rows} of the {BH * N} rows x {P} partials"
    elif args.row == "ulysses":
        P, B, Nl, H, d = 8, 1, 23552, 16, 64
        Hl = H // P
        ins = [torch.randn((B, Nl, H, d), device=dev, generator=g).to(torch.bfloat16) for _ in range(3)]
        send = [torch.empty((P, B, Hl, Nl, d), device=dev, dtype=torch.bfloat16) for _ in range(3)]
        att = [torch.empty((B, Hl, P * Nl, d), device=dev, dtype=torch.bfloat16) for _ in range(3)]
        o_att = torch.randn((B, Hl, P * Nl, d), device=dev, generator=g)
        o_send = torch.empty((P, B, Hl, Nl, d), device=dev)
        o_back = torch.empty((B, Nl, H, d), device=dev)

        def step():
            # the all-to-all itself moves send -> recv between ranks; on one GPU
            # recv is the send buffer
            for x, s_, y in zip(ins, send, att):
                va.ulysses_pack(x, P, out=s_)
                va.ulysses_unpack(s_, out=y)
            va.ulysses_pack_out(o_att, P, out=o_send)
            va.ulysses_unpack_out(o_send, out=o_back)

        ms = time_events(step, args.steps)
        nbytes = 3 * 2 * 2 * B * Nl * H * d * 2 + 2 * 2 * B * Nl * H * d * 4
        dom, dom_ms, dom_bytes = "ulysses_layout_kernel", ms, nbytes
        xs = [x[:, :2048].view(torch.int16).cpu().numpy().view(np.uint16) for x in ins]
        oo = o_send[:, :, :, :256].cpu().numpy()

        def cpu_step():
            for x in xs:
                oracle.ulysses.unpack(oracle.ulysses.pack(x, P))
            oracle.ulysses.unpack_out(oracle.ulysses.pack_out(oracle.ulysses.unpack(oo), P))

        cpu_fn, cpu_bytes = cpu_step, 3 * 2 * 2 * xs[0].size * 2 + 3 * 2 * oo.size * 4
        sample = f"numpy layouts of 2,048 of the {Nl} tokens per rank (Q, K, V) and 256 per rank of O"
    else:
        M, H, C, d = 8192, 16, 92, 64
        q = torch.randn((H, d), device=dev, generator=g).to(torch.bfloat16)
        k = torch.randn((M, H, C, d), device=dev, generator=g).to(torch.bfloat16)
        v = torch.randn((M, H, C, d), device=dev, generator=g).to(torch.bfloat16)
        dout = torch.randn((M, H, d), device=dev, generator=g).to(torch.bfloat16)
        o, lse = va.agg_fwd(q, k, v)
        kv = M * H * C * d
        fwd_bytes = 2 * kv * 2 + M * H * (d + 1) * 4  # read K, V; write O, LSE
        bwd_bytes = 2 * kv * 2 + M * H * (d * 4 + d * 2 + 4) + 2 * kv * 4  # + O, dO, LSE; write dK, dV
        fwd_ms = time_events(lambda: va.agg_fwd(q, k, v), args.steps)
        bwd_ms = time_events(lambda: va.agg_bwd(q, k, v, o, lse, dout), args.steps)
        ms, nbytes = fwd_ms + bwd_ms, fwd_bytes + bwd_bytes
        per_kernel = {"agg_fwd": {"ms": fwd_ms, "GB_s": fwd_bytes / fwd_ms / 1e6},
                      "agg_bwd": {"ms": bwd_ms, "GB_s": bwd_bytes / bwd_ms / 1e6}}
        dom, dom_ms, dom_bytes = "attn_agg_bwd_kernel (+ the dq partial sum)", bwd_ms, bwd_bytes
        m_s = 64
        xs = workloads.make_aggregation_inputs(m_s, H, C, d, seed=1)
        cpu_fn = lambda: oracle.aggregation.backward(xs["q"], xs["k"], xs["v"], xs["dout"], 0.125)  # noqa: E731
        cpu_bytes = nbytes * m_s // M
        sample = f"fp64 forward+backward of {m_s} of the {M} patch positions"
    gbs = nbytes / (ms * 1e-3) / 1e9
    dom_gbs = dom_bytes / (dom_ms * 1e-3) / 1e9
    line = {
        "metric": f"{args.row} HBM throughput", "value": gbs, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": 2, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": {"ulysses": "u8"}.get(args.row, "f32"), "data": "synthetic",
        "config": {"workload": ROW_DOC[args.row]},
        "roofline": {"bound": "hbm", "achieved": dom_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": dom_gbs / PEAK_HBM_GBS, "traffic": stored_traffic(dom.split()[0], args.row, args.row),
                     "kernel": dom, "algorithmic_bytes": dom_bytes},
        "per_kernel": per_kernel,
        "kernel_sources": kernel_sources_digest(args.row),
    }
    if not args.no_cpu_baseline:
        n, dt = timed_cpu(cpu_fn, budget)
        # these oracles are element-wise numpy and einsum without BLAS: one thread
        line["cpu_baseline"] = {"value": n * cpu_bytes / dt / 1e9, "unit": "GB/s", "cores": 1,
                                "kind": "oracle", "sample": f"{sample}, {n} times in {dt:.1f} s"}
    print(json.dumps(line), flush=True)


# Attention workloads beside the headline one: the paper's other head dims
# (Table I's ViT-10B, d = 72 with 64 heads; the 2560-wide 16-head model of
# Sec. V-C, d = 160) as one GPU's Ulysses shard, and the headline workload
# with every operand in the sequence-major layout an all-to-all produces.
ATT_ROWS = {
    "d64": dict(B=4, H=1, N=188416, d=64, bnhd=False,
                doc="ViT-Base heads (d=64), the per-GPU shard of the paper's 188K run: B=4, H=1, N=188,416"),
    "m1": dict(B=1, H=1, N=1048576, d=64, bnhd=False,
               doc="ViT-Base heads at 1M tokens (d=64; 1 head per GPU at 16 Ulysses ranks), B=1, H=1, N=1,048,576"),
    "d72": dict(B=1, H=2, N=65536, d=72, bnhd=False,
                doc="ViT-10B heads (d=72; 64 heads, 2 per GPU at 32 Ulysses ranks), B=1, N=65,536"),
    "d160": dict(B=1, H=1, N=65536, d=160, bnhd=False,
                 doc="2560-wide 16-head model (d=160; 1 head per GPU at 16 Ulysses ranks), B=1, N=65,536"),
    "bnhd": dict(B=1, H=2, N=188416, d=128, bnhd=True,
                 doc="B=1, H=2, N=188,416, d=128 with q, k, v, dO, O, dQ, dK, dV all sequence-major [B,N,H,d]"),
}


def bench_attention_row(args):
    """Forward + backward attention on one of ATT_ROWS: counted TFLOP/s (the
    headline convention, at the real head dim), the dominant kernel against
    the bf16 MFMA peak, and the oracle beside it."""
    import types

    import numpy as np
    import torch

    import paper_2405_15780_amd as va
    import workloads

    cfg = ATT_ROWS[args.row]
    B, H, N, d = cfg["B"], cfg["H"], cfg["N"], cfg["d"]
    scale = 1.0 / np.sqrt(d)
    x = workloads.make_small_inputs(B, H, N, d, seed=4000 + d)
    dev = torch.device("cuda:0")
    f32 = dict(dtype=torch.float32, device=dev)

    def put(bits):
        t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16)
        if cfg["bnhd"]:  # stored [B, N, H, d], handed over as its [B, H, N, d] view
            return t.transpose(1, 2).contiguous().to(dev).transpose(1, 2)
        return t.to(dev)

    def out4():
        if cfg["bnhd"]:
            return torch.empty((B, N, H, d), **f32).transpose(1, 2)
        return torch.empty((B, H, N, d), **f32)

    t = {n: put(a) for n, a in x.items()}
    o, dq, dk, dv = out4(), out4(), out4(), out4()
    lse = torch.empty((B, H, N), **f32)
    ws = torch.empty(va.workspace_bytes(B, H, N, d) // 4, **f32)
    nn = float(B * H) * N * N * d
    if cfg["bnhd"]:  # the strided backward is one entry point (three kernels)
        segs = [("fwd", lambda: va.fwd(t["q"], t["k"], t["v"], scale, out=(o, lse)), "mfma", 4.0 * nn),
                ("bwd", lambda: va.bwd(t["q"], t["k"], t["v"], o, lse, t["dout"], scale, workspace=ws,
                                       out=(dq, dk, dv)), "mfma", 14.0 * nn)]
    else:
        segs = [("fwd", lambda: va.fwd(t["q"], t["k"], t["v"], scale, out=(o, lse)), "mfma", 4.0 * nn),
                ("rowdot", lambda: va.bwd_rowdot(o, t["dout"], lse, ws), "hbm", float(B * H * N) * (6 * d + 12)),
                ("dkdv", lambda: va.bwd_dkdv(t["q"], t["k"], t["v"], t["dout"], lse, dk, dv, ws, scale), "mfma",
                 8.0 * nn),
                ("dq", lambda: va.bwd_dq(t["q"], t["k"], t["v"], t["dout"], lse, dq, ws, scale), "mfma", 6.0 * nn)]
    for _ in range(args.warmup):
        for _, fn, _, _ in segs:
            fn()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(segs) + 1)] for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(args.steps):
        for j, (_, fn, _, _) in enumerate(segs):
            ev[i][j].record()
            fn()
        ev[i][-1].record()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    seg_ms = {name: float(np.mean([e[j].elapsed_time(e[j + 1]) for e in ev])) for j, (name, *_) in enumerate(segs)}
    value = 14.0 * nn / (ms * 1e-3) / 1e12
    dom = max(seg_ms, key=seg_ms.get)
    _, _, bound, work = next(s_ for s_ in segs if s_[0] == dom)
    achieved = work / (seg_ms[dom] * 1e-3) / 1e12
    per_kernel = {}
    for name, _, b_, wk in segs:
        per_kernel[name] = {"ms": seg_ms[name]}
        if b_ == "mfma":
            per_kernel[name]["tflops"] = wk / (seg_ms[name] * 1e-3) / 1e12
        else:
            per_kernel[name]["gbs"] = wk / (seg_ms[name] * 1e-3) / 1e9
    line = {
        "metric": f"attention fwd+bwd TFLOP/s, {cfg['doc']}", "value": value, "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": cfg["doc"], "B": B, "H": H, "N": N, "d": d,
                   "layout": "[B,N,H,d]" if cfg["bnhd"] else "[B,H,N,d]",
                   "tile_width": 64 if d <= 64 else 96 if d <= 96 else 128 if d <= 128 else 160},
        "pct_of_peak": 100.0 * value / PEAK_BF16_TFLOPS,
        "kernels": per_kernel,
        "roofline": {"bound": bound, "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": stored_traffic(dom, args.row, args.row),
                     "kernel": dom if dom != "bwd" else "bwd (rowdot + dkdv + dq)",
                     "algorithmic_flops": work},
        "kernel_sources": kernel_sources_digest(args.row),
    }
    if not args.no_cpu_baseline:
        w = types.SimpleNamespace(N=N, d=d, scale=scale, backward=True, B=B, H=H)
        line["cpu_baseline"] = cpu_baseline(w, x, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.hbm_reference:
        hbm_reference()
        return
    if args.mfma_reference:
        mfma_reference()
        return
    if args.row in ATT_ROWS:
        if args.gpus != 1:
            print(json.dumps({"error": "one GPU per run: the library has no multi-GPU path; use --gpus 1", "n_gpus": args.gpus}))
            sys.exit(2)
        bench_attention_row(args)
        return
    if args.row != "attention":
        if args.gpus != 1:
            print(json.dumps({"error": "one GPU per run: the library has no multi-GPU path; use --gpus 1", "n_gpus": args.gpus}))
            sys.exit(2)
        bench_row(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "one GPU per run: the library has no multi-GPU path; use --gpus 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2405_15780_amd as va
    import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = workloads.WORKLOADS[args.workload]
    B, H, N, d = w.shape
    x = workloads.make_inputs(w)
    dev = torch.device("cuda:0")
    t = {n: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev) for n, a in x.items()}
    f32 = dict(dtype=torch.float32, device=dev)
    o = torch.empty((B, H, N, d), **f32)
    lse = torch.empty((B, H, N), **f32)
    dq, dk, dv = (torch.empty((B, H, N, d), **f32) for _ in range(3))
    scale = w.scale
    # backward mode: recompute (O(N d) memory) unless the opt-in dS mode is
    # asked for, which needs B*H*N^2*2 bytes of workspace (142 GB at N=188,416)
    ds_bytes = va.workspace_bytes_kv(B, H, N, N, d, va.VITATTN_BWD_STORE_DS)
    free_bytes = torch.cuda.mem_get_info(dev)[0]
    fits = ds_bytes > 0 and ds_bytes + (8 << 30) < free_bytes
    mode = args.bwd_mode if w.backward else "none"
    if mode == "stored-ds" and not fits:
        print(json.dumps({"error": f"the dS-mode workspace ({ds_bytes / 1e9:.0f} GB) does not fit"}))
        sys.exit(2)
    ws = torch.empty(max(ds_bytes if mode == "stored-ds" else va.workspace_bytes(B, H, N, d), 4) // 4, **f32)
    workspace_gb = ws.numel() * 4 / 1e9  # of the timed mode (the comparison below may enlarge ws)

    def step(ev=None, m=None):
        m = m or mode
        if ev is not None:
            ev[0].record()
        va.fwd(t["q"], t["k"], t["v"], scale, out=(o, lse))
        if w.backward:
            if ev is not None:
                ev[1].record()
            va.bwd_rowdot(o, t["dout"], lse, ws)
            if ev is not None:
                ev[2].record()
            if m == "stored-ds":
                va.bwd_dkdv_ds(t["q"], t["k"], t["v"], t["dout"], lse, dk, dv, ws, scale)
            else:
                va.bwd_dkdv(t["q"], t["k"], t["v"], t["dout"], lse, dk, dv, ws, scale)
            if ev is not None:
                ev[3].record()
            if m == "stored-ds":
                va.bwd_dq_from_ds(t["k"], dq, ws, scale)
            else:
                va.bwd_dq(t["q"], t["k"], t["v"], t["dout"], lse, dq, ws, scale)
        if ev is not None:
            ev[4].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with SmiSampler() as smi:
        wall0 = time.perf_counter()
        start.record()
        for i in range(args.steps):
            step(events[i])
        stop.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
    step_ms = [e[0].elapsed_time(e[4]) for e in events]
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps

    names = ["fwd", "rowdot", "dkdv", "dq"] if w.backward else ["fwd"]
    spans = {"fwd": (0, 1 if w.backward else 4), "rowdot": (1, 2), "dkdv": (2, 3), "dq": (3, 4)}
    kern_ms = {n: float(np.mean([e[spans[n][0]].elapsed_time(e[spans[n][1]]) for e in events])) for n in names}

    flops = w.counted_flops()
    value = flops["total"] / (ms_per_step * 1e-3) / 1e12
    nn = float(B * H) * N * N * d
    # algorithmic work of one launch of each kernel
    kern_work = {
        "fwd": ("mfma", 4.0 * nn),                       # S = QK^T and O = PV
        "dkdv": ("mfma", 8.0 * nn),                      # S, dP recomputed; dV += P^T dO; dK += dS^T Q
        "dq": ("mfma", 6.0 * nn),                        # S, dP recomputed; dQ += dS K
        "rowdot": ("hbm", float(B * H * N) * (2 * d + 4 * d + 12)),  # read dO bf16, O fp32, LSE; write D, LSE2
    }
    if mode == "stored-ds":  # dK/dV also writes dS; dQ = dS K reads it (bound by HBM: 2 bytes per score)
        kern_work["dkdv"] = ("mfma", 8.0 * nn)
        kern_work["dq"] = ("hbm", float(B * H) * N * N * 2 + float(B * H * N) * d * 4)
    dom = max(names, key=lambda n: kern_ms[n])
    bound, work = kern_work[dom]
    traffic_key = w.name if mode == "recompute" else w.name + "+stored-ds"
    if bound == "mfma":
        achieved = work / (kern_ms[dom] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_BF16_TFLOPS, "traffic": stored_traffic(dom, traffic_key), "kernel": dom}
    else:
        achieved = work / (kern_ms[dom] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS, "traffic": stored_traffic(dom, traffic_key), "kernel": dom}

    per_kernel = {}
    for n in names:
        b_, wk = kern_work[n]
        per_kernel[n] = {"ms": kern_ms[n]}
        if b_ == "mfma":
            per_kernel[n]["tflops"] = wk / (kern_ms[n] * 1e-3) / 1e12
            per_kernel[n]["frac_of_peak"] = per_kernel[n]["tflops"] / PEAK_BF16_TFLOPS
        else:
            per_kernel[n]["gbs"] = wk / (kern_ms[n] * 1e-3) / 1e9

    # the other backward mode, outside the timed region, for comparison
    alt = None
    if w.backward and fits and not args.no_compare:
        other = "recompute" if mode == "stored-ds" else "stored-ds"
        if other == "stored-ds" and ws.numel() * 4 < ds_bytes:
            ws = torch.empty(ds_bytes // 4, **f32)
        for _ in range(max(1, args.warmup)):
            step(m=other)
        ev2 = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
        for i in range(args.steps):
            step(ev2[i], m=other)
        torch.cuda.synchronize()
        alt_ms = float(np.mean([e[0].elapsed_time(e[4]) for e in ev2]))
        alt = {"bwd_mode": other, "ms_per_step": alt_ms, "value": flops["total"] / (alt_ms * 1e-3) / 1e12,
               "workspace_gb": (ds_bytes if other == "stored-ds" else va.workspace_bytes(B, H, N, d)) / 1e9,
               "kernels_ms": {n: float(np.mean([e[spans[n][0]].elapsed_time(e[spans[n][1]]) for e in ev2]))
                              for n in names}}

    # the vendor bf16 GEMM on random operands in the same process, after the
    # timed region: the power-limited rate that dense matrix-core work reaches
    ceiling = None
    if not args.no_compare:
        g = torch.Generator(device="cuda:0").manual_seed(w.seed)
        ga, gb = (torch.randn(16384, 16384, device="cuda:0", generator=g).to(torch.bfloat16) for _ in range(2))
        g_ms, g_tf = vendor_gemm_tflops(ga, gb, 60)
        del ga, gb
        ceiling = {"kind": "torch.matmul bf16 16384^3, random normal operands", "tflops": g_tf,
                   "value_frac": value / g_tf,
                   "kernel_frac": {n: per_kernel[n]["tflops"] / g_tf for n in names if "tflops" in per_kernel[n]}}

    smi_summary = smi.summary()
    clock = None
    if smi_summary:
        # peak at the clock the chip actually held: 256 CU x 4096 flop/clk x sclk
        peak_at_sclk = 256 * 4096 * smi_summary["sclk_mhz_median"] * 1e6 / 1e12
        clock = dict(smi_summary, peak_tflops_at_sclk=peak_at_sclk, pct_of_peak_at_sclk=100.0 * value / peak_at_sclk)
    if args.workload == 4:
        metric = "attention fwd+bwd TFLOP/s and % of bf16 MFMA peak at N=188,416, d=128"
    else:
        metric = (f"attention {'fwd+bwd' if w.backward else 'fwd'} TFLOP/s and % of bf16 MFMA peak, "
                  f"B={B}, H={H}, N={N:,}, d={d}")
    result = {
        "metric": metric,
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": B, "H": H, "N": N, "d": d, "passes": "fwd+bwd" if w.backward else "fwd",
                   "grid": f"{w.grid[0]}x{w.grid[1]}", "seed": w.seed, "bwd_mode": mode,
                   "workspace_gb": workspace_gb},
        "other_bwd_mode": alt,
        "pct_of_peak": 100.0 * value / PEAK_BF16_TFLOPS,
        "counted_tflop_per_step": flops["total"] / 1e12,
        "step_ms_median": float(np.median(step_ms)),
        "step_ms_min": float(np.min(step_ms)),
        "clock": clock,
        "kernels": per_kernel,
        "practical_ceiling": ceiling,
        "wall_s_timed": wall,
        "roofline": roof,
        "kernel_sources": kernel_sources_digest(args.row),
    }
    if not args.no_cpu_baseline:
        print(f"# timing the oracle for ~{args.cpu_seconds:.0f} s", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(w, x, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
