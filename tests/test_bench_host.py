"""Host-side behaviour of bench.py that needs no GPU: more than one GPU is
refused with a JSON message (and exit status 2) before anything touches a
device, for the default workload and the other rows; and the host logic around
the measurement (source digests, defaults, the CPU baseline's sampling, the
clock summary)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("extra", [[], ["--row", "merge"], ["--row", "d72"]])
def test_more_than_one_gpu_is_refused(extra):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2", *extra],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2, (r.returncode, r.stdout, r.stderr)
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


def test_kernel_source_digests_are_per_family():
    sys.path.insert(0, ROOT)
    import bench

    d = {row: bench.kernel_sources_digest(row) for row in bench.KERNEL_FILES}
    assert d["attention"] == d["d72"] == d["d160"] == d["bnhd"] == d["d64"] == d["m1"]
    assert len({d["attention"], d["merge"], d["ulysses"], d["agg"]}) == 4


def test_default_backward_is_the_recompute_mode():
    sys.path.insert(0, ROOT)
    import bench

    old = sys.argv
    try:
        sys.argv = ["bench.py"]
        assert bench.parse().bwd_mode == "recompute"
    finally:
        sys.argv = old


def test_cpu_baseline_walks_the_workload_and_repeats_a_small_one():
    import types

    sys.path.insert(0, ROOT)
    import bench
    import workloads

    for backward in (True, False):
        w = types.SimpleNamespace(B=1, H=2, N=64, d=16, scale=0.25, backward=backward)
        x = workloads.make_small_inputs(1, 2, 64, 16, seed=3)
        bench.cpu_baseline(w, x, 0.0)  # one block: warms up the BLAS threads
        r = bench.cpu_baseline(w, x, 0.5)
        assert r["kind"] == "oracle" and r["unit"] == "TFLOP/s" and r["value"] > 0 and r["cores"] >= 1
        assert "times over" in r["sample"], r["sample"]  # 128 tiny rows take far less than the budget
        assert ("forward+backward" in r["sample"]) == backward


def test_clock_summary_ignores_idle_samples():
    # readings below 500 MHz are the GPU idle or ramping; a timed region too
    # short to catch the GPU busy reports no clock rather than idle readings
    sys.path.insert(0, ROOT)
    import bench

    s = bench.SmiSampler()
    s.samples = [(253.0, 157.0), (252.0, 158.0)]
    assert s.summary() is None
    s.samples = [(253.0, 157.0), (1300.0, 1900.0), (1320.0, 2000.0)]
    got = s.summary()
    assert got["samples"] == 2 and got["sclk_mhz_min"] == 1900.0 and got["power_w_median"] == 1310.0


def test_source_digest_ignores_comments_but_not_code(tmp_path):
    # stored counter readings stay valid across comment edits and are
    # invalidated by any change to the code they were taken on
    import shutil

    sys.path.insert(0, ROOT)
    import bench

    src = os.path.join(ROOT, "paper_2405_15780_amd", "csrc")
    for name in os.listdir(src):
        shutil.copy(os.path.join(src, name), tmp_path / name)
    base = bench.kernel_sources_digest("attention", str(tmp_path))
    assert base == bench.kernel_sources_digest("attention")
    path = tmp_path / "vitattn_bwd.hip"
    code = path.read_text()
    path.write_text("// a new comment line\n" + code.replace("\n}", "  /* inline */\n}", 1) + "\n\n// trailing\n")
    assert bench.kernel_sources_digest("attention", str(tmp_path)) == base
    path.write_text(code.replace("constexpr int RING = 3;", "constexpr int RING = 4;", 1))
    assert bench.kernel_sources_digest("attention", str(tmp_path)) != base
    assert bench.strip_comments('a = "//x"; // c\nb = 1; /* d */ c\n\n') == 'a = "//x";\nb = 1;   c'
