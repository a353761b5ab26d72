"""Host-side behaviour of bench.py that needs no GPU: more than one GPU is
refused with a JSON message (and exit status 2) before anything touches a
device, for the default workload and the other rows."""
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
