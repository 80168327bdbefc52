"""The block-timeline diagnostics build on the GPU: `bench.py --block-timeline`
runs one step of a small matrix on libedkm_stamps.so, in a child process (this
process keeps the product library), and writes a timeline whose launches are
the library's, in order, with their blocks and positive spans."""
import os
import re
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

STEP = (["k_init_zero", "k_hist", "k_hist_merge", "k_window"] + ["k_fwd_iter"] * 5 +
        ["k_fwd_out", "k_gather_wt", "k_keyed_grad", "k_grad_top"] + ["k_bwd_iter"] * 5 + ["k_gather_grad"])


def test_block_timeline_of_a_small_matrix(tmp_path):
    from paper_2309_00964_amd import build
    if not os.path.exists(build.OUT_STAMPS):
        pytest.skip("the diagnostics build is not built")
    out = tmp_path / "timeline.md"
    print("[gpu-case] block timeline, 256x256, child process", flush=True)
    r = subprocess.run([sys.executable, "bench.py", "--workload", "single_256x256", "--warmup", "2",
                        "--block-timeline", str(out)], cwd=ROOT, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-3000:]
    text = out.read_text()
    table = text.split("| # | Kernel | Blocks |", 1)[1].split("\n\n", 1)[0]
    rows = re.findall(r"^\| (\d+) \| (k_\w+) \| (\d+) \| ([\d.]+) \| ([\d.]+) \| ([\d.]+) \|", table, re.M)
    assert [x[1] for x in rows] == STEP
    assert all(int(x[2]) > 0 and float(x[4]) > 0 for x in rows)
    starts = [float(x[3]) for x in rows]
    assert starts == sorted(starts)          # launches in stream order
    assert "| 1 | k_hist | " in text.split("Phases", 1)[1]   # phase marks recorded
