"""The block-timeline diagnostics build (libedkm_stamps.so, the library's
sources compiled with EDKM_BLOCK_STAMPS): it exports every entry point of
include/edkm.h plus the three calls of include/edkm_stamps.h, the product
library exports none of the latter, and bench.py reads the record with the
header's shape.  No GPU: the libraries are only loaded."""
import json
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2309_00964_amd import build  # noqa: E402


def declared(header):
    text = open(os.path.join(ROOT, "include", header)).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(edkm_[a-z_]+)\s*\(", text)))


def exported(lib_path, names):
    code = ("import json, sys; from paper_2309_00964_amd import edkm; "
            "print(json.dumps([edkm.LIB_PATH, [n for n in sys.argv[1:] if hasattr(edkm._lib, n)]]))")
    env = dict(os.environ, EDKM_LIBRARY=lib_path)
    r = subprocess.run([sys.executable, "-c", code, *names], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    path, found = json.loads(r.stdout.strip().splitlines()[-1])
    assert os.path.abspath(path) == os.path.abspath(lib_path)
    return set(found)


@pytest.mark.skipif(not (os.path.exists(build.OUT) and os.path.exists(build.OUT_STAMPS)),
                    reason="libraries not built (run __graft_entry__.build())")
def test_stamps_build_exports_the_product_abi_and_the_stamp_calls():
    api, stamps = declared("edkm.h"), declared("edkm_stamps.h")
    assert stamps == ["edkm_stamps_clock_khz", "edkm_stamps_dump", "edkm_stamps_reset"]
    assert exported(build.OUT_STAMPS, api + stamps) == set(api + stamps)
    assert exported(build.OUT, api + stamps) == set(api)


def test_bench_reads_the_record_with_the_header_shape():
    import bench
    text = open(os.path.join(ROOT, "include", "edkm_stamps.h")).read()
    got = {k: int(v) for k, v in re.findall(r"EDKM_STAMP_(LAUNCHES|BLOCKS|WORDS)\s*=\s*(\d+)", text)}
    assert got == {"LAUNCHES": bench.STAMP_LAUNCHES, "BLOCKS": bench.STAMP_BLOCKS, "WORDS": bench.STAMP_WORDS}
    kernels = open(os.path.join(ROOT, "paper_2309_00964_amd", "csrc", "edkm_kernels.hip")).read()
    for name, labels in bench.TIMELINE_PHASES.items():   # each kernel stamps as many phases as named
        body = kernels[kernels.index(" %s(BatchArgs b" % name):]
        body = body[:body.index("\n}\n")]
        marks = sorted(set(int(x) for x in re.findall(r"EDKM_STAMP_MARK\(b, (\d)\)", body)))
        assert marks == list(range(2, 2 + len(labels))), (name, marks)
    assert all(len(v) <= 5 for v in bench.TIMELINE_PHASES.values())   # record words 2..6


def test_timeline_report_on_a_synthetic_record():
    """Two launches, 128 and 4 blocks, stamps in 100 MHz ticks: the report's
    spans, gaps, phases and per-XCC ends are the ones planted."""
    import numpy as np
    import bench
    W = bench.STAMP_WORDS
    raw = []
    for rep in range(3):
        ts = np.zeros((2, bench.STAMP_BLOCKS, W), np.uint64)
        base = 10_000 + 977 * rep
        for blk in range(128):                     # k_hist: 1 us to 21 us, XCC = blk % 8
            x = blk % 8
            ts[0, blk] = [base + 100, base + 100 + 1000 + 100 * x, base + 600, base + 700, 0, 0, 0, x]
        for blk in range(4):                       # k_window: starts 2 us after the last k_hist block
            ts[1, blk] = [base + 2000 + 200, base + 2200 + 300, base + 2210, base + 2220, base + 2230, 0, 0, 0]
        ts[1, 0, 4] = 0                            # one block never chose a window: left out of the phases
        raw.append((["k_hist", "k_window"], ts))
    text = bench.timeline_report(raw, 100e6, "synthetic", "cmd", 2)
    lines = text.splitlines()
    row = lambda q: next(l_ for l_ in lines if l_.startswith("| %d | " % q))
    assert row(0) == "| 0 | k_hist | 128 | 0.0 | 17.0 | 0.0 | 13.5 | 17.0 |"
    assert row(1) == "| 1 | k_window | 4 | 21.0 | 3.0 | 4.0 | 3.0 | 3.0 |"
    assert "Step 24.0 us: launch spans 20.0 us, gaps 4.0 us." in text
    assert "| 0 | k_hist | 128 | entry -> keys streamed 5.00; keys streamed -> span found 1.00; span found -> end" in text
    assert ("| 1 | k_window | 3 | entry -> wave 0 scanned 0.10; wave 0 scanned -> block totals combined 0.10; block totals combined -> windows chosen 0.10; "
            "windows chosen -> end 2.70") in text
    xcc = next(l_ for l_ in lines if "0:16/10.0" in l_)
    assert xcc.endswith("7:16/17.0 | 7.0 |")
