"""bench.py host logic, no GPU: the one-GPU refusal, the two roofline
formulas, the rocprof counter summary and the CPU-baseline record."""
import csv
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


def test_hbm_roofline_uses_algorithmic_bytes():
    n = 1_000_000
    avg_ms = {"k_hist": 0.001, "k_gather_wt": 0.002, "k_keyed_grad": 0.002, "k_gather_grad": 0.004}
    r = bench.hbm_roofline(avg_ms, n)
    assert r["kernel"] == "k_gather_grad" and r["bound"] == "hbm" and r["unit"] == "GB/s"
    assert r["achieved"] == pytest.approx(10 * n / 4e-6 / 1e9)
    assert r["frac"] == pytest.approx(r["achieved"] / 8000.0)
    total = (2 + 6 + 6 + 10) * n / (9e-6) / 1e9
    assert r["n_pass_total_GBps"] == pytest.approx(total)


def test_alu_roofline_counts_ops_per_map_entry():
    n, k = 1_000_000, 16
    r = bench.alu_roofline({"k_dense_iter": 0.1, "k_dense_biter": 0.2}, n, k)
    assert r["kernel"] == "k_dense_biter" and r["bound"] == "alu" and r["unit"] == "TFLOP/s"
    assert r["achieved"] == pytest.approx(15 * n * k / 2e-4 / 1e12)
    assert r["peak"] == 157.3 and r["frac"] == pytest.approx(r["achieved"] / 157.3)


def _write_counters(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def test_pmc_summary_scales_by_the_copy_calibration(tmp_path, monkeypatch):
    fetch, write = tmp_path / "fetch", tmp_path / "write"
    fetch.mkdir()
    write.mkdir()
    gib = float(bench.COPY_BYTES) / 1024.0
    # the copy reads as half its bytes on FETCH_SIZE and all of them on WRITE_SIZE
    _write_counters(fetch / "copy_counter_collection.csv", [
        dict(Dispatch_Id=1, Kernel_Name="__amd_rocclr_copyBuffer", Counter_Name="FETCH_SIZE", Counter_Value=gib / 2),
        dict(Dispatch_Id=2, Kernel_Name="__amd_rocclr_copyBuffer", Counter_Name="FETCH_SIZE", Counter_Value=1.0)])
    _write_counters(write / "copy_counter_collection.csv", [
        dict(Dispatch_Id=1, Kernel_Name="__amd_rocclr_copyBuffer", Counter_Name="WRITE_SIZE", Counter_Value=gib)])
    _write_counters(fetch / "bench_counter_collection.csv", [
        dict(Dispatch_Id=5, Kernel_Name="edkm::k_gather_grad(edkm::BatchArgs)", Counter_Name="FETCH_SIZE", Counter_Value=100.0),
        dict(Dispatch_Id=9, Kernel_Name="edkm::k_gather_grad(edkm::BatchArgs)", Counter_Name="FETCH_SIZE", Counter_Value=300.0),
        # the merge kernel's name starts with the histogram's: it must not count as k_hist
        dict(Dispatch_Id=3, Kernel_Name="edkm::k_hist(edkm::BatchArgs)", Counter_Name="FETCH_SIZE", Counter_Value=1000.0),
        dict(Dispatch_Id=4, Kernel_Name="edkm::k_hist_merge(edkm::BatchArgs)", Counter_Name="FETCH_SIZE", Counter_Value=10.0)])
    _write_counters(write / "bench_counter_collection.csv", [
        dict(Dispatch_Id=5, Kernel_Name="edkm::k_gather_grad(edkm::BatchArgs)", Counter_Name="WRITE_SIZE", Counter_Value=50.0),
        dict(Dispatch_Id=3, Kernel_Name="edkm::k_hist(edkm::BatchArgs)", Counter_Name="WRITE_SIZE", Counter_Value=4.0),
        dict(Dispatch_Id=4, Kernel_Name="edkm::k_hist_merge(edkm::BatchArgs)", Counter_Name="WRITE_SIZE", Counter_Value=8.0)])
    out = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(out))
    bench.pmc_summary(str(fetch), str(write))
    res = json.load(open(out))
    assert res["fetch_scale"] == pytest.approx(2.0) and res["write_scale"] == pytest.approx(1.0)
    kg = res["kernels"]["k_gather_grad"]
    assert kg["fetch_bytes"] == pytest.approx(200.0 * 1024 * 2)
    assert kg["write_bytes"] == pytest.approx(50.0 * 1024)
    kh = res["kernels"]["k_hist"]
    assert kh["fetch_bytes"] == pytest.approx(1000.0 * 1024 * 2) and kh["write_bytes"] == pytest.approx(4.0 * 1024)
    assert res["source_hash"] == bench.source_hash()
    # the counters belong to the workload they were taken on, and to no other line
    avg_ms = {"k_hist": 0.001, "k_gather_wt": 0.002, "k_keyed_grad": 0.002, "k_gather_grad": 0.004}
    r = bench.hbm_roofline(avg_ms, 10, workload=bench.TRAFFIC_WORKLOAD)
    assert r["traffic"] == pytest.approx(kg["bytes_per_launch"])
    assert bench.hbm_roofline(avg_ms, 10, workload=bench.TRAFFIC_WORKLOAD + "_half_grads")["traffic"] is None
    assert bench.hbm_roofline(avg_ms, 10)["traffic"] is None


def test_kernel_base_name():
    assert bench.kernel_base_name("edkm::k_hist(edkm::BatchArgs)") == "k_hist"
    assert bench.kernel_base_name("edkm::k_hist_merge(edkm::BatchArgs)") == "k_hist_merge"
    assert bench.kernel_base_name("void edkm::k_fwd_iter<8>(edkm::BatchArgs)") == "k_fwd_iter"
    assert bench.kernel_base_name("__amd_rocclr_copyBuffer") == "__amd_rocclr_copyBuffer"


def test_cpu_baseline_record():
    from paper_2309_00964_amd import inputs
    samples = []
    for i, name in enumerate(("q_proj", "k_proj")):
        keys = inputs.fp16_weights(20_000 + i, 97 + i)
        samples.append((name, keys, inputs.quantile_init(keys, 8), inputs.upstream_grad(keys.size, 99 + i)))
    r = bench.cpu_baseline(samples, 8)
    assert r["kind"] == "oracle" and r["unit"] == "weights/s" and r["value"] > 0 and r["cores"] >= 1
    assert r["single_thread"]["cores"] == 1 and r["single_thread"]["value"] > 0
    assert r["table_form"]["value"] > 0 and "q_proj" in r["table_form"]["sample"]


def test_source_hash_ignores_comments_only(tmp_path, monkeypatch):
    src = os.path.join(ROOT, "paper_2309_00964_amd", "csrc")
    dst = tmp_path / "paper_2309_00964_amd" / "csrc"
    dst.mkdir(parents=True)
    for f in os.listdir(src):
        (dst / f).write_text(open(os.path.join(src, f)).read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    base = bench.source_hash()
    k = dst / "edkm_kernels.hip"
    k.write_text("// a new comment line\n" + k.read_text().replace("namespace edkm {", "namespace edkm {  /* x */", 1))
    assert bench.source_hash() == base
    # the block-timeline instrumentation is not product code either
    body = k.read_text()
    i = body.index("EDKM_STAMP_ENTRY(b);", body.index("k_hist(BatchArgs b)"))
    k.write_text(body[:i] + "EDKM_STAMP_MARK(b, 6);\n    " + body[i:] +
                 "\n#ifdef EDKM_BLOCK_STAMPS\nstatic int stamp_only_value = 2;\n#endif\n")
    assert bench.source_hash() == base
    k.write_text(k.read_text() + "\nstatic int unused_probe_value = 1;\n")
    assert bench.source_hash() != base


def test_pass_bytes_per_weight():
    """Algorithmic bytes per weight over the four N-sized passes: 24 with
    fp32 W~ and gradients, 22 with 16-bit W~, 18 with 16-bit gradients (dL/dW~
    read twice, dL/dw written once), 16 with both (the training step in the
    weights' own precision)."""
    import bench
    passes = ("k_hist", "k_gather_wt", "k_keyed_grad", "k_gather_grad")
    total = {(h, g): sum(bench.pass_bytes(p, h, g) for p in passes)
             for h in (False, True) for g in (False, True)}
    assert total == {(False, False): 24, (True, False): 22, (False, True): 18, (True, True): 16}
