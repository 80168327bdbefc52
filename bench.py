#!/usr/bin/env python3
"""Throughput of uniquified DKM forward + backward on one MI355X.

One step is the whole hot path over one LLaMA-7B decoder layer at 3 bits
(q, k, v, o 4096x4096; gate, up 11008x4096; down 4096x11008: 202,375,168 fp16
weights, each matrix with its own 8 centroids, tau = 2e-3, 5 iterations):
init_unique + forward + backward for the seven matrices, issued as the batched
C-ABI calls on one stream.  Inputs (weights, initial centroids, dL/dW~) are
synthetic, seeded, and resident in HBM before the timed region.

Output: one JSON line with weights/s, the HBM roofline of the dominant
N-sized kernel (timed live with HIP events around its launches), and the CPU
oracle timed on a bounded sample on this host.

Other modes (measurement helpers):
  --copy-calibration          run a plain 1 GiB device copy (HBM counter calibration)
  --pmc-summary FETCH WRITE   turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE)
                              into profiles/hbm_traffic.json
"""
import argparse
import ctypes
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "weights clustered/s (DKM fwd+bwd, LLaMA-7B layer shapes, 3-bit); HBM GB/s"
PEAK_HBM_GBS = 8000.0
# algorithmic bytes per weight of each N-sized pass (fp32 W~ output)
PASS_BYTES = {"k_hist": 2, "k_gather_wt": 6, "k_keyed_grad": 6, "k_gather_grad": 10}
PASS_IDS = {"k_hist": 0, "k_gather_wt": 1, "k_keyed_grad": 2, "k_gather_grad": 3}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
COPY_BYTES = 1 << 30


def source_hash():
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2309_00964_amd", "csrc", "*"))):
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


class HipEvents:
    """Timing events straight from the HIP runtime torch uses."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so.7")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        e = ctypes.c_void_p()
        if self.lib.hipEventCreate(ctypes.byref(e)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return e.value

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, e):
        self.lib.hipEventDestroy(e)


def cpu_baseline(host, names):
    """The fp64 dense oracle, as it stands, on the named matrices of the layer."""
    from oracle import dense
    from paper_2309_00964_amd import inputs
    n = 0
    t0 = time.perf_counter()
    for name in names:
        keys, c0, g = host[name]
        f = dense.forward(keys, c0.astype("float64"), inputs.TAU, inputs.ITERS)
        dense.backward(keys, f, g.astype("float64"))
        n += keys.size
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "weights/s", "cores": dense.threads(), "kind": "oracle",
            "sample": "fp64 dense DKM forward+backward (5 iterations, k=8) of %s (%d weights) "
                      "in %.1f s" % ("+".join(names), n, dt)}


def bench(args):
    import numpy as np
    import torch
    from paper_2309_00964_amd import edkm, inputs

    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    w = inputs.WORKLOADS[4]
    bits, k = 3, 8
    plans, keys, c_in, c_out, wt, iters, grads, gw, gc, host = [], [], [], [], [], [], [], [], [], {}
    total = 0
    for i, (name, r, c) in enumerate(w["mats"]):
        n = r * c
        total += n
        kh = inputs.fp16_weights(n, inputs.weight_seed(4, i))
        c0 = inputs.quantile_init(kh, k)
        g = inputs.upstream_grad(n, inputs.grad_seed(4, i))
        if name in args.cpu_sample:
            host[name] = (kh, c0, g)
        plans.append(edkm.Plan(n, bits, inputs.ITERS, device=dev))
        keys.append(torch.from_numpy(kh.view(np.int16)).to(dev))
        c_in.append(torch.from_numpy(c0).to(dev))
        c_out.append(torch.empty(k, device=dev))
        wt.append(torch.empty(n, device=dev))
        iters.append(torch.zeros(1, dtype=torch.int32, device=dev))
        grads.append(torch.from_numpy(g).to(dev))
        gw.append(torch.empty(n, device=dev))
        gc.append(torch.empty(k, device=dev))
    torch.cuda.synchronize()

    def step():
        edkm.init_unique_batch(plans, keys)
        edkm.forward_batch(plans, keys, inputs.TAU, 0.0, c_in, c_out, wt, False, iters)
        edkm.backward_batch(plans, keys, grads, gw, gc)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    hip = HipEvents()
    ev = {p: [(hip.create(), hip.create()) for _ in range(args.steps)] for p in PASS_IDS}
    t_start, t_stop = hip.create(), hip.create()
    stream = torch.cuda.current_stream().cuda_stream
    hip.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    hip.lib.hipEventRecord(t_start, stream)
    for s in range(args.steps):
        for p, pid in PASS_IDS.items():
            edkm.plan_set_pass_events(plans[0], pid, ev[p][s][0], ev[p][s][1])
        step()
    hip.lib.hipEventRecord(t_stop, stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    for pid in PASS_IDS.values():
        edkm.plan_set_pass_events(plans[0], pid, None, None)
    gpu_ms = hip.elapsed_ms(t_start, t_stop)
    elapsed = max(wall, gpu_ms / 1000.0)

    passes = {}
    for p in PASS_IDS:
        d = [hip.elapsed_ms(a, b) for a, b in ev[p]]
        avg = sum(d) / len(d)
        nbytes = PASS_BYTES[p] * total
        passes[p] = {"avg_us": avg * 1000.0, "bytes": nbytes, "GBps": nbytes / (avg * 1e-3) / 1e9}
    dom = max(passes, key=lambda p: passes[p]["avg_us"])
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        tf = json.load(open(TRAFFIC_FILE))
        if tf.get("source_hash") == source_hash() and dom in tf.get("kernels", {}):
            traffic = tf["kernels"][dom]["bytes_per_launch"]
    n_bytes_all = sum(v["bytes"] for v in passes.values())
    t_all = sum(v["avg_us"] for v in passes.values()) * 1e-6
    roof = {"bound": "hbm", "kernel": dom, "achieved": passes[dom]["GBps"], "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": passes[dom]["GBps"] / PEAK_HBM_GBS, "traffic": traffic,
            "n_pass_total_GBps": n_bytes_all / t_all / 1e9,
            "n_pass_total_frac": n_bytes_all / t_all / 1e9 / PEAK_HBM_GBS,
            "passes": {p: {"avg_us": round(v["avg_us"], 2), "GBps": round(v["GBps"], 1)}
                       for p, v in passes.items()}}
    for e in [t_start, t_stop] + [x for p in ev for pair in ev[p] for x in pair]:
        hip.destroy(e)

    out = {
        "metric": METRIC,
        "value": total * args.steps / elapsed,
        "unit": "weights/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1000.0 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic",
        "config": {"workload": "llama7b_decoder_layer_3bit", "matrices": len(plans),
                   "weights": total, "bits": bits, "k": k, "tau": inputs.TAU,
                   "iters": inputs.ITERS, "w_tilde": "fp32", "weights_dtype": "fp16",
                   "parallelism": "single_gpu"},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(host, args.cpu_sample)
    print(json.dumps(out), flush=True)


def copy_calibration():
    import torch
    a = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES}), flush=True)


def _pmc_rows(d, prefix):
    import csv
    files = glob.glob(os.path.join(d, "**", prefix + "*counter_collection.csv"), recursive=True)
    if not files:
        sys.exit("no %s*counter_collection.csv under %s" % (prefix, d))
    rows = []
    for f in files:
        rows += [dict(r, _file=f) for r in csv.DictReader(open(f))]
    return rows


def pmc_summary(fetch_dir, write_dir):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of the pass kernels (run "bench"),
    scaled by what the same counters read for the 1 GiB copies of the calibration
    run ("copy")."""
    def per_dispatch(d, prefix, counter):
        acc = {}
        for r in _pmc_rows(d, prefix):
            if r.get("Counter_Name") != counter:
                continue
            key = (r["_file"], r.get("Dispatch_Id"), r.get("Kernel_Name", ""))
            acc[key] = acc.get(key, 0.0) + float(r["Counter_Value"])
        return acc

    def passes(d, counter):
        out = {}
        for (_, _, name), v in per_dispatch(d, "bench", counter).items():
            p = next((p for p in PASS_IDS if p in name), None)
            if p:
                out.setdefault(p, []).append(v)
        return {p: sum(v) / len(v) for p, v in out.items()}

    def copy(d, counter):
        vals = [v for (_, _, name), v in per_dispatch(d, "copy", counter).items()
                if "copyBuffer" in name]
        big = [v for v in vals if v >= 0.5 * max(vals)]
        return sum(big) / len(big)

    fetch, write = passes(fetch_dir, "FETCH_SIZE"), passes(write_dir, "WRITE_SIZE")
    cf, cw = copy(fetch_dir, "FETCH_SIZE"), copy(write_dir, "WRITE_SIZE")
    f_scale = COPY_BYTES / (cf * 1024.0)
    w_scale = COPY_BYTES / (cw * 1024.0)
    res = {"source_hash": source_hash(), "copy_bytes": COPY_BYTES,
           "copy_fetch_kib": cf, "copy_write_kib": cw,
           "fetch_scale": f_scale, "write_scale": w_scale, "kernels": {}}
    for p in PASS_IDS:
        if p in fetch and p in write:
            fb, wb = fetch[p] * 1024.0 * f_scale, write[p] * 1024.0 * w_scale
            res["kernels"][p] = {"fetch_kib": fetch[p], "write_kib": write[p],
                                 "bytes_per_launch": fb + wb, "fetch_bytes": fb, "write_bytes": wb,
                                 "algorithmic_bytes": None}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    json.dump(res, open(TRAFFIC_FILE, "w"), indent=1)
    print(json.dumps(res))


def main():
    from paper_2309_00964_amd.inputs import LLAMA7B_LAYER
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", nargs="+", default=[m[0] for m in LLAMA7B_LAYER],
                    help="matrices of the layer the CPU oracle is timed on (default: all seven)")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    args = ap.parse_args()
    if args.pmc_summary:
        return pmc_summary(*args.pmc_summary)
    if args.gpus != 1:
        sys.exit("bench.py runs on one GPU: this build has no multi-GPU path (--gpus %d asked)"
                 % args.gpus)
    if args.copy_calibration:
        return copy_calibration()
    bench(args)


if __name__ == "__main__":
    main()
