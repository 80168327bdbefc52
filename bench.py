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

Weight format: --key-format fp16 (default) or bf16 (any workload).
16-bit arrays (decoder layer): --w-tilde half (W~), --grads half (dL/dW~ and
dL/dw), in the weight format.
Cold-cache passes only: --evict-between-calls (decoder layer; pass times only).

The per-pass times are measured twice: back to back (the line's roofline) and
with the Infinity Cache evicted between the three calls
(roofline.evicted_between_calls; --no-evicted-passes skips it).

Other workloads (--workload; one JSON line each, same fields):
  single_256x256 [--bits]     one 256x256 matrix (65,536 weights; launch-bound)
  attn_proj_4096x4096 [--bits]  one 4096x4096 attention projection (16.8M weights)
  mlp_outliers [--bits 3|4]   the 11008x4096 MLP matrix with 0.1% outliers
                              (single-matrix workloads: the dense per-weight-map
                              path is timed beside the uniquified one, "dense")
  stack [--bits 2|3|4]        32 decoder layers (224 matrices, 6.48e9 weights,
                              drawn on the GPU), one step over every matrix
  palettize [--bits 1..4]     export of the decoder layer after a clustering step:
                              packed b-bit nearest-centroid indices per weight
  unique_inverse              the decoder layer's distinct patterns and 16-bit inverse
                              index per weight (the uniquification's lists)

Other modes (measurement helpers):
  --copy-calibration          run a plain 1 GiB device copy (HBM counter calibration)
  --pmc-summary FETCH WRITE   turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE)
                              into profiles/hbm_traffic.json
  --dram-summary DIR...       turn rocprofv3 --pmc runs of the DRAM request counters into
                              profiles/dram_traffic.json (HBM bytes vs Infinity Cache hits)
  --block-timeline OUT.md     run the workload (decoder_layer, attn_proj_4096x4096,
                              mlp_outliers, single_256x256) on the diagnostics build
                              libedkm_stamps.so and write each launch's block timeline
                              of one step (start, span, gap, phases, per-XCC ends)
"""
import argparse
import ctypes
import gc
import glob
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "weights clustered/s (DKM fwd+bwd, LLaMA-7B layer shapes, 3-bit); HBM GB/s"
PEAK_HBM_GBS = 8000.0
# algorithmic bytes per weight of each N-sized pass (fp32 W~ output)
PASS_BYTES = {"k_hist": 2, "k_gather_wt": 6, "k_keyed_grad": 6, "k_gather_grad": 10}
PASS_IDS = {"k_hist": 0, "k_gather_wt": 1, "k_keyed_grad": 2, "k_gather_grad": 3}
# dense comparison path: timed kernels and algorithmic fp32 operations per map
# entry (weight, centroid).  Map row: difference, absolute value, scale,
# exponential, row sum, normalisation (6).  Forward iteration adds S_j += a and
# P_j += a v (3).  Backward iteration adds alpha_j = gamma_j / S_j (v - C_j) (2),
# sum a alpha (2), a (alpha - mean) (2), sign product (1), row and column sums (2).
DENSE_PASS_IDS = {"k_dense_iter": 4, "k_dense_biter": 5}
DENSE_OPS_PER_ENTRY = {"k_dense_iter": 9, "k_dense_biter": 15}
PEAK_FP32_TFLOPS = 157.3
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
# the counter runs behind TRAFFIC_FILE time the default decoder-layer step; its
# figures are attached to that workload's line only
TRAFFIC_WORKLOAD = "llama7b_decoder_layer_3bit"
COPY_BYTES = 1 << 30


def source_hash():
    """Hash of the product build's kernel code: comments, blank lines and the
    block-timeline instrumentation (the EDKM_BLOCK_STAMPS sections and the
    EDKM_STAMP_* statements, which the product build compiles to nothing) are
    left out, so the counters stay tied to what the product compiles."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2309_00964_amd", "csrc", "*"))):
        text = open(f).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        text = re.sub(r"#ifdef EDKM_BLOCK_STAMPS\n.*?#endif", "", text, flags=re.S)
        text = re.sub(r"(?m)^\s*EDKM_STAMP_\w+\([^;]*\);\s*\\?$", "", text)
        h.update("\n".join(l.rstrip() for l in text.splitlines() if l.strip()).encode())
    return h.hexdigest()[:16]


class HipEvents:
    """Timing events straight from the HIP runtime torch uses."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so.7")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    def create(self):
        e = ctypes.c_void_p()
        if self.lib.hipEventCreate(ctypes.byref(e)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return e.value

    def record(self, e, stream):
        if self.lib.hipEventRecord(e, stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, e):
        self.lib.hipEventDestroy(e)


def cpu_model():
    """The host CPU's model name (Linux /proc/cpuinfo), or the platform's."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or platform.machine()


def _repeat_until(fn, min_s):
    """Run fn() at least once and until min_s seconds have passed; (runs, seconds)."""
    runs = 0
    t0 = time.perf_counter()
    while True:
        fn()
        runs += 1
        dt = time.perf_counter() - t0
        if dt >= min_s:
            return runs, dt


def cpu_baseline(samples, k, table_names=("q_proj", "gate_proj", "w", "L0.q_proj"), fmt="fp16",
                 min_s=3.0):
    """The fp64 oracles, as they stand, on bounded samples of the workload:
    ``samples`` is a list of (name, keys, c0, g) host arrays.  The headline
    value is the dense oracle on all host threads over every sample (repeated
    until ``min_s`` seconds have passed, for samples too small to time once);
    beside it the same on one thread (first 2^20 weights of the first sample)
    and the table-form oracle (numpy) on the samples named in ``table_names``."""
    import numpy as np
    from oracle import dense, table
    from paper_2309_00964_amd import inputs

    def dense_all():
        for _, keys, c0, g in samples:
            f = dense.forward(keys, c0.astype("float64"), inputs.TAU, inputs.ITERS, fmt=fmt)
            dense.backward(keys, f, g.astype("float64"))
    n1 = sum(x[1].size for x in samples)
    runs, dt = _repeat_until(dense_all, min_s)
    n = n1 * runs
    out = {"value": n / dt, "unit": "weights/s", "cores": dense.threads(), "kind": "oracle",
           "cpu_model": cpu_model(), "logical_cpus": os.cpu_count(),
           "sample": "fp64 dense DKM forward+backward (%d iterations, k=%d) of %s (%d weights)%s "
                     "in %.1f s" % (inputs.ITERS, k, "+".join(s[0] for s in samples), n1,
                                    " x %d runs" % runs if runs > 1 else "", dt)}
    name, keys, c0, g = samples[0]
    m = min(keys.size, 1 << 20)
    nth = dense.threads()
    dense.set_threads(1)

    def dense_one():
        f = dense.forward(keys[:m], c0.astype("float64"), inputs.TAU, inputs.ITERS, fmt=fmt)
        dense.backward(keys[:m], f, g[:m].astype("float64"))
    runs1, dt1 = _repeat_until(dense_one, min(min_s, 1.0))
    dense.set_threads(nth)
    out["single_thread"] = {"value": m * runs1 / dt1, "unit": "weights/s", "cores": 1,
                            "sample": "the same oracle on the first %d weights of %s%s in %.1f s"
                                      % (m, name, " x %d runs" % runs1 if runs1 > 1 else "", dt1)}
    tab = [x for x in samples if x[0] in table_names] or samples[:1]

    def table_all():
        for _, keys, c0, g in tab:
            f = table.forward(keys, c0.astype(np.float64), inputs.TAU, inputs.ITERS, fmt=fmt)
            table.backward(keys, f, g.astype(np.float64))
    nt1 = sum(x[1].size for x in tab)
    runs2, dt2 = _repeat_until(table_all, min(min_s, 1.0))
    out["table_form"] = {"value": nt1 * runs2 / dt2, "unit": "weights/s", "kind": "oracle (table form, numpy)",
                         "sample": "fp64 uniquified DKM forward+backward of %s (%d weights)%s in %.1f s"
                                   % ("+".join(x[0] for x in tab), nt1,
                                      " x %d runs" % runs2 if runs2 > 1 else "", dt2)}
    return out


LAST_TIMING = {}   # the first timed region of the last timed() call: GPU and host clocks


def timed(step, plan, pass_ids, steps, warmup):
    """Warm up, then run `steps` calls of step() twice on the current stream:
    first as the library runs them, timed between two HIP events (the step
    time), then with the library recording per-pass events on `plan` around
    each timed pass (the per-launch kernel times of the roofline).  The event
    records add a few microseconds per pass, so they stay out of the step time.
    Returns (seconds for `steps` steps, {pass: average launch ms},
    {pass: median launch ms})."""
    import torch
    from paper_2309_00964_amd import edkm
    # Python's cyclic garbage collector stays off while steps are enqueued (as
    # timeit does): a full collection of this process's objects stops the
    # host for ~35 ms, which a 20-step region would count as 1.7 ms per step
    # of idle GPU.
    gc.collect()
    gc_was_on = gc.isenabled()
    gc.disable()
    try:
        return _timed(step, plan, pass_ids, steps, warmup, torch, edkm)
    finally:
        if gc_was_on:
            gc.enable()


def _timed(step, plan, pass_ids, steps, warmup, torch, edkm):
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    hip = HipEvents()
    stream = torch.cuda.current_stream().cuda_stream
    t_start, t_stop = hip.create(), hip.create()
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    hip.record(t_start, stream)
    for _ in range(steps):
        step()
    hip.record(t_stop, stream)
    enq = time.perf_counter() - wall0
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    gpu_s = hip.elapsed_ms(t_start, t_stop) / 1000.0
    ev = {p: [(hip.create(), hip.create()) for _ in range(steps)] for p in pass_ids}
    for s in range(steps):
        for p, pid in pass_ids.items():
            edkm.plan_set_pass_events(plan, pid, ev[p][s][0], ev[p][s][1])
        step()
    torch.cuda.synchronize()
    for pid in pass_ids.values():
        edkm.plan_set_pass_events(plan, pid, None, None)
    per = {p: [hip.elapsed_ms(a, b) for a, b in ev[p]] for p in pass_ids}
    avg = {p: sum(v) / steps for p, v in per.items()}
    med = {p: statistics.median(v) for p, v in per.items()}
    for e in [t_start, t_stop] + [x for p in ev for pair in ev[p] for x in pair]:
        hip.destroy(e)
    LAST_TIMING.update(gpu_ms_per_step=gpu_s * 1000.0 / steps, host_wall_ms_per_step=wall * 1000.0 / steps,
                       host_enqueue_ms_per_step=enq * 1000.0 / steps)
    return max(wall, gpu_s), avg, med


def pass_bytes(p, out_half=False, grads_half=False):
    """Algorithmic bytes per weight of an N-sized pass: 16-bit W~ takes 2 of
    the W~ gather's 6; 16-bit gradients take 2 of the keyed sum's 6 (dL/dW~)
    and 4 of the gradient gather's 10 (dL/dW~ and dL/dw)."""
    if out_half and p == "k_gather_wt":
        return 4
    if grads_half and p == "k_keyed_grad":
        return 4
    if grads_half and p == "k_gather_grad":
        return 6
    return PASS_BYTES[p]


def hbm_roofline(avg_ms, total, out_half=False, med_ms=None, grads_half=False, workload=None):
    """Roofline of the dominant N-sized pass (HBM-bound) plus all passes:
    achieved from the average launch time (as the kernel trace reports it),
    the median beside it.  `traffic` comes from the counter summary only for
    the workload and build it was taken on."""
    passes = {}
    for p, ms in avg_ms.items():
        nbytes = pass_bytes(p, out_half, grads_half) * total
        passes[p] = {"avg_us": ms * 1000.0, "bytes": nbytes, "GBps": nbytes / (ms * 1e-3) / 1e9}
        if med_ms:
            passes[p]["median_us"] = med_ms[p] * 1000.0
    dom = max(passes, key=lambda p: passes[p]["avg_us"])
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        tf = json.load(open(TRAFFIC_FILE))
        if (tf.get("source_hash") == source_hash() and tf.get("workload") == workload
                and dom in tf.get("kernels", {})):
            traffic = tf["kernels"][dom]["bytes_per_launch"]
    n_bytes_all = sum(v["bytes"] for v in passes.values())
    t_all = sum(v["avg_us"] for v in passes.values()) * 1e-6
    return {"bound": "hbm", "kernel": dom, "achieved": passes[dom]["GBps"], "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": passes[dom]["GBps"] / PEAK_HBM_GBS, "traffic": traffic,
            "traffic_kind": "L2-to-fabric bytes per launch (FETCH_SIZE + WRITE_SIZE, scaled by a 1 GiB "
                            "copy): Infinity Cache hits included; the L2's DRAM-request counters count "
                            "them too (profiles/dram_traffic.json)",
            "n_pass_total_GBps": n_bytes_all / t_all / 1e9,
            "n_pass_total_frac": n_bytes_all / t_all / 1e9 / PEAK_HBM_GBS,
            "passes": {p: dict({"avg_us": round(v["avg_us"], 2), "GBps": round(v["GBps"], 1)},
                               **({"median_us": round(v["median_us"], 2)} if "median_us" in v else {}))
                       for p, v in passes.items()}}


def alu_roofline(avg_ms, n, k):
    """Roofline of the dominant dense kernel (fp32 VALU-bound): algorithmic
    fp32 operations per map entry x n*k entries per launch."""
    kern = {p: {"avg_us": ms * 1000.0,
                "TFLOPs": DENSE_OPS_PER_ENTRY[p] * n * k / (ms * 1e-3) / 1e12}
            for p, ms in avg_ms.items()}
    dom = max(kern, key=lambda p: kern[p]["avg_us"])
    return {"bound": "alu", "kernel": dom, "achieved": kern[dom]["TFLOPs"], "peak": PEAK_FP32_TFLOPS,
            "unit": "TFLOP/s", "frac": kern[dom]["TFLOPs"] / PEAK_FP32_TFLOPS, "traffic": None,
            # the code is built without packed-fp32 instructions, so one lane issues one fp32
            # operation (two for an FMA) per cycle: half the headline peak
            "peak_without_packed_fp32": PEAK_FP32_TFLOPS / 2,
            "frac_without_packed_fp32": kern[dom]["TFLOPs"] / (PEAK_FP32_TFLOPS / 2),
            "ops_note": "the exponential counts as one operation (one transcendental instruction, "
                        "issued at a quarter of the FMA rate)",
            "ops_per_entry": DENSE_OPS_PER_ENTRY[dom],
            "kernels": {p: {"avg_us": round(v["avg_us"], 2), "TFLOPs": round(v["TFLOPs"], 2)}
                        for p, v in kern.items()}}


class Matrices:
    """Device inputs and outputs of a list of (name, rows, cols) matrices, each
    with its own plan and centroids."""

    def __init__(self, config, mats, bits, outliers=False, on_device=False, keep_host=(), fmt="fp16",
                 out_half=False, evict=False, grads_half=False):
        import numpy as np
        import torch
        from paper_2309_00964_amd import edkm, inputs
        dev = torch.device("cuda:0")
        k = 1 << bits
        self.names, self.plans, self.keys, self.c_in, self.c_out = [], [], [], [], []
        self.wt, self.iters, self.grads, self.gw, self.gc, self.host = [], [], [], [], [], []
        self.total = 0
        for i, (name, r, c) in enumerate(mats):
            n = r * c
            self.total += n
            if on_device:
                kt = inputs.fp16_weights_device(n, inputs.weight_seed(config, i), dev, outliers, fmt)
                c0 = inputs.quantile_init_device(kt, k, fmt)
                gt = inputs.upstream_grad_device(n, inputs.grad_seed(config, i), dev)
                if name in keep_host:
                    self.host.append((name, kt.cpu().numpy().view(np.uint16), c0.cpu().numpy(),
                                      gt.cpu().numpy()))
            else:
                kh = inputs.weights(n, inputs.weight_seed(config, i), outliers, fmt)
                c0h = inputs.quantile_init(kh, k, fmt)
                g = inputs.upstream_grad(n, inputs.grad_seed(config, i))
                if name in keep_host:
                    self.host.append((name, kh, c0h, g))
                kt = torch.from_numpy(kh.view(np.int16)).to(dev)
                c0 = torch.from_numpy(c0h).to(dev)
                gt = torch.from_numpy(g).to(dev)
            self.names.append(name)
            self.plans.append(edkm.Plan(n, bits, inputs.ITERS, device=dev, key_format=fmt))
            self.keys.append(kt)
            self.c_in.append(c0)
            self.c_out.append(torch.empty(k, device=dev))
            self.wt.append(torch.empty(n, dtype=torch.int16 if out_half else torch.float32, device=dev))
            self.iters.append(torch.zeros(1, dtype=torch.int32, device=dev))
            if grads_half:   # dL/dW~ rounded to the weights' format; dL/dw written in it
                self.grads.append(gt.to(torch.float16 if fmt == "fp16" else torch.bfloat16).view(torch.int16))
                self.gw.append(torch.empty(n, dtype=torch.int16, device=dev))
            else:
                self.grads.append(gt)
                self.gw.append(torch.empty(n, device=dev))
            self.gc.append(torch.empty(k, device=dev))
        self.fmt = fmt
        self.out_half = out_half
        self.evict_buf = torch.ones(1 << 28, device="cuda") if evict else None
        self.evict_sink = torch.zeros((), device="cuda")
        self.evicting = evict
        torch.cuda.synchronize()

    def step(self):
        from paper_2309_00964_amd import edkm, inputs
        edkm.init_unique_batch(self.plans, self.keys)
        self.evict()
        edkm.forward_batch(self.plans, self.keys, inputs.TAU, 0.0, self.c_in, self.c_out, self.wt,
                           self.out_half, self.iters)
        self.evict()
        edkm.backward_batch(self.plans, self.keys, self.grads, self.gw, self.gc)
        self.evict()

    def evict(self):
        """With an eviction buffer: read 1 GiB between calls, so that no call
        finds the previous call's data in the 256 MB Infinity Cache (as when a
        model's own work runs between them)."""
        if self.evict_buf is not None and self.evicting:
            self.evict_sink += self.evict_buf.sum()

    def dense_step(self):
        from paper_2309_00964_amd import edkm, inputs
        for i, p in enumerate(self.plans):
            edkm.forward_dense(p, self.keys[i], inputs.TAU, 0.0, self.c_in[i], self.c_out[i],
                               self.wt[i], False, self.iters[i])
            edkm.backward_dense(p, self.keys[i], self.grads[i], self.gw[i], self.gc[i])


def _fmt_tag(args):
    return "" if args.key_format == "fp16" else "_" + args.key_format


def result_line(args, workload, m, bits, elapsed, roof, extra_cfg=None):
    from paper_2309_00964_amd import inputs
    cfg = {"workload": workload, "matrices": len(m.plans), "weights": m.total, "bits": bits,
           "k": 1 << bits, "tau": inputs.TAU, "iters": inputs.ITERS, "w_tilde": "fp32",
           "weights_dtype": m.fmt, "parallelism": "single_gpu"}
    cfg.update(extra_cfg or {})
    return {
        "metric": METRIC,
        "value": m.total * args.steps / elapsed,
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
        "config": cfg,
        "roofline": roof,
        "timing": {k: round(v, 4) for k, v in LAST_TIMING.items()},
    }


def bench_decoder_layer(args):
    """One LLaMA-7B decoder layer at 3 bits: the seven matrices as batched calls.

    The step runs init_unique, forward and backward back to back, so a pass
    can find the tail of what the previous call read in the Infinity Cache.
    Unless --no-evicted-passes is given, the per-pass times are measured a
    second time with 1 GiB read between the three calls (no call then finds
    its predecessor's data, as when a model's own work runs in between) and
    reported beside the back-to-back figures in roofline.evicted_between_calls."""
    from paper_2309_00964_amd import inputs
    bits = 3
    keep = () if args.no_cpu_baseline else tuple(args.cpu_sample)
    half = args.w_tilde == "half"
    ghalf = args.grads == "half"
    want_evicted = args.evict_between_calls or not args.no_evicted_passes
    m = Matrices(4, inputs.WORKLOADS[4]["mats"], bits, keep_host=keep, fmt=args.key_format, out_half=half,
                 evict=want_evicted, grads_half=ghalf)
    m.evicting = args.evict_between_calls
    elapsed, avg, med = timed(m.step, m.plans[0], PASS_IDS, args.steps, args.warmup)
    extra = {"w_tilde": m.fmt if half else "fp32"}
    if ghalf:
        extra["grads"] = m.fmt
    if args.evict_between_calls:
        # the step time then includes three 1 GiB eviction reads; the pass
        # times (roofline) are the figures this mode is for
        extra["evict_between_calls"] = True
    workload = ("llama7b_decoder_layer_3bit" + _fmt_tag(args) + ("_half_wtilde" if half else "")
                + ("_half_grads" if ghalf else "") + ("_evicted" if args.evict_between_calls else ""))
    roof = hbm_roofline(avg, m.total, half, med, ghalf, workload)
    line_timing = dict(LAST_TIMING)
    if want_evicted and not args.evict_between_calls:
        m.evicting = True
        _, eavg, emed = timed(m.step, m.plans[0], PASS_IDS, args.steps, 1)
        m.evicting = False
        ev = hbm_roofline(eavg, m.total, half, emed, ghalf)
        roof["evicted_between_calls"] = {
            "kernel": ev["kernel"], "achieved": ev["achieved"], "frac": ev["frac"],
            "n_pass_total_GBps": ev["n_pass_total_GBps"], "n_pass_total_frac": ev["n_pass_total_frac"],
            "passes": ev["passes"],
            "note": "same passes with 1 GiB read between init_unique, forward and backward "
                    "(no Infinity Cache reuse across calls); the gradient gather keeps the "
                    "reuse inside the backward"}
    LAST_TIMING.clear()
    LAST_TIMING.update(line_timing)
    out = result_line(args, workload, m, bits, elapsed, roof, extra)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(m.host, 1 << bits, fmt=m.fmt)
    return out


def bench_single_matrix(args, cfg, default_bits):
    """One matrix of the synthetic workloads: 256x256 (config 1), 4096x4096
    (config 2, an attention projection) or 11008x4096 with 0.1% outliers
    (config 3, an MLP matrix).  The uniquified path is the line; the dense
    (per-weight map) path is timed beside it on the same inputs."""
    from paper_2309_00964_amd import inputs
    bits = args.bits or default_bits
    w = inputs.WORKLOADS[cfg]
    keep = () if args.no_cpu_baseline else ("w",)
    m = Matrices(cfg, w["mats"], bits, outliers=w["outliers"], keep_host=keep, fmt=args.key_format)
    elapsed, avg, med = timed(m.step, m.plans[0], PASS_IDS, args.steps, args.warmup)
    name = "%s_%dbit%s" % (SINGLE_NAMES[cfg], bits, _fmt_tag(args))
    extra = {"outliers": inputs.OUTLIER_P} if w["outliers"] else {}
    out = result_line(args, name, m, bits, elapsed, hbm_roofline(avg, m.total, med_ms=med), extra)
    d_el, d_avg, _ = timed(m.dense_step, m.plans[0], DENSE_PASS_IDS, args.steps, args.warmup)
    out["dense"] = {"value": m.total * args.steps / d_el, "unit": "weights/s",
                    "ms_per_step": d_el * 1000.0 / args.steps,
                    "unique_speedup": d_el / elapsed,
                    "roofline": alu_roofline(d_avg, m.total, 1 << bits)}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(m.host, 1 << bits, fmt=m.fmt)
    return out


SINGLE_NAMES = {1: "single_256x256", 2: "attn_proj_4096x4096", 3: "llama7b_mlp_11008x4096_outliers"}


def bench_mlp_outliers(args):
    """The 11008x4096 MLP matrix with 0.1% outliers (4 bits unless --bits 3)."""
    return bench_single_matrix(args, 3, 4)


def bench_palettize(args):
    """Export of the decoder layer: after one clustering step, the packed b-bit
    nearest-entry indices of every weight against its matrix's final centroids
    (edkm_palettize_batch: one table launch and one packing launch for the
    seven matrices).  Pass events time the packing kernel; the roofline is its
    2 + b/8 bytes per weight."""
    import torch
    from paper_2309_00964_amd import edkm, inputs
    bits = args.bits or 3
    m = Matrices(4, inputs.WORKLOADS[4]["mats"], bits, fmt=args.key_format)
    m.step()
    outs = [torch.empty((p.n * bits + 7) // 8, dtype=torch.uint8, device="cuda") for p in m.plans]

    def step():
        edkm.palettize_batch(m.plans, m.keys, m.c_out, outs)
    elapsed, avg, _ = timed(step, m.plans[0], {"k_palettize": edkm.PASS_PALETTIZE}, args.steps, args.warmup)
    per_w = 2.0 + bits / 8.0
    kern_s = avg["k_palettize"] / 1000.0
    achieved = per_w * m.total / kern_s / 1e9
    roof = {"bound": "hbm", "kernel": "k_palettize", "achieved": achieved, "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": None,
            "bytes_per_weight": per_w, "kernel_us_per_step": kern_s * 1e6}
    return result_line(args, "llama7b_decoder_layer_palettize_%dbit%s" % (bits, _fmt_tag(args)), m,
                       bits, elapsed, roof, {"w_tilde": None, "output": "packed %d-bit indices" % bits})


def bench_unique_inverse(args):
    """The uniquification's lists for the decoder layer (edkm_unique_inverse_batch
    after one init_unique): the sorted distinct patterns and the 16-bit inverse
    index of every weight, one ranking launch and one N-sized launch for the
    seven matrices.  Pass events time the inverse-index kernel; the roofline is
    its 2 + 2 bytes per weight."""
    import torch
    from paper_2309_00964_amd import edkm, inputs
    bits = args.bits or 3
    m = Matrices(4, inputs.WORKLOADS[4]["mats"], bits, fmt=args.key_format)
    m.step()
    uniq = [torch.empty(edkm.NKEYS, dtype=torch.int16, device="cuda") for _ in m.plans]
    inv = [torch.empty(p.n, dtype=torch.int16, device="cuda") for p in m.plans]

    def step():
        edkm.unique_inverse_batch(m.plans, m.keys, uniq, inv)
    elapsed, avg, _ = timed(step, m.plans[0], {"k_inverse": edkm.PASS_INVERSE}, args.steps, args.warmup)
    per_w = 4.0
    kern_s = avg["k_inverse"] / 1000.0
    achieved = per_w * m.total / kern_s / 1e9
    roof = {"bound": "hbm", "kernel": "k_inverse", "achieved": achieved, "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": None,
            "bytes_per_weight": per_w, "kernel_us_per_step": kern_s * 1e6}
    return result_line(args, "llama7b_decoder_layer_unique_inverse%s" % _fmt_tag(args), m,
                       bits, elapsed, roof, {"w_tilde": None, "output": "distinct patterns + 16-bit inverse index"})


def bench_stack(args):
    """A 32-layer stack of decoder-layer shapes (224 matrices, 6.48e9 weights),
    drawn on the device; one step clusters every matrix forward and backward."""
    from paper_2309_00964_amd import inputs
    bits = args.bits or 3
    w = inputs.WORKLOADS[5]
    # the CPU oracle's rate on two of the 32 layers (14 matrices, 405M weights)
    keep = () if args.no_cpu_baseline else tuple(n for n, _, _ in w["mats"] if n.split(".")[0] in ("L0", "L1"))
    m = Matrices(5, w["mats"], bits, on_device=True, keep_host=keep, fmt=args.key_format)
    elapsed, avg, med = timed(m.step, m.plans[0], PASS_IDS, args.steps, args.warmup)
    # the pass events bracket the first launch group of each step: its first
    # LAUNCH_GROUP matrices (layers 0-3)
    from paper_2309_00964_amd import edkm
    group = edkm.LAUNCH_GROUP
    roof = hbm_roofline(avg, sum(r * c for _, r, c in w["mats"][:group]), med_ms=med)
    roof["note"] = "pass events cover the first launch group (%d matrices) of each step" % group
    out = result_line(args, "llama7b_32_layer_stack_%dbit%s" % (bits, _fmt_tag(args)), m, bits, elapsed, roof)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(m.host, 1 << bits, fmt=m.fmt)
    return out


def copy_calibration():
    import torch
    a = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES}), flush=True)


def kernel_base_name(name):
    """'edkm::k_hist(edkm::BatchArgs)' -> 'k_hist'; 'void edkm::k_fwd_iter<8>(...)' -> 'k_fwd_iter'."""
    return name.split("(")[0].split("<")[0].split("::")[-1].split(" ")[-1]


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
            p = kernel_base_name(name)   # exact: k_hist is not k_hist_merge
            if p in PASS_IDS:
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
    res = {"source_hash": source_hash(), "workload": TRAFFIC_WORKLOAD, "copy_bytes": COPY_BYTES,
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


DRAM_FILE = os.path.join(ROOT, "profiles", "dram_traffic.json")
DRAM_COUNTERS = ("TCC_EA0_RDREQ_DRAM_sum", "TCC_EA0_WRREQ_DRAM_sum", "TCC_EA0_RDREQ_sum", "TCC_EA0_WRREQ_sum")


def dram_summary(dirs):
    """Which of the L2's fabric requests the counters see as bound for DRAM.
    Each directory holds a rocprofv3 --pmc run of the four DRAM_COUNTERS over
    "bench" (a workload run) and "copy" (--copy-calibration).  Of the read
    (write) requests the L2 sends to the fabric, TCC_EA0_RDREQ_DRAM
    (WRREQ_DRAM) counts those addressed to the memory controller.  The
    summary gives that share per pass and, with the fabric bytes of
    profiles/hbm_traffic.json (same kernels), the DRAM-addressed bytes.  On
    MI355X the Infinity Cache sits behind that interface, so its hits are
    counted as DRAM requests too: the share is 1 for every pass, and the
    split of HBM bytes from Infinity Cache hits is not observable with these
    counters (the evicted-between-calls pass times measure the reuse instead)."""
    def per_pass(d, prefix, counter):
        acc = {}
        for r in _pmc_rows(d, prefix):
            if r.get("Counter_Name") != counter:
                continue
            key = (r["_file"], r.get("Dispatch_Id"), r.get("Kernel_Name", ""))
            acc[key] = acc.get(key, 0.0) + float(r["Counter_Value"])
        out = {}
        for (_, _, name), v in acc.items():
            p = kernel_base_name(name)
            if p in PASS_IDS or "copyBuffer" in name:
                out.setdefault("copy" if "copyBuffer" in name else p, []).append(v)
        return {p: sum(v) / len(v) for p, v in out.items()}

    fabric = json.load(open(TRAFFIC_FILE)) if os.path.exists(TRAFFIC_FILE) else {}
    same_build = fabric.get("source_hash") == source_hash()
    res = {"source_hash": source_hash(), "counters": list(DRAM_COUNTERS), "runs": {}}
    for d in dirs:
        label = os.path.basename(os.path.normpath(d))
        rd = per_pass(d, "bench", "TCC_EA0_RDREQ_DRAM_sum")
        wd = per_pass(d, "bench", "TCC_EA0_WRREQ_DRAM_sum")
        ra = per_pass(d, "bench", "TCC_EA0_RDREQ_sum")
        wa = per_pass(d, "bench", "TCC_EA0_WRREQ_sum")
        cp = {c: per_pass(d, "copy", c).get("copy") for c in DRAM_COUNTERS}
        run = {"copy_read_dram_share": cp["TCC_EA0_RDREQ_DRAM_sum"] / cp["TCC_EA0_RDREQ_sum"]
               if cp["TCC_EA0_RDREQ_sum"] else None,
               "copy_write_dram_share": cp["TCC_EA0_WRREQ_DRAM_sum"] / cp["TCC_EA0_WRREQ_sum"]
               if cp["TCC_EA0_WRREQ_sum"] else None,
               "passes": {}}
        for p in PASS_IDS:
            if p not in ra:
                continue
            q = {"read_requests": ra[p], "read_dram_requests": rd.get(p, 0.0),
                 "write_requests": wa.get(p, 0.0), "write_dram_requests": wd.get(p, 0.0),
                 "read_dram_share": rd.get(p, 0.0) / ra[p] if ra[p] else None,
                 "write_dram_share": wd.get(p, 0.0) / wa[p] if wa.get(p) else None}
            k = fabric.get("kernels", {}).get(p)
            if same_build and k:
                q["fabric_read_bytes"] = k["fetch_bytes"]
                q["fabric_write_bytes"] = k["write_bytes"]
                q["dram_addressed_read_bytes"] = k["fetch_bytes"] * q["read_dram_share"]
                q["dram_addressed_write_bytes"] = k["write_bytes"] * (q["write_dram_share"] or 0.0)
            run["passes"][p] = q
        res["runs"][label] = run
    os.makedirs(os.path.dirname(DRAM_FILE), exist_ok=True)
    json.dump(res, open(DRAM_FILE, "w"), indent=1)
    print(json.dumps(res))


# record shape of the diagnostics build (EDKM_STAMP_* of include/edkm_stamps.h)
STAMP_LAUNCHES, STAMP_BLOCKS, STAMP_WORDS = 96, 4096, 8
TIMELINE_PHASES = {   # phase marks (record words 2..5) of the instrumented kernels
    "k_hist": ("keys streamed", "span found"),
    "k_window": ("wave 0 scanned", "block totals combined", "windows chosen"),
    "k_hist_merge": ("rows summed",),
    "k_grad_top": ("rows summed (G loaded)", "patterns done", "block summed"),
    "k_fwd_iter": ("loads issued", "partials summed, C formed", "patterns done", "block summed"),
    "k_bwd_iter": ("loads issued", "partials summed, gamma formed", "patterns done", "block summed"),
}


def block_timeline(args):
    """Per-block wall-clock stamps of one step, from the diagnostics build
    (libedkm_stamps.so: the product sources compiled with EDKM_BLOCK_STAMPS),
    summarised per launch: when its first block started and its last block
    ended relative to the step's first block, the gap after the previous
    launch, block durations, the phase marks of the instrumented kernels and,
    for the kernels with one block per CU or more, when the blocks of each XCC
    had finished.  Medians over `reps` steps after `warmup` untimed ones."""
    import numpy as np
    import torch
    from paper_2309_00964_amd import build, edkm, inputs
    if os.path.abspath(edkm.LIB_PATH) != os.path.abspath(build.OUT_STAMPS):
        sys.exit("--block-timeline: %s is loaded, not the diagnostics build %s"
                 % (edkm.LIB_PATH, build.OUT_STAMPS))
    lib = edkm._lib
    lib.edkm_stamps_dump.argtypes = [ctypes.c_void_p, ctypes.c_char_p]
    L, B, W = STAMP_LAUNCHES, STAMP_BLOCKS, STAMP_WORDS
    work = {"decoder_layer": (4, 3, False), "attn_proj_4096x4096": (2, 3, False),
            "mlp_outliers": (3, 4, True), "single_256x256": (1, 3, False)}
    if args.workload not in work:
        sys.exit("--block-timeline: workload %s has no timeline" % args.workload)
    cfg, bits, outl = work[args.workload]
    bits = args.bits or bits
    m = Matrices(cfg, inputs.WORKLOADS[cfg]["mats"], bits, outliers=outl, fmt=args.key_format)
    for _ in range(args.warmup):
        m.step()
    torch.cuda.synchronize()
    rate = lib.edkm_stamps_clock_khz() * 1e3
    if rate <= 0:
        sys.exit("--block-timeline: no stamp clock rate")
    reps = 7
    raw = []
    for _ in range(reps):
        if lib.edkm_stamps_reset() != 0:
            sys.exit("--block-timeline: edkm_stamps_reset failed")
        m.step()
        torch.cuda.synchronize()
        buf = np.zeros(L * B * W, np.uint64)
        names = ctypes.create_string_buffer(L * 32)
        n = lib.edkm_stamps_dump(buf.ctypes.data, names)
        if n < 0 or n > L:
            sys.exit("--block-timeline: %d launches (record holds %d)" % (n, L))
        nm = [names.raw[i * 32:(i + 1) * 32].split(b"\0")[0].decode() for i in range(n)]
        raw.append((nm, buf.reshape(L, B, W)[:n]))
    cmd = "python bench.py --workload %s%s --block-timeline %s" % (
        args.workload, "" if args.key_format == "fp16" else " --key-format " + args.key_format,
        args.block_timeline)
    title = "%s (%d weights, %d-bit, %s)" % (args.workload, m.total, bits, m.fmt)
    text = timeline_report(raw, rate, title, cmd, args.warmup)
    with open(args.block_timeline, "w") as f:
        f.write(text)
    print(text, flush=True)
    return None


def timeline_report(raw, rate, title, cmd, warmup):
    """Markdown summary of stamp records: raw = [(launch names, uint64 array
    [launches, blocks, STAMP_WORDS]) per step], rate = stamp clock in Hz."""
    import numpy as np
    W = STAMP_WORDS
    reps = len(raw)
    names0 = raw[0][0]
    if any(r[0] != names0 for r in raw):
        raise ValueError("the launch sequence changed between steps")
    scale = np.where(np.arange(W) < 7, 1e6 / rate, 1.0)
    steps, blocks = [], []
    for _, ts in raw:
        recs = [ts[q][ts[q][:, 0] > 0].astype(np.float64) for q in range(len(names0))]
        blocks.append([np.nonzero(ts[q][:, 0] > 0)[0] for q in range(len(names0))])
        if any(len(r) == 0 for r in recs):
            raise ValueError("a launch has no block records")
        t0 = min(r[:, 0].min() for r in recs)
        # words 0..6 to microseconds from the step's first block start (a phase
        # mark that was not reached becomes negative); word 7 (XCC id) as is
        steps.append([(r - np.where(np.arange(W) < 7, t0, 0.0)) * scale for r in recs])
    med = lambda xs: float(np.median(xs))
    rows = []
    for q, name in enumerate(names0):
        start = med([s_[q][:, 0].min() for s_ in steps])
        end = med([s_[q][:, 1].max() for s_ in steps])
        gap = med([s_[q][:, 0].min() - s_[q - 1][:, 1].max() for s_ in steps]) if q else 0.0
        dur = med([med(s_[q][:, 1] - s_[q][:, 0]) for s_ in steps])
        dmax = med([(s_[q][:, 1] - s_[q][:, 0]).max() for s_ in steps])
        rows.append((name, len(steps[0][q]), start, end - start, gap, dur, dmax))
    span = med([max(r_[:, 1].max() for r_ in s_) for s_ in steps])
    out = ["# Block timeline of one step: " + title,
           "", "```", cmd, "```", "",
           "Diagnostics build libedkm_stamps.so (the product sources with EDKM_BLOCK_STAMPS): every block "
           "stamps the GPU wall clock (%.0f MHz) at entry and exit and its XCC id.  Medians over %d steps "
           "after %d warm-up steps; times in microseconds from the step's first block start.  A launch's "
           "span runs from its first block start to its last block end; its gap from the previous launch's "
           "last block end to its first block start." % (rate / 1e6, reps, warmup), "",
           "| # | Kernel | Blocks | Start | Span | Gap before | Block median | Block max |",
           "|---|---|---|---|---|---|---|---|"]
    for q, r in enumerate(rows):
        out.append("| %d | %s | %d | %.1f | %.1f | %.1f | %.1f | %.1f |" % ((q,) + r))
    tot = {}
    for r in rows:
        t = tot.setdefault(r[0], [0, 0.0, 0.0])
        t[0] += 1
        t[1] += r[3]
        t[2] += r[4]
    out += ["", "Step %.1f us: launch spans %.1f us, gaps %.1f us." % (
        span, sum(r[3] for r in rows), sum(r[4] for r in rows)), "",
        "| Kernel | Launches | Spans | Gaps before |", "|---|---|---|---|"]
    for k_, (c, sp, gp) in sorted(tot.items(), key=lambda kv: -kv[1][1]):
        out.append("| %s | %d | %.1f | %.1f |" % (k_, c, sp, gp))
    mid = steps[reps // 2]
    mid_blocks = blocks[reps // 2]
    ph = []
    for q, name in enumerate(names0):
        labels = TIMELINE_PHASES.get(name)
        if not labels:
            continue
        v = mid[q]
        v = v[(v[:, 2:2 + len(labels)] > 0).all(axis=1)]   # blocks that reached every mark
        if not len(v):
            continue
        cols = [0] + [2 + i for i in range(len(labels))] + [1]
        lab = lambda c: "entry" if c == 0 else "end" if c == 1 else labels[c - 2]
        seg = ["%s -> %s %.2f" % (lab(a), lab(b_), med(v[:, b_] - v[:, a])) for a, b_ in zip(cols[:-1], cols[1:])]
        ph.append("| %d | %s | %d | %s |" % (q, name, len(v), "; ".join(seg)))
    if ph:
        out += ["", "Phases (medians over the blocks of the middle step that reached every mark, us):", "",
                "| # | Kernel | Blocks | Phases |", "|---|---|---|---|"] + ph
    xr, dist = [], []
    for q, name in enumerate(names0):
        v = mid[q]
        if len(v) < 64:
            continue
        blk = mid_blocks[q]
        x = v[:, 7].astype(np.int64) & 0xF
        s0 = v[:, 0].min()
        ends = {c: v[x == c, 1].max() - s0 for c in range(16) if (x == c).any()}
        blocks = {c: int((x == c).sum()) for c in ends}
        xr.append("| %d | %s | %s | %.1f |" % (q, name, " ".join("%d:%d/%.1f" % (c, blocks[c], ends[c])
                                                                    for c in ends),
                                            max(ends.values()) - min(ends.values())))
        d = v[:, 1] - v[:, 0]
        slow = np.argsort(-d)[:6]
        dist.append("| %d | %s | %.1f | %.1f | %.1f | %.1f | %s |" % (
            q, name, np.percentile(d, 10), np.median(d), np.percentile(d, 90), d.max(),
            " ".join("%d:%.1f" % (blk[i], d[i]) for i in slow)))
    if dist:
        out += ["", "Block durations of the same launches (us): percentiles, and the six slowest blocks "
                "(linear block index: duration).", "", "| # | Kernel | p10 | p50 | p90 | Max | Slowest |",
                "|---|---|---|---|---|---|---|"] + dist
    if xr:
        out += ["", "Per-XCC finish of the launches with 64 blocks or more (middle step): XCC:blocks/last block "
                "end from the launch's first block start (us), and the spread between the first and last XCC "
                "to finish.", "", "| # | Kernel | XCC:blocks/end | Spread |", "|---|---|---|---|"] + xr
    return "\n".join(out) + "\n"


def main():
    from paper_2309_00964_amd.inputs import LLAMA7B_LAYER
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", choices=("decoder_layer", "single_256x256", "attn_proj_4096x4096",
                                           "mlp_outliers", "stack", "palettize", "unique_inverse"),
                    default="decoder_layer")
    ap.add_argument("--bits", type=int, choices=(1, 2, 3, 4), default=None,
                    help="mlp_outliers: 3 or 4 (default 4); stack: 2, 3 or 4 (default 3); "
                         "palettize: 1-4 (default 3)")
    ap.add_argument("--key-format", choices=("fp16", "bf16"), default="fp16",
                    help="weight format (default fp16, the metric's; bf16 is the paper's training format)")
    ap.add_argument("--w-tilde", choices=("fp32", "half"), default="fp32",
                    help="decoder_layer: W~ output as fp32 (default, 24 B per weight) or in the "
                         "16-bit weight format (22 B per weight)")
    ap.add_argument("--grads", choices=("fp32", "half"), default="fp32",
                    help="decoder_layer: dL/dW~ in and dL/dw out as fp32 (default) or in the 16-bit "
                         "weight format (18 B per weight; with --w-tilde half, 16 B: "
                         "a training step in the weights' precision)")
    ap.add_argument("--evict-between-calls", action="store_true",
                    help="decoder layer: read 1 GiB between init_unique, forward and backward, so that "
                         "no call finds its predecessor's data in the Infinity Cache (pass times only)")
    ap.add_argument("--no-evicted-passes", action="store_true",
                    help="decoder layer: skip the second per-pass measurement with the Infinity Cache "
                         "evicted between the calls")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", nargs="+", default=[m[0] for m in LLAMA7B_LAYER],
                    help="matrices of the layer the CPU oracle is timed on (default: all seven)")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--dram-summary", nargs="+", metavar="DIR")
    ap.add_argument("--block-timeline", metavar="OUT_MD")
    args = ap.parse_args()
    if args.block_timeline:
        # the diagnostics build, loaded in place of the product library
        from paper_2309_00964_amd import build
        os.environ["EDKM_LIBRARY"] = build.OUT_STAMPS
    if args.pmc_summary:
        return pmc_summary(*args.pmc_summary)
    if args.dram_summary:
        return dram_summary(args.dram_summary)
    if args.gpus != 1:
        sys.exit("bench.py runs on one GPU: the library has no multi-GPU path (--gpus %d asked)"
                 % args.gpus)
    if args.copy_calibration:
        return copy_calibration()
    import torch
    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    fn = {"decoder_layer": bench_decoder_layer, "mlp_outliers": bench_mlp_outliers,
          "single_256x256": lambda a: bench_single_matrix(a, 1, 3),
          "attn_proj_4096x4096": lambda a: bench_single_matrix(a, 2, 3),
          "stack": bench_stack, "palettize": bench_palettize,
          "unique_inverse": bench_unique_inverse}[args.workload]
    if args.workload == "decoder_layer" and args.bits not in (None, 3):
        sys.exit("the decoder-layer workload is 3-bit")
    if args.block_timeline:
        return block_timeline(args)
    print(json.dumps(fn(args)), flush=True)


if __name__ == "__main__":
    main()
