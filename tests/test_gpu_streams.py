"""Streams and graphs: distinct plans run concurrently on distinct streams, and
a whole batched step (init_unique + forward + backward) captured in a HIP graph
replays to the eager results, also with the weights changed in place between
replays and an early stop that moves with them, as do the export calls
(distinct-pattern list, inverse index, palettization).

Forward outputs are compared bitwise (fixed-order reductions).  Backward
outputs within 1e-6 relative: the keyed sum's fp32 fallback and merge atomics
vary in the last bits between runs.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2309_00964_amd import edkm, inputs                     # noqa: E402
from parity_util import assert_close                              # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda"
TAU, ITERS = inputs.TAU, inputs.ITERS


def say(*a):
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


class Batch:
    """Device inputs/outputs and plans of a few matrices."""

    def __init__(self, sizes, seed, bits=3):
        k = 1 << bits
        self.keys, self.c0, self.g = [], [], []
        for i, n in enumerate(sizes):
            kh = inputs.fp16_weights(n, seed + i, outliers=(i == 1))
            self.keys.append(torch.from_numpy(kh.view(np.int16)).to(DEV))
            self.c0.append(torch.from_numpy(inputs.quantile_init(kh, k)).to(DEV))
            self.g.append(torch.from_numpy(inputs.upstream_grad(n, seed + 50 + i)).to(DEV))
        self.plans = [edkm.Plan(n, bits, ITERS) for n in sizes]
        self.c_out = [torch.empty(k, device=DEV) for _ in sizes]
        self.wt = [torch.empty(n, device=DEV) for n in sizes]
        self.it = [torch.zeros(1, dtype=torch.int32, device=DEV) for _ in sizes]
        self.gw = [torch.empty(n, device=DEV) for n in sizes]
        self.gc = [torch.empty(k, device=DEV) for _ in sizes]

    def step(self, stream=None):
        edkm.init_unique_batch(self.plans, self.keys, stream=stream)
        edkm.forward_batch(self.plans, self.keys, TAU, 0.0, self.c0, self.c_out, self.wt, False, self.it,
                           stream=stream)
        edkm.backward_batch(self.plans, self.keys, self.g, self.gw, self.gc, stream=stream)

    def outputs(self):
        return [dict(c_out=a.cpu().numpy(), wt=b.cpu().numpy(), it=c.cpu().numpy(),
                     gw=d.cpu().numpy(), gc=e.cpu().numpy())
                for a, b, c, d, e in zip(self.c_out, self.wt, self.it, self.gw, self.gc)]

    def poison(self):
        for t in self.c_out + self.wt + self.gw + self.gc:
            t.fill_(float("nan"))
        for t in self.it:
            t.fill_(-1)


def same(got, ref, what):
    for i, (a, b) in enumerate(zip(got, ref)):
        for name in ("c_out", "wt", "it"):
            assert np.array_equal(a[name], b[name]), "%s %d %s" % (what, i, name)
        assert_close(a["gw"], b["gw"], 1e-6, "%s %d gw" % (what, i))
        assert_close(a["gc"], b["gc"], 1e-6, "%s %d gc" % (what, i))


def test_two_plans_on_two_streams_concurrently():
    a = Batch([65536, 300_007], 300)
    b = Batch([100_003, 1_000_003], 310)
    say("streams: references")
    a.step()
    b.step()
    torch.cuda.synchronize()
    ref_a, ref_b = a.outputs(), b.outputs()
    a.poison()
    b.poison()
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()     # default priority
    say("streams: concurrent")
    for _ in range(3):
        a.step(stream=s1)
        b.step(stream=s2)
    torch.cuda.synchronize()
    same(a.outputs(), ref_a, "stream a")
    same(b.outputs(), ref_b, "stream b")


def test_graph_capture_replays_the_eager_step():
    x = Batch([65536, 300_007, 1_000_003], 320)
    other = Batch([50_000], 330)
    say("graph: eager reference")
    x.step()
    torch.cuda.synchronize()
    ref = x.outputs()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        x.step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    say("graph: capture")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        x.step()
    torch.cuda.synchronize()
    for rep in range(3):
        other.step()                 # eager work of the program between replays
        x.poison()
        torch.cuda.synchronize()
        say("graph: replay", rep)
        graph.replay()
        torch.cuda.synchronize()
        same(x.outputs(), ref, "replay %d" % rep)


def _step_sizes(keys, c0, iters):
    """max_j |C^(t)_j - C^(t-1)_j| for t = 1..iters, from the fp64 oracle."""
    from oracle import dense
    h = dense.forward(keys, c0.astype(np.float64), TAU, iters)["c_hist"]
    return np.max(np.abs(np.diff(h, axis=0)), axis=1)


def _stop_iteration(st, eps, iters):
    """Iteration at which a run with step sizes st stops for eps, or None when
    a step size lies within 5% of eps (fp32 and fp64 could then disagree)."""
    if np.any(np.abs(np.log(st / eps)) < np.log(1.05)):
        return None
    return int(np.argmax(st <= eps)) + 1 if np.any(st <= eps) else iters


def test_graph_replay_follows_new_weights_with_early_stop():
    """A training loop's use of a captured step: the weights and the starting
    centroids change in place between replays (two sets in turn, the second
    the first halved, so it converges at another pace) and eps > 0, so the
    matrices stop at iterations that differ from one replay to the next.  Every
    replay must equal the eager step on the same inputs: the counts, windows,
    convergence state and partial blocks that the previous replay left in the
    workspaces must not leak into the next."""
    sizes, iters = [65536, 100_003, 70_001], 12
    k1 = [inputs.fp16_weights(n, 360 + i, outliers=(i == 1)) for i, n in enumerate(sizes)]
    sets = [k1, [(inputs.values(k) * 0.5).astype(np.float16).view(np.uint16) for k in k1]]
    c0s = [[inputs.quantile_init(k, 8) for k in keys] for keys in sets]
    steps = [[_step_sizes(k, c, iters) for k, c in zip(keys, cs)] for keys, cs in zip(sets, c0s)]
    eps, stops = None, None
    for cand in np.geomspace(1e-4, 1e-2, 200):
        t = [[_stop_iteration(st, float(cand), iters) for st in row] for row in steps]
        if any(x is None for row in t for x in row):
            continue
        if any(a != b for a, b in zip(t[0], t[1])):
            eps, stops = float(cand), t
            break
    assert eps is not None, "no eps gives different stopping points for the two sets"
    say("graph eps: eps", eps, "stops", stops)
    kd = [torch.empty(n, dtype=torch.int16, device=DEV) for n in sizes]
    host = [[torch.from_numpy(k.view(np.int16)) for k in keys] for keys in sets]
    host_c = [[torch.from_numpy(c) for c in cs] for cs in c0s]
    ci = [torch.empty(8, device=DEV) for _ in sizes]
    g = [torch.from_numpy(inputs.upstream_grad(n, 380 + i)).to(DEV) for i, n in enumerate(sizes)]
    plans = [edkm.Plan(n, 3, iters) for n in sizes]
    co = [torch.empty(8, device=DEV) for _ in sizes]
    wt = [torch.empty(n, device=DEV) for n in sizes]
    it = [torch.zeros(1, dtype=torch.int32, device=DEV) for _ in sizes]
    gw = [torch.empty(n, device=DEV) for n in sizes]
    gc = [torch.empty(8, device=DEV) for _ in sizes]

    def load(j):
        for d, h in zip(kd + ci, host[j] + host_c[j]):
            d.copy_(h)

    def step():
        edkm.init_unique_batch(plans, kd)
        edkm.forward_batch(plans, kd, TAU, eps, ci, co, wt, False, it)
        edkm.backward_batch(plans, kd, g, gw, gc)

    def poison():
        for t in co + wt + gw + gc:
            t.fill_(float("nan"))
        for t in it:
            t.fill_(-1)

    def outputs():
        return [dict(c_out=a.cpu().numpy(), wt=b.cpu().numpy(), it=c.cpu().numpy(),
                     gw=d.cpu().numpy(), gc=e.cpu().numpy())
                for a, b, c, d, e in zip(co, wt, it, gw, gc)]

    refs = []
    for j in range(2):
        say("graph eps: eager reference", j)
        load(j)
        poison()
        step()
        torch.cuda.synchronize()
        refs.append(outputs())
        assert [int(r["it"][0]) for r in refs[j]] == stops[j], j
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    say("graph eps: capture")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(4):
        j = rep % 2                      # the capture ran on set 1: start on set 0
        load(j)
        poison()
        torch.cuda.synchronize()
        say("graph eps: replay", rep, "set", j)
        graph.replay()
        torch.cuda.synchronize()
        same(outputs(), refs[j], "replay %d set %d" % (rep, j))


def test_graph_capture_of_the_export_calls():
    """init_unique, the distinct-pattern list with the inverse index, and the
    packed palettization indices, captured in one graph: every replay (with
    the outputs poisoned and other eager work in between) matches the eager
    results exactly (integer outputs)."""
    x = Batch([65536, 300_007], 340)
    other = Batch([50_000], 350)
    uo = [torch.empty(edkm.NKEYS, dtype=torch.int16, device=DEV) for _ in x.plans]
    io = [torch.empty(p.n, dtype=torch.int16, device=DEV) for p in x.plans]
    po = [torch.empty((p.n * p.bits + 7) // 8, dtype=torch.uint8, device=DEV) for p in x.plans]

    def poison():
        for t in uo + io:
            t.fill_(0x5A5A)
        for t in po:
            t.fill_(0xAB)

    def step():
        edkm.init_unique_batch(x.plans, x.keys)
        edkm.unique_inverse_batch(x.plans, x.keys, uo, io)
        edkm.palettize_batch(x.plans, x.keys, x.c0, po)

    def outs():
        return [t.cpu().numpy().copy() for t in uo + io + po]

    say("graph export: eager reference")
    poison()
    step()
    torch.cuda.synchronize()
    ref = outs()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    say("graph export: capture")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        other.step()
        poison()
        torch.cuda.synchronize()
        say("graph export: replay", rep)
        graph.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(outs(), ref)):
            assert np.array_equal(a, b), "replay %d output %d" % (rep, i)
