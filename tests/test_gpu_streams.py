"""Streams and graphs: distinct plans run concurrently on distinct streams, and
a whole batched step (init_unique + forward + backward) captured in a HIP graph
replays to the eager results, as do the export calls (distinct-pattern list,
inverse index, palettization).

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
