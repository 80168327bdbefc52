"""Seeded random batch compositions (1-28 matrices of 1 to 2.5M weights, 1-4
bits, fp16 and bf16): batched calls against one call per matrix, and the table
oracle on the small matrices.  The forward and the counts are bitwise equal
either way.  The backward is within 1e-4: a matrix's N-pass workgroups differ
between a batch and a single call, so its keyed-sum partial rows, and with
them the last bits of G, differ too (Sec. 2.2: the uniquified backward need
only match autograd to rounding).  A dL/dC^(0) that cancels to almost zero
(rms below 1e-6, e.g. a matrix of one weight) has no relative error to test
and is skipped in the oracle comparison."""
import random
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import table                                          # noqa: E402
from paper_2309_00964_amd import edkm, inputs                     # noqa: E402
from paper_2309_00964_amd.runner import run                       # noqa: E402
from parity_util import TOL_BWD, TOL_FWD, assert_close            # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def cases(seed, count):
    rng = random.Random(seed)
    for case in range(count):
        cnt = rng.choice([1, 2, 3, 5, 7, 12, 28])
        bits = rng.choice([1, 2, 3, 4])
        fmt = rng.choice(["fp16", "bf16"])
        sizes = [rng.choice([1, 7, 1000, 65536, 300_007, 1 << 20, 2_500_001]) for _ in range(cnt)]
        yield case, bits, fmt, sizes


@pytest.mark.parametrize("case,bits,fmt,sizes", list(cases(7, 8)))
def test_random_batch_matches_single_calls_and_oracle(case, bits, fmt, sizes):
    say("batch sweep", case, "bits", bits, fmt, "sizes", sizes)
    k = 1 << bits
    keys_h = [inputs.weights(n, 9000 + 17 * case + i, False, fmt) for i, n in enumerate(sizes)]
    c0_h = [inputs.quantile_init(x, k, fmt) for x in keys_h]
    g_h = [inputs.upstream_grad(n, 500 + case * 31 + i) for i, n in enumerate(sizes)]
    keys = [torch.from_numpy(x.view(np.int16)).to(DEV) for x in keys_h]
    c0 = [torch.from_numpy(x).to(DEV) for x in c0_h]
    gs = [torch.from_numpy(x).to(DEV) for x in g_h]
    plans = [edkm.Plan(n, bits, inputs.ITERS, device=DEV, key_format=fmt) for n in sizes]
    co = [torch.empty(k, device=DEV) for _ in sizes]
    wt = [torch.empty(n, device=DEV) for n in sizes]
    it = [torch.zeros(1, dtype=torch.int32, device=DEV) for _ in sizes]
    gw = [torch.empty(n, device=DEV) for n in sizes]
    gc = [torch.empty(k, device=DEV) for _ in sizes]
    cnts = [torch.empty(edkm.NKEYS, dtype=torch.int32, device=DEV) for _ in sizes]
    edkm.init_unique_batch(plans, keys, cnts)
    edkm.forward_batch(plans, keys, inputs.TAU, 0.0, c0, co, wt, False, it)
    edkm.backward_batch(plans, keys, gs, gw, gc)
    torch.cuda.synchronize()
    for i, n in enumerate(sizes):
        s = run(keys[i], c0[i], bits, inputs.TAU, inputs.ITERS, grad=gs[i], want_counts=True, key_format=fmt)
        torch.cuda.synchronize()
        what = "case %d matrix %d (n=%d)" % (case, i, n)
        assert np.array_equal(cnts[i].cpu().numpy(), s["counts"].cpu().numpy()), what
        assert np.array_equal(co[i].cpu().numpy(), s["c_out"].cpu().numpy()), what
        assert np.array_equal(wt[i].cpu().numpy(), s["w_tilde"].cpu().numpy()), what
        assert_close(gw[i].cpu().numpy(), s["grad_w"].cpu().numpy(), 1e-4, what + " grad_w")
        assert_close(gc[i].cpu().numpy(), s["grad_c"].cpu().numpy(), 1e-4, what + " grad_c")
        if n <= 300_007:
            f = table.forward(keys_h[i], c0_h[i].astype(np.float64), inputs.TAU, inputs.ITERS, fmt=fmt)
            gw_o, gc_o, _ = table.backward(keys_h[i], f, g_h[i].astype(np.float64))
            assert_close(co[i].cpu().numpy(), f["c_out"], TOL_FWD, what + " c_out")
            assert_close(wt[i].cpu().numpy(), f["w_tilde"], TOL_FWD, what + " w_tilde")
            assert_close(gw[i].cpu().numpy(), gw_o, TOL_BWD, what + " grad_w")
            if np.sqrt(np.mean(gc_o ** 2)) >= 1e-6:
                assert_close(gc[i].cpu().numpy(), gc_o, TOL_BWD, what + " grad_c")
