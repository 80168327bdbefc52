"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Counts and occupied-pattern numbers are compared bit-exactly; floating point
uses the rules in parity_util (1e-4 forward, 1e-3 gradients).  Sizes run from
single weights through several workgroup slices with ragged tails up to the
full workload shapes (4096x4096, 11008x4096 with outliers at 3 and 4 bits, and
the seven matrices of a LLaMA-7B decoder layer in one batch, which is the call
the benchmark times).  The dense oracle checks everything up to a few hundred
thousand weights; the full shapes use the table-form oracle, itself pinned to
the dense one in test_oracle_pins.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import dense, table                                  # noqa: E402
from paper_2309_00964_amd import edkm, inputs                     # noqa: E402
from paper_2309_00964_amd.runner import run                       # noqa: E402
from parity_util import (EMPTY_THEN_LIVE, TOL_BWD, TOL_FWD,  # noqa: E402
                         assert_bf16_within_ulp, assert_close, assert_close_conditioned,
                         assert_fp16_within_ulp, empty_then_live_inputs, iterate_sensitivity,
                         _bf16_bits, _bf16_values)

pytestmark = pytest.mark.gpu
DEV = "cuda"
TAU, ITERS = inputs.TAU, inputs.ITERS


def say(*a):
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def dkeys(keys):
    return torch.from_numpy(np.ascontiguousarray(keys).view(np.int16)).to(DEV)


def gpu(keys, c0, bits, g=None, tau=TAU, iters=ITERS, eps=0.0, **kw):
    out = run(dkeys(keys), torch.from_numpy(np.asarray(c0, np.float32)), bits, tau, iters, eps,
              grad=None if g is None else torch.from_numpy(np.asarray(g, np.float32)), **kw)
    torch.cuda.synchronize()
    res = {}
    for k, v in out.items():
        if isinstance(v, torch.Tensor):
            if v.dtype == torch.bfloat16:      # numpy has no bfloat16: hand back the patterns
                v = v.view(torch.int16)
            res[k] = v.cpu().numpy()
    return res


def oracle(keys, c0, g=None, tau=TAU, iters=ITERS, eps=0.0, form="dense", fmt="fp16"):
    mod = dense if form == "dense" else table
    f = mod.forward(keys, np.asarray(c0, np.float64), tau, iters, eps=eps, fmt=fmt)
    if g is not None:
        r = mod.backward(keys, f, np.asarray(g, np.float64))
        f["gw"], f["gc"] = r[0], r[1]
    return f


def check(res, ref, g=True, what=""):
    assert int(res["iters"][0]) == ref["T"], what
    assert_close(res["c_out"], ref["c_out"], TOL_FWD, what + " c_out")
    assert_close(res["w_tilde"], ref["w_tilde"], TOL_FWD, what + " w_tilde")
    if g:
        assert_close(res["grad_w"], ref["gw"], TOL_BWD, what + " grad_w")
        assert_close(res["grad_c"], ref["gc"], TOL_BWD, what + " grad_c")


def special_keys(n, seed):
    """Gaussian weights mixed with signed zeros, subnormals, |w| >= 16 and tiny values."""
    keys = inputs.fp16_weights(n, seed)
    rng = np.random.default_rng(seed)
    extra = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x03FF, 0x83FF, 0x0400, 0x4C00, 0xCC00,
                      0x7BFF, 0xFBFF, 0x5A00, 0xDA00], dtype=np.uint16)
    pos = rng.choice(n, size=min(n, 4 * extra.size), replace=False)
    keys[pos] = np.resize(extra, pos.size)
    return keys


# ------------------------------------------------------------------ histogram

@pytest.mark.parametrize("n,seed,outl,special", [
    (65536, inputs.weight_seed(1, 0), False, False),
    (3 * 65536 + 37, 11, True, False),
    (100003, 12, False, True),
    (1, 13, False, False),
    (7, 14, False, True),
    (9, 15, False, False),
])
def test_counts_bit_exact(n, seed, outl, special):
    keys = special_keys(n, seed) if special else inputs.fp16_weights(n, seed, outliers=outl)
    c0 = inputs.quantile_init(keys, 8)
    say("counts", n, seed)
    res = gpu(keys, c0, 3, want_counts=True)
    ref = table.histogram(keys)
    assert np.array_equal(res["counts"].view(np.uint32), ref)
    assert int(res["num_unique"].view(np.uint32)[0]) == int(np.count_nonzero(ref))


def test_counts_single_pattern_overflow_path():
    """17M copies of one pattern: every workgroup's bin passes 2^16."""
    n = 17_000_000
    keys = np.full(n, 0x2000, dtype=np.uint16)
    c0 = inputs.quantile_init(keys, 8)
    say("single pattern", n)
    res = gpu(keys, c0, 3, g=np.ones(n, np.float32), want_counts=True)
    ref = table.histogram(keys)
    assert np.array_equal(res["counts"].view(np.uint32), ref)
    v = float(np.uint16(0x2000).view(np.float16))
    assert np.allclose(res["c_out"], v, rtol=1e-6)
    assert np.allclose(res["w_tilde"], v, rtol=1e-6)


@pytest.mark.parametrize("case", ["constant", "signed_zeros", "on_centroids"])
def test_degenerate_inputs_match_oracle(case):
    """Inputs where the method degenerates: one repeated value (every quantile
    centroid equals it, so rows are uniform and C never moves), a random mix of
    +0 and -0 (two keys, one value, every distance 0), and two values sitting
    exactly on their starting centroids (d|x|/dx at 0 taken as 0).  Counts are
    bit-exact and C, W~ and dL/dw are held to the usual tolerances.  dL/dC^(0)
    is zero or underflow-sized in fp64 here (the centroids settle onto isolated
    values, so C^(T) hardly depends on C^(0)); it is held to an absolute bound,
    1e-6 of sum |g|, the scale a centroid gradient could take."""
    n = 50_003
    rng = np.random.default_rng(490)
    if case == "constant":
        keys = np.full(n, np.float16(0.01).view(np.uint16), dtype=np.uint16)
        c0 = inputs.quantile_init(keys, 4)
    elif case == "signed_zeros":
        keys = np.where(rng.random(n) < 0.5, 0x0000, 0x8000).astype(np.uint16)
        c0 = inputs.quantile_init(keys, 4)
    else:
        a, b = np.float16(-0.02), np.float16(0.03)
        keys = np.where(rng.random(n) < 0.3, a.view(np.uint16), b.view(np.uint16)).astype(np.uint16)
        c0 = np.array([float(a), float(b), 0.0, 0.05], np.float32)
    g = inputs.upstream_grad(n, 491)
    say("degenerate", case)
    res = gpu(keys, c0, 2, g=g, want_counts=True)
    assert np.array_equal(res["counts"].view(np.uint32), table.histogram(keys))
    ref = oracle(keys, c0, g)
    check(res, ref, g=False, what=case)
    assert_close(res["grad_w"], ref["gw"], TOL_BWD, case + " grad_w")
    assert np.all(np.abs(res["grad_c"] - ref["gc"]) <= 1e-6 * float(np.abs(g).sum())), case


# ------------------------------------------------------------------ forward / backward

CASES = [
    # n, bits, outliers, seed
    (65536, 3, False, inputs.weight_seed(1, 0)),
    (65536, 1, False, 21),
    (65536, 2, False, 22),
    (65536, 4, False, 23),
    (2 * 65536 + 37, 3, True, 24),
    (300007, 4, True, 25),
    (1, 3, False, 26),
    (7, 2, False, 27),
    (1000, 3, False, 28),
]


@pytest.mark.parametrize("n,bits,outl,seed", CASES)
def test_unique_path_matches_oracle(n, bits, outl, seed):
    keys = inputs.fp16_weights(n, seed, outliers=outl)
    c0 = inputs.quantile_init(keys, 1 << bits)
    g = inputs.upstream_grad(n, seed + 500)
    say("unique", n, bits, outl, seed)
    res = gpu(keys, c0, bits, g=g)
    check(res, oracle(keys, c0, g), what="unique n=%d bits=%d" % (n, bits))


@pytest.mark.parametrize("n,bits,outl,seed", [c for c in CASES if c[0] <= 300007])
def test_dense_path_matches_oracle(n, bits, outl, seed):
    keys = inputs.fp16_weights(n, seed, outliers=outl)
    c0 = inputs.quantile_init(keys, 1 << bits)
    g = inputs.upstream_grad(n, seed + 500)
    say("dense", n, bits, outl, seed)
    res = gpu(keys, c0, bits, g=g, dense=True, want_attn=n <= 70000)
    ref = oracle(keys, c0, g)
    check(res, ref, what="dense n=%d bits=%d" % (n, bits))
    if "attn" in res:
        fa = dense.forward(keys, c0.astype(np.float64), TAU, ITERS, want_attn=True)["attn"]
        assert_close(res["attn"], fa, TOL_FWD, "attention map")
        assert np.allclose(res["attn"].sum(axis=1), 1.0, atol=1e-5)


def test_dense_and_unique_agree_on_gpu():
    keys = inputs.fp16_weights(200_000, 31, outliers=True)
    c0 = inputs.quantile_init(keys, 8)
    g = inputs.upstream_grad(keys.size, 32)
    say("dense vs unique")
    u = gpu(keys, c0, 3, g=g)
    d = gpu(keys, c0, 3, g=g, dense=True)
    assert_close(u["c_out"], d["c_out"], TOL_FWD, "c_out")
    assert_close(u["w_tilde"], d["w_tilde"], TOL_FWD, "w_tilde")
    assert_close(u["grad_w"], d["grad_w"], TOL_BWD, "grad_w")
    assert_close(u["grad_c"], d["grad_c"], TOL_BWD, "grad_c")


@pytest.mark.parametrize("dense_path", [False, True])
def test_fp16_output_within_one_ulp(dense_path):
    keys = inputs.fp16_weights(65536 + 5, 41)
    c0 = inputs.quantile_init(keys, 8)
    say("fp16 out", dense_path)
    res = gpu(keys, c0, 3, out_half=True, dense=dense_path)
    ref = oracle(keys, c0)
    assert_fp16_within_ulp(res["w_tilde"].view(np.uint16), ref["w_tilde"])


def test_special_values_and_wide_range():
    """Signed zeros, subnormals, |w| >= 16 up to 65504: exact decode, global
    fallbacks outside the LDS windows."""
    keys = special_keys(100003, 51)
    c0 = inputs.quantile_init(keys, 16)
    g = inputs.upstream_grad(keys.size, 52)
    say("special values")
    res = gpu(keys, c0, 4, g=g)
    check(res, oracle(keys, c0, g), what="special")


def test_wide_magnitude_span_exceeds_windows():
    """Occupied magnitudes spanning more than the LDS windows: the densest part
    is windowed, the rest is read through the global table.  With centroids out
    to 3.7e4 and tau = 2e-3, one fp32 ulp of an iterate shifts the softmax
    boundaries by up to ulp(C)/tau: patterns near a boundary have gradients
    that move by up to about 1e-3 of their size when the iterates are rounded
    (fp64 oracle, see iterate_sensitivity).  Elementwise, each output is
    compared within the tolerance plus that conditioning; rel-L2 and the counts
    are held to the usual bars."""
    rng = np.random.default_rng(61)
    n = 150_000
    logs = rng.uniform(-24, 15.9, n)
    vals = np.sign(rng.standard_normal(n)) * np.exp2(logs)
    keys = vals.astype(np.float16).view(np.uint16)
    keys[: n // 2] = inputs.fp16_weights(n // 2, 62)
    c0 = inputs.quantile_init(keys, 8)
    g = inputs.upstream_grad(n, 63)
    say("wide span")
    res = gpu(keys, c0, 3, g=g, want_counts=True)
    assert np.array_equal(res["counts"].view(np.uint32), table.histogram(keys))
    ref = oracle(keys, c0, g)
    dwt, dgw, dgc = iterate_sensitivity(keys, c0, g, TAU, ITERS)
    assert int(res["iters"][0]) == ref["T"]
    assert_close(res["c_out"], ref["c_out"], TOL_FWD, "wide span c_out")
    assert_close_conditioned(res["w_tilde"], ref["w_tilde"], dwt, TOL_FWD, "wide span w_tilde")
    assert_close_conditioned(res["grad_w"], ref["gw"], dgw, TOL_BWD, "wide span grad_w")
    assert_close_conditioned(res["grad_c"], ref["gc"], dgc, TOL_BWD, "wide span grad_c")


def test_nonfinite_weights():
    keys = inputs.fp16_weights(50_000, 71)
    bad = keys.copy()
    bad[[5, 777, 40_000]] = [0x7C00, 0xFC00, 0x7E00]
    c0 = inputs.quantile_init(keys, 8)
    say("non-finite checked")
    with pytest.raises(edkm.EdkmError) as e:
        gpu(bad, c0, 3, check_finite=True)
    assert e.value.status == edkm.ERR_NONFINITE
    say("non-finite unchecked")
    g = inputs.upstream_grad(bad.size, 72)
    res = gpu(bad, c0, 3, g=g)
    finite = np.ones(bad.size, bool)
    finite[[5, 777, 40_000]] = False
    ref = oracle(bad[finite], c0, g[finite])
    assert np.all(np.isnan(res["w_tilde"][~finite]))
    assert np.all(np.isnan(res["grad_w"][~finite]))
    assert_close(res["c_out"], ref["c_out"], TOL_FWD, "c_out")
    assert_close(res["w_tilde"][finite], ref["w_tilde"], TOL_FWD, "w_tilde")
    assert_close(res["grad_w"][finite], ref["gw"], TOL_BWD, "grad_w")
    assert_close(res["grad_c"], ref["gc"], TOL_BWD, "grad_c")


def test_batch_nonfinite_check_is_per_matrix():
    """init_unique_batch with check_finite = 1 on [finite, Inf/NaN, finite]:
    the call reports EDKM_ERR_NONFINITE, as the single form would for the
    middle matrix, and, as the single form on each would, leaves only that
    plan uncounted: the other two go on through forward and backward and
    equal fresh single calls, while the middle plan's forward is a state
    error."""
    sizes = [50_000, 60_001, 70_003]
    ks = [inputs.fp16_weights(n, 73 + i) for i, n in enumerate(sizes)]
    ks[1][[3, 999, 60_000]] = [0x7C00, 0xFC00, 0x7E00]
    c0s = [inputs.quantile_init(k, 8) for k in ks]
    gs = [inputs.upstream_grad(n, 76 + i) for i, n in enumerate(sizes)]
    plans = [edkm.Plan(n, 3, ITERS) for n in sizes]
    kd = [dkeys(k) for k in ks]
    say("batch non-finite check")
    with pytest.raises(edkm.EdkmError) as e:
        edkm.init_unique_batch(plans, kd, check_finite=True)
    assert e.value.status == edkm.ERR_NONFINITE
    co = torch.empty(8, device=DEV)
    wt = torch.empty(sizes[1], device=DEV)
    with pytest.raises(edkm.EdkmError) as e:
        edkm.forward(plans[1], kd[1], TAU, 0.0, torch.from_numpy(c0s[1]).to(DEV), co, wt)
    assert e.value.status == edkm.ERR_STATE
    good = [0, 2]
    ci = [torch.from_numpy(c0s[i]).to(DEV) for i in good]
    co = [torch.empty(8, device=DEV) for _ in good]
    wt = [torch.empty(sizes[i], device=DEV) for i in good]
    it = [torch.zeros(1, dtype=torch.int32, device=DEV) for _ in good]
    gd = [torch.from_numpy(gs[i]).to(DEV) for i in good]
    gw = [torch.empty(sizes[i], device=DEV) for i in good]
    gc = [torch.empty(8, device=DEV) for _ in good]
    pg, kg = [plans[i] for i in good], [kd[i] for i in good]
    edkm.forward_batch(pg, kg, TAU, 0.0, ci, co, wt, False, it)
    edkm.backward_batch(pg, kg, gd, gw, gc)
    torch.cuda.synchronize()
    for q, i in enumerate(good):
        ref = gpu(ks[i], c0s[i], 3, g=gs[i])
        assert int(it[q].item()) == int(ref["iters"][0]), i
        assert np.array_equal(co[q].cpu().numpy(), ref["c_out"]), i
        assert np.array_equal(wt[q].cpu().numpy(), ref["w_tilde"]), i
        # a batch splits the N-sized passes differently from a single call,
        # so the keyed sums' last bits differ (as in the batch-versus-single tests)
        assert_close(gw[q].cpu().numpy(), ref["grad_w"], 1e-4, "grad_w %d" % i)
        assert_close(gc[q].cpu().numpy(), ref["grad_c"], 1e-4, "grad_c %d" % i)


def test_keyed_sum_wraps_fixed_point_range():
    """Five patterns repeated over a million weights; dL/dW~ is a small bulk
    (N(0, 1e-3^2)) with 5% of entries +-0.75.  The fixed-point scale follows
    the bulk, so each +-0.75 is about 2^29.6 quanta and the per-workgroup sum
    of every pattern wanders past the 32-bit range in both directions: the wrap
    (carry) path of the keyed reduction is taken thousands of times.  (Random
    signs keep dL/dC^(0) well conditioned; with dL/dW~ all positive it is a
    1e-6 residual of the sums, below what fp32 resolves.)"""
    vals = np.array([-0.011, -0.004, 0.0005, 0.006, 0.013], dtype=np.float16)
    n = 1_000_003
    rng = np.random.default_rng(81)
    keys = vals.view(np.uint16)[rng.integers(0, vals.size, n)]
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    big = rng.random(n) < 0.05
    g[big] = np.where(rng.random(int(big.sum())) < 0.5, -0.75, 0.75).astype(np.float32)
    c0 = np.array([-0.01, -0.002, 0.004, 0.012], np.float32)
    say("keyed sum: fixed-point wraps")
    plan = edkm.Plan(n, 2, ITERS)     # five patterns would choose the 64-bit mode: force 32-bit
    edkm.plan_set_keyed_mode(plan, edkm.KEYED_I32)
    res = gpu(keys, c0, 2, g=g, plan=plan)
    check(res, oracle(keys, c0, g, form="table"), what="fixed-point wraps")


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
@pytest.mark.parametrize("mode", ["auto", "i32", "u64"])
def test_keyed_sum_modes_match_oracle(fmt, mode):
    """Both keyed-sum accumulator modes, forced or chosen from the data (fp16
    patterns choose 32-bit, bf16 ones 64-bit), give the oracle's gradients."""
    n = 300_007
    keys = inputs.weights(n, 86, True, fmt)
    c0 = inputs.quantile_init(keys, 8, fmt)
    g = inputs.upstream_grad(n, 87)
    plan = edkm.Plan(n, 3, ITERS, key_format=fmt)
    edkm.plan_set_keyed_mode(plan, {"auto": edkm.KEYED_AUTO, "i32": edkm.KEYED_I32,
                                    "u64": edkm.KEYED_U64}[mode])
    say("keyed modes", fmt, mode)
    res = gpu(keys, c0, 3, g=g, plan=plan, key_format=fmt)
    check(res, oracle(keys, c0, g, fmt=fmt), what="keyed %s %s" % (fmt, mode))


def test_keyed_sum_heavy_tailed_gradient():
    """dL/dW~ with rare huge values (1e6 times the bulk), exact zeros and
    subnormals: the fixed-point scale must follow the bulk, the huge values
    take the exact fp32 path."""
    n = 300_007
    keys = inputs.fp16_weights(n, 82, outliers=True)
    c0 = inputs.quantile_init(keys, 8)
    rng = np.random.default_rng(83)
    g = inputs.upstream_grad(n, 84)
    g[rng.random(n) < 5e-4] *= np.float32(1e6)
    g[rng.random(n) < 1e-2] = 0.0
    g[rng.random(n) < 1e-3] = np.float32(1e-40)
    say("keyed sum: heavy-tailed gradient")
    res = gpu(keys, c0, 3, g=g)
    check(res, oracle(keys, c0, g), what="heavy-tailed g")


def test_unit_upstream_gradient_identity():
    """With dL/dW~ = 1 the loss is sum_i w_i whatever the centroids (sum_i W~_i =
    sum_j S_j C_j = sum_j P_j), so dL/dw_i = 1 and dL/dC^(0) = 0."""
    keys = inputs.fp16_weights(200_003, 75, outliers=True)
    c0 = inputs.quantile_init(keys, 8)
    say("unit gradient")
    res = gpu(keys, c0, 3, g=np.ones(keys.size, np.float32))
    assert np.max(np.abs(res["grad_w"] - 1.0)) <= 1e-3
    rnd = gpu(keys, c0, 3, g=inputs.upstream_grad(keys.size, 76))
    assert np.max(np.abs(res["grad_c"])) <= 1e-3 * np.max(np.abs(rnd["grad_c"]))


def test_early_stop_matches_oracle():
    keys = inputs.fp16_weights(65536, 81)
    c0 = inputs.quantile_init(keys, 8)
    g = inputs.upstream_grad(keys.size, 82)
    full = dense.forward(keys, c0.astype(np.float64), TAU, 12)
    steps = np.max(np.abs(np.diff(full["c_hist"], axis=0)), axis=1)
    s = np.sort(steps)
    # an eps between two step sizes that differ by >= 10%, far from fp32 rounding
    i = next(i for i in range(len(s) // 3, len(s) - 1) if s[i + 1] > 1.1 * s[i])
    eps = float(np.sqrt(s[i] * s[i + 1]))
    say("early stop", eps)
    for dense_path in (False, True):
        res = gpu(keys, c0, 3, g=g, iters=12, eps=eps, dense=dense_path)
        check(res, oracle(keys, c0, g, iters=12, eps=eps), what="eps dense=%s" % dense_path)


def test_batch_early_stop_at_different_iterations():
    """One eps for a batch whose matrices converge at different speeds: each
    stops at its own iteration, the backward unrolls its own T, and every matrix
    equals its single call and the oracle.  eps is chosen so that no matrix has
    a step size within 5% of it (no fp32-versus-fp64 ambiguity)."""
    spec = [(65536, 90, False), (100_003, 91, True), (70_001, 92, False)]
    ks = [inputs.fp16_weights(n, seed, outliers=o) for n, seed, o in spec]
    c0s = [inputs.quantile_init(k, 8) for k in ks]
    gs = [inputs.upstream_grad(n, seed + 10) for n, seed, _ in spec]
    steps = []
    for k, c0 in zip(ks, c0s):
        h = dense.forward(k, c0.astype(np.float64), TAU, 12)["c_hist"]
        steps.append(np.max(np.abs(np.diff(h, axis=0)), axis=1))
    eps, ts = None, None
    for cand in np.geomspace(1e-4, 1e-2, 400):
        if any(np.any(np.abs(np.log(st / cand)) < np.log(1.05)) for st in steps):
            continue
        t = [int(np.argmax(st <= cand)) + 1 if np.any(st <= cand) else 12 for st in steps]
        if len(set(t)) > 1:
            eps, ts = float(cand), t
            break
    assert eps is not None, "no eps separates the matrices' stopping points"
    say("batch early stop", eps, ts)
    plans = [edkm.Plan(n, 3, 12) for n, _, _ in spec]
    kd = [dkeys(k) for k in ks]
    ci = [torch.from_numpy(c).to(DEV) for c in c0s]
    co = [torch.empty(8, device=DEV) for _ in spec]
    wt = [torch.empty(n, device=DEV) for n, _, _ in spec]
    it = [torch.zeros(1, dtype=torch.int32, device=DEV) for _ in spec]
    gd = [torch.from_numpy(g).to(DEV) for g in gs]
    gw = [torch.empty(n, device=DEV) for n, _, _ in spec]
    gc = [torch.empty(8, device=DEV) for _ in spec]
    edkm.init_unique_batch(plans, kd)
    edkm.forward_batch(plans, kd, TAU, eps, ci, co, wt, False, it)
    edkm.backward_batch(plans, kd, gd, gw, gc)
    torch.cuda.synchronize()
    for i in range(len(spec)):
        single = gpu(ks[i], c0s[i], 3, g=gs[i], iters=12, eps=eps)
        assert int(it[i].item()) == int(single["iters"][0]), i
        assert np.array_equal(co[i].cpu().numpy(), single["c_out"]), i
        res = dict(iters=it[i].cpu().numpy(), c_out=co[i].cpu().numpy(), w_tilde=wt[i].cpu().numpy(),
                   grad_w=gw[i].cpu().numpy(), grad_c=gc[i].cpu().numpy())
        check(res, oracle(ks[i], c0s[i], gs[i], iters=12, eps=eps), what="batch eps %d" % i)
    assert len({int(t.item()) for t in it}) > 1


def test_empty_cluster_keeps_centroid():
    keys = inputs.fp16_weights(30_000, 91)
    c0 = np.append(inputs.quantile_init(keys, 7), np.float32(2.0))   # fp64 underflows too
    g = inputs.upstream_grad(keys.size, 92)
    say("empty cluster")
    for dense_path in (False, True):
        res = gpu(keys, c0, 3, g=g, dense=dense_path)
        ref = oracle(keys, c0, g)
        assert res["c_out"][7] == np.float32(2.0)
        check(res, ref, what="empty cluster dense=%s" % dense_path)


@pytest.mark.parametrize("dense_path", [False, True])
def test_empty_then_live_cluster(dense_path):
    """A centroid that is empty at t = 1 (its attention underflows for every
    weight, in fp32 as in fp64) and occupied at t = 2: it keeps its value, and
    dL/dC^(0) for it is the whole gradient that reaches C^(1) through the kept
    value (about -325 here, where dropping the identity gradient would give 0).
    Both the uniquified and the dense path against the oracle."""
    keys, c0, g = empty_then_live_inputs()
    e = EMPTY_THEN_LIVE
    say("empty then live", "dense" if dense_path else "unique")
    res = gpu(keys, c0, 1, g=g, tau=e["tau"], iters=e["T"], dense=dense_path)
    ref = oracle(keys, c0, g, tau=e["tau"], iters=e["T"])
    assert ref["s_hist"][1, 1] == 0.0 and ref["s_hist"][2, 1] > 1.0 and abs(ref["gc"][1]) > 100.0
    check(res, ref, what="empty then live")


@pytest.mark.parametrize("bits,eps", [(3, 0.0), (2, 1.0)])
def test_backward_repeated_after_one_forward(bits, eps):
    """Backward twice after one forward, with different upstream gradients:
    each matches the oracle (the backward's first table partials are added
    into a block that the forward clears and each backward clears after use).
    eps = 1 stops after one iteration, where the gradient gather itself reads
    that block."""
    n = 300_007
    keys = inputs.fp16_weights(n, 131)
    k = 1 << bits
    c0 = inputs.quantile_init(keys, k)
    say("repeated backward", bits, eps)
    plan = edkm.Plan(n, bits, ITERS)
    kd = dkeys(keys)
    c_in = torch.from_numpy(c0).to(DEV)
    c_out = torch.empty(k, device=DEV)
    wt = torch.empty(n, device=DEV)
    it = torch.zeros(1, dtype=torch.int32, device=DEV)
    edkm.init_unique(plan, kd)
    edkm.forward(plan, kd, TAU, eps, c_in, c_out, wt, False, it)
    ref_f = oracle(keys, c0, eps=eps)
    assert int(it.item()) == ref_f["T"] and (eps == 0.0 or ref_f["T"] == 1)
    for seed in (132, 133):
        g = inputs.upstream_grad(n, seed)
        gw = torch.empty(n, device=DEV)
        gc = torch.empty(k, device=DEV)
        edkm.backward(plan, kd, torch.from_numpy(g).to(DEV), gw, gc)
        torch.cuda.synchronize()
        ref = oracle(keys, c0, g, eps=eps)
        assert_close(gw.cpu().numpy(), ref["gw"], TOL_BWD, "grad_w seed %d" % seed)
        assert_close(gc.cpu().numpy(), ref["gc"], TOL_BWD, "grad_c seed %d" % seed)


def test_forward_repeatable_and_exact_scaling():
    """Forward results are bitwise repeatable.  Scaling w, C^(0) and tau by 2 scales
    C and W~ by 2: bitwise on the dense path (same reduction order), and to
    rounding on the table path, where doubling moves every pattern to another
    table row (key + 0x400) and so reorders the fixed-order sums."""
    keys = inputs.fp16_weights(65536 * 2 + 3, 101)
    c0 = inputs.quantile_init(keys, 8)
    k2 = (keys.view(np.float16) * np.float16(2)).view(np.uint16)
    assert np.array_equal(k2.view(np.float16).astype(np.float64), 2 * keys.view(np.float16).astype(np.float64))
    say("repeat/scale")
    for dense_path in (False, True):
        a = gpu(keys, c0, 3, dense=dense_path)
        b = gpu(keys, c0, 3, dense=dense_path)
        assert np.array_equal(a["c_out"], b["c_out"]) and np.array_equal(a["w_tilde"], b["w_tilde"])
        s = gpu(k2, 2 * c0, 3, tau=2 * TAU, dense=dense_path)
        if dense_path:
            assert np.array_equal(s["c_out"], 2 * a["c_out"])
            assert np.array_equal(s["w_tilde"], 2 * a["w_tilde"])
        else:
            assert_close(s["c_out"], 2 * a["c_out"].astype(np.float64), 1e-6, "scaled c_out")
            assert_close(s["w_tilde"], 2 * a["w_tilde"].astype(np.float64), 1e-6, "scaled w_tilde")


def test_negation_symmetry_on_gpu():
    """w, C^(0) -> -w, -C^(0): C and W~ negate, dL/dw and dL/dC^(0) are
    unchanged (the map depends on |w - c| only).  Bitwise for the dense
    forward, whose sums keep their order; to rounding elsewhere: on the table
    path negation moves every pattern to the other sign half (key ^ 0x8000),
    which reorders the fixed-order sums, and the keyed gradient sum uses
    atomics."""
    n, bits = 65536 * 3 + 5, 3
    keys = inputs.fp16_weights(n, 102)
    c0 = inputs.quantile_init(keys, 1 << bits)
    g = inputs.upstream_grad(n, 103)
    kn = keys ^ np.uint16(0x8000)
    say("negation symmetry")
    for dense_path in (True, False):
        a = gpu(keys, c0, bits, g=g, dense=dense_path)
        b = gpu(kn, -c0, bits, g=g, dense=dense_path)
        what = "dense" if dense_path else "table"
        if dense_path:
            assert np.array_equal(b["c_out"], -a["c_out"]) and np.array_equal(b["w_tilde"], -a["w_tilde"])
        else:
            assert_close(b["c_out"], -a["c_out"].astype(np.float64), 1e-6, what + " c_out")
            assert_close(b["w_tilde"], -a["w_tilde"].astype(np.float64), 1e-6, what + " w_tilde")
        assert_close(b["grad_w"], a["grad_w"].astype(np.float64), 1e-5, what + " grad_w")
        assert_close(b["grad_c"], a["grad_c"].astype(np.float64), 1e-4, what + " grad_c")


def test_misaligned_buffers_take_the_scalar_path():
    n = 65536 + 11
    keys = inputs.fp16_weights(n + 1, 111)
    c0 = inputs.quantile_init(keys[1:], 8)
    g = inputs.upstream_grad(n + 1, 112)
    say("misaligned")
    kd = dkeys(keys)[1:]
    gd = torch.from_numpy(g).to(DEV)[1:]
    plan = edkm.Plan(n, 3, ITERS)
    c_in = torch.from_numpy(c0).to(DEV)
    c_out = torch.empty(8, device=DEV)
    wt = torch.empty(n + 1, device=DEV)[1:]
    gw = torch.empty(n + 1, device=DEV)[1:]
    gc = torch.empty(8, device=DEV)
    it = torch.zeros(1, dtype=torch.int32, device=DEV)
    edkm.init_unique(plan, kd)
    edkm.forward(plan, kd, TAU, 0.0, c_in, c_out, wt, False, it)
    edkm.backward(plan, kd, gd, gw, gc)
    torch.cuda.synchronize()
    res = dict(iters=it.cpu().numpy(), c_out=c_out.cpu().numpy(), w_tilde=wt.cpu().numpy(),
               grad_w=gw.cpu().numpy(), grad_c=gc.cpu().numpy())
    check(res, oracle(keys[1:], c0, g[1:]), what="misaligned")


def test_batch_equals_single_calls():
    sizes = [65536, 100003, 7, 300000]
    bits = 3
    ks = [inputs.fp16_weights(n, 120 + i, outliers=(i == 3)) for i, n in enumerate(sizes)]
    c0s = [inputs.quantile_init(k, 8) for k in ks]
    gs = [inputs.upstream_grad(n, 130 + i) for i, n in enumerate(sizes)]
    say("batch")
    plans = [edkm.Plan(n, bits, ITERS) for n in sizes]
    kd = [dkeys(k) for k in ks]
    ci = [torch.from_numpy(c).to(DEV) for c in c0s]
    co = [torch.empty(8, device=DEV) for _ in sizes]
    wt = [torch.empty(n, device=DEV) for n in sizes]
    it = [torch.zeros(1, dtype=torch.int32, device=DEV) for _ in sizes]
    gd = [torch.from_numpy(g).to(DEV) for g in gs]
    gw = [torch.empty(n, device=DEV) for n in sizes]
    gc = [torch.empty(8, device=DEV) for _ in sizes]
    edkm.init_unique_batch(plans, kd)
    edkm.forward_batch(plans, kd, TAU, 0.0, ci, co, wt, False, it)
    edkm.backward_batch(plans, kd, gd, gw, gc)
    torch.cuda.synchronize()
    for i, n in enumerate(sizes):
        single = gpu(ks[i], c0s[i], bits, g=gs[i])
        assert np.array_equal(co[i].cpu().numpy(), single["c_out"])
        assert np.array_equal(wt[i].cpu().numpy(), single["w_tilde"])
        assert_close(gw[i].cpu().numpy(), single["grad_w"], 1e-5, "batch grad_w")
        res = dict(iters=it[i].cpu().numpy(), c_out=co[i].cpu().numpy(), w_tilde=wt[i].cpu().numpy(),
                   grad_w=gw[i].cpu().numpy(), grad_c=gc[i].cpu().numpy())
        check(res, oracle(ks[i], c0s[i], gs[i]), what="batch %d" % i)


def test_batch_spanning_launch_groups():
    """31 matrices: one full launch group of LAUNCH_GROUP matrices and one of 3
    (cut by size).  Every matrix equals its single-matrix call (forward
    bitwise) and the oracle."""
    assert edkm.LAUNCH_GROUP == 28
    sizes = [4096 + 1531 * i for i in range(31)]
    ks = [inputs.fp16_weights(n, 400 + i, outliers=(i % 5 == 2)) for i, n in enumerate(sizes)]
    c0s = [inputs.quantile_init(k, 8) for k in ks]
    gs = [inputs.upstream_grad(n, 440 + i) for i, n in enumerate(sizes)]
    say("batch over two launch groups")
    plans = [edkm.Plan(n, 3, ITERS) for n in sizes]
    kd = [dkeys(k) for k in ks]
    ci = [torch.from_numpy(c).to(DEV) for c in c0s]
    co = [torch.empty(8, device=DEV) for _ in sizes]
    wt = [torch.empty(n, device=DEV) for n in sizes]
    it = [torch.zeros(1, dtype=torch.int32, device=DEV) for _ in sizes]
    gd = [torch.from_numpy(g).to(DEV) for g in gs]
    gw = [torch.empty(n, device=DEV) for n in sizes]
    gc = [torch.empty(8, device=DEV) for _ in sizes]
    edkm.init_unique_batch(plans, kd)
    edkm.forward_batch(plans, kd, TAU, 0.0, ci, co, wt, False, it)
    edkm.backward_batch(plans, kd, gd, gw, gc)
    torch.cuda.synchronize()
    for i in range(len(sizes)):
        single = gpu(ks[i], c0s[i], 3, g=gs[i])
        assert np.array_equal(co[i].cpu().numpy(), single["c_out"]), i
        assert np.array_equal(wt[i].cpu().numpy(), single["w_tilde"]), i
        res = dict(iters=it[i].cpu().numpy(), c_out=co[i].cpu().numpy(), w_tilde=wt[i].cpu().numpy(),
                   grad_w=gw[i].cpu().numpy(), grad_c=gc[i].cpu().numpy())
        check(res, oracle(ks[i], c0s[i], gs[i]), what="group batch %d" % i)


class _Mats:
    """Device buffers of a list of (n, bits) matrices for the batched calls."""

    def __init__(self, spec, seed):
        self.spec = spec
        self.ks = [inputs.fp16_weights(n, seed + i, outliers=(i % 3 == 1)) for i, (n, _) in enumerate(spec)]
        self.c0s = [inputs.quantile_init(k, 1 << b) for k, (_, b) in zip(self.ks, spec)]
        self.gs = [inputs.upstream_grad(n, seed + 40 + i) for i, (n, _) in enumerate(spec)]
        self.plans = [edkm.Plan(n, b, ITERS) for n, b in spec]
        self.kd = [dkeys(k) for k in self.ks]
        self.ci = [torch.from_numpy(c).to(DEV) for c in self.c0s]
        self.co = [torch.empty(1 << b, device=DEV) for _, b in spec]
        self.wt = [torch.empty(n, device=DEV) for n, _ in spec]
        self.it = [torch.zeros(1, dtype=torch.int32, device=DEV) for _ in spec]
        self.gd = [torch.from_numpy(g).to(DEV) for g in self.gs]
        self.gw = [torch.empty(n, device=DEV) for n, _ in spec]
        self.gc = [torch.empty(1 << b, device=DEV) for _, b in spec]

    def sub(self, name, idx):
        return [getattr(self, name)[i] for i in idx]

    def result(self, i):
        return dict(iters=self.it[i].cpu().numpy(), c_out=self.co[i].cpu().numpy(),
                    w_tilde=self.wt[i].cpu().numpy(), grad_w=self.gw[i].cpu().numpy(),
                    grad_c=self.gc[i].cpu().numpy())


def test_batch_mixed_bit_widths():
    """Matrices of 1 to 4 bits in one batched step: launch groups are cut where
    the bit width changes.  Each matrix equals its single call (forward
    bitwise) and the oracle."""
    spec = [(70_001, 3), (65536, 1), (100_003, 4), (30_000, 4), (5000, 2), (90_000, 3)]
    m = _Mats(spec, 470)
    say("batch, mixed bit widths")
    edkm.init_unique_batch(m.plans, m.kd)
    edkm.forward_batch(m.plans, m.kd, TAU, 0.0, m.ci, m.co, m.wt, False, m.it)
    edkm.backward_batch(m.plans, m.kd, m.gd, m.gw, m.gc)
    torch.cuda.synchronize()
    for i, (n, b) in enumerate(spec):
        single = gpu(m.ks[i], m.c0s[i], b, g=m.gs[i])
        assert np.array_equal(m.co[i].cpu().numpy(), single["c_out"]), i
        assert np.array_equal(m.wt[i].cpu().numpy(), single["w_tilde"]), i
        check(m.result(i), oracle(m.ks[i], m.c0s[i], m.gs[i]), what="mixed bits %d" % i)


def test_backward_batch_over_forwards_with_different_tau():
    """Two forward_batch calls with different tau, then one backward_batch over
    all plans: the backward splits its launch groups where tau changes, and each
    matrix's gradients match the oracle at its own tau."""
    spec = [(65536, 3), (100_003, 3), (70_001, 3), (30_000, 3)]
    taus = [TAU, TAU, 5e-3, 5e-3]
    m = _Mats(spec, 480)
    say("backward batch, two taus")
    edkm.init_unique_batch(m.plans, m.kd)
    for idx, tau in (([0, 1], TAU), ([2, 3], 5e-3)):
        edkm.forward_batch(m.sub("plans", idx), m.sub("kd", idx), tau, 0.0, m.sub("ci", idx), m.sub("co", idx),
                           m.sub("wt", idx), False, m.sub("it", idx))
    edkm.backward_batch(m.plans, m.kd, m.gd, m.gw, m.gc)
    torch.cuda.synchronize()
    for i in range(len(spec)):
        check(m.result(i), oracle(m.ks[i], m.c0s[i], m.gs[i], tau=taus[i]), what="tau %g matrix %d" % (taus[i], i))


@pytest.mark.parametrize("tau", [2e-4, 5e-2])
def test_unique_path_at_other_temperatures(tau):
    """Near-hard assignment (tau = 2e-4, a tenth of the workload's) and a soft
    one (tau = 5e-2, most weights spread over several centroids)."""
    keys = inputs.fp16_weights(300_007, 490, outliers=True)
    c0 = inputs.quantile_init(keys, 8)
    g = inputs.upstream_grad(keys.size, 491)
    say("tau", tau)
    check(gpu(keys, c0, 3, g=g, tau=tau), oracle(keys, c0, g, tau=tau), what="tau %g" % tau)


def test_call_order_and_key_buffer_checks():
    keys = inputs.fp16_weights(4096, 141)
    c0 = torch.from_numpy(inputs.quantile_init(keys, 8)).to(DEV)
    kd = dkeys(keys)
    other = kd.clone()
    plan = edkm.Plan(keys.size, 3, ITERS)
    c_out = torch.empty(8, device=DEV)
    wt = torch.empty(keys.size, device=DEV)
    g = torch.ones(keys.size, device=DEV)
    gw, gc = torch.empty_like(wt), torch.empty(8, device=DEV)
    with pytest.raises(edkm.EdkmError):
        edkm.forward(plan, kd, TAU, 0.0, c0, c_out, wt)
    edkm.init_unique(plan, kd)
    with pytest.raises(edkm.EdkmError) as e:
        edkm.forward(plan, other, TAU, 0.0, c0, c_out, wt)
    assert e.value.status == edkm.ERR_STATE
    with pytest.raises(edkm.EdkmError):
        edkm.backward(plan, kd, g, gw, gc)
    edkm.forward(plan, kd, TAU, 0.0, c0, c_out, wt)
    edkm.backward(plan, kd, g, gw, gc)
    first = gw.clone()
    edkm.backward(plan, kd, g, gw, gc)       # a second backward reuses the forward state
    torch.cuda.synchronize()
    assert_close(gw.cpu().numpy(), first.cpu().numpy(), 1e-6, "repeat backward")



def test_plan_reused_across_weight_distributions():
    """One plan and its workspace carried through matrices with very different
    pattern sets in turn: narrow Gaussian, a span wider than the LDS windows,
    special values, one repeated value, then the narrow one again.  Each must
    give what a fresh plan gives on the same inputs (counts, occupied-pattern
    count and forward outputs bitwise; backward within 1e-6 relative, as
    between any two runs), so nothing one matrix left in the workspace
    (windows, keyed-sum mode, table entries of patterns the next one lacks, G,
    partial rows) reaches the next."""
    n = 150_000
    rng = np.random.default_rng(401)
    wide = (np.sign(rng.standard_normal(n)) * np.exp2(rng.uniform(-24, 15.9, n))).astype(np.float16).view(np.uint16)
    wide[: n // 2] = inputs.fp16_weights(n // 2, 402)
    narrow = inputs.fp16_weights(n, 400)
    sets = [("narrow", narrow), ("wide", wide), ("special", special_keys(n, 403)),
            ("constant", np.full(n, np.float16(0.01).view(np.uint16), dtype=np.uint16)),
            ("narrow again", narrow)]
    plan = edkm.Plan(n, 3, ITERS)
    for i, (name, keys) in enumerate(sets):
        c0 = inputs.quantile_init(keys, 8)
        g = inputs.upstream_grad(n, 410 + i)
        say("plan reuse", name)
        got = gpu(keys, c0, 3, g=g, want_counts=True, plan=plan)
        ref = gpu(keys, c0, 3, g=g, want_counts=True)
        for f in ("counts", "num_unique", "iters", "c_out", "w_tilde"):
            assert np.array_equal(got[f], ref[f]), (name, f)
        assert_close(got["grad_w"], ref["grad_w"], 1e-6, name + " grad_w")
        slack = 1e-6 * np.abs(ref["grad_c"]) + 1e-9 * float(np.abs(g).sum())
        assert np.all(np.abs(got["grad_c"] - ref["grad_c"]) <= slack), name + " grad_c"



# ------------------------------------------------------------------ 16-bit gradients

def bits16(x, fmt):
    """float32 -> 16-bit patterns of the weight format, round to nearest even."""
    x = np.asarray(x, np.float32)
    return x.astype(np.float16).view(np.uint16) if fmt == "fp16" else _bf16_bits(x)


def value16(b, fmt):
    b = np.asarray(b, np.uint16)
    return b.view(np.float16).astype(np.float64) if fmt == "fp16" else _bf16_values(b)


def assert16(bits, ref, fmt, tol, what):
    check = assert_fp16_within_ulp if fmt == "fp16" else assert_bf16_within_ulp
    check(np.asarray(bits).view(np.uint16), ref, what, tol=tol)


HALF_GRAD_CASES = [(65536, 3, False, 700), (300_007, 4, True, 701), (1_000_003, 2, False, 702)]


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
@pytest.mark.parametrize("flags", [1, 2, 3])
@pytest.mark.parametrize("n,bits,outl,seed", HALF_GRAD_CASES)
def test_half_gradients(n, bits, outl, seed, fmt, flags):
    """edkm_backward_ex with 16-bit dL/dW~ (flag 1), 16-bit dL/dw (flag 2) or
    both, in the weights' format.  A 16-bit dL/dW~ is the fp32 one rounded to
    that format: the oracle takes those rounded values.  A 16-bit dL/dw is
    within one ulp of the fp32 path's result rounded (same inputs, another run:
    the keyed sum's float atomics may flip a rounding) and within one ulp of
    the oracle's, or its fp32 bar where g_i H + R cancels."""
    k = 1 << bits
    keys = inputs.weights(n, seed, outl, fmt)
    c0 = inputs.quantile_init(keys, k, fmt)
    g = inputs.upstream_grad(n, seed + 1)
    g_eff = value16(bits16(g, fmt), fmt).astype(np.float32) if flags & 1 else g
    say("half gradients", n, bits, fmt, flags)
    plan = edkm.Plan(n, bits, ITERS, key_format=fmt)
    kd = dkeys(keys)
    ci = torch.from_numpy(c0).to(DEV)
    co, wt = torch.empty(k, device=DEV), torch.empty(n, device=DEV)
    edkm.init_unique(plan, kd)
    edkm.forward(plan, kd, TAU, 0.0, ci, co, wt)
    g32 = torch.from_numpy(g_eff).to(DEV)
    gw32, gc32 = torch.empty(n, device=DEV), torch.empty(k, device=DEV)
    edkm.backward(plan, kd, g32, gw32, gc32)
    gin = torch.from_numpy(bits16(g, fmt).view(np.int16)).to(DEV) if flags & 1 else g32
    gw = torch.empty(n, dtype=torch.int16 if flags & 2 else torch.float32, device=DEV)
    gc = torch.empty(k, device=DEV)
    edkm.backward(plan, kd, gin, gw, gc)
    torch.cuda.synchronize()
    a32 = gw32.cpu().numpy()
    ref = oracle(keys, c0, g_eff, form="dense" if n <= 300_007 else "table", fmt=fmt)
    what = "n=%d bits=%d %s flags=%d" % (n, bits, fmt, flags)
    if flags & 2:
        got = gw.cpu().numpy().view(np.uint16)
        r32 = bits16(a32, fmt)
        ulp = np.abs(value16(r32 + np.uint16(1), fmt) - value16(r32, fmt))
        assert np.all(np.abs(value16(got, fmt) - value16(r32, fmt)) <= ulp), what + " vs fp32 path"
        assert16(got, ref["gw"], fmt, TOL_BWD, what + " grad_w")
    else:
        assert_close(gw.cpu().numpy(), a32, 1e-6, what + " vs fp32 path")
        assert_close(gw.cpu().numpy(), ref["gw"], TOL_BWD, what + " grad_w")
    assert_close(gc.cpu().numpy(), ref["gc"], TOL_BWD, what + " grad_c")


def test_half_gradients_misaligned_take_the_scalar_path():
    """16-bit gradient arrays one element off 16-byte alignment (the scalar
    path of both N-sized passes) equal the aligned call's results."""
    n = 100_003
    keys = inputs.fp16_weights(n, 710)
    c0 = inputs.quantile_init(keys, 8)
    g16 = bits16(inputs.upstream_grad(n, 711), "fp16").view(np.int16)
    plan = edkm.Plan(n, 3, ITERS)
    kd = dkeys(keys)
    co, wt = torch.empty(8, device=DEV), torch.empty(n, device=DEV)
    edkm.init_unique(plan, kd)
    edkm.forward(plan, kd, TAU, 0.0, torch.from_numpy(c0).to(DEV), co, wt)
    say("half gradients misaligned")
    outs = []
    for off in (0, 1):
        gbuf = torch.zeros(n + 8, dtype=torch.int16, device=DEV)
        gbuf[off:off + n] = torch.from_numpy(g16).to(DEV)
        wbuf = torch.zeros(n + 8, dtype=torch.int16, device=DEV)
        gc = torch.empty(8, device=DEV)
        edkm.backward(plan, kd, gbuf[off:off + n], wbuf[off:off + n], gc)
        torch.cuda.synchronize()
        outs.append((wbuf[off:off + n].cpu().numpy().view(np.uint16), gc.cpu().numpy()))
    (a, ga), (b, gb) = outs
    ulp = np.abs(value16(a + np.uint16(1), "fp16") - value16(a, "fp16"))
    assert np.all(np.abs(value16(b, "fp16") - value16(a, "fp16")) <= ulp)
    assert_close(gb, ga, 1e-6, "grad_c")


# ------------------------------------------------------------------ full workload shapes

@pytest.mark.parametrize("cfg,bits,fmt", [(2, 3, "fp16"), (3, 3, "fp16"), (3, 4, "fp16"),
                                          (2, 3, "bf16"), (3, 4, "bf16")])
def test_full_size_matrix(cfg, bits, fmt):
    w = inputs.WORKLOADS[cfg]
    _, r, c = w["mats"][0]
    n = r * c
    keys = inputs.weights(n, inputs.weight_seed(cfg, 0), w["outliers"], fmt)
    c0 = inputs.quantile_init(keys, 1 << bits, fmt)
    g = inputs.upstream_grad(n, inputs.grad_seed(cfg, 0))
    say("full", cfg, bits, fmt, n)
    res = gpu(keys, c0, bits, g=g, want_counts=True, key_format=fmt)
    assert np.array_equal(res["counts"].view(np.uint32), table.histogram(keys))
    check(res, oracle(keys, c0, g, form="table", fmt=fmt), what="cfg%d bits=%d %s" % (cfg, bits, fmt))


@pytest.mark.parametrize("cfg,bits", [(2, 3), (3, 3), (3, 4)])
def test_full_size_dense_path(cfg, bits):
    """The dense comparison path at the sizes the benchmark times it (4096x4096,
    and 11008x4096 with outliers at 3 and 4 bits): 1,024 workgroups of up to
    44,032 weights each, every partial row summed by the one-block finishing
    kernels.  Against the table-form oracle (pinned to the dense one)."""
    w = inputs.WORKLOADS[cfg]
    _, r, c = w["mats"][0]
    n = r * c
    keys = inputs.fp16_weights(n, inputs.weight_seed(cfg, 0), w["outliers"])
    c0 = inputs.quantile_init(keys, 1 << bits)
    g = inputs.upstream_grad(n, inputs.grad_seed(cfg, 0))
    say("full dense", cfg, bits, n)
    res = gpu(keys, c0, bits, g=g, dense=True)
    check(res, oracle(keys, c0, g, form="table"), what="dense cfg%d bits=%d" % (cfg, bits))


@pytest.mark.parametrize("fmt,out_half", [("fp16", False), ("fp16", True), ("bf16", False), ("bf16", True)])
def test_decoder_layer_batch_full_size(fmt, out_half):
    """The seven matrices of one LLaMA-7B decoder layer in one batch (the call the
    benchmark times, also in its 16-bit W~ and bf16-weight modes), each against
    the table-form oracle.  16-bit W~ (fp16 or bf16, the weights' format) is
    held to one ulp of the oracle value rounded to that format; bf16 entries
    near a zero crossing of W~, where one bf16 ulp is below fp32 accuracy, to
    the fp32 forward bar instead."""
    w = inputs.WORKLOADS[4]
    say("decoder layer", fmt, "half W~" if out_half else "fp32 W~")
    plans, kd, ci, co, wt, it, gd, gw, gc, host = [], [], [], [], [], [], [], [], [], []
    for i, (name, r, c) in enumerate(w["mats"]):
        n = r * c
        keys = inputs.weights(n, inputs.weight_seed(4, i), False, fmt)
        c0 = inputs.quantile_init(keys, 8, fmt)
        g = inputs.upstream_grad(n, inputs.grad_seed(4, i))
        host.append((keys, c0, g))
        plans.append(edkm.Plan(n, 3, ITERS, key_format=fmt))
        kd.append(dkeys(keys))
        ci.append(torch.from_numpy(c0).to(DEV))
        co.append(torch.empty(8, device=DEV))
        wt.append(torch.empty(n, dtype=torch.int16 if out_half else torch.float32, device=DEV))
        it.append(torch.zeros(1, dtype=torch.int32, device=DEV))
        gd.append(torch.from_numpy(g).to(DEV))
        gw.append(torch.empty(n, device=DEV))
        gc.append(torch.empty(8, device=DEV))
    edkm.init_unique_batch(plans, kd)
    edkm.forward_batch(plans, kd, TAU, 0.0, ci, co, wt, out_half, it)
    edkm.backward_batch(plans, kd, gd, gw, gc)
    torch.cuda.synchronize()
    for i, (keys, c0, g) in enumerate(host):
        what = "%s %s" % (w["mats"][i][0], fmt)
        ref = oracle(keys, c0, g, form="table", fmt=fmt)
        wv = wt[i].cpu().numpy()
        assert int(it[i].item()) == ref["T"], what
        assert_close(co[i].cpu().numpy(), ref["c_out"], TOL_FWD, what + " c_out")
        if out_half and fmt == "bf16":
            assert_bf16_within_ulp(wv.view(np.uint16), ref["w_tilde"], what + " bf16 W~", tol=TOL_FWD)
        elif out_half:
            assert_fp16_within_ulp(wv.view(np.uint16), ref["w_tilde"], what + " fp16 W~")
        else:
            assert_close(wv, ref["w_tilde"], TOL_FWD, what + " w_tilde")
        assert_close(gw[i].cpu().numpy(), ref["gw"], TOL_BWD, what + " grad_w")
        assert_close(gc[i].cpu().numpy(), ref["gc"], TOL_BWD, what + " grad_c")



@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
def test_decoder_layer_training_in_16_bits_full_size(fmt):
    """The decoder layer's seven matrices with every N-sized array in the
    weights' format, as a 16-bit training step has them: 16-bit W~ out,
    16-bit dL/dW~ in (the fp32 draw rounded), 16-bit dL/dw out.  Each matrix
    against the table-form oracle on the rounded gradient: W~ and dL/dw within
    one ulp (or, where the result cancels towards 0, the fp32 bar)."""
    w = inputs.WORKLOADS[4]
    say("decoder layer 16-bit training", fmt)
    plans, kd, ci, co, wt, it, gd, gw, gc, host = [], [], [], [], [], [], [], [], [], []
    for i, (name, r, c) in enumerate(w["mats"]):
        n = r * c
        keys = inputs.weights(n, inputs.weight_seed(4, i), False, fmt)
        c0 = inputs.quantile_init(keys, 8, fmt)
        g16 = bits16(inputs.upstream_grad(n, inputs.grad_seed(4, i)), fmt)
        host.append((keys, c0, value16(g16, fmt)))
        plans.append(edkm.Plan(n, 3, ITERS, key_format=fmt))
        kd.append(dkeys(keys))
        ci.append(torch.from_numpy(c0).to(DEV))
        co.append(torch.empty(8, device=DEV))
        wt.append(torch.empty(n, dtype=torch.int16, device=DEV))
        it.append(torch.zeros(1, dtype=torch.int32, device=DEV))
        gd.append(torch.from_numpy(g16.view(np.int16)).to(DEV))
        gw.append(torch.empty(n, dtype=torch.int16, device=DEV))
        gc.append(torch.empty(8, device=DEV))
    edkm.init_unique_batch(plans, kd)
    edkm.forward_batch(plans, kd, TAU, 0.0, ci, co, wt, True, it)
    edkm.backward_batch(plans, kd, gd, gw, gc)
    torch.cuda.synchronize()
    for i, (keys, c0, g) in enumerate(host):
        what = "%s %s" % (w["mats"][i][0], fmt)
        ref = oracle(keys, c0, g, form="table", fmt=fmt)
        assert int(it[i].item()) == ref["T"], what
        assert_close(co[i].cpu().numpy(), ref["c_out"], TOL_FWD, what + " c_out")
        assert16(wt[i].cpu().numpy(), ref["w_tilde"], fmt, TOL_FWD, what + " W~")
        assert16(gw[i].cpu().numpy(), ref["gw"], fmt, TOL_BWD, what + " grad_w")
        assert_close(gc[i].cpu().numpy(), ref["gc"], TOL_BWD, what + " grad_c")


# ------------------------------------------------------------------ bf16 weights

BF16_CASES = [(1, 3, False, 31), (4097, 2, True, 32), (65573, 3, True, 33), (300_007, 4, True, 34),
              (1_000_003, 3, False, 35)]


@pytest.mark.parametrize("n,bits,outl,seed", BF16_CASES)
def test_bf16_unique_path_matches_oracle(n, bits, outl, seed):
    """bfloat16 weights: the same table machinery with the bf16 decode."""
    keys = inputs.bf16_weights(n, seed, outl)
    c0 = inputs.quantile_init(keys, 1 << bits, "bf16")
    g = inputs.upstream_grad(n, seed + 1)
    say("bf16 unique", n, bits)
    res = gpu(keys, c0, bits, g=g, want_counts=True, key_format="bf16")
    np.testing.assert_array_equal(res["counts"].view(np.uint32), table.histogram(keys))
    assert int(res["num_unique"][0]) == np.unique(keys).size
    form = "dense" if n <= 300_007 else "table"
    check(res, oracle(keys, c0, g, form=form, fmt="bf16"), what="bf16 n=%d" % n)


def test_bf16_dense_path_matches_oracle():
    keys = inputs.bf16_weights(65573, 36, outliers=True)
    c0 = inputs.quantile_init(keys, 8, "bf16")
    g = inputs.upstream_grad(keys.size, 37)
    say("bf16 dense")
    res = gpu(keys, c0, 3, g=g, dense=True, key_format="bf16")
    check(res, oracle(keys, c0, g, fmt="bf16"), what="bf16 dense")


@pytest.mark.parametrize("dense_path", [False, True])
def test_bf16_output_within_one_ulp(dense_path):
    """16-bit W~ outputs take the weight format: bf16, round to nearest even."""
    keys = inputs.bf16_weights(65536 + 5, 38)
    c0 = inputs.quantile_init(keys, 8, "bf16")
    say("bf16 out", dense_path)
    res = gpu(keys, c0, 3, out_half=True, dense=dense_path, key_format="bf16")
    assert_bf16_within_ulp(res["w_tilde"].view(np.uint16), oracle(keys, c0, fmt="bf16")["w_tilde"])


def test_bf16_special_values():
    """Signed zeros, bf16 subnormals (fp32 subnormals), the smallest normals and
    +-1: exact decode, and the zero/subnormal magnitudes fall outside the 8-byte
    window (global fallback)."""
    keys = inputs.bf16_weights(100_003, 39)
    rng = np.random.default_rng(39)
    extra = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x007F, 0x807F, 0x0080, 0x8080, 0x3F80,
                      0xBF80], dtype=np.uint16)
    pos = rng.choice(keys.size, size=4 * extra.size, replace=False)
    keys[pos] = np.resize(extra, pos.size)
    c0 = inputs.quantile_init(keys, 16, "bf16")
    g = inputs.upstream_grad(keys.size, 40)
    say("bf16 special")
    res = gpu(keys, c0, 4, g=g, key_format="bf16")
    check(res, oracle(keys, c0, g, fmt="bf16"), what="bf16 special")


def test_bf16_far_values_take_the_global_tables():
    """2,000 weights at +-1e30 (magnitudes far outside both LDS windows) with a
    centroid on each: every lookup of theirs goes to the global tables.  (Values
    that drag a centroid into the empty space between clusters are avoided: once
    every attention to a centroid is below fp32's range but not fp64's, the
    two precisions legitimately take different empty-cluster decisions.)"""
    keys = inputs.bf16_weights(100_003, 44)
    rng = np.random.default_rng(44)
    pos = rng.choice(keys.size, size=2000, replace=False)
    keys[pos[:1000]] = 0x7149
    keys[pos[1000:]] = 0xF149
    normal = np.ones(keys.size, bool)
    normal[pos] = False
    far = float(inputs.values(np.array([0x7149], np.uint16), "bf16")[0])
    c0 = np.sort(np.concatenate([inputs.quantile_init(keys[normal], 14, "bf16"),
                                 np.float32([far, -far])])).astype(np.float32)
    g = inputs.upstream_grad(keys.size, 45)
    say("bf16 far values")
    res = gpu(keys, c0, 4, g=g, key_format="bf16")
    check(res, oracle(keys, c0, g, fmt="bf16"), what="bf16 far values")


def test_bf16_nonfinite_weights():
    keys = inputs.bf16_weights(50_000, 42)
    bad = keys.copy()
    idx = [5, 777, 40_000, 49_999]
    bad[idx] = [0x7F80, 0xFF80, 0x7FC0, 0x7F81]
    c0 = inputs.quantile_init(keys, 8, "bf16")
    say("bf16 non-finite checked")
    with pytest.raises(edkm.EdkmError) as e:
        gpu(bad, c0, 3, check_finite=True, key_format="bf16")
    assert e.value.status == edkm.ERR_NONFINITE
    say("bf16 non-finite unchecked")
    g = inputs.upstream_grad(bad.size, 43)
    res = gpu(bad, c0, 3, g=g, key_format="bf16")
    finite = np.ones(bad.size, bool)
    finite[idx] = False
    ref = oracle(bad[finite], c0, g[finite], fmt="bf16")
    assert np.all(np.isnan(res["w_tilde"][~finite]))
    assert np.all(np.isnan(res["grad_w"][~finite]))
    assert_close(res["c_out"], ref["c_out"], TOL_FWD, "c_out")
    assert_close(res["w_tilde"][finite], ref["w_tilde"], TOL_FWD, "w_tilde")
    assert_close(res["grad_w"][finite], ref["gw"], TOL_BWD, "grad_w")
    assert_close(res["grad_c"], ref["gc"], TOL_BWD, "grad_c")


def test_mixed_format_batch_equals_single_calls():
    """A batch mixing fp16 and bf16 matrices is cut into launch groups of one
    format each; every matrix equals its single-matrix call bitwise in the
    forward."""
    spec = [(65536, "fp16"), (100_003, "bf16"), (70_001, "bf16"), (30_000, "fp16")]
    ks = [inputs.weights(n, 150 + i, i == 1, fmt) for i, (n, fmt) in enumerate(spec)]
    c0s = [inputs.quantile_init(k, 8, fmt) for k, (_, fmt) in zip(ks, spec)]
    gs = [inputs.upstream_grad(n, 160 + i) for i, (n, _) in enumerate(spec)]
    say("mixed-format batch")
    plans = [edkm.Plan(n, 3, ITERS, key_format=fmt) for n, fmt in spec]
    kd = [dkeys(k) for k in ks]
    ci = [torch.from_numpy(c).to(DEV) for c in c0s]
    co = [torch.empty(8, device=DEV) for _ in spec]
    wt = [torch.empty(n, device=DEV) for n, _ in spec]
    it = [torch.zeros(1, dtype=torch.int32, device=DEV) for _ in spec]
    gd = [torch.from_numpy(g).to(DEV) for g in gs]
    gw = [torch.empty(n, device=DEV) for n, _ in spec]
    gc = [torch.empty(8, device=DEV) for _ in spec]
    edkm.init_unique_batch(plans, kd)
    edkm.forward_batch(plans, kd, TAU, 0.0, ci, co, wt, False, it)
    edkm.backward_batch(plans, kd, gd, gw, gc)
    torch.cuda.synchronize()
    for i, (n, fmt) in enumerate(spec):
        single = gpu(ks[i], c0s[i], 3, g=gs[i], key_format=fmt)
        assert np.array_equal(co[i].cpu().numpy(), single["c_out"])
        assert np.array_equal(wt[i].cpu().numpy(), single["w_tilde"])
        res = dict(iters=it[i].cpu().numpy(), c_out=co[i].cpu().numpy(), w_tilde=wt[i].cpu().numpy(),
                   grad_w=gw[i].cpu().numpy(), grad_c=gc[i].cpu().numpy())
        check(res, oracle(ks[i], c0s[i], gs[i], fmt=fmt), what="mixed %d %s" % (i, fmt))
