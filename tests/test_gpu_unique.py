"""GPU distinct-pattern list and inverse index (edkm_unique_inverse) against
the oracle's uniquification (numpy.unique of the uint16 keys, with
return_inverse).

Integer work, compared bit for bit.  Every output buffer carries guard
elements after its end (and unique_out's entries past the distinct count are
guards too), which must come back untouched.  Sizes run from one weight
through ragged multi-workgroup slices to the 4096x4096 workload shape, plus
every 16-bit pattern at once (ranks up to 65,535), non-finite patterns and
signed zeros, misaligned buffers (the scalar path), bf16 keys and batches
that span launch groups.  At the decoder layer's size, in the batched call,
the outputs are checked by properties that hold at any size.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import table                                          # noqa: E402
from paper_2309_00964_amd import edkm, inputs                     # noqa: E402
from parity_util import TOL_BWD, TOL_FWD, assert_close            # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda"
GUARD = 64
FILL = 0x5A5A          # guard pattern (int16 and uint16 alike)
NKEYS = edkm.NKEYS


def say(*a):
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def dkeys(keys, offset=0):
    buf = torch.zeros(keys.size + offset, dtype=torch.int16, device=DEV)
    buf[offset:] = torch.from_numpy(np.ascontiguousarray(keys).view(np.int16)).to(DEV)
    return buf[offset:]


def out16(n, offset=0):
    buf = torch.full((offset + n + GUARD,), FILL, dtype=torch.int16, device=DEV)
    return buf, buf[offset:offset + n]


def host16(t):
    return t.cpu().numpy().view(np.uint16)


def gpu_unique(keys, fmt="fp16", key_offset=0, out_offset=0, want_unique=True, want_inverse=True):
    """init_unique then unique_inverse; returns (unique list, inverse,
    num_unique, unique buffer past the list, inverse guard)."""
    n = keys.size
    kd = dkeys(keys, key_offset)
    plan = edkm.Plan(n, 3, inputs.ITERS, key_format=fmt)
    nu = torch.zeros(1, dtype=torch.int32, device=DEV)
    edkm.init_unique(plan, kd, num_unique_out=nu)
    ubuf, uview = out16(NKEYS)
    ibuf, iview = out16(n, out_offset)
    edkm.unique_inverse(plan, kd, uview if want_unique else None, iview if want_inverse else None)
    torch.cuda.synchronize()
    U = int(nu.item())
    u = host16(ubuf)
    i = host16(ibuf)
    return u[:U], i[out_offset:out_offset + n], U, u[U:], np.concatenate([i[:out_offset], i[out_offset + n:]])


def check(keys, got, what):
    u_ref, inv_ref = table.unique_keys(keys)
    u, inv, U, u_rest, guard = got
    assert U == u_ref.size, what
    np.testing.assert_array_equal(u, u_ref, err_msg=what)
    np.testing.assert_array_equal(inv.astype(np.uint32), inv_ref, err_msg=what)
    assert np.all(u_rest == FILL) and np.all(guard == FILL), what + ": wrote past its outputs"


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
@pytest.mark.parametrize("n", [1, 7, 65_536, 1_000_003])
def test_unique_inverse_matches_numpy_unique(fmt, n):
    keys = inputs.weights(n, 300 + n % 97, True, fmt)
    say("unique_inverse", fmt, n)
    check(keys, gpu_unique(keys, fmt), "%s n=%d" % (fmt, n))


def test_every_pattern_present():
    """All 65,536 patterns occur (Inf/NaN included): 65,536 distinct keys, the
    largest rank 65,535, unique_out written in full."""
    rng = np.random.default_rng(301)
    keys = np.concatenate([rng.permutation(NKEYS), rng.integers(0, NKEYS, 98_307)]).astype(np.uint16)
    rng.shuffle(keys)
    say("unique_inverse all patterns", keys.size)
    got = gpu_unique(keys)
    assert got[2] == NKEYS
    check(keys, got, "all patterns")


def test_nonfinite_and_signed_zero_patterns():
    """Inf/NaN patterns are keys like any other; +0 and -0 are distinct."""
    keys = inputs.fp16_weights(200_001, 302)
    keys[[0, 5, 77, 200_000]] = [0x7C00, 0xFC00, 0x7E00, 0xFFFF]
    keys[[1, 2, 3]] = [0x0000, 0x8000, 0x8000]
    say("unique_inverse non-finite, signed zeros")
    check(keys, gpu_unique(keys), "special patterns")


@pytest.mark.parametrize("key_offset,out_offset", [(1, 0), (0, 1), (3, 5)])
def test_misaligned_buffers(key_offset, out_offset):
    keys = inputs.fp16_weights(123_457, 303)
    say("unique_inverse misaligned", key_offset, out_offset)
    check(keys, gpu_unique(keys, key_offset=key_offset, out_offset=out_offset), "misaligned")


def test_one_output_only():
    keys = inputs.fp16_weights(500_009, 304)
    u_ref, inv_ref = table.unique_keys(keys)
    say("unique_inverse unique only")
    u, inv, U, u_rest, _ = gpu_unique(keys, want_inverse=False)
    np.testing.assert_array_equal(u, u_ref)
    assert np.all(inv == FILL) and np.all(u_rest == FILL)
    say("unique_inverse inverse only")
    u, inv, U, u_rest, guard = gpu_unique(keys, want_unique=False)
    np.testing.assert_array_equal(inv.astype(np.uint32), inv_ref)
    assert np.all(u == FILL) and np.all(guard == FILL)


def test_workload_shape_4096x4096():
    keys = inputs.weights(4096 * 4096, 305, False, "fp16")
    say("unique_inverse 4096x4096")
    check(keys, gpu_unique(keys), "4096x4096")


def test_between_forward_and_backward_leaves_the_path_intact():
    """unique_inverse after forward, then backward: W~ and the gradients still
    match the oracle (the ranking uses its own part of the workspace)."""
    n, bits = 65_536, 3
    keys = inputs.fp16_weights(n, 306)
    c0 = inputs.quantile_init(keys, 1 << bits)
    g = inputs.upstream_grad(n, 307)
    kd = dkeys(keys)
    plan = edkm.Plan(n, bits, inputs.ITERS)
    edkm.init_unique(plan, kd)
    c_out = torch.empty(1 << bits, device=DEV)
    wt = torch.empty(n, device=DEV)
    edkm.forward(plan, kd, inputs.TAU, 0.0, torch.from_numpy(c0).to(DEV), c_out, wt)
    ubuf, uview = out16(NKEYS)
    ibuf, iview = out16(n)
    say("unique_inverse between forward and backward")
    edkm.unique_inverse(plan, kd, uview, iview)
    gw = torch.empty(n, device=DEV)
    gc = torch.empty(1 << bits, device=DEV)
    edkm.backward(plan, kd, torch.from_numpy(g).to(DEV), gw, gc)
    torch.cuda.synchronize()
    ref = table.forward(keys, c0.astype(np.float64), inputs.TAU, inputs.ITERS)
    gw_ref, gc_ref, _ = table.backward(keys, ref, g.astype(np.float64))
    assert_close(wt.cpu().numpy(), ref["w_tilde"], TOL_FWD, "w_tilde")
    assert_close(gw.cpu().numpy(), gw_ref, TOL_BWD, "grad_w")
    assert_close(gc.cpu().numpy(), gc_ref, TOL_BWD, "grad_c")
    u_ref, inv_ref = table.unique_keys(keys)
    np.testing.assert_array_equal(host16(ubuf)[:u_ref.size], u_ref)
    np.testing.assert_array_equal(host16(ibuf)[:n].astype(np.uint32), inv_ref)


def test_wrong_key_buffer_is_a_state_error():
    keys = inputs.fp16_weights(10_000, 308)
    kd, other = dkeys(keys), dkeys(keys)
    plan = edkm.Plan(keys.size, 3, inputs.ITERS)
    edkm.init_unique(plan, kd)
    _, iview = out16(keys.size)
    with pytest.raises(edkm.EdkmError) as e:
        edkm.unique_inverse(plan, other, None, iview)
    assert e.value.status == edkm.ERR_STATE


def test_batch_across_launch_groups():
    """31 matrices (two launch groups), mixed sizes and formats' worth of
    patterns, some wanting only one output."""
    sizes = [1, 2, 3, 31, 33, 4097, 65_536, 65_537] + [10_000 + 997 * i for i in range(23)]
    keys = [inputs.fp16_weights(n, 320 + i) for i, n in enumerate(sizes)]
    kd = [dkeys(k) for k in keys]
    plans = [edkm.Plan(n, 3, inputs.ITERS) for n in sizes]
    edkm.init_unique_batch(plans, kd)
    ub = [out16(NKEYS) for _ in sizes]
    ib = [out16(n) for n in sizes]
    uo = [None if i % 5 == 1 else ub[i][1] for i in range(len(sizes))]
    io = [None if i % 5 == 3 else ib[i][1] for i in range(len(sizes))]
    say("unique_inverse batch", len(sizes))
    edkm.unique_inverse_batch(plans, kd, uo, io)
    torch.cuda.synchronize()
    for i, k in enumerate(keys):
        u_ref, inv_ref = table.unique_keys(k)
        u, inv = host16(ub[i][0]), host16(ib[i][0])
        if uo[i] is None:
            assert np.all(u == FILL), i
        else:
            np.testing.assert_array_equal(u[:u_ref.size], u_ref, err_msg=str(i))
            assert np.all(u[u_ref.size:] == FILL), i
        if io[i] is None:
            assert np.all(inv == FILL), i
        else:
            np.testing.assert_array_equal(inv[:k.size].astype(np.uint32), inv_ref, err_msg=str(i))
            assert np.all(inv[k.size:] == FILL), i


def test_decoder_layer_batch_properties():
    """The seven matrices of a LLaMA-7B decoder layer in one batched call: the
    list is strictly ascending with num_unique entries, covers exactly the
    occupied patterns of the counts, and unique[inverse] rebuilds the keys."""
    mats = inputs.WORKLOADS[4]["mats"]
    kd, plans, cnt, nus = [], [], [], []
    for j, (name, rows, cols) in enumerate(mats):
        n = rows * cols
        kd.append(inputs.fp16_weights_device(n, 4000 + j, DEV).view(torch.int16))
        plans.append(edkm.Plan(n, 3, inputs.ITERS))
        cnt.append(torch.empty(NKEYS, dtype=torch.int32, device=DEV))
        nus.append(torch.empty(1, dtype=torch.int32, device=DEV))
    edkm.init_unique_batch(plans, kd, counts_out=cnt, num_unique_out=nus)
    uo = [torch.empty(NKEYS, dtype=torch.int16, device=DEV) for _ in mats]
    io = [torch.empty(p.n, dtype=torch.int16, device=DEV) for p in plans]
    say("unique_inverse decoder layer batch")
    edkm.unique_inverse_batch(plans, kd, uo, io)
    torch.cuda.synchronize()
    for j in range(len(mats)):
        U = int(nus[j].item())
        u = uo[j][:U].to(torch.int32) & 0xFFFF
        assert bool(torch.all(u[1:] > u[:-1])), mats[j][0]
        occupied = torch.nonzero(cnt[j] != 0).flatten().to(torch.int32)
        assert occupied.numel() == U and bool(torch.equal(occupied, u)), mats[j][0]
        inv = io[j].to(torch.int64) & 0xFFFF
        assert int(inv.max()) < U, mats[j][0]
        assert bool(torch.equal(uo[j][inv], kd[j])), mats[j][0]
