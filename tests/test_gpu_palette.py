"""GPU palettization (edkm_palettize) against the palettization oracle.

The indices are integers decided by fp32 comparisons; both sides decide them
in fp32 on the same lookup table, so the packed bytes must match bit for bit.
The tables come from the input recipe (quantiles) or from the fp64 oracle's
final centroids, never from the GPU path.  Bytes past the packed output are
checked untouched.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import dense, palette                                 # noqa: E402
from paper_2309_00964_amd import edkm, inputs                     # noqa: E402
from parity_util import TOL_BWD, TOL_FWD, assert_close            # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda"
GUARD = 64


def say(*a):
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def gpu_palettize(keys, lut, bits, fmt, key_offset=0, out_offset=0):
    """Run edkm_palettize with the keys and the output placed key_offset
    elements / out_offset bytes into their buffers; returns (packed bytes,
    the guard bytes after them)."""
    n = keys.size
    nbytes = (n * bits + 7) // 8
    kbuf = torch.zeros(n + key_offset, dtype=torch.int16, device=DEV)
    kbuf[key_offset:] = torch.from_numpy(keys.view(np.int16)).to(DEV)
    obuf = torch.full((out_offset + nbytes + GUARD,), 0xAB, dtype=torch.uint8, device=DEV)
    plan = edkm.Plan(n, bits, inputs.ITERS, key_format=fmt)
    edkm.palettize(plan, kbuf[key_offset:], torch.from_numpy(np.asarray(lut, np.float32)).to(DEV),
                   obuf[out_offset:])
    torch.cuda.synchronize()
    o = obuf.cpu().numpy()
    return o[out_offset:out_offset + nbytes], o[out_offset + nbytes:]


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
@pytest.mark.parametrize("bits", [1, 2, 3, 4])
@pytest.mark.parametrize("n", [1, 31, 33, 65537, 1_000_003])
def test_palettize_bit_exact(fmt, bits, n):
    keys = inputs.weights(n, 200 + bits, True, fmt)
    lut = inputs.quantile_init(keys, 1 << bits, fmt)
    say("palettize", fmt, bits, n)
    got, guard = gpu_palettize(keys, lut, bits, fmt)
    np.testing.assert_array_equal(got, palette.palettize(keys, lut, bits, fmt))
    assert np.all(guard == 0xAB)


@pytest.mark.parametrize("bits", [2, 3])
def test_palettize_unaligned_buffers(bits):
    """Keys one element and the output one byte off alignment: the scalar path."""
    keys = inputs.fp16_weights(100_003, 210)
    lut = inputs.quantile_init(keys, 1 << bits)
    say("palettize unaligned", bits)
    got, guard = gpu_palettize(keys, lut, bits, "fp16", key_offset=1, out_offset=1)
    np.testing.assert_array_equal(got, palette.palettize(keys, lut, bits))
    assert np.all(guard == 0xAB)


def test_palettize_nonfinite_and_ties():
    """Inf/NaN weights get index 0; a weight equidistant from two entries gets
    the lower one."""
    keys = inputs.fp16_weights(10_000, 211)
    keys[[0, 17, 9999]] = [0x7C00, 0xFC00, 0x7E00]
    keys[[1, 2]] = np.array([0.5, 0.5], np.float16).view(np.uint16)
    lut = np.array([0.25, 0.75, -0.01, 0.01], np.float32)
    say("palettize special")
    got, _ = gpu_palettize(keys, lut, 2, "fp16")
    ref = palette.palettize(keys, lut, 2)
    np.testing.assert_array_equal(got, ref)
    idx = palette.unpack(got, keys.size, 2)
    assert idx[0] == idx[17] == idx[9999] == 0 and idx[1] == idx[2] == 0


def test_palettize_with_final_centroids_between_forward_and_backward():
    """The export of a clustering step: the fp64 oracle's C^(T) (as fp32) is the
    table.  Palettizing between forward and backward leaves the plan's state
    alone: the backward that follows still matches the oracle."""
    n, bits = 300_007, 3
    keys = inputs.fp16_weights(n, 212, outliers=True)
    c0 = inputs.quantile_init(keys, 8)
    g = inputs.upstream_grad(n, 213)
    ref = dense.forward(keys, c0.astype(np.float64), inputs.TAU, inputs.ITERS)
    gw_ref, gc_ref = dense.backward(keys, ref, g.astype(np.float64))
    lut = ref["c_out"].astype(np.float32)
    say("palettize mid-step")
    plan = edkm.Plan(n, bits, inputs.ITERS)
    kd = torch.from_numpy(keys.view(np.int16)).to(DEV)
    c_out = torch.empty(8, device=DEV)
    wt = torch.empty(n, device=DEV)
    edkm.init_unique(plan, kd)
    edkm.forward(plan, kd, inputs.TAU, 0.0, torch.from_numpy(c0).to(DEV), c_out, wt)
    out = torch.zeros((n * bits + 7) // 8, dtype=torch.uint8, device=DEV)
    edkm.palettize(plan, kd, torch.from_numpy(lut).to(DEV), out)
    gw = torch.empty(n, device=DEV)
    gc = torch.empty(8, device=DEV)
    edkm.backward(plan, kd, torch.from_numpy(g).to(DEV), gw, gc)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy(), palette.palettize(keys, lut, bits))
    assert_close(c_out.cpu().numpy(), ref["c_out"], TOL_FWD, "c_out")
    assert_close(gw.cpu().numpy(), gw_ref, TOL_BWD, "grad_w")
    assert_close(gc.cpu().numpy(), gc_ref, TOL_BWD, "grad_c")


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
def test_palettize_full_size(fmt):
    """The 11008x4096 MLP matrix with outliers at 3 bits."""
    w = inputs.WORKLOADS[3]
    _, r, c = w["mats"][0]
    keys = inputs.weights(r * c, inputs.weight_seed(3, 0), True, fmt)
    lut = inputs.quantile_init(keys, 8, fmt)
    say("palettize full", fmt)
    got, guard = gpu_palettize(keys, lut, 3, fmt)
    np.testing.assert_array_equal(got, palette.palettize(keys, lut, 3, fmt))
    assert np.all(guard == 0xAB)


def gpu_palettize_batch(keys_list, luts, bits_list, fmt, offsets=None):
    """edkm_palettize_batch over several matrices; offsets[i] = (key_offset,
    out_offset) places matrix i off alignment.  Returns [(packed, guard)]."""
    offsets = offsets or [(0, 0)] * len(keys_list)
    plans, kv, lv, ov, obufs, nb = [], [], [], [], [], []
    for keys, lut, bits, (ko, oo) in zip(keys_list, luts, bits_list, offsets):
        n = keys.size
        nbytes = (n * bits + 7) // 8
        kbuf = torch.zeros(n + ko, dtype=torch.int16, device=DEV)
        kbuf[ko:] = torch.from_numpy(keys.view(np.int16)).to(DEV)
        obuf = torch.full((oo + nbytes + GUARD,), 0xAB, dtype=torch.uint8, device=DEV)
        plans.append(edkm.Plan(n, bits, inputs.ITERS, key_format=fmt))
        kv.append(kbuf[ko:])
        lv.append(torch.from_numpy(np.asarray(lut, np.float32)).to(DEV))
        ov.append(obuf[oo:])
        obufs.append((obuf, oo))
        nb.append(nbytes)
    edkm.palettize_batch(plans, kv, lv, ov)
    torch.cuda.synchronize()
    out = []
    for (obuf, oo), nbytes in zip(obufs, nb):
        o = obuf.cpu().numpy()
        out.append((o[oo:oo + nbytes], o[oo + nbytes:]))
    return out


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
def test_palettize_batch_bit_exact(fmt):
    """Thirty-two matrices in four launch groups: 28 + 2 at 3 bits (cut by
    size), then one each at 2 and 4 bits (cut by bit width); ragged sizes, one
    matrix off alignment (its scalar path beside vectorised neighbours)."""
    sizes = [1, 31, 65537, 1_000_003, 33, 300_007, 16, 2_000_001] + [999 + 4099 * i for i in range(22)] + [70_000, 8]
    bits = [3] * 30 + [2, 4]
    assert edkm.LAUNCH_GROUP == 28
    offsets = [(0, 0)] * len(sizes)
    offsets[5] = (1, 1)
    keys = [inputs.weights(n, 220 + i, i % 2 == 1, fmt) for i, n in enumerate(sizes)]
    luts = [inputs.quantile_init(k, 1 << b, fmt) for k, b in zip(keys, bits)]
    say("palettize batch", fmt)
    got = gpu_palettize_batch(keys, luts, bits, fmt, offsets)
    for i, ((packed, guard), k, lut, b) in enumerate(zip(got, keys, luts, bits)):
        np.testing.assert_array_equal(packed, palette.palettize(k, lut, b, fmt), err_msg="matrix %d" % i)
        assert np.all(guard == 0xAB), i


def test_palettize_batch_layer_shapes():
    """The seven decoder-layer matrices at 3 bits in one batched call: every
    matrix's bytes equal its single-matrix call, and q_proj and gate_proj equal
    the oracle."""
    mats = inputs.WORKLOADS[4]["mats"]
    keys = [inputs.weights(r * c, inputs.weight_seed(4, i), False, "fp16") for i, (_, r, c) in enumerate(mats)]
    luts = [inputs.quantile_init(k, 8) for k in keys]
    say("palettize batch, decoder layer")
    got = gpu_palettize_batch(keys, luts, [3] * len(keys), "fp16")
    for i, (k, lut) in enumerate(zip(keys, luts)):
        single, _ = gpu_palettize(k, lut, 3, "fp16")
        np.testing.assert_array_equal(got[i][0], single, err_msg=mats[i][0])
        assert np.all(got[i][1] == 0xAB), mats[i][0]
    for i in (0, 4):
        np.testing.assert_array_equal(got[i][0], palette.palettize(keys[i], luts[i], 3), err_msg=mats[i][0])
