"""Pins of the palettization oracle (oracle/palette.py): the packing against a
worked example and a round trip, the nearest-entry rule against a brute-force
loop in fp32 scalars, ties and non-finite weights."""
import numpy as np
import pytest

from oracle import palette
from paper_2309_00964_amd import inputs


def test_packing_worked_example():
    # b = 3: 5 = 101b and 3 = 011b, least significant bit first: stream 1,0,1, 1,1,0
    # -> byte 0b00011101 = 0x1D; b = 4: 0xA, 0x3 -> 0x3A
    np.testing.assert_array_equal(palette.pack(np.array([5, 3]), 3), [0x1D])
    np.testing.assert_array_equal(palette.pack(np.array([0xA, 0x3]), 4), [0x3A])
    # b = 1: eight indices fill one byte, the ninth starts the next
    np.testing.assert_array_equal(palette.pack(np.array([1, 0, 0, 0, 0, 0, 0, 1, 1]), 1), [0x81, 0x01])
    # b = 2: 3, 2, 1, 0 -> 11 01 10 00 read from the top = 0b00011011
    np.testing.assert_array_equal(palette.pack(np.array([3, 2, 1, 0]), 2), [0x1B])


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
@pytest.mark.parametrize("n", [1, 7, 8, 31, 33, 1000])
def test_pack_round_trip_and_size(bits, n):
    idx = np.random.default_rng(bits * 100 + n).integers(0, 1 << bits, n).astype(np.uint8)
    p = palette.pack(idx, bits)
    assert p.size == (n * bits + 7) // 8
    np.testing.assert_array_equal(palette.unpack(p, n, bits), idx)


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
def test_nearest_entry_matches_brute_force(fmt):
    keys = inputs.weights(3000, 7, True, fmt)
    lut = inputs.quantile_init(keys, 8, fmt) + np.float32(1e-4)
    got = palette.indices(keys, lut, fmt)
    vals = palette.values32(keys, fmt)
    for i in range(keys.size):
        best, bd = 0, abs(np.float32(vals[i]) - np.float32(lut[0]))
        for j in range(1, lut.size):
            d = abs(np.float32(vals[i]) - np.float32(lut[j]))
            if d < bd:
                best, bd = j, d
        assert got[i] == best


def test_ties_take_the_lowest_entry_and_nonfinite_get_zero():
    keys = np.array([0.5, 0.25, np.inf, np.nan, -np.inf], dtype=np.float16).view(np.uint16)
    lut = np.array([0.25, 0.75, 0.25], np.float32)     # 0.5 is equidistant from entries 0 and 1
    np.testing.assert_array_equal(palette.indices(keys, lut), [0, 0, 0, 0, 0])
    lut = np.array([0.75, 0.25], np.float32)
    np.testing.assert_array_equal(palette.indices(keys, lut), [0, 1, 0, 0, 0])


def test_nearest_final_centroid_versus_largest_final_attention():
    """The two readings of the export rule (the paper names the artefact, a
    table of centroids plus an index per weight, but not how a weight picks
    its entry).  This library takes the entry of the given table nearest to
    the weight; passing C^(T) as the table gives the nearest final centroid.
    The other reading, the largest entry of the weight's final attention row
    A^(T), is the nearest entry of C^(T-1), since A^(T) is built from C^(T-1)
    and softmax(-|v - c| / tau) decreases with the distance.  The two differ
    exactly on weights whose nearest centroid changes in the last update:
    about 3% of the config-1 weights after five iterations."""
    from oracle import table
    keys = inputs.fp16_weights(65536, inputs.weight_seed(1, 0))
    c0 = inputs.quantile_init(keys, 8)
    f = table.forward(keys, c0, 2e-3, 5)
    T = f["T"]
    v = keys.view(np.float16).astype(np.float64)
    d = -np.abs(v[:, None] - f["c_hist"][T - 1][None, :]) / 2e-3
    a = np.exp(d - d.max(axis=1, keepdims=True))
    a /= a.sum(axis=1, keepdims=True)
    largest = np.argmax(a, axis=1)
    prev = palette.indices(keys, f["c_hist"][T - 1].astype(np.float32))
    final = palette.indices(keys, f["c_hist"][T].astype(np.float32))
    np.testing.assert_array_equal(largest, prev)
    differ = final != largest
    assert 0.005 < differ.mean() < 0.1
    # where they differ, the weight lies between the old and the new midpoint
    # of two neighbouring centroids
    for c in (f["c_hist"][T - 1], f["c_hist"][T]):
        assert np.all(np.diff(c) > 0)
    m_old = (f["c_hist"][T - 1][1:] + f["c_hist"][T - 1][:-1]) / 2
    m_new = (f["c_hist"][T][1:] + f["c_hist"][T][:-1]) / 2
    lo, hi = np.minimum(m_old, m_new), np.maximum(m_old, m_new)
    between = np.any((v[:, None] >= lo[None, :] - 1e-7) & (v[:, None] <= hi[None, :] + 1e-7), axis=1)
    assert np.all(between[differ])
