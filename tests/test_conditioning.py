"""The conditioning-aware comparison used where a case is ill-conditioned at
fp32 resolution (tests/parity_util.py: iterate_sensitivity,
assert_close_conditioned), checked on the CPU against the oracle alone.

The DKM iteration of Sec. 2 forms each C^(t) as P/S; an fp32 implementation
rounds every iterate.  Where a softmax boundary between far-apart centroids
falls next to occupied patterns, that rounding alone moves the exact
gradients of those patterns by a sizable fraction of themselves."""
import numpy as np

from oracle import table
from paper_2309_00964_amd import inputs
from parity_util import TOL_BWD, assert_close_conditioned, iterate_sensitivity, rel_errors


def _wide():
    """The GPU parity test's wide-span case (test_wide_magnitude_span_exceeds_windows)."""
    n = 150_000
    rng = np.random.default_rng(61)
    logs = rng.uniform(-24, 15.9, n)
    vals = np.sign(rng.standard_normal(n)) * np.exp2(logs)
    keys = vals.astype(np.float16).view(np.uint16)
    keys[: n // 2] = inputs.fp16_weights(n // 2, 62)
    return keys


def _rel(d, ref):
    ref = np.asarray(ref, np.float64)
    return d / (np.abs(ref) + np.median(np.abs(ref)))


def test_gaussian_weights_are_well_conditioned():
    """Gaussian fp16 weights: rounding the iterates moves the oracle's
    gradients by far less than the parity tolerance, so the conditioned
    comparison is the plain one there."""
    keys = inputs.fp16_weights(20_000, 5)
    c0 = inputs.quantile_init(keys, 8)
    g = inputs.upstream_grad(keys.size, 6)
    f = table.forward(keys, c0.astype(np.float64), inputs.TAU, inputs.ITERS)
    gw, gc, _ = table.backward(keys, f, g.astype(np.float64))
    dwt, dgw, dgc = iterate_sensitivity(keys, c0, g, inputs.TAU, inputs.ITERS)
    assert np.max(_rel(dgw, gw)) < 1e-2 * TOL_BWD
    assert np.max(_rel(dgc, gc)) < 1e-2 * TOL_BWD
    assert np.max(_rel(dwt, f["w_tilde"])) < 1e-6


def test_wide_span_is_ill_conditioned_and_planted_errors_still_fail():
    """The wide-span case: some gradients move by more than a tenth of the
    tolerance under one-ulp rounding of the iterates (the reason for the
    conditioned comparison).  A 1% error planted on a well-conditioned element
    still fails it, and so does a 1e-3 rel-L2 shift of the whole vector."""
    keys = _wide()
    c0 = inputs.quantile_init(keys, 8)
    g = inputs.upstream_grad(keys.size, 63)
    f = table.forward(keys, c0.astype(np.float64), inputs.TAU, inputs.ITERS)
    gw, gc, _ = table.backward(keys, f, g.astype(np.float64))
    _, dgw, _ = iterate_sensitivity(keys, c0, g, inputs.TAU, inputs.ITERS)
    r = _rel(dgw, gw)
    assert np.max(r) > 0.1 * TOL_BWD
    assert_close_conditioned(gw, gw, dgw, TOL_BWD, "exact")
    i = int(np.argmin(r + (np.abs(gw) < np.median(np.abs(gw)))))   # well conditioned, not tiny
    bad = gw.copy()
    bad[i] *= 1.01
    try:
        assert_close_conditioned(bad, gw, dgw, TOL_BWD, "planted")
    except AssertionError:
        pass
    else:
        raise AssertionError("a 1% error on a well-conditioned element passed")
    shifted = gw * (1 + 2e-3)
    assert rel_errors(shifted, gw)[0] > TOL_BWD
    try:
        assert_close_conditioned(shifted, gw, dgw, TOL_BWD, "shifted")
    except AssertionError:
        pass
    else:
        raise AssertionError("a 2e-3 relative shift passed")


def test_bf16_bar_near_zero_crossing():
    """The bf16 W~ bar (parity_util.assert_bf16_within_ulp with tol): a value
    next to a zero crossing of W~ that is off by about 1e-8 of the centroid
    scale (fp32 arithmetic) passes through the fp32 floor, while an entry of
    ordinary size two bf16 ulps away still fails, floor or not."""
    import pytest
    from parity_util import TOL_FWD, _bf16_bits, _bf16_values, assert_bf16_within_ulp
    ref = np.array([-3.12000202627e-09, 0.0213, -0.0375, 0.0042])
    near = ref.copy()
    near[0] = -3.49245965e-09                 # 3.7e-10 away: many bf16 ulps of 3e-9
    bits = _bf16_bits(near.astype(np.float32))
    with pytest.raises(AssertionError):
        assert_bf16_within_ulp(bits, ref)
    assert_bf16_within_ulp(bits, ref, tol=TOL_FWD)
    far = _bf16_bits(ref.astype(np.float32))
    far[1] += np.uint16(2)                    # two ulps of 0.0213: about 2.4e-4
    assert abs(_bf16_values(far[1:2])[0] - ref[1]) > TOL_FWD * (abs(ref[1]) + np.median(np.abs(ref)))
    with pytest.raises(AssertionError):
        assert_bf16_within_ulp(far, ref, tol=TOL_FWD)
