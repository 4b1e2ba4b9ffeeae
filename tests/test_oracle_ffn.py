"""Pins of the FFN oracle (dense, threshold sparsity, calibration, RMSNorm stack).

None of these tests compares the oracle with itself: each checks it against a
hand-computed value, a brute-force scalar loop, an independent library
(PyTorch float64), or an invariant that a dropped term, a wrong sign, a
wrong index or a transposed operand would break.
"""

import math

import numpy as np
import pytest

import oracle
from synth import bf16_bits, ffn_weights, decode_inputs, calibration_inputs, TINY


def _brute_ffn(x, wg, wu, wd, active=None):
    """Scalar triple loop with math.exp (no numpy arithmetic)."""
    d = len(x)
    f = len(wg)
    y = [0.0] * d
    for i in range(f):
        if active is not None and i not in active:
            continue
        g = sum(float(wg[i][k]) * float(x[k]) for k in range(d))
        u = sum(float(wu[i][k]) * float(x[k]) for k in range(d))
        a = g / (1.0 + math.exp(-g))
        h = a * u
        for c in range(d):
            y[c] += h * float(wd[i][c])
    return y


def _small(seed, b, d, f):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((b, d))
    wg, wu, wd = (rng.standard_normal((f, d)) / math.sqrt(d) for _ in range(3))
    return x, wg, wu, wd


def test_hand_case_single_neuron():
    # x = (1, 0); gate row (ln 3, 0) -> g = ln 3, sigmoid(ln 3) = 3/4,
    # SiLU = 0.75 ln 3; up row (2, 5) -> u = 2; h = 1.5 ln 3; down row (1, -1).
    x = np.array([[1.0, 0.0]])
    wg = np.array([[math.log(3.0), 0.0]])
    wu = np.array([[2.0, 5.0]])
    wd = np.array([[1.0, -1.0]])
    y = oracle.ffn_dense(x, wg, wu, wd)
    h = 1.5 * math.log(3.0)
    np.testing.assert_allclose(y, [[h, -h]], rtol=1e-15, atol=0)


def test_hand_case_threshold_two_neurons():
    # Neuron 0: g = ln 3 -> a = 0.75 ln 3 = 0.824; neuron 1: g = -ln 3 -> a = -0.25 ln 3 = -0.275.
    x = np.array([[1.0, 0.0]])
    wg = np.array([[math.log(3.0), 0.0], [-math.log(3.0), 0.0]])
    wu = np.array([[1.0, 0.0], [1.0, 0.0]])
    wd = np.array([[1.0, 0.0], [0.0, 1.0]])
    for t, want_set, want_y in [
        (0.5, [0], [0.75 * math.log(3.0), 0.0]),
        (0.2, [0, 1], [0.75 * math.log(3.0), -0.25 * math.log(3.0)]),
        (0.9, [], [0.0, 0.0]),
    ]:
        y, sets = oracle.ffn_cats(x, wg, wu, wd, t)
        assert sets[0].tolist() == want_set
        np.testing.assert_allclose(y[0], want_y, rtol=1e-15, atol=1e-300)


def test_silu_identities():
    z = np.linspace(-30, 30, 601)
    s = oracle.silu(z)
    # SiLU(z) - SiLU(-z) = z and SiLU(0) = 0, SiLU(z) -> z for large z, -> 0 for very negative z.
    np.testing.assert_allclose(s - oracle.silu(-z), z, atol=1e-12)
    assert oracle.silu(np.array([0.0]))[0] == 0.0
    assert abs(oracle.silu(np.array([40.0]))[0] - 40.0) < 1e-12
    assert abs(oracle.silu(np.array([-800.0]))[0]) < 1e-300


def test_dense_matches_bruteforce_loops():
    x, wg, wu, wd = _small(1, 2, 8, 12)
    y = oracle.ffn_dense(x, wg, wu, wd)
    for b in range(2):
        np.testing.assert_allclose(y[b], _brute_ffn(x[b], wg, wu, wd), rtol=1e-12, atol=1e-14)


def test_dense_matches_torch_float64_on_tiny_layer():
    torch = pytest.importorskip("torch")
    wg, wu, wd = ffn_weights(3, TINY.d_model, TINY.d_ff, TINY.weight_std)
    x = decode_inputs(3, 4, TINY.d_model)
    y = oracle.ffn_dense(x, wg, wu, wd)

    def tw(bits):
        return torch.from_numpy(bits.astype(np.int16)).view(torch.bfloat16).to(torch.float64)

    xt = torch.from_numpy(x).to(torch.float64)
    g = torch.nn.functional.linear(xt, tw(wg))
    u = torch.nn.functional.linear(xt, tw(wu))
    ref = torch.nn.functional.linear(torch.nn.functional.silu(g) * u, tw(wd).T.contiguous())
    np.testing.assert_allclose(y, ref.numpy(), rtol=1e-10, atol=1e-12)


def test_widen_bf16_exact():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    a = (rng.standard_normal(10000) * 10.0).astype(np.float32)
    bits = bf16_bits(a)
    via_torch = torch.from_numpy(bits.astype(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.widen_bf16(bits), via_torch)


def test_neuron_permutation_invariance():
    x, wg, wu, wd = _small(2, 3, 16, 40)
    perm = np.random.default_rng(0).permutation(40)
    y = oracle.ffn_dense(x, wg, wu, wd)
    yp = oracle.ffn_dense(x, wg[perm], wu[perm], wd[perm])
    np.testing.assert_allclose(y, yp, rtol=1e-12, atol=1e-14)
    # Permuting only the down rows must change the result (catches a down/up index mix-up).
    yq = oracle.ffn_dense(x, wg, wu, wd[perm])
    assert np.max(np.abs(y - yq)) > 1e-3


def test_linearity_and_sign():
    x, wg, wu, wd = _small(4, 2, 16, 24)
    y = oracle.ffn_dense(x, wg, wu, wd)
    np.testing.assert_allclose(oracle.ffn_dense(x, wg, wu, 2.0 * wd), 2.0 * y, rtol=1e-13)
    np.testing.assert_allclose(oracle.ffn_dense(x, wg, -wu, wd), -y, rtol=1e-13)
    # Flipping the gate is NOT a sign flip (SiLU is not odd): catches a dropped sigmoid.
    assert np.max(np.abs(oracle.ffn_dense(x, -wg, wu, wd) + y)) > 1e-3


def test_cats_negative_threshold_is_dense_bitwise():
    wg, wu, wd = ffn_weights(7, TINY.d_model, TINY.d_ff, TINY.weight_std)
    x = decode_inputs(7, 3, TINY.d_model)
    y, sets = oracle.ffn_cats(x, wg, wu, wd, -1.0)
    assert all(len(s) == TINY.d_ff for s in sets)
    np.testing.assert_array_equal(y, oracle.ffn_dense(x, wg, wu, wd))


def test_cats_infinite_threshold_is_zero():
    wg, wu, wd = ffn_weights(7, TINY.d_model, TINY.d_ff, TINY.weight_std)
    x = decode_inputs(8, 2, TINY.d_model)
    y, sets = oracle.ffn_cats(x, wg, wu, wd, float("inf"))
    assert all(len(s) == 0 for s in sets)
    assert np.all(y == 0.0)


def test_cats_sets_match_bruteforce_threshold_and_sort():
    x, wg, wu, wd = _small(9, 2, 12, 30)
    t = 0.15
    sets, _ = oracle.cats_active_sets(x, wg, t)
    for b in range(2):
        brute = []
        for i in range(30):
            g = sum(float(wg[i][k]) * float(x[b][k]) for k in range(12))
            a = g / (1.0 + math.exp(-g))
            if abs(a) > t:
                brute.append(i)
        assert sorted(brute) == sets[b].tolist()
        y_b = oracle.ffn_masked(x[b:b + 1], wg, wu, wd, [sets[b]])[0]
        np.testing.assert_allclose(y_b, _brute_ffn(x[b], wg, wu, wd, set(brute)), rtol=1e-12, atol=1e-14)


def test_cats_sets_nested_in_threshold():
    wg, wu, wd = ffn_weights(11, TINY.d_model, TINY.d_ff, TINY.weight_std)
    x = decode_inputs(11, 2, TINY.d_model)
    prev = None
    for t in [0.0, 0.05, 0.1, 0.2, 0.4, 0.8]:
        sets, _ = oracle.cats_active_sets(x, wg, t)
        if prev is not None:
            for b in range(2):
                assert set(sets[b].tolist()) <= set(prev[b].tolist())
        prev = sets


def test_calibration_nearest_rank_count():
    wg, _, _ = ffn_weights(12, TINY.d_model, TINY.d_ff, TINY.weight_std)
    xc = calibration_inputs(12, 64, TINY.d_model)
    a = np.abs(oracle.gate_activations(xc, wg)).ravel()
    m = a.size
    assert np.unique(a).size == m  # no ties on this draw
    for q in [0.4, 0.5, 0.65]:
        t = oracle.calibrate_threshold(xc, wg, q)
        assert int(np.sum(a > t)) == m - math.ceil(q * m)
        assert int(np.sum(a <= t)) == math.ceil(q * m)


def test_masked_ffn_drops_exactly_the_unselected_neurons():
    x, wg, wu, wd = _small(13, 1, 10, 20)
    keep = [1, 4, 5, 19]
    y = oracle.ffn_masked(x, wg, wu, wd, [np.array(keep)])
    np.testing.assert_allclose(y[0], _brute_ffn(x[0], wg, wu, wd, set(keep)), rtol=1e-12, atol=1e-14)
    # Equivalent to the dense FFN of the kept rows (row gather).
    y2 = oracle.ffn_dense(x, wg[keep], wu[keep], wd[keep])
    np.testing.assert_allclose(y, y2, rtol=1e-12, atol=1e-14)


def test_rmsnorm_closed_form_and_torch():
    h = np.array([[3.0, 4.0]])
    np.testing.assert_allclose(oracle.rmsnorm(h, 1e-5), h / math.sqrt(12.5 + 1e-5), rtol=1e-15)
    c = np.full((1, 64), -7.5)
    np.testing.assert_allclose(oracle.rmsnorm(c, 0.0), -np.ones((1, 64)), rtol=1e-15)
    torch = pytest.importorskip("torch")
    r = np.random.default_rng(14).standard_normal((3, 128))
    ref = torch.nn.functional.rms_norm(torch.from_numpy(r), (128,), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(r, 1e-5), ref, rtol=1e-12)


def test_stack_layer_is_residual_plus_ffn_of_norm():
    x, wg, wu, wd = _small(15, 2, 16, 24)
    out = oracle.stack_layer(x, lambda z: oracle.ffn_dense(z, wg, wu, wd))
    # With a zero down projection the layer is the identity (residual path only).
    ident = oracle.stack_layer(x, lambda z: oracle.ffn_dense(z, wg, wu, 0.0 * wd))
    np.testing.assert_array_equal(ident, x)
    # Brute force: normalise by hand, then the scalar FFN loop.
    for b in range(2):
        rms = math.sqrt(sum(v * v for v in x[b]) / 16 + 1e-5)
        xn = [v / rms for v in x[b]]
        want = [x[b][c] + v for c, v in enumerate(_brute_ffn(xn, wg, wu, wd))]
        np.testing.assert_allclose(out[b], want, rtol=1e-12, atol=1e-13)


def test_threshold_is_strict():
    # A neuron with gate pre-activation 0 has SiLU = 0 exactly; at t = 0 it must be dropped,
    # and every neuron with a nonzero activation kept.
    x = np.array([[1.0, 0.0]])
    wg = np.array([[0.0, 0.0], [math.log(3.0), 0.0], [0.0, 5.0]])
    sets, a = oracle.cats_active_sets(x, wg, 0.0)
    assert a[0, 0] == 0.0 and a[0, 2] == 0.0
    assert sets[0].tolist() == [1]
    # At t equal to the exact activation of neuron 1, neuron 1 is dropped too.
    sets, _ = oracle.cats_active_sets(x, wg, float(a[0, 1]))
    assert sets[0].tolist() == []
