"""The seeded generators are deterministic, correctly shaped and round to bf16 correctly."""

import numpy as np
import pytest

import synth


def test_determinism_and_streams():
    a = synth.ffn_weights(1, 64, 48, 0.02)
    b = synth.ffn_weights(1, 64, 48, 0.02)
    c = synth.ffn_weights(2, 64, 48, 0.02)
    for u, v in zip(a, b):
        assert u.dtype == np.uint16 and u.shape == (48, 64)
        np.testing.assert_array_equal(u, v)
    assert not np.array_equal(a[0], c[0])
    assert not np.array_equal(a[0], a[1])
    x1 = synth.decode_inputs(1, 3, 64)
    x2 = synth.calibration_inputs(1, 3, 64)
    assert x1.dtype == np.float32 and not np.array_equal(x1, x2)


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    a = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    want = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    np.testing.assert_array_equal(synth.bf16_bits(a), want)


def test_verify_generator_shapes_and_boost():
    lg, dr = synth.verify_inputs(3, 2, 4, 100, 2.0, rows=5)
    assert lg.shape == (2, 5, 100) and lg.dtype == np.float32
    assert dr.shape == (2, 4) and dr.dtype == np.int32
    assert dr.min() >= 0 and dr.max() < 100
    lg2, dr2 = synth.verify_inputs(3, 2, 4, 100, 2.0, rows=5, calibrated=True)
    np.testing.assert_array_equal(dr, dr2)
    for b in range(2):
        for j in range(4):
            assert lg2[b, j, dr2[b, j]] == lg2[b, j].max()


def test_attention_generator_shapes_and_types():
    from synth import attn_inputs
    q, kn, vn, kc, vc = attn_inputs(3, 2, 4, 8, 2, 16, 50)
    assert q.shape == (2, 4, 8, 16) and q.dtype == np.float32
    assert kn.shape == vn.shape == (2, 4, 2, 16) and kn.dtype == np.uint16
    assert kc.shape == vc.shape == (2, 50, 2, 16) and kc.dtype == np.uint16
    q2, *_ = attn_inputs(3, 2, 4, 8, 2, 16, 50)
    assert np.array_equal(q, q2)
