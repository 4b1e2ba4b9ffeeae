"""GPU parity: RMSNorm, the bf16 normal fill, and a small FFN-only layer stack."""

import numpy as np
import pytest

import oracle
from synth import ffn_weights, decode_inputs, calibration_inputs
from gpu_util import say, dev_bf16, dev_f32, host, check_cats_sets, check_ffn

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


@pytest.mark.parametrize("bsz,d", [(1, 4096), (3, 264), (16, 8192), (2, 1), (2, 1001)])
def test_rmsnorm(sr, bsz, d):
    h = decode_inputs(bsz + d, bsz, d) * 5.0
    out = host(sr.sirius_rmsnorm(dev_f32(h), 1e-5))
    np.testing.assert_allclose(out, oracle.rmsnorm(h, 1e-5), rtol=2e-6, atol=1e-7)


def test_fill_normal_is_seeded_and_normal(sr):
    import torch
    a = torch.empty(1 << 20, dtype=torch.bfloat16, device="cuda")
    b = torch.empty(1000, dtype=torch.bfloat16, device="cuda")
    sr.sirius_fill_normal_bf16(a, 42, 0.0, 0.02)
    sr.sirius_fill_normal_bf16(b, 42, 0.0, 0.02)
    ha, hb = host(a), host(b)
    assert np.array_equal(ha[:1000], hb)  # element e depends only on (seed, e)
    v = oracle.widen_bf16(ha)
    assert abs(v.mean()) < 1e-4 and abs(v.std() - 0.02) < 2e-4
    c = torch.empty(1 << 20, dtype=torch.bfloat16, device="cuda")
    sr.sirius_fill_normal_bf16(c, 43, 0.0, 0.02)
    assert not np.array_equal(host(c), ha)
    # tail fraction beyond 3 sigma is that of a normal (0.27%)
    frac = float(np.mean(np.abs(v) > 0.06))
    assert 0.0020 < frac < 0.0034


def test_four_layer_cats_stack_per_layer_parity(sr):
    d, f, nl = 256, 688, 4
    layers = [ffn_weights(900 + l, d, f, 1 / 16) for l in range(nl)]
    dev_layers = [[dev_bf16(w) for w in ws] for ws in layers]
    ts = [oracle.calibrate_threshold(calibration_inputs(900 + l, 64, d), layers[l][0], 0.5) for l in range(nl)]
    h = dev_f32(decode_inputs(900, 2, d))
    for l in range(nl):
        say(f"stack layer {l}")
        h_in = host(h).copy()
        sr.sirius_ffn_cats(h, *dev_layers[l], ts[l], norm_eps=1e-5, resid=h, y=h, want_active=False)
        # the library's own active sets (second call, same input) define the masked reference
        _, idx, cnt = sr.sirius_ffn_cats(dev_f32(h_in), *dev_layers[l], ts[l], norm_eps=1e-5)
        xn = oracle.rmsnorm(h_in, 1e-5)
        sets, _ = check_cats_sets(xn, layers[l][0], ts[l], host(idx), host(cnt))
        wg, wu, wd = layers[l]
        check_ffn(host(h), oracle.ffn_masked(xn, wg, wu, wd, sets), resid=h_in)
