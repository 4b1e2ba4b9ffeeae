"""GPU parity: per-token top-k sparse FFN (the paper's FSparse implementation, Sec. 3
footnote) vs the fp64 oracle."""

import numpy as np
import pytest

import oracle
from synth import ffn_weights, decode_inputs, TINY, LLAMA3_8B
from gpu_util import say, dev_bf16, dev_f32, host, check_topk_sets, check_ffn

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


def _layer(seed, d, f, std):
    wg, wu, wd = ffn_weights(seed, d, f, std)
    return (wg, wu, wd), tuple(dev_bf16(w) for w in (wg, wu, wd))


@pytest.mark.parametrize("k", [1, 172, 344, 687, 688])
def test_tiny_layer_batch_one(sr, k):
    (wg, wu, wd), W = _layer(501, TINY.d_model, TINY.d_ff, TINY.weight_std)
    xs = decode_inputs(501, 8, TINY.d_model)
    nb_total = 0
    for i in range(8):
        say(f"topk tiny k={k} token {i}")
        x = xs[i:i + 1]
        y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x), *W, k)
        sets, nb = check_topk_sets(x, wg, k, host(idx), host(cnt))
        nb_total += nb
        check_ffn(host(y), oracle.ffn_masked(x, wg, wu, wd, sets))
    say(f"  boundary neurons: {nb_total}")


@pytest.mark.parametrize("bsz", [2, 3, 8, 13])
def test_tiny_layer_batches(sr, bsz):
    (wg, wu, wd), W = _layer(600 + bsz, TINY.d_model, TINY.d_ff, TINY.weight_std)
    x = decode_inputs(600 + bsz, bsz, TINY.d_model)
    say(f"topk tiny B={bsz}")
    y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x), *W, 344)
    sets, _ = check_topk_sets(x, wg, 344, host(idx), host(cnt))
    check_ffn(host(y), oracle.ffn_masked(x, wg, wu, wd, sets))


@pytest.mark.parametrize("d,f,bsz,k", [(264, 1000, 1, 500), (264, 1000, 3, 1), (512, 97, 5, 48),
                                       (4096, 33, 1, 33), (8, 1, 2, 1), (1024, 2049, 1, 1024),
                                       (8192, 300, 2, 150), (256, 40000, 1, 20000)])
def test_ragged_shapes_norm_resid(sr, d, f, bsz, k):
    say(f"topk ragged d={d} f={f} B={bsz} k={k}")
    (wg, wu, wd), W = _layer(700 + d + f + bsz, d, f, 1.0 / np.sqrt(d))
    x = decode_inputs(9 + bsz, bsz, d) * 3.0
    res = decode_inputs(10 + bsz, bsz, d)
    xn = oracle.rmsnorm(x, 1e-5)
    y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x), *W, k, norm_eps=1e-5, resid=dev_f32(res))
    sets, _ = check_topk_sets(xn, wg, k, host(idx), host(cnt))
    check_ffn(host(y), oracle.ffn_masked(xn, wg, wu, wd, sets), resid=res)


def test_all_neurons_is_dense(sr):
    (wg, wu, wd), W = _layer(800, TINY.d_model, TINY.d_ff, TINY.weight_std)
    for bsz in (1, 4):
        x = decode_inputs(800 + bsz, bsz, TINY.d_model)
        y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x), *W, TINY.d_ff)
        assert np.array_equal(host(idx), np.tile(np.arange(TINY.d_ff, dtype=np.int32), (bsz, 1)))
        check_ffn(host(y), oracle.ffn_dense(x, wg, wu, wd))


def test_ties_keep_the_lower_index(sr):
    # repeated gate rows give equal activations: the lower neuron indices must be kept
    d, f = 64, 4000
    wg, wu, wd = ffn_weights(900, d, f, 1.0 / 8.0)
    wg = wg.copy()
    wg[1000:1100] = wg[5]  # 101 neurons with the gate of neuron 5
    W = tuple(dev_bf16(w) for w in (wg, wu, wd))
    x = decode_inputs(900, 1, d)
    a = np.abs(oracle.gate_activations(x, wg)[0])
    rank5 = int(np.sum(a > a[5]))  # neurons strictly above the tied value
    for extra in (1, 50, 101):
        k = rank5 + extra
        y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x), *W, k)
        g = set(host(idx)[0, :k].tolist())
        tied = [5] + list(range(1000, 1100))
        assert set(t for t in tied if t in g) == set(tied[:extra])
        check_ffn(host(y), oracle.ffn_masked(x, wg, wu, wd, [sorted(g)]))


def test_all_equal_activations_keep_the_first_k(sr):
    # every gate row equal: one value everywhere, so the cut falls back to the index order
    d, f = 64, 4000
    wg, wu, wd = ffn_weights(950, d, f, 1.0 / 8.0)
    wg = np.tile(wg[:1], (f, 1))
    W = tuple(dev_bf16(w) for w in (wg, wu, wd))
    x = decode_inputs(950, 1, d)
    for k in (1, 999, 3999):
        say(f"topk all-equal k={k}")
        y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x), *W, k)
        assert host(idx)[0, :k].tolist() == list(range(k)) and int(host(cnt)[0]) == k
        check_ffn(host(y), oracle.ffn_masked(x, wg, wu, wd, [np.arange(k)]))


def test_largest_layer_width(sr):
    # d_ff = 65536: the widest bin of the first digit pass holds more than can be ranked
    # directly, so a second digit pass runs
    (wg, wu, wd), W = _layer(960, 256, 65536, 1.0 / 16.0)
    x = decode_inputs(960, 2, 256)
    for bsz in (1, 2):
        say(f"topk d_ff=65536 B={bsz}")
        y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x[:bsz]), *W, 32768)
        sets, _ = check_topk_sets(x[:bsz], wg, 32768, host(idx), host(cnt))
        check_ffn(host(y), oracle.ffn_masked(x[:bsz], wg, wu, wd, sets))


def test_llama3_8b_layer_half_density(sr):
    s = LLAMA3_8B
    (wg, wu, wd), W = _layer(1000, s.d_model, s.d_ff, s.weight_std)
    xs = decode_inputs(1000, 4, s.d_model)
    for i in range(4):
        say(f"topk 8B token {i}")
        x = xs[i:i + 1]
        y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x), *W, s.d_ff // 2)
        sets, nb = check_topk_sets(x, wg, s.d_ff // 2, host(idx), host(cnt))
        check_ffn(host(y), oracle.ffn_masked(x, wg, wu, wd, sets))
    say("topk 8B B=4")
    y, idx, cnt = sr.sirius_ffn_topk(dev_f32(xs), *W, s.d_ff // 2)
    sets, _ = check_topk_sets(xs, wg, s.d_ff // 2, host(idx), host(cnt))
    check_ffn(host(y), oracle.ffn_masked(xs, wg, wu, wd, sets))


def test_repeatable_and_without_lists(sr):
    (wg, wu, wd), W = _layer(1100, TINY.d_model, TINY.d_ff, TINY.weight_std)
    x = decode_inputs(1100, 1, TINY.d_model)
    y1, _, _ = sr.sirius_ffn_topk(dev_f32(x), *W, 300)
    y2, i2, c2 = sr.sirius_ffn_topk(dev_f32(x), *W, 300, want_active=False)
    assert i2 is None and c2 is None
    assert np.array_equal(host(y1), host(y2))
