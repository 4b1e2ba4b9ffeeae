"""GPU parity: threshold-sparse (CATS-style) and dense FFN decode vs the fp64 oracle."""

import numpy as np
import pytest

import oracle
from synth import ffn_weights, decode_inputs, calibration_inputs, TINY, LLAMA3_8B
from gpu_util import (say, dev_bf16, dev_f32, host, check_cats_sets, check_topk_sets, check_ffn)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


def _layer(seed, d, f, std):
    wg, wu, wd = ffn_weights(seed, d, f, std)
    return (wg, wu, wd), tuple(dev_bf16(w) for w in (wg, wu, wd))


def test_tiny_config_sixteen_tokens(sr):
    """Tiny layer, batch 1, 16 decode tokens, t = q50 over 64 calibration vectors."""
    (wg, wu, wd), W = _layer(101, TINY.d_model, TINY.d_ff, TINY.weight_std)
    t = oracle.calibrate_threshold(calibration_inputs(101, 64, TINY.d_model), wg, 0.5)
    xs = decode_inputs(101, 16, TINY.d_model)
    total_b = 0
    for i in range(16):
        say(f"tiny cats token {i}")
        x = xs[i:i + 1]
        y, idx, cnt = sr.sirius_ffn_cats(dev_f32(x), *W, t)
        sets, nb = check_cats_sets(x, wg, t, host(idx), host(cnt))
        total_b += nb
        check_ffn(host(y), oracle.ffn_masked(x, wg, wu, wd, sets))
    say(f"boundary neurons excluded: {total_b} of {16 * TINY.d_ff}")
    assert total_b < 0.02 * 16 * TINY.d_ff


@pytest.mark.parametrize("d,f,bsz", [(264, 1000, 1), (264, 1000, 3), (256, 688, 16), (512, 97, 5),
                                     (4096, 33, 4), (4096, 40, 5), (8, 1, 2),
                                     (8192, 300, 2)])
def test_ragged_shapes_norm_resid(sr, d, f, bsz):
    say(f"cats ragged d={d} f={f} B={bsz}")
    (wg, wu, wd), W = _layer(200 + d + f + bsz, d, f, 1.0 / np.sqrt(d))
    x = decode_inputs(7 + bsz, bsz, d) * 3.0
    res = decode_inputs(8 + bsz, bsz, d)
    xn = oracle.rmsnorm(x, 1e-5)
    t = float(np.median(np.abs(oracle.gate_activations(xn, wg))))
    y, idx, cnt = sr.sirius_ffn_cats(dev_f32(x), *W, t, norm_eps=1e-5, resid=dev_f32(res))
    sets, _ = check_cats_sets(xn, wg, t, host(idx), host(cnt))
    check_ffn(host(y), oracle.ffn_masked(xn, wg, wu, wd, sets), resid=res)


@pytest.mark.parametrize("d,f", [(8, 1), (264, 1000), (512, 97), (1024, 3000), (2048, 4099), (4096, 33),
                                 (4096, 5000), (8192, 300)])
def test_batch1_dense_ragged_norm_resid(sr, d, f):
    """Batch-1 dense decode (every neuron kept: the gate and up rows of a neuron are read together
    for d_model <= 4096) at ragged shapes, with RMSNorm and residual, against the oracle; and
    bitwise equal to the threshold path with t < 0, which reads them in separate phases."""
    say(f"dense B=1 ragged d={d} f={f}")
    (wg, wu, wd), W = _layer(400 + d + f, d, f, 1.0 / np.sqrt(d))
    x = decode_inputs(9 + d, 1, d) * 3.0
    res = decode_inputs(10 + d, 1, d)
    xn = oracle.rmsnorm(x, 1e-5)
    yd = sr.sirius_ffn_dense(dev_f32(x), *W, norm_eps=1e-5, resid=dev_f32(res))
    check_ffn(host(yd), oracle.ffn_dense(xn, wg, wu, wd), resid=res)
    yc, idx, cnt = sr.sirius_ffn_cats(dev_f32(x), *W, -1.0, norm_eps=1e-5, resid=dev_f32(res))
    assert int(host(cnt)[0]) == f
    assert np.array_equal(host(yd), host(yc))


@pytest.mark.parametrize("bsz", [1, 2, 4, 7])
def test_negative_threshold_is_dense(sr, bsz):
    say(f"cats t<0 B={bsz}")
    (wg, wu, wd), W = _layer(300 + bsz, TINY.d_model, TINY.d_ff, TINY.weight_std)
    x = decode_inputs(300 + bsz, bsz, TINY.d_model)
    y, idx, cnt = sr.sirius_ffn_cats(dev_f32(x), *W, -1.0)
    assert np.all(host(cnt) == TINY.d_ff)
    assert np.array_equal(host(idx), np.tile(np.arange(TINY.d_ff, dtype=np.int32), (bsz, 1)))
    ref = oracle.ffn_dense(x, wg, wu, wd)
    check_ffn(host(y), ref)
    yd = sr.sirius_ffn_dense(dev_f32(x), *W)
    assert np.array_equal(host(yd), host(y))  # same kernels, same order: bitwise


@pytest.mark.parametrize("d,f,bsz,norm", [(2048, 3000, 2, False), (4096, 1000, 4, True), (6144, 777, 3, False),
                                          (2048, 14000, 4, True), (8192, 3000, 3, True)])
def test_wide_small_batches_every_mode(sr, d, f, bsz, norm):
    """At most 4 tokens with d_model a multiple of 2048 (one to four K spans; one to seven row
    tiles per segment): threshold sets and outputs, a threshold below 0 equal to the dense call
    bit for bit, the dense call against the oracle, and per-token top-k, with and without RMSNorm
    and residual."""
    say(f"wide small batch d={d} f={f} B={bsz} norm={norm}")
    (wg, wu, wd), W = _layer(1200 + d + f + bsz, d, f, 1.0 / np.sqrt(d))
    x = decode_inputs(1300 + bsz, bsz, d) * (3.0 if norm else 1.0)
    res = decode_inputs(1400 + bsz, bsz, d) if norm else None
    xn = oracle.rmsnorm(x, 1e-5) if norm else x
    kw = dict(norm_eps=1e-5, resid=dev_f32(res)) if norm else {}
    t = float(np.median(np.abs(oracle.gate_activations(xn, wg))))
    y, idx, cnt = sr.sirius_ffn_cats(dev_f32(x), *W, t, **kw)
    sets, _ = check_cats_sets(xn, wg, t, host(idx), host(cnt))
    check_ffn(host(y), oracle.ffn_masked(xn, wg, wu, wd, sets), resid=res)
    yneg, _, cneg = sr.sirius_ffn_cats(dev_f32(x), *W, -1.0, **kw)
    assert np.all(host(cneg) == f)
    yd = sr.sirius_ffn_dense(dev_f32(x), *W, **kw)
    assert np.array_equal(host(yd), host(yneg))  # same kernel, same sums: bitwise
    check_ffn(host(yd), oracle.ffn_dense(xn, wg, wu, wd), resid=res)
    k = max(1, f // 3)
    y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x), *W, k, **kw)
    sets, _ = check_topk_sets(xn, wg, k, host(idx), host(cnt))
    check_ffn(host(y), oracle.ffn_masked(xn, wg, wu, wd, sets), resid=res)


@pytest.mark.parametrize("mode,bsz", [("dense", 16), ("cats", 4), ("dense", 4), ("dense", 64)])
def test_batched_calls_under_graph_capture(sr, mode, bsz):
    """Batched calls at a width the unit kernels take (the 16-token gate/up kernel, the exact-input
    kernel of at most 4 tokens in threshold and every-neuron-kept mode, and the 64-token pass with
    its one-output-per-thread reduce) record into a HIP graph; every replay, with eager calls in
    between, equals the eager result bit for bit (kept lists included)."""
    import torch
    d, f = 2048, 3000
    (wg, wu, wd), W = _layer(1500 + bsz, d, f, 1.0 / np.sqrt(d))
    x = dev_f32(decode_inputs(1600 + bsz, bsz, d))
    res = dev_f32(decode_inputs(1700 + bsz, bsz, d))
    op = sr.OP_FFN_DENSE if mode == "dense" else sr.OP_FFN_CATS
    ws = torch.empty((int(sr.lib().sirius_workspace_size(op, bsz, d, f, 0, 0)),), dtype=torch.uint8,
                     device="cuda")
    y = torch.empty_like(x)
    idx = torch.empty((bsz, f), dtype=torch.int32, device="cuda")
    cnt = torch.empty((bsz,), dtype=torch.int32, device="cuda")
    t = 0.02

    def call():
        if mode == "dense":
            sr.sirius_ffn_dense(x, *W, norm_eps=1e-5, resid=res, y=y, ws=ws)
        else:
            sr.sirius_ffn_cats(x, *W, t, norm_eps=1e-5, resid=res, y=y, active_idx=idx, active_cnt=cnt,
                               ws=ws)

    say(f"graph capture {mode} B={bsz}")
    call()
    torch.cuda.synchronize()
    want, want_cnt = host(y).copy(), host(cnt).copy()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            call()
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        y.fill_(float("nan"))
        cnt.fill_(-1)
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host(y), want), f"replay {rep}"
        if mode == "cats":
            assert np.array_equal(host(cnt), want_cnt), f"replay {rep} counts"
        call()  # eager work between replays
        torch.cuda.synchronize()


def test_infinite_threshold_is_residual(sr):
    (wg, wu, wd), W = _layer(400, TINY.d_model, TINY.d_ff, TINY.weight_std)
    x = decode_inputs(400, 2, TINY.d_model)
    res = decode_inputs(401, 2, TINY.d_model)
    y, idx, cnt = sr.sirius_ffn_cats(dev_f32(x), *W, float("inf"), resid=dev_f32(res))
    assert np.all(host(cnt) == 0)
    assert np.array_equal(host(y), res)


def test_run_twice_bitwise_and_in_place(sr):
    (wg, wu, wd), W = _layer(500, 512, 1000, 1.0 / np.sqrt(512))
    x = decode_inputs(500, 3, 512)
    t = 0.05
    y1, i1, c1 = sr.sirius_ffn_cats(dev_f32(x), *W, t)
    y2, i2, c2 = sr.sirius_ffn_cats(dev_f32(x), *W, t)
    assert np.array_equal(host(y1), host(y2)) and np.array_equal(host(c1), host(c2))
    # in-place residual layer: h <- h + FFN(RMSNorm(h))
    h = dev_f32(x)
    y_sep, _, _ = sr.sirius_ffn_cats(dev_f32(x), *W, t, norm_eps=1e-5, resid=dev_f32(x))
    sr.sirius_ffn_cats(h, *W, t, norm_eps=1e-5, resid=h, y=h)
    assert np.array_equal(host(h), host(y_sep))


def test_llama3_8b_layer_batch1(sr):
    """Full 8B FFN shape, bf16 weights N(0, 0.02), t calibrated to 50% from 256 N(0,1) inputs."""
    say("8B cats: generating weights")
    (wg, wu, wd), W = _layer(600, LLAMA3_8B.d_model, LLAMA3_8B.d_ff, LLAMA3_8B.weight_std)
    t = oracle.calibrate_threshold(calibration_inputs(600, 256, LLAMA3_8B.d_model), wg, 0.5)
    xs = decode_inputs(600, 4, LLAMA3_8B.d_model)
    fracs = []
    for i in range(4):
        say(f"8B cats token {i}")
        x = xs[i:i + 1]
        y, idx, cnt = sr.sirius_ffn_cats(dev_f32(x), *W, t)
        sets, nb = check_cats_sets(x, wg, t, host(idx), host(cnt))
        check_ffn(host(y), oracle.ffn_masked(x, wg, wu, wd, sets))
        fracs.append(len(sets[0]) / LLAMA3_8B.d_ff)
        say(f"  kept {fracs[-1]:.3f}, boundary {nb}")
    assert 0.4 < float(np.mean(fracs)) < 0.6
    # dense path at the same shape
    say("8B dense B=1")
    y = sr.sirius_ffn_dense(dev_f32(xs[:1]), *W)
    check_ffn(host(y), oracle.ffn_dense(xs[:1], wg, wu, wd))


def test_llama3_8b_batch4_union(sr):
    say("8B cats B=4")
    (wg, wu, wd), W = _layer(601, LLAMA3_8B.d_model, LLAMA3_8B.d_ff, LLAMA3_8B.weight_std)
    x = decode_inputs(601, 4, LLAMA3_8B.d_model)
    t = float(np.median(np.abs(oracle.gate_activations(x, wg))))
    y, idx, cnt = sr.sirius_ffn_cats(dev_f32(x), *W, t)
    sets, _ = check_cats_sets(x, wg, t, host(idx), host(cnt))
    check_ffn(host(y), oracle.ffn_masked(x, wg, wu, wd, sets))


def test_calibration_matches_oracle(sr):
    for (d, f, n, q) in [(256, 688, 64, 0.5), (264, 1000, 7, 0.4), (4096, 14336, 16, 0.65)]:
        say(f"calibrate d={d} f={f} N={n} q={q}")
        wg, _, _ = ffn_weights(700 + d, d, f, 1.0 / np.sqrt(d))
        xc = calibration_inputs(700 + d, n, d)
        t_gpu = float(host(sr.sirius_cats_calibrate(dev_f32(xc), dev_bf16(wg), q))[0])
        t_ref = oracle.calibrate_threshold(xc, wg, q)
        assert abs(t_gpu - t_ref) <= 1e-5 * t_ref, (t_gpu, t_ref)


def test_kernel_timing_changes_nothing(sr):
    """With per-kernel timing on, the kernels carry the events on their own dispatches: the
    results are bitwise those of a plain launch and each kernel name records one launch with
    a positive duration."""
    (wg, wu, wd), W = _layer(107, TINY.d_model, TINY.d_ff, TINY.weight_std)
    t = oracle.calibrate_threshold(calibration_inputs(107, 64, TINY.d_model), wg, 0.5)
    x = dev_f32(decode_inputs(107, 1, TINY.d_model))
    y0, idx0, cnt0 = sr.sirius_ffn_cats(x, *W, t)
    sr.sirius_profile_reset()
    sr.sirius_profile_enable(True)
    try:
        y1, idx1, cnt1 = sr.sirius_ffn_cats(x, *W, t)
    finally:
        sr.sirius_profile_enable(False)
    for name in ("cats_decode", "cats_reduce"):
        ms, n = sr.sirius_profile_query(name)
        say(f"{name}: {n} launch, {ms * 1e3:.2f} us")
        assert n == 1 and 0.0 < ms < 100.0
    assert sr.sirius_profile_query("no_such_kernel") == (0.0, 0)
    sr.sirius_profile_reset()
    assert np.array_equal(host(y0), host(y1))
    assert np.array_equal(host(cnt0), host(cnt1))
    n0 = int(host(cnt0)[0])
    assert np.array_equal(host(idx0)[0, :n0], host(idx1)[0, :n0])
