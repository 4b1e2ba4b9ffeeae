"""GPU parity: the multi-token dense FFN (batch >= 8, gate/up products on MFMA) vs the fp64 oracle.

This path is the full model's parallel pass over a drafted chunk (the chunk of
tokens the full model checks at once). The gate and up products take the
normalised input rounded to bf16, so the precision-matched reference is the
oracle's dense FFN on that rounded input: the MFMA products are exact and
accumulate in fp32, and h enters the down product as a bf16 pair (hi + lo,
relative error below 2^-17), so the fp32-path tolerance applies to it. Against
the unrounded input the stated bound of the method holds as well.
"""

import numpy as np
import pytest

import oracle
from synth import ffn_weights, decode_inputs, griffin_prompt, TINY, LLAMA3_8B
from gpu_util import (say, dev_bf16, dev_f32, host, check_ffn, check_ffn_rounded_norm, rel_err,
                      rounded_bf16, FP32_PATH_TOL, METHOD_TOL)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


def _layer(seed, d, f, std):
    wg, wu, wd = ffn_weights(seed, d, f, std)
    return (wg, wu, wd), tuple(dev_bf16(w) for w in (wg, wu, wd))


@pytest.mark.parametrize("d,f,bsz", [(256, 688, 8), (264, 1000, 9), (256, 688, 16), (512, 97, 17),
                                     (4096, 40, 33), (8, 1, 8), (264, 1000, 64), (520, 33, 48),
                                     (8192, 100, 16),
                                     # one 16-token tile with d_model % 128 == 0: the LDS-ring gate/up
                                     # kernel (ragged d_ff, partial last segments, a single K block)
                                     (1024, 5000, 16), (4096, 14000, 13), (128, 8, 8), (256, 1000, 10),
                                     (4096, 40, 16),
                                     # d_model a multiple of 2048 and at most 16 tokens: the gate/up
                                     # kernel on 16-row x 2048-column units (one, three and four K
                                     # spans, one and seven tiles per segment, rows past d_ff)
                                     (2048, 3000, 8), (6144, 777, 11), (2048, 90, 9), (8192, 3000, 16)])
def test_ragged_batches(sr, d, f, bsz):
    say(f"dense mfma d={d} f={f} B={bsz}")
    (wg, wu, wd), W = _layer(500 + d + f + bsz, d, f, 1.0 / np.sqrt(d))
    x = decode_inputs(40 + bsz, bsz, d)
    y = host(sr.sirius_ffn_dense(dev_f32(x), *W))
    check_ffn(y, oracle.ffn_dense(rounded_bf16(x), wg, wu, wd), tol=FP32_PATH_TOL)
    e = rel_err(y, oracle.ffn_dense(x, wg, wu, wd))
    say(f"  error vs unrounded input: {e:.2e} x RMS")
    assert e <= METHOD_TOL


@pytest.mark.parametrize("bsz", [8, 24])
def test_norm_and_residual(sr, bsz):
    d, f = 264, 1000
    say(f"dense mfma norm+resid B={bsz}")
    (wg, wu, wd), W = _layer(600 + bsz, d, f, 1.0 / np.sqrt(d))
    x = decode_inputs(60 + bsz, bsz, d) * 3.0
    res = decode_inputs(61 + bsz, bsz, d)
    y = host(sr.sirius_ffn_dense(dev_f32(x), *W, norm_eps=1e-5, resid=dev_f32(res)))
    xn = oracle.rmsnorm(x, 1e-5)
    e, nb = check_ffn_rounded_norm(y, xn, wg, wu, wd, resid=res)
    say(f"  error {e:.2e} x RMS, {nb} inputs with ambiguous rounding")
    assert rel_err(y - res, oracle.ffn_dense(xn, wg, wu, wd)) <= METHOD_TOL


def test_run_twice_bitwise_and_in_place(sr):
    import torch
    d, f, bsz = TINY.d_model, TINY.d_ff, 16
    (wg, wu, wd), W = _layer(700, d, f, TINY.weight_std)
    x = decode_inputs(700, bsz, d)
    a = host(sr.sirius_ffn_dense(dev_f32(x), *W, norm_eps=1e-5, resid=dev_f32(x)))
    b = host(sr.sirius_ffn_dense(dev_f32(x), *W, norm_eps=1e-5, resid=dev_f32(x)))
    assert np.array_equal(a, b)
    h = dev_f32(x)
    sr.sirius_ffn_dense(h, *W, norm_eps=1e-5, resid=h, y=h)  # residual layer in place
    torch.cuda.synchronize()
    assert np.array_equal(host(h), a)


def test_condensed_batch(sr):
    """Condensed decode of 12 tokens equals the FFN restricted to the selected neurons."""
    d, f, k, bsz = 256, 688, 300, 12
    say(f"condensed mfma B={bsz}")
    (wg, wu, wd), W = _layer(800, d, f, TINY.weight_std)
    sel, _, wgc, wuc, wdc = sr.sirius_griffin_select(dev_bf16(griffin_prompt(800, 32, d)), *W, k)
    sel = host(sel).astype(np.int64)
    x = decode_inputs(800, bsz, d)
    y = host(sr.sirius_ffn_condensed(dev_f32(x), wgc, wuc, wdc))
    check_ffn(y, oracle.ffn_masked(rounded_bf16(x), wg, wu, wd, [sel] * bsz), tol=FP32_PATH_TOL)


def test_llama3_8b_verify_chunk(sr):
    """The full model's 16-token pass over one Llama-3-8B-shaped FFN layer."""
    d, f, bsz = LLAMA3_8B.d_model, LLAMA3_8B.d_ff, 16
    say("8B dense mfma B=16")
    (wg, wu, wd), W = _layer(900, d, f, LLAMA3_8B.weight_std)
    x = decode_inputs(900, bsz, d)
    res = decode_inputs(901, bsz, d)
    y = host(sr.sirius_ffn_dense(dev_f32(x), *W, norm_eps=1e-5, resid=dev_f32(res)))
    xn = oracle.rmsnorm(x, 1e-5)
    e, nb = check_ffn_rounded_norm(y, xn, wg, wu, wd, resid=res)
    say(f"  error vs precision-matched oracle: {e:.2e} x RMS ({nb} inputs with ambiguous rounding)")
    assert rel_err(y - res, oracle.ffn_dense(xn, wg, wu, wd)) <= METHOD_TOL


@pytest.mark.parametrize("bsz", [64, 40])
def test_llama3_8b_tree_pass(sr, bsz):
    """The full model's pass over a drafted tree of about 64 nodes (kernel size 16 x width 4, the
    paper's hardware-friendly tree) on one Llama-3-8B-shaped FFN layer, with RMSNorm and residual:
    four (or a ragged two and a half) 16-token MFMA tiles over the full 4096 x 14336 layer."""
    d, f = LLAMA3_8B.d_model, LLAMA3_8B.d_ff
    say(f"8B dense mfma B={bsz}")
    (wg, wu, wd), W = _layer(910 + bsz, d, f, LLAMA3_8B.weight_std)
    x = decode_inputs(910 + bsz, bsz, d)
    res = decode_inputs(911 + bsz, bsz, d)
    y = host(sr.sirius_ffn_dense(dev_f32(x), *W, norm_eps=1e-5, resid=dev_f32(res)))
    xn = oracle.rmsnorm(x, 1e-5)
    e, nb = check_ffn_rounded_norm(y, xn, wg, wu, wd, resid=res)
    say(f"  error vs precision-matched oracle: {e:.2e} x RMS ({nb} inputs with ambiguous rounding)")
    assert rel_err(y - res, oracle.ffn_dense(xn, wg, wu, wd)) <= METHOD_TOL


@pytest.mark.parametrize("d,f", [(256, 1000), (256, 97), (512, 3100), (2048, 1000)])
@pytest.mark.parametrize("bsz,mode", [(4, "dense"), (16, "dense"), (64, "dense"), (16, "cats")])
def test_segment_tail_on_dirty_workspace(sr, d, f, bsz, mode):
    """Batched calls whose segment layout ends inside a 64-position down block (250 segments of
    16 positions at d_ff = 1000, 25 at 97, 194 at 3100): the positions past the last segment must
    read h = 0 whatever the workspace held. The workspace is filled with 0xFF bytes (NaN as bf16
    and fp32) before the call."""
    import torch
    say(f"segment tail d={d} f={f} B={bsz} {mode}")
    (wg, wu, wd), W = _layer(800 + d + f + bsz, d, f, 1.0 / np.sqrt(d))
    x = decode_inputs(80 + bsz, bsz, d)
    op = sr.OP_FFN_DENSE if mode == "dense" else sr.OP_FFN_CATS
    n = int(sr.lib().sirius_workspace_size(op, bsz, d, f, 0, 0))
    ws = torch.full((n,), 255, dtype=torch.uint8, device="cuda")
    if mode == "dense":
        y = host(sr.sirius_ffn_dense(dev_f32(x), *W, ws=ws))
    else:  # t < 0 keeps every neuron: the dense FFN on the exact input
        y = host(sr.sirius_ffn_cats(dev_f32(x), *W, -1.0, want_active=False, ws=ws)[0])
    assert np.all(np.isfinite(y))
    x_ref = rounded_bf16(x) if (mode == "dense" and bsz >= 8) else x
    check_ffn(y, oracle.ffn_dense(x_ref, wg, wu, wd), tol=FP32_PATH_TOL)
