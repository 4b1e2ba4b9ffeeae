"""GPU parity: prompt-fixed top-k neuron selection, condensation and condensed decode."""

import numpy as np
import pytest

import oracle
from synth import ffn_weights, griffin_prompt, decode_inputs, TINY, LLAMA3_8B
from gpu_util import say, dev_bf16, dev_f32, host, check_ffn

pytestmark = pytest.mark.gpu

SCORE_BAND = 1e-4  # relative guard band around the k-th score


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


def _check(sr, seed, t_n, d, f, k, std, normalize=False, decode_b=2):
    say(f"griffin T={t_n} d={d} f={f} k={k} normalize={normalize}")
    wg, wu, wd = ffn_weights(seed, d, f, std)
    xp = griffin_prompt(seed, t_n, d)
    W = [dev_bf16(w) for w in (wg, wu, wd)]
    sel, scores, wgc, wuc, wdc = sr.sirius_griffin_select(dev_bf16(xp), *W, k, normalize_tokens=normalize)
    sel, scores = host(sel).astype(np.int64), host(scores)
    s_ref = oracle.griffin_scores(xp, wg, wu, normalize)
    np.testing.assert_allclose(scores, s_ref, rtol=2e-5, atol=1e-30)
    assert np.all(np.diff(sel) > 0)
    ref = oracle.griffin_topk(s_ref, k)
    kth = np.sort(s_ref)[::-1][k - 1]
    near = np.abs(s_ref - kth) <= SCORE_BAND * kth
    sym = np.setxor1d(sel, ref)
    assert np.all(near[sym]), f"{int((~near[sym]).sum())} selection mismatches outside the band"
    # condensed rows are exact copies of the selected rows
    for w, c in ((wg, wgc), (wu, wuc), (wd, wdc)):
        assert np.array_equal(host(c), w[sel])
    # decode with the condensed weights equals the FFN masked to the selected set
    x = decode_inputs(seed, decode_b, d)
    y = sr.sirius_ffn_condensed(dev_f32(x), wgc, wuc, wdc)
    check_ffn(host(y), oracle.ffn_masked(x, wg, wu, wd, [sel] * decode_b))
    return int(near.sum())


def test_tiny(sr):
    _check(sr, 1, 64, TINY.d_model, TINY.d_ff, TINY.d_ff // 2, TINY.weight_std)


def test_ragged(sr):
    _check(sr, 2, 100, 264, 1000, 333, 1.0 / np.sqrt(264))
    _check(sr, 3, 1, 8, 5, 2, 0.5)


@pytest.mark.parametrize("normalize", [False, True])
def test_several_ragged_tiles(sr, normalize):
    # two token tiles of 256 (the last ragged), ten neuron tiles of 112 (eight placed one per
    # XCD and two left over, the last ragged), and a K tail of 8 past the last 32-wide stage
    _check(sr, 7, 300, 520, 1100, 400, 1.0 / np.sqrt(520), normalize=normalize)
    # three token tiles, eighteen neuron tiles (two rounds of eight, two left over), a K of
    # fewer stages than the ring holds, and one of exactly one stage
    _check(sr, 8, 600, 96, 2000, 1000, 1.0 / np.sqrt(96), normalize=normalize)
    _check(sr, 9, 257, 32, 113, 50, 1.0 / np.sqrt(32), normalize=normalize)


def test_normalized_variant(sr):
    _check(sr, 4, 70, 256, 688, 300, TINY.weight_std, normalize=True)


def test_k_equals_dff_is_dense(sr):
    d, f = 256, 300
    wg, wu, wd = ffn_weights(5, d, f, 1 / 16)
    xp = griffin_prompt(5, 16, d)
    W = [dev_bf16(w) for w in (wg, wu, wd)]
    sel, _, wgc, wuc, wdc = sr.sirius_griffin_select(dev_bf16(xp), *W, f)
    assert np.array_equal(host(sel), np.arange(f))
    x = decode_inputs(5, 3, d)
    assert np.array_equal(host(sr.sirius_ffn_condensed(dev_f32(x), wgc, wuc, wdc)),
                          host(sr.sirius_ffn_dense(dev_f32(x), *W)))


def test_llama3_8b_prompt512(sr):
    nb = _check(sr, 6, 512, LLAMA3_8B.d_model, LLAMA3_8B.d_ff, LLAMA3_8B.d_ff // 2, LLAMA3_8B.weight_std,
                decode_b=1)
    say(f"8B griffin boundary neurons: {nb}")


def test_long_prompt_full_width_sampled(sr):
    """A 2000-token prompt at Llama-3-8B FFN width: 8 token tiles of 256 (the last ragged) over
    128 neuron tiles of 112. The oracle recomputes 64 sampled neurons' scores from their own rows; the
    selection must be exactly the top-k of the returned scores (equal scores: lower index), and
    sampled condensed rows must be the selected rows."""
    import torch
    d, f, t_n = LLAMA3_8B.d_model, LLAMA3_8B.d_ff, 2000
    k = f // 2
    say(f"griffin T={t_n} d={d} f={f} k={k} (sampled)")
    ws = []
    for m in range(3):
        w = torch.empty((f, d), dtype=torch.bfloat16, device="cuda")
        sr.sirius_fill_normal_bf16(w, 9100 + m, 0.0, LLAMA3_8B.weight_std)
        ws.append(w)
    xp = griffin_prompt(9103, t_n, d)
    sel, scores, wgc, wuc, wdc = sr.sirius_griffin_select(dev_bf16(xp), *ws, k)
    sel, scores = host(sel).astype(np.int64), host(scores)
    np.testing.assert_array_equal(sel, oracle.griffin_topk(scores, k))
    rng = np.random.default_rng(9104)
    idx = np.sort(rng.choice(f, 64, replace=False))
    rows = torch.from_numpy(idx).cuda()
    s_ref = oracle.griffin_scores(xp, host(ws[0][rows]), host(ws[1][rows]))
    np.testing.assert_allclose(scores[idx], s_ref, rtol=2e-5, atol=1e-30)
    j = np.sort(rng.choice(k, 16, replace=False))
    src = torch.from_numpy(sel[j]).cuda()
    dst = torch.from_numpy(j).cuda()
    for w, c in zip(ws, (wgc, wuc, wdc)):
        assert torch.equal(c[dst], w[src])
