"""GPU parity on full FFN stacks at their real sizes, checked layer by layer against the oracle.

  * Llama-3-8B FFN stack: 32 layers of 4096 x 14336 bf16 (11.3 GB), h <- h + FFN(RMSNorm(h)),
    batch 1 / 4 / 16, per-token threshold sparsity calibrated per layer to 40 / 50 / 65 %;
    and the prompt-fixed variant: per-layer 512-token prompt, top-50 % neurons condensed,
    condensed stack at batch 1 / 4 / 16.
  * Llama-3-70B FFN stack: 80 layers of 8192 x 28672 bf16 (112.7 GB resident), batch 1,
    thresholds calibrated per layer to 50 / 65 % sparsity.

Weights are filled on the device by the library's seeded generator. Every layer runs through
the library in place (resid = y = h) exactly as a decode step would; at sampled layers the
layer's input is copied out first and the oracle recomputes that layer from it (the active
sets must match outside the guard band, the output must match the oracle's FFN on the
library's own sets). End-to-end agreement over many layers is not asserted, since a single
boundary flip early on changes every later input.
"""

import numpy as np
import pytest

import oracle
from synth import decode_inputs, calibration_inputs, griffin_prompt, LLAMA3_8B, LLAMA3_70B
from gpu_util import (say, dev_f32, dev_bf16, host, check_cats_sets, check_ffn, check_ffn_rounded_norm,
                      MFMA_MIN_BATCH)

pytestmark = pytest.mark.gpu

EPS = 1e-5
SCORE_BAND = 1e-4


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


class Stack:
    """A stack of device-filled FFN layers with per-layer calibrated thresholds."""

    def __init__(self, sr, shape, n_layers, seed, n_cal, sparsities):
        import torch
        d, f = shape.d_model, shape.d_ff
        self.d, self.f = d, f
        self.layers = []
        for l in range(n_layers):
            ws = []
            for m in range(3):
                w = torch.empty((f, d), dtype=torch.bfloat16, device="cuda")
                sr.sirius_fill_normal_bf16(w, seed + 3 * l + m, 0.0, shape.weight_std)
                ws.append(w)
            self.layers.append(ws)
        x_cal = dev_f32(calibration_inputs(seed, n_cal, d))
        self.t = {}
        for s in sparsities:
            ts = [sr.sirius_cats_calibrate(x_cal, self.layers[l][0], s) for l in range(n_layers)]
            self.t[s] = [float(v) for v in torch.cat(ts).cpu().numpy()]
        self._host = {}

    def host_layer(self, l):
        if l not in self._host:
            self._host[l] = [host(w) for w in self.layers[l]]
        return self._host[l]

    def free(self):
        import torch
        self.layers = []
        self._host = {}
        torch.cuda.empty_cache()


def run_cats_stack(sr, st, h0, s, check_layers):
    """Runs the threshold-sparse stack in place; checks the sampled layers. Returns the kept
    fraction at each checked layer."""
    import torch
    bsz = h0.shape[0]
    h = dev_f32(h0)
    idx = torch.empty((bsz, st.f), dtype=torch.int32, device="cuda")
    cnt = torch.empty(bsz, dtype=torch.int32, device="cuda")
    kept = []
    for l, (wg, wu, wd) in enumerate(st.layers):
        t = st.t[s][l]
        if l not in check_layers:
            sr.sirius_ffn_cats(h, wg, wu, wd, t, norm_eps=EPS, resid=h, y=h, want_active=False)
            continue
        h_in = host(h).copy()
        sr.sirius_ffn_cats(h, wg, wu, wd, t, norm_eps=EPS, resid=h, y=h, active_idx=idx, active_cnt=cnt)
        hwg, hwu, hwd = st.host_layer(l)
        xn = oracle.rmsnorm(h_in, EPS)
        sets, nb = check_cats_sets(xn, hwg, t, host(idx), host(cnt))
        e = check_ffn(host(h), oracle.ffn_masked(xn, hwg, hwu, hwd, sets), resid=h_in)
        frac = float(np.mean([len(x) for x in sets])) / st.f
        kept.append(frac)
        say(f"  layer {l}: kept {frac:.3f}, boundary {nb}, error {e:.2e} x RMS")
    assert np.all(np.isfinite(host(h)))
    return kept


# ---------------------------------------------------------------------------------------- 8B

@pytest.fixture(scope="module")
def stack8b(sr):
    say("8B stack: filling 32 layers, calibrating 40/50/65 %")
    st = Stack(sr, LLAMA3_8B, 32, 7000, 256, (0.40, 0.50, 0.65))
    yield st
    st.free()


CHECK_8B = (0, 15, 31)


@pytest.mark.parametrize("bsz", [1, 4, 16])
@pytest.mark.parametrize("s", [0.40, 0.50, 0.65])
def test_llama3_8b_cats_stack(sr, stack8b, s, bsz):
    say(f"8B CATS stack s={s} B={bsz}")
    kept = run_cats_stack(sr, stack8b, decode_inputs(7100 + bsz, bsz, LLAMA3_8B.d_model), s, CHECK_8B)
    # the calibrated threshold keeps about 1 - s of the neurons on the stack's own inputs
    assert all(abs(k - (1.0 - s)) < 0.1 for k in kept), kept


@pytest.fixture(scope="module")
def condensed8b(sr, stack8b):
    """Per-layer prompt top-k (k = d_ff / 2) and condensed weights; selection checked at the
    sampled layers."""
    d, f = LLAMA3_8B.d_model, LLAMA3_8B.d_ff
    k = f // 2
    cond, sels = [], {}
    for l, (wg, wu, wd) in enumerate(stack8b.layers):
        xp = griffin_prompt(7200 + l, 512, d)
        sel, scores, wgc, wuc, wdc = sr.sirius_griffin_select(dev_bf16(xp), wg, wu, wd, k,
                                                              want_scores=l in CHECK_8B)
        cond.append((wgc, wuc, wdc))
        if l in CHECK_8B:
            say(f"8B griffin layer {l}: checking the selection")
            hwg, hwu, _ = stack8b.host_layer(l)
            s_ref = oracle.griffin_scores(xp, hwg, hwu)
            np.testing.assert_allclose(host(scores), s_ref, rtol=2e-5, atol=1e-30)
            sel_h = host(sel).astype(np.int64)
            kth = np.sort(s_ref)[::-1][k - 1]
            near = np.abs(s_ref - kth) <= SCORE_BAND * kth
            sym = np.setxor1d(sel_h, oracle.griffin_topk(s_ref, k))
            assert np.all(near[sym]), f"{int((~near[sym]).sum())} selection mismatches outside the band"
            sels[l] = sel_h
    return cond, sels


@pytest.mark.parametrize("bsz", [1, 4, 16])
def test_llama3_8b_condensed_stack(sr, stack8b, condensed8b, bsz):
    say(f"8B condensed stack B={bsz}")
    cond, sels = condensed8b
    h = dev_f32(decode_inputs(7300 + bsz, bsz, LLAMA3_8B.d_model))
    for l, (wgc, wuc, wdc) in enumerate(cond):
        if l not in CHECK_8B:
            sr.sirius_ffn_condensed(h, wgc, wuc, wdc, norm_eps=EPS, resid=h, y=h)
            continue
        h_in = host(h).copy()
        sr.sirius_ffn_condensed(h, wgc, wuc, wdc, norm_eps=EPS, resid=h, y=h)
        hwg, hwu, hwd = stack8b.host_layer(l)
        xn = oracle.rmsnorm(h_in, EPS)
        if bsz >= MFMA_MIN_BATCH:  # gate/up on MFMA from the bf16-rounded normalised input
            e, nb = check_ffn_rounded_norm(host(h), xn, hwg, hwu, hwd, sets=[sels[l]] * bsz, resid=h_in)
        else:
            e, nb = check_ffn(host(h), oracle.ffn_masked(xn, hwg, hwu, hwd, [sels[l]] * bsz), resid=h_in), 0
        say(f"  layer {l}: error {e:.2e} x RMS ({nb} inputs with ambiguous bf16 rounding)")
    assert np.all(np.isfinite(host(h)))


def test_llama3_8b_dense_verify_chunk_stack(sr, stack8b):
    """The full model's 16-token pass through all 32 dense layers (MFMA path)."""
    say("8B dense stack B=16")
    bsz = 16
    h = dev_f32(decode_inputs(7400, bsz, LLAMA3_8B.d_model))
    for l, (wg, wu, wd) in enumerate(stack8b.layers):
        if l not in CHECK_8B:
            sr.sirius_ffn_dense(h, wg, wu, wd, norm_eps=EPS, resid=h, y=h)
            continue
        h_in = host(h).copy()
        sr.sirius_ffn_dense(h, wg, wu, wd, norm_eps=EPS, resid=h, y=h)
        hwg, hwu, hwd = stack8b.host_layer(l)
        xn = oracle.rmsnorm(h_in, EPS)
        e, nb = check_ffn_rounded_norm(host(h), xn, hwg, hwu, hwd, resid=h_in)
        say(f"  layer {l}: error {e:.2e} x RMS ({nb} inputs with ambiguous bf16 rounding)")


def test_llama3_8b_dense_tree_pass_stack(sr, stack8b):
    """The full model's pass over a 64-node drafted tree (kernel size 16 x width 4) through all
    32 dense layers: four 16-token MFMA tiles per layer."""
    say("8B dense stack B=64")
    bsz = 64
    h = dev_f32(decode_inputs(7500, bsz, LLAMA3_8B.d_model))
    for l, (wg, wu, wd) in enumerate(stack8b.layers):
        if l not in CHECK_8B:
            sr.sirius_ffn_dense(h, wg, wu, wd, norm_eps=EPS, resid=h, y=h)
            continue
        h_in = host(h).copy()
        sr.sirius_ffn_dense(h, wg, wu, wd, norm_eps=EPS, resid=h, y=h)
        hwg, hwu, hwd = stack8b.host_layer(l)
        xn = oracle.rmsnorm(h_in, EPS)
        e, nb = check_ffn_rounded_norm(host(h), xn, hwg, hwu, hwd, resid=h_in)
        say(f"  layer {l}: error {e:.2e} x RMS ({nb} inputs with ambiguous bf16 rounding)")
    assert np.all(np.isfinite(host(h)))


# --------------------------------------------------------------------------------------- 70B

@pytest.fixture(scope="module")
def stack70b(sr, stack8b):
    stack8b.free()  # release the 8B stack's 17 GB first
    say("70B stack: filling 80 layers (112.7 GB), calibrating 50/65 %")
    st = Stack(sr, LLAMA3_70B, 80, 8000, 64, (0.50, 0.65))
    yield st
    st.free()


@pytest.mark.parametrize("s", [0.50, 0.65])
def test_llama3_70b_cats_stack(sr, stack70b, s):
    say(f"70B CATS stack s={s} B=1")
    kept = run_cats_stack(sr, stack70b, decode_inputs(8100, 1, LLAMA3_70B.d_model), s, (0, 39, 79))
    assert all(abs(k - (1.0 - s)) < 0.1 for k in kept), kept


def test_llama3_70b_dense_verify_chunk_layers(sr, stack70b):
    """The full model's 16-token pass over Llama-3-70B-shaped layers (MFMA path: 8 neuron ranges x
    32 column tiles of the down product), with RMSNorm and residual, checked on three layers."""
    bsz = 16
    for l in (0, 39, 79):
        say(f"70B dense B=16 layer {l}")
        h_in = decode_inputs(8200 + l, bsz, LLAMA3_70B.d_model)
        wg, wu, wd = stack70b.layers[l]
        y = host(sr.sirius_ffn_dense(dev_f32(h_in), wg, wu, wd, norm_eps=EPS, resid=dev_f32(h_in)))
        hwg, hwu, hwd = stack70b.host_layer(l)
        xn = oracle.rmsnorm(h_in, EPS)
        e, nb = check_ffn_rounded_norm(y, xn, hwg, hwu, hwd, resid=h_in)
        say(f"  error {e:.2e} x RMS ({nb} inputs with ambiguous bf16 rounding)")


@pytest.mark.parametrize("bsz", [32, 64])
def test_llama3_70b_dense_tree_pass_layer(sr, stack70b, bsz):
    """The full model's pass over a drafted tree of 32 or 64 nodes on a Llama-3-70B-shaped layer
    (two or four 16-token MFMA tiles), with RMSNorm and residual."""
    l = 40
    say(f"70B dense B={bsz} layer {l}")
    h_in = decode_inputs(8300 + bsz, bsz, LLAMA3_70B.d_model)
    wg, wu, wd = stack70b.layers[l]
    y = host(sr.sirius_ffn_dense(dev_f32(h_in), wg, wu, wd, norm_eps=EPS, resid=dev_f32(h_in)))
    hwg, hwu, hwd = stack70b.host_layer(l)
    xn = oracle.rmsnorm(h_in, EPS)
    e, nb = check_ffn_rounded_norm(y, xn, hwg, hwu, hwd, resid=h_in)
    say(f"  error {e:.2e} x RMS ({nb} inputs with ambiguous bf16 rounding)")
