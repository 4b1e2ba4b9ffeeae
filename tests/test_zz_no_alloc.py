"""GPU: the allocation-free threshold-sparse FFN (sirius_ffn_cats_noalloc) against the workspace
entry point sirius_ffn_cats and the oracle.

The two entry points run the same kernels, so their outputs and kept lists must agree bit for
bit; the oracle checks the allocation-free call to the parity bar of the threshold path (sets
outside the 1e-3 guard band, output within 1e-4 x RMS of the oracle's FFN on the GPU's own
sets). Two calls in a row share the library's device scratch, the second with a smaller input,
so that leftovers of the first call cannot leak into the second.
"""

import ctypes

import numpy as np
import pytest

import oracle
from synth import ffn_weights, decode_inputs, calibration_inputs, TINY, LLAMA3_8B
from gpu_util import say, dev_bf16, dev_f32, host, check_cats_sets, check_ffn

pytestmark = pytest.mark.gpu

EPS = 1e-5


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


def _case(sr, shape, seed, bsz):
    wg, wu, wd = ffn_weights(seed, shape.d_model, shape.d_ff, shape.weight_std)
    W = tuple(dev_bf16(w) for w in (wg, wu, wd))
    t = float(host(sr.sirius_cats_calibrate(dev_f32(calibration_inputs(seed, 64, shape.d_model)), W[0], 0.5))[0])
    x = decode_inputs(seed + 1, bsz, shape.d_model) * 2.0
    res = decode_inputs(seed + 2, bsz, shape.d_model)
    return (wg, wu, wd), W, t, x, res


def _noalloc_c_abi(sr, x, W, t, resid, y, idx, cnt):
    """The allocation-free call straight through the C ABI (ctypes), on torch's current stream."""
    import torch
    L = sr.lib()
    f, d = int(W[0].shape[0]), int(W[0].shape[1])
    p = lambda a: ctypes.c_void_p(a.data_ptr())
    rc = L.sirius_ffn_cats_noalloc(p(x), int(x.shape[0]), p(W[0]), p(W[1]), p(W[2]), d, f, float(t), EPS,
                                   p(resid), p(y), p(idx), p(cnt),
                                   ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0, L.sirius_last_error().decode()


def test_noalloc_matches_workspace_entry_twice(sr):
    import torch
    cases = [(LLAMA3_8B, 9100, 16), (TINY, 9200, 1)]  # the second call is smaller
    results = []
    for shape, seed, bsz in cases:
        say(f"noalloc cats {shape.name} B={bsz}")
        (wg, wu, wd), W, t, x, res = _case(sr, shape, seed, bsz)
        xd, rd = dev_f32(x), dev_f32(res)
        y = torch.full_like(xd, float("nan"))
        idx = torch.full((bsz, shape.d_ff), -7, dtype=torch.int32, device="cuda")
        cnt = torch.full((bsz,), -7, dtype=torch.int32, device="cuda")
        _noalloc_c_abi(sr, xd, W, t, rd, y, idx, cnt)
        y_na, idx_na, cnt_na = host(y), host(idx), host(cnt)
        results.append((shape, W, t, x, res, y_na, idx_na, cnt_na))
    for shape, W, t, x, res, y_na, idx_na, cnt_na in results:
        bsz = x.shape[0]
        say(f"  compare {shape.name} B={bsz} with sirius_ffn_cats and the oracle")
        y_ws, idx_ws, cnt_ws = sr.sirius_ffn_cats(dev_f32(x), *W, t, norm_eps=EPS, resid=dev_f32(res))
        y_ws, idx_ws, cnt_ws = host(y_ws), host(idx_ws), host(cnt_ws)
        np.testing.assert_array_equal(cnt_na, cnt_ws)
        for b in range(bsz):
            np.testing.assert_array_equal(idx_na[b, : cnt_na[b]], idx_ws[b, : cnt_ws[b]])
        assert np.array_equal(y_na, y_ws), "allocation-free output differs from sirius_ffn_cats"
        hw = [host(w) for w in W]
        xn = oracle.rmsnorm(x, EPS)
        sets, nb = check_cats_sets(xn, hw[0], t, idx_na, cnt_na)
        e = check_ffn(y_na, oracle.ffn_masked(xn, *hw, sets), resid=res)
        say(f"  kept {np.mean(cnt_na) / shape.d_ff:.3f}, boundary {nb}, error {e:.2e} x RMS")


def test_noalloc_under_graph_capture(sr):
    """The call records into a HIP graph (nothing to allocate) and every replay matches an eager
    call bit for bit."""
    import torch
    shape, bsz = TINY, 3
    (wg, wu, wd), W, t, x, res = _case(sr, shape, 9300, bsz)
    xd, rd = dev_f32(x), dev_f32(res)
    y = torch.empty_like(xd)
    idx = torch.empty((bsz, shape.d_ff), dtype=torch.int32, device="cuda")
    cnt = torch.empty((bsz,), dtype=torch.int32, device="cuda")
    _noalloc_c_abi(sr, xd, W, t, rd, y, idx, cnt)
    want = host(y).copy()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            _noalloc_c_abi(sr, xd, W, t, rd, y, idx, cnt)
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host(y), want), f"replay {rep}"
        # eager work between replays
        _noalloc_c_abi(sr, xd, W, t, rd, y, idx, cnt)
        torch.cuda.synchronize()
