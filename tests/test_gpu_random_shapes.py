"""GPU parity over seeded random shapes: the dense, threshold-sparse (CATS) and per-token top-k FFN
calls through the one FFN dispatcher -- the batch-1 decode kernel, the batched MFMA engine at every
token class and at short and long segments (d_model % 256 == 0, 2..64 tokens, d_ff up to 14336),
the small-batch kernels of other widths -- with and without RMSNorm and residual, against the fp64
oracle."""

import numpy as np
import pytest

import oracle
from synth import ffn_weights, decode_inputs
from gpu_util import (say, dev_bf16, dev_f32, host, rounded_bf16, check_cats_sets, check_topk_sets,
                      check_ffn, check_ffn_rounded_norm, FP32_PATH_TOL, MFMA_MIN_BATCH)

pytestmark = pytest.mark.gpu

_WIDTHS = (256, 512, 768, 1024, 136, 264, 520)   # the first four take the batched engine
_BATCHES = (1, 2, 3, 4, 5, 7, 8, 9, 12, 16, 17, 24, 31, 33, 48, 64)


def _cases(n=18, seed=2409):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        d = int(rng.choice(_WIDTHS))
        # even cases: short segments (d_ff <= 4200: at most 20 neurons); odd: up to 56 neurons
        f = int(rng.integers(1, 4201)) if i % 2 == 0 else int(rng.integers(7200, 14337))
        b = int(rng.choice(_BATCHES))
        out.append((i, d, f, b, bool(rng.integers(0, 2))))
    return out


CASES = _cases()


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


def _setup(case):
    i, d, f, b, norm = case
    wg, wu, wd = ffn_weights(9000 + i, d, f, 1.0 / np.sqrt(d))
    W = tuple(dev_bf16(w) for w in (wg, wu, wd))
    x = decode_inputs(9100 + i, b, d) * (3.0 if norm else 1.0)
    res = decode_inputs(9200 + i, b, d) if norm else None
    xn = oracle.rmsnorm(x, 1e-5) if norm else x
    kw = dict(norm_eps=1e-5, resid=dev_f32(res)) if norm else {}
    return (wg, wu, wd), W, x, res, xn, kw


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"c{c[0]}-d{c[1]}-f{c[2]}-B{c[3]}-{'norm' if c[4] else 'plain'}")
def test_dense(sr, case):
    i, d, f, b, norm = case
    say(f"random dense {case}")
    (wg, wu, wd), W, x, res, xn, kw = _setup(case)
    y = host(sr.sirius_ffn_dense(dev_f32(x), *W, **kw))
    if b < MFMA_MIN_BATCH:  # the exact input
        check_ffn(y, oracle.ffn_dense(xn, wg, wu, wd), resid=res)
    elif norm:  # the GPU's normalised input rounded to bf16
        check_ffn_rounded_norm(y, xn, wg, wu, wd, resid=res)
    else:
        check_ffn(y, oracle.ffn_dense(rounded_bf16(x), wg, wu, wd), tol=FP32_PATH_TOL)


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"c{c[0]}-d{c[1]}-f{c[2]}-B{c[3]}-{'norm' if c[4] else 'plain'}")
def test_cats(sr, case):
    i, d, f, b, norm = case
    say(f"random cats {case}")
    (wg, wu, wd), W, x, res, xn, kw = _setup(case)
    t = float(np.median(np.abs(oracle.gate_activations(xn, wg))))
    y, idx, cnt = sr.sirius_ffn_cats(dev_f32(x), *W, t, **kw)
    sets, _ = check_cats_sets(xn, wg, t, host(idx), host(cnt))
    check_ffn(host(y), oracle.ffn_masked(xn, wg, wu, wd, sets), resid=res)


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"c{c[0]}-d{c[1]}-f{c[2]}-B{c[3]}-{'norm' if c[4] else 'plain'}")
def test_topk(sr, case):
    i, d, f, b, norm = case
    say(f"random topk {case}")
    (wg, wu, wd), W, x, res, xn, kw = _setup(case)
    k = int(np.random.default_rng(9300 + i).integers(1, f + 1))
    y, idx, cnt = sr.sirius_ffn_topk(dev_f32(x), *W, k, **kw)
    sets, _ = check_topk_sets(xn, wg, k, host(idx), host(cnt))
    check_ffn(host(y), oracle.ffn_masked(xn, wg, wu, wd, sets), resid=res)
