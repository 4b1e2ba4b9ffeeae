"""Pins of the coarse-grained (Griffin) oracle: prompt statistic, top-k, condensation."""

import math

import numpy as np

import oracle
from synth import ffn_weights, griffin_prompt, decode_inputs, TINY


def _small(seed, t, d, f):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((t, d))
    wg, wu, wd = (rng.standard_normal((f, d)) / math.sqrt(d) for _ in range(3))
    return x, wg, wu, wd


def _brute_scores(x, wg, wu, normalize=False):
    t_n, d = len(x), len(x[0])
    f = len(wg)
    z = [[0.0] * f for _ in range(t_n)]
    for t in range(t_n):
        for i in range(f):
            g = sum(float(wg[i][k]) * float(x[t][k]) for k in range(d))
            u = sum(float(wu[i][k]) * float(x[t][k]) for k in range(d))
            z[t][i] = g / (1.0 + math.exp(-g)) * u
    if normalize:
        for t in range(t_n):
            n = math.sqrt(sum(v * v for v in z[t]))
            z[t] = [v / n for v in z[t]]
    return [math.sqrt(sum(z[t][i] ** 2 for t in range(t_n))) for i in range(f)]


def test_single_token_score_is_abs_activation_product():
    # T = 1: s_i = |SiLU(g_i) u_i|. Hand case: gate (ln 3), up (-2) -> |0.75 ln3 * -2| = 1.5 ln 3.
    x = np.array([[1.0, 0.0]])
    wg = np.array([[math.log(3.0), 0.0], [0.0, 1.0]])
    wu = np.array([[-2.0, 0.0], [0.0, 1.0]])
    s = oracle.griffin_scores(x, wg, wu)
    np.testing.assert_allclose(s, [1.5 * math.log(3.0), 0.0], rtol=1e-15, atol=0)


def test_scores_match_bruteforce():
    x, wg, wu, _ = _small(21, 5, 8, 14)
    np.testing.assert_allclose(oracle.griffin_scores(x, wg, wu), _brute_scores(x, wg, wu), rtol=1e-12)
    np.testing.assert_allclose(oracle.griffin_scores(x, wg, wu, True), _brute_scores(x, wg, wu, True),
                               rtol=1e-12)


def test_scores_are_token_order_invariant_and_scale_quadratically():
    x, wg, wu, _ = _small(22, 6, 8, 10)
    s = oracle.griffin_scores(x, wg, wu)
    np.testing.assert_allclose(oracle.griffin_scores(x[::-1], wg, wu), s, rtol=1e-13)
    # Doubling W_up doubles every z, so doubles every score (a squared-sum without the sqrt would quadruple).
    np.testing.assert_allclose(oracle.griffin_scores(x, wg, 2 * wu), 2 * s, rtol=1e-13)
    # Repeating the prompt twice multiplies each score by sqrt(2).
    np.testing.assert_allclose(oracle.griffin_scores(np.vstack([x, x]), wg, wu), math.sqrt(2) * s, rtol=1e-13)


def test_topk_matches_bruteforce_sort_with_ties():
    s = np.array([0.5, 2.0, 2.0, 0.1, 2.0, 1.0, 1.0])
    # Ranking by (-score, index): 1, 2, 4 (score 2), 5, 6 (score 1), 0, 3.
    assert oracle.griffin_topk(s, 2).tolist() == [1, 2]
    assert oracle.griffin_topk(s, 4).tolist() == [1, 2, 4, 5]
    assert oracle.griffin_topk(s, 7).tolist() == list(range(7))
    rng = np.random.default_rng(23)
    for _ in range(20):
        v = rng.integers(0, 6, size=40).astype(float)  # many ties
        k = int(rng.integers(1, 41))
        brute = sorted(sorted(range(40), key=lambda i: (-v[i], i))[:k])
        assert oracle.griffin_topk(v, k).tolist() == brute


def test_condense_is_row_gather_and_full_k_is_dense():
    wg, wu, wd = ffn_weights(24, TINY.d_model, TINY.d_ff, TINY.weight_std)
    xp = griffin_prompt(24, 16, TINY.d_model)
    s = oracle.griffin_scores(xp, wg, wu)
    sel = oracle.griffin_topk(s, TINY.d_ff)
    assert sel.tolist() == list(range(TINY.d_ff))
    x = decode_inputs(24, 2, TINY.d_model)
    y_full = oracle.ffn_condensed(x, oracle.condense(wg, sel), oracle.condense(wu, sel), oracle.condense(wd, sel))
    np.testing.assert_array_equal(y_full, oracle.ffn_dense(x, wg, wu, wd))
    sel = oracle.griffin_topk(s, TINY.d_ff // 2)
    c = oracle.condense(wd, sel)
    assert c.dtype == wd.dtype
    for j, i in enumerate(sel):
        assert np.array_equal(c[j], wd[i])


def test_condensed_ffn_equals_masked_ffn():
    wg, wu, wd = ffn_weights(25, TINY.d_model, TINY.d_ff, TINY.weight_std)
    xp = griffin_prompt(25, 32, TINY.d_model)
    sel = oracle.griffin_topk(oracle.griffin_scores(xp, wg, wu), 344)
    x = decode_inputs(25, 3, TINY.d_model)
    yc = oracle.ffn_condensed(x, oracle.condense(wg, sel), oracle.condense(wu, sel), oracle.condense(wd, sel))
    ym = oracle.ffn_masked(x, wg, wu, wd, [sel] * 3)
    np.testing.assert_allclose(yc, ym, rtol=1e-12, atol=1e-14)
    # The selected neurons carry the largest prompt statistic.
    s = oracle.griffin_scores(xp, wg, wu)
    rest = np.setdiff1d(np.arange(TINY.d_ff), sel)
    assert s[sel].min() >= s[rest].max()
