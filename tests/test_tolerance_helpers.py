"""CPU checks of the GPU tests' tolerance helpers (no GPU): the rounding allowance of the
fused-RMSNorm MFMA check accepts every admissible rounding of the ambiguous inputs and still
rejects a planted output error."""

import numpy as np
import pytest

import oracle
from synth import ffn_weights, decode_inputs, bf16_bits
from gpu_util import check_ffn_rounded_norm, check_tree_build


def _widen(v):
    return oracle.widen_bf16(bf16_bits(np.asarray(v, dtype=np.float32)))


@pytest.fixture(scope="module")
def case():
    d, f, bsz = 256, 688, 4
    wg, wu, wd = ffn_weights(11, d, f, 1 / 16)
    xn = oracle.rmsnorm(decode_inputs(11, bsz, d) * 2.0, 1e-5)
    return wg, wu, wd, xn


def test_other_rounding_of_ambiguous_inputs_is_accepted(case):
    wg, wu, wd, xn = case
    band = 2e-4  # wider than the GPU needs, so that a fair number of inputs are ambiguous
    lo, hi = _widen(xn * (1 - band)), _widen(xn * (1 + band))
    near = _widen(xn)
    other = np.where(near == lo, hi, lo)  # round every ambiguous input the other way
    alt = np.where(lo != hi, other, near)
    y_alt = oracle.ffn_dense(alt, wg, wu, wd)
    e, nb = check_ffn_rounded_norm(y_alt, xn, wg, wu, wd, band=band)
    assert nb > 10 and e > 1e-4  # the flips are visible, and allowed


def test_planted_error_is_rejected(case):
    wg, wu, wd, xn = case
    y = oracle.ffn_dense(_widen(xn), wg, wu, wd)
    rms = float(np.sqrt(np.mean(y * y)))
    y[1, 7] += 3e-4 * rms
    with pytest.raises(AssertionError):
        check_ffn_rounded_norm(y, xn, wg, wu, wd)


def _tree_case(seed=4, wc=3, v=500, w=6):
    rng = np.random.default_rng(seed)
    lg = rng.normal(size=(wc, v)) * 2.0
    cum = -np.sort(rng.exponential(3.0, size=wc))
    tok, par, sc = oracle.tree_build_step(lg, cum, w)
    return lg, cum, w, tok, par, sc


def test_tree_build_check_accepts_the_oracle_and_rounded_scores():
    lg, cum, w, tok, par, sc = _tree_case()
    assert check_tree_build(lg, cum, w, 1.0, tok, par, sc.astype(np.float32)) == 0


@pytest.mark.parametrize("plant", ["swap", "token", "parent", "score", "repeat"])
def test_tree_build_check_rejects_planted_mistakes(plant):
    lg, cum, w, tok, par, sc = _tree_case()
    tok, par, sc = tok.copy(), par.copy(), sc.copy()
    if plant == "swap":       # two well-separated ranks exchanged
        tok[[1, 2]], par[[1, 2]], sc[[1, 2]] = tok[[2, 1]], par[[2, 1]], sc[[2, 1]]
    elif plant == "token":    # a neighbouring token id
        tok[0] = (tok[0] + 1) % lg.shape[1]
    elif plant == "parent":   # the right token under another leaf
        par[0] = (par[0] + 1) % lg.shape[0]
    elif plant == "score":
        sc[3] += 1e-3
    else:
        tok[4], par[4] = tok[3], par[3]
    with pytest.raises(AssertionError):
        check_tree_build(lg, cum, w, 1.0, tok, par, sc)


def test_tree_build_check_allows_either_order_of_a_near_tie():
    lg, cum, w, tok, par, sc = _tree_case()
    # make ranks 1 and 2 tie within the band by moving one logit
    lg = lg.copy()
    ls = oracle.log_softmax(lg)
    target = sc[1] - 3e-6
    lg[par[2], tok[2]] += target - (cum[par[2]] + ls[par[2], tok[2]])
    tok2, par2, sc2 = oracle.tree_build_step(lg, cum, w)
    assert abs(sc2[1] - sc2[2]) < 1e-5
    tok2, par2, sc2 = tok2.copy(), par2.copy(), sc2.copy()
    tok2[[1, 2]], par2[[1, 2]], sc2[[1, 2]] = tok2[[2, 1]], par2[[2, 1]], sc2[[2, 1]]
    assert check_tree_build(lg, cum, w, 1.0, tok2, par2, sc2) == 2
