"""CPU checks of the GPU tests' tolerance helpers (no GPU): the rounding allowance of the
fused-RMSNorm MFMA check accepts every admissible rounding of the ambiguous inputs and still
rejects a planted output error."""

import numpy as np
import pytest

import oracle
from synth import ffn_weights, decode_inputs, bf16_bits
from gpu_util import check_ffn_rounded_norm


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
