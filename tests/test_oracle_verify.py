"""Pins of the correction-check oracle (Algorithm 1: first rejection below r, interleaved token)."""

import json
import math
import os

import numpy as np
import pytest

import oracle
from synth import verify_inputs, VERIFY_TINY

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "verify_hand_cases.json")


def _num(s):
    if s == "ln4":
        return math.log(4.0)
    return float(s)


def _expr(s):
    return float(eval(s, {"__builtins__": {}}, {"exp": math.exp}))  # fixture expressions only


def _cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_hand_cases(case):
    rows = np.array([[_num(v) for v in row] for row in case["rows"]], dtype=np.float64)[None]
    drafted = np.array([case["drafted"]])
    acc, nxt, q = oracle.verify_accept(rows, drafted, case["r"], case["temperature"])
    assert int(acc[0]) == case["accept_len"]
    assert int(nxt[0]) == case["next_token"]
    np.testing.assert_allclose(q[0], [_expr(e) for e in case["q"]], rtol=1e-12, atol=1e-300)


def test_uniform_logits_probability_is_one_over_v():
    v = VERIFY_TINY.vocab
    lg = np.zeros((1, 4, v))
    dr = np.array([[3, 999, 0, 500]])
    for r, want in [(0.9 / v, 4), (1.1 / v, 0)]:
        acc, nxt, q = oracle.verify_accept(lg, dr, r)
        np.testing.assert_allclose(q, 1.0 / v, rtol=1e-12)
        assert acc[0] == want
        assert nxt[0] == (-1 if want == 4 else 0)


def test_probabilities_match_torch_softmax():
    torch = pytest.importorskip("torch")
    lg, dr = verify_inputs(31, 2, 4, 1000, 2.0, rows=5)
    for tau in (1.0, 0.6):
        _, _, q = oracle.verify_accept(lg, dr, 0.1, tau)
        p = torch.softmax(torch.from_numpy(lg).to(torch.float64) / tau, dim=-1).numpy()
        want = np.take_along_axis(p[:, :4, :], dr[:, :, None].astype(np.int64), axis=2)[:, :, 0]
        np.testing.assert_allclose(q, want, rtol=1e-12)


def test_accept_len_is_first_rejection_by_bruteforce_and_monotone_in_r():
    lg, dr = verify_inputs(32, 6, 16, 1000, 2.0, rows=17, calibrated=True)
    prev = None
    for r in [0.0, 0.05, 0.1, 0.3, 0.5, 0.9, 1.0]:
        acc, nxt, q = oracle.verify_accept(lg, dr, r)
        for b in range(6):
            j = next((k for k in range(16) if q[b, k] < r), 16)
            assert acc[b] == j
            row = lg[b, j]
            assert nxt[b] == int(np.flatnonzero(row == row.max())[0])
            if prev is not None:
                assert acc[b] <= prev[b]  # a larger threshold never lengthens the advance
        prev = acc


def test_calibrated_generator_spreads_acceptance():
    # Guards the test workload itself: the literal recipe at a large vocabulary rejects at 0 almost always.
    lg, dr = verify_inputs(33, 8, 16, 4096, 3.0, calibrated=True)
    acc, _, _ = oracle.verify_accept(lg, dr, 0.1)
    assert len(set(acc.tolist())) >= 3
