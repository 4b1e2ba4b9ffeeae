"""GPU parity: correction check (likelihood of drafted tokens, first rejection, corrected token)."""

import json
import math
import os

import numpy as np
import pytest

import oracle
from synth import verify_inputs, VERIFY_TINY, VERIFY_8B
from gpu_util import say, dev_f32, dev_i32, host, verify_boundary_rows, MAX_BOUNDARY_ROWS

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "verify_hand_cases.json")


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


def _run_and_check(sr, lg, dr, r, tau):
    acc, nxt, p = sr.sirius_verify_accept(dev_f32(lg), dev_i32(dr), r, tau)
    acc, nxt, p = host(acc), host(nxt), host(p)
    acc_o, nxt_o, q_o = oracle.verify_accept(lg, dr, r, tau)
    skip = set(verify_boundary_rows(q_o, acc_o, r))
    assert len(skip) <= MAX_BOUNDARY_ROWS, f"{len(skip)} rows inside the guard band of r"
    for b in range(lg.shape[0]):
        if b in skip:
            continue
        assert acc[b] == acc_o[b], (b, acc[b], acc_o[b])
        assert nxt[b] == nxt_o[b], (b, nxt[b], nxt_o[b])
    np.testing.assert_allclose(p, q_o, rtol=1e-5, atol=1e-12)
    return acc, len(skip)


def test_hand_cases_on_gpu(sr):
    with open(GOLDEN) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        say(f"verify hand case: {c['name']}")
        rows = np.array([[math.log(4.0) if v == "ln4" else float(v) for v in row] for row in c["rows"]],
                        dtype=np.float32)[None]
        dr = np.array([c["drafted"]], dtype=np.int32)
        acc, nxt, p = sr.sirius_verify_accept(dev_f32(rows), dev_i32(dr), c["r"], c["temperature"])
        assert int(host(acc)[0]) == c["accept_len"], c["name"]
        assert int(host(nxt)[0]) == c["next_token"], c["name"]


@pytest.mark.parametrize("rows_extra", [0, 1])
@pytest.mark.parametrize("tau", [1.0, 0.6])
def test_tiny_config(sr, rows_extra, tau):
    k, v = VERIFY_TINY.k, VERIFY_TINY.vocab
    for seed in range(4):
        say(f"verify tiny seed={seed} R=K+{rows_extra} tau={tau}")
        lg, dr = verify_inputs(seed, 3, k, v, VERIFY_TINY.logit_var, rows=k + rows_extra, calibrated=(seed % 2 == 1))
        _run_and_check(sr, lg, dr, 0.1, tau)


def test_odd_vocab_scalar_path_and_out_of_range_ids(sr):
    lg, dr = verify_inputs(11, 4, 5, 1001, 2.0, rows=6, calibrated=True)
    dr[0, 2] = -3
    dr[1, 0] = 1001
    say("verify odd vocab")
    _run_and_check(sr, lg, dr, 0.1, 1.0)
    lg2, dr2 = verify_inputs(12, 2, 3, 7, 1.0)
    _run_and_check(sr, lg2, dr2, 0.3, 1.0)


@pytest.mark.parametrize("calibrated", [False, True])
def test_llama3_vocab(sr, calibrated):
    s = VERIFY_8B
    for r in (0.05, 0.1, 0.3):
        for tau in (1.0, 0.6):
            say(f"verify 8x16x128256 calibrated={calibrated} r={r} tau={tau}")
            lg, dr = verify_inputs(20, s.batch, s.k, s.vocab, s.logit_var, rows=s.k + 1, calibrated=calibrated)
            acc, nskip = _run_and_check(sr, lg, dr, r, tau)
            say(f"  accept_len={acc.tolist()} boundary rows={nskip}")


def test_ties_in_argmax_across_segments(sr):
    # the maximum appears in several segments of a long row: the lowest index must win
    v = 128256
    lg = np.zeros((1, 2, v), dtype=np.float32)
    for pos in (100000, 70001, 9000, 127999):
        lg[0, 0, pos] = 5.0
    lg[0, 1, 5] = 1.0
    dr = np.array([[3]], dtype=np.int32)
    acc, nxt, _ = sr.sirius_verify_accept(dev_f32(lg), dev_i32(dr), 0.5, 1.0)
    assert int(host(acc)[0]) == 0 and int(host(nxt)[0]) == 9000


def test_long_rows_cap_the_segment_count(sr):
    # a single long row: more than 64 segments of 2048 would be wanted; the count is capped
    for v, rows in ((300000, 2), (262147, 2)):
        say(f"verify V={v}")
        lg, dr = verify_inputs(40, 2, 1, v, 3.0, rows=rows, calibrated=True)
        _run_and_check(sr, lg, dr, 0.1, 1.0)


@pytest.mark.parametrize("bsz", [255, 256, 257, 300])
def test_many_batch_entries(sr, bsz):
    """Hundreds of batch entries (one scan workgroup each), two calls in a row."""
    k, v = VERIFY_TINY.k, VERIFY_TINY.vocab
    for rep in range(2):
        say(f"verify B={bsz} rep={rep}")
        lg, dr = verify_inputs(900 + bsz + rep, bsz, k, v, VERIFY_TINY.logit_var, rows=k + 1)
        _run_and_check(sr, lg, dr, 0.1, 1.0)
