"""Pins of the tree oracle (Sec. 4, hardware-friendly tree building and tree verification)."""

import json
import math
import os

import numpy as np
import pytest

import oracle
from synth import verify_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tree_hand_cases.json")


def _num(s):
    if s.startswith("ln"):
        return math.log(float(s[2:]))
    return float(s)


def _expr(s):
    return float(eval(s, {"__builtins__": {}}, {"log": math.log}))  # fixture expressions only


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("case", _golden()["build"], ids=lambda c: c["name"])
def test_build_hand_cases(case):
    lg = np.array([[_num(v) for v in row] for row in case["logits"]])
    cum = None if case["cum"] is None else np.array([_expr(e) for e in case["cum"]])
    tok, par, out = oracle.tree_build_step(lg, cum, case["width"])
    assert tok.tolist() == case["tokens"]
    assert par.tolist() == case["parents"]
    np.testing.assert_allclose(out, [_expr(e) for e in case["cum_out"]], rtol=1e-12)


@pytest.mark.parametrize("case", _golden()["verify"], ids=lambda c: c["name"])
def test_verify_hand_cases(case):
    lg = np.array([[[_num(v) for v in row] for row in step] for step in case["logits"]])
    bonus = None
    if "bonus" in case:
        bonus = np.array([[_num(v) for v in row] for row in case["bonus"]])
    best, acc, nxt, q, adv = oracle.tree_verify(lg, np.array(case["tokens"]), np.array(case["parents"]),
                                                case["r"], case["temperature"], bonus)
    assert (best, acc, nxt) == (case["best_leaf"], case["accept_len"], case["next_token"])
    assert adv.tolist() == case["advance"]
    np.testing.assert_allclose(q, [[_expr(e) for e in row] for row in case["q"]], rtol=1e-12)


def test_width_one_build_is_greedy():
    rng = np.random.default_rng(3)
    lg = rng.normal(size=(1, 500)) * 2.0
    tok, par, cum = oracle.tree_build_step(lg, None, 1)
    assert tok.tolist() == [int(np.argmax(lg[0]))] and par.tolist() == [0]
    np.testing.assert_allclose(cum[0], np.max(lg[0]) - np.log(np.sum(np.exp(lg[0]))), rtol=1e-12)


def test_width_one_verify_is_the_chain_check():
    """W = 1: the tree is a chain and tree_verify must agree with verify_accept exactly."""
    for seed in range(6):
        lg, dr = verify_inputs(70 + seed, 1, 6, 300, 2.0, rows=7, calibrated=True)
        for r in (0.05, 0.3):
            acc, nxt, q = oracle.verify_accept(lg, dr, r, 0.6)
            best, a2, n2, q2, _ = oracle.tree_verify(lg[0, :6, None, :], dr[0][:, None], np.zeros((6, 1), int),
                                                     r, 0.6, bonus=lg[0, 6:7])
            assert best == 0 and a2 == int(acc[0]) and n2 == int(nxt[0])
            np.testing.assert_allclose(q2[:, 0], q[0], rtol=1e-12)


def test_build_step_is_the_top_w_of_all_expansions_by_brute_force():
    rng = np.random.default_rng(5)
    for trial in range(5):
        wc, v, w = 3, 7, 5
        lg = rng.normal(size=(wc, v))
        cum = -np.abs(rng.normal(size=wc))
        if trial == 0:
            lg[1] = lg[0]  # ties across parents
            cum[1] = cum[0]
        tok, par, out = oracle.tree_build_step(lg, cum, w)
        cands = []
        for p in range(wc):
            z = lg[p] - np.max(lg[p])
            lp = z - math.log(sum(math.exp(t) for t in z))
            for t in range(v):
                cands.append((-(cum[p] + lp[t]), p, t))
        cands.sort()
        assert [(c[1], c[2]) for c in cands[:w]] == list(zip(par.tolist(), tok.tolist()))
        np.testing.assert_allclose(out, [-c[0] for c in cands[:w]], rtol=1e-12)
        assert np.all(np.diff(out) <= 0) and np.all(out <= cum[par] + 1e-15)


def test_each_path_advances_like_the_chain_check_of_its_own_rows():
    """Every leaf's advance equals verify_accept on the rows along its path."""
    rng = np.random.default_rng(9)
    k_n, w_n, v_n = 5, 4, 50
    for trial in range(8):
        lg = rng.normal(size=(k_n, w_n, v_n)) * 2.0
        tok = rng.integers(0, v_n, size=(k_n, w_n))
        for i in range(k_n):  # make most drafted tokens likely so that advances vary
            for w in range(w_n):
                if rng.random() < 0.8:
                    lg[i, w, tok[i, w]] = lg[i, w].max() + rng.uniform(0, 6)
        par = np.vstack([np.full(w_n, -1), rng.integers(0, w_n, size=(k_n - 1, w_n))])
        best, acc, nxt, q, adv = oracle.tree_verify(lg, tok, par, 0.3, 1.0)
        path = oracle.tree_paths(par)
        for leaf in range(w_n):
            rows = lg[np.arange(k_n), path[leaf]][None]
            dr = tok[np.arange(k_n), path[leaf]][None]
            a, n, _ = oracle.verify_accept(rows, dr, 0.3, 1.0)
            assert adv[leaf] == a[0]
            if leaf == best and a[0] < k_n:
                assert nxt == n[0]
        assert acc == adv.max() and best == int(np.flatnonzero(adv == adv.max())[0])


def test_paths_follow_parent_links():
    # K = 3, W = 3; leaf 0: step-2 slot 0 -> parent 1 at step 1 -> parent 0 at step 0
    par = np.array([[-1, -1, -1], [2, 0, 0], [1, 1, 2]])
    assert oracle.tree_paths(par).tolist() == [[0, 1, 0], [0, 1, 1], [0, 2, 2]]
