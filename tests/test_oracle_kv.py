"""Pins of the KV-cache oracle (Algorithm 1; Sec. 4, how to correct): attention over the shared
cache with the direct rewrite, and the rollback after the check."""

import math

import numpy as np
import pytest

import oracle


def _rand(seed, bsz, n, h, hkv, hd, lmax):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((bsz, n, h, hd))
    kn, vn = rng.standard_normal((2, bsz, n, hkv, hd))
    kc, vc = rng.standard_normal((2, bsz, lmax, hkv, hd))
    return q, kn, vn, kc, vc


def test_hand_case_two_positions():
    # scale 1/sqrt(2); q = (sqrt(2) ln 3, 0): score 0 against k0 = (0, 0) and ln 3 against the new
    # key (1, 0), so the weights are 1/4 and 3/4 and the output mixes v0 = (4, 0), v1 = (0, 8)
    q = np.array([[[[math.sqrt(2.0) * math.log(3.0), 0.0]]]])
    kc = np.array([[[[0.0, 0.0]], [[9.0, 9.0]]]])  # row 1 is overwritten by the new key
    vc = np.array([[[[4.0, 0.0]], [[7.0, 7.0]]]])
    kn = np.array([[[[1.0, 0.0]]]])
    vn = np.array([[[[0.0, 8.0]]]])
    out, k2, v2 = oracle.attn_kv(q, kn, vn, kc, vc, [1])
    np.testing.assert_allclose(out[0, 0, 0], [1.0, 6.0], rtol=1e-14)
    assert k2[0, 1, 0].tolist() == [1.0, 0.0] and v2[0, 1, 0].tolist() == [0.0, 8.0]


def test_one_visible_position_returns_its_value():
    q, kn, vn, kc, vc = _rand(1, 2, 1, 4, 2, 8, 6)
    out, _, _ = oracle.attn_kv(q, kn, vn, kc, vc, [0, 0])
    for h in range(4):
        np.testing.assert_allclose(out[:, 0, h], vn[:, 0, h // 2], rtol=1e-14)


def test_equal_keys_average_the_visible_values():
    q, kn, vn, kc, vc = _rand(2, 1, 3, 2, 1, 4, 9)
    kc[:] = 0.5
    kn[:] = 0.5
    out, _, v2 = oracle.attn_kv(q, kn, vn, kc, vc, [4])
    for i in range(3):
        want = v2[0, :4 + i + 1, 0].mean(axis=0)
        for h in range(2):
            np.testing.assert_allclose(out[0, i, h], want, rtol=1e-13)


def test_matches_scalar_loops():
    q, kn, vn, kc, vc = _rand(3, 2, 3, 4, 2, 8, 10)
    pos = [2, 5]
    out, _, _ = oracle.attn_kv(q, kn, vn, kc, vc, pos)
    for b in range(2):
        keys, vals = kc[b].copy(), vc[b].copy()
        keys[pos[b]:pos[b] + 3] = kn[b]
        vals[pos[b]:pos[b] + 3] = vn[b]
        for i in range(3):
            for h in range(4):
                kvh = h // 2
                s = [sum(q[b, i, h, c] * keys[j, kvh, c] for c in range(8)) / math.sqrt(8.0)
                     for j in range(pos[b] + i + 1)]
                m = max(s)
                w = [math.exp(x - m) for x in s]
                z = sum(w)
                want = [sum(w[j] * vals[j, kvh, c] for j in range(len(w))) / z for c in range(8)]
                np.testing.assert_allclose(out[b, i, h], want, rtol=1e-12)


def test_grouped_heads_equal_repeated_heads():
    q, kn, vn, kc, vc = _rand(4, 1, 2, 4, 2, 8, 7)
    out, _, _ = oracle.attn_kv(q, kn, vn, kc, vc, [3])
    rep = lambda a: np.repeat(a, 2, axis=2)  # kv head h // 2 for query head h
    out2, _, _ = oracle.attn_kv(q, rep(kn), rep(vn), rep(kc), rep(vc), [3])
    np.testing.assert_allclose(out, out2, rtol=1e-14)


def test_causal_and_rewrite_only_the_chunk():
    q, kn, vn, kc, vc = _rand(5, 1, 4, 2, 1, 8, 12)
    out, k2, v2 = oracle.attn_kv(q, kn, vn, kc, vc, [5])
    kn2, vn2 = kn.copy(), vn.copy()
    kn2[0, 3] += 1.0
    vn2[0, 3] -= 2.0
    out3, _, _ = oracle.attn_kv(q, kn2, vn2, kc, vc, [5])
    np.testing.assert_array_equal(out3[0, :3], out[0, :3])  # earlier tokens do not see token 3
    assert not np.allclose(out3[0, 3], out[0, 3])
    np.testing.assert_array_equal(k2[0, :5], kc[0, :5])
    np.testing.assert_array_equal(k2[0, 9:], kc[0, 9:])
    np.testing.assert_array_equal(k2[0, 5:9], kn[0])
    np.testing.assert_array_equal(v2[0, 5:9], vn[0])


def test_shifting_every_key_changes_nothing():
    # q . (k + c) adds the same q . c to every score of a row: softmax is unchanged
    q, kn, vn, kc, vc = _rand(6, 1, 2, 2, 1, 8, 6)
    out, _, _ = oracle.attn_kv(q, kn, vn, kc, vc, [2])
    c = np.linspace(-1.0, 1.0, 8)
    out2, _, _ = oracle.attn_kv(q, kn + c, vn, kc + c, vc, [2])
    np.testing.assert_allclose(out2, out, rtol=1e-12, atol=1e-12)


def test_rollback_hand_cases():
    # chunk of n = 16 at position 10: rejecting the first drafted token keeps one input row
    assert oracle.kv_rollback([10, 10, 10, 10], [0, 5, 15, 16], 16).tolist() == [11, 16, 26, 26]
    assert oracle.kv_rollback([0], [0], 1).tolist() == [1]


def test_out_of_range_position_is_rejected():
    q, kn, vn, kc, vc = _rand(7, 1, 3, 2, 1, 4, 5)
    with pytest.raises(ValueError):
        oracle.attn_kv(q, kn, vn, kc, vc, [3])
