"""Pins of the per-token top-k oracle (the paper's own fine-grained implementation, Sec. 3
footnote): hand-computed selections, ties, reductions to the dense FFN and to threshold
sparsity, and a brute-force sort."""

import math

import numpy as np
import pytest

import oracle


def _one_hot_layer(gates):
    """d_model = F = len(gates); x = e_0; gate row i = (g_i, 0, ...); up rows (1, 0, ...);
    down row i = e_i, so y_i = a_i = SiLU(g_i) for a kept neuron i and 0 otherwise."""
    f = len(gates)
    x = np.zeros((1, f))
    x[0, 0] = 1.0
    wg = np.zeros((f, f))
    wg[:, 0] = gates
    wu = np.zeros((f, f))
    wu[:, 0] = 1.0
    wd = np.eye(f)
    return x, wg, wu, wd


def test_hand_case_five_neurons():
    # SiLU(ln 3) = 0.75 ln 3 = 0.824; SiLU(-ln 3) = -0.25 ln 3 = -0.275; SiLU(ln 9) = 0.9 ln 9
    # = 1.978; SiLU(0) = 0; SiLU(-ln 9) = -0.1 ln 9 = -0.220. Order by |a|: 2, 0, 1, 4, 3.
    l3, l9 = math.log(3.0), math.log(9.0)
    x, wg, wu, wd = _one_hot_layer([l3, -l3, l9, 0.0, -l9])
    a = [0.75 * l3, -0.25 * l3, 0.9 * l9, 0.0, -0.1 * l9]
    for k, want in [(1, [2]), (2, [0, 2]), (3, [0, 1, 2]), (4, [0, 1, 2, 4]), (5, [0, 1, 2, 3, 4])]:
        y, sets = oracle.ffn_topk(x, wg, wu, wd, k)
        assert sets[0].tolist() == want, k
        np.testing.assert_allclose(y[0], [a[i] if i in want else 0.0 for i in range(5)], rtol=1e-14, atol=1e-300)


def test_ties_go_to_the_lower_index():
    g = math.log(3.0)
    x, wg, wu, wd = _one_hot_layer([0.1, g, 0.2, g, g])
    assert oracle.topk_active_sets(x, wg, 1)[0][0].tolist() == [1]
    assert oracle.topk_active_sets(x, wg, 2)[0][0].tolist() == [1, 3]
    assert oracle.topk_active_sets(x, wg, 4)[0][0].tolist() == [1, 2, 3, 4]


def _small(seed, b, d, f):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((b, d))
    wg, wu, wd = (rng.standard_normal((f, d)) / math.sqrt(d) for _ in range(3))
    return x, wg, wu, wd


def test_all_neurons_is_the_dense_ffn_bitwise():
    x, wg, wu, wd = _small(1, 3, 24, 40)
    y, sets = oracle.ffn_topk(x, wg, wu, wd, 40)
    assert all(s.tolist() == list(range(40)) for s in sets)
    assert np.array_equal(y, oracle.ffn_dense(x, wg, wu, wd))


def test_matches_a_brute_force_sort():
    x, wg, wu, wd = _small(2, 4, 16, 50)
    for k in (1, 7, 25, 49):
        sets, _ = oracle.topk_active_sets(x, wg, k)
        for b in range(4):
            act = []
            for i in range(50):
                g = sum(float(wg[i][c]) * float(x[b][c]) for c in range(16))
                act.append((-abs(g / (1.0 + math.exp(-g))), i))
            want = sorted(i for _, i in sorted(act)[:k])
            assert sets[b].tolist() == want


def test_equals_threshold_sparsity_at_the_next_value():
    # with distinct magnitudes, top-k keeps exactly the neurons above the (k+1)-th largest |a|
    x, wg, wu, wd = _small(3, 3, 32, 64)
    a = np.abs(oracle.gate_activations(x, wg))
    for k in (1, 10, 32, 63):
        sets, _ = oracle.topk_active_sets(x, wg, k)
        for b in range(3):
            t = np.sort(a[b])[::-1][k]
            cats, _ = oracle.cats_active_sets(x, wg, t)  # the same batched gate product
            assert sets[b].tolist() == cats[b].tolist()


def test_sets_are_nested_and_exactly_k():
    x, wg, wu, wd = _small(4, 2, 16, 30)
    prev = [set() for _ in range(2)]
    for k in range(1, 31):
        sets, _ = oracle.topk_active_sets(x, wg, k)
        for b in range(2):
            assert len(sets[b]) == k and prev[b] <= set(sets[b].tolist())
            prev[b] = set(sets[b].tolist())


def test_k_outside_the_layer_is_rejected():
    x, wg, wu, wd = _small(5, 1, 8, 10)
    for k in (0, 11):
        with pytest.raises(ValueError):
            oracle.topk_active_sets(x, wg, k)
