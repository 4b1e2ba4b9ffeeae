"""Pins for the generation-loop oracle (Algorithm 1 on a small random-weight decoder).

The loop oracle keeps one shared KV cache, rewrites it with the full model's pass and rolls
it back. These tests restate the same procedure without any cache: every logit is recomputed
from the whole token sequence with plain per-position loops, the positions before the
period's first input taking the full model's path and the drafted positions the sparse
model's (that is the cache's content in Algorithm 1: the full model rewrote every committed
row). A wrong rollback position, a stale sparse row left in the cache, a wrong row-to-token
alignment or a lost corrected token changes the committed tokens and fails them. Two special
cases reduce to plain greedy decoding by the full model: r > 1 rejects every draft, and a
sparse model with every neuron kept and r <= 0 accepts every draft.
"""

import dataclasses
import math

import numpy as np
import pytest

from oracle import loop
from oracle.ffn import widen_bf16
from synth import model_weights, prompt_tokens, ModelShape, bf16_bits

SMALL = ModelShape("small-decoder", 2, 32, 48, 4, 2, 8, 50, 64, 6.0)


def _model(shape=SMALL, seed=3, q=0.5):
    bits = model_weights(seed, shape)
    m = loop.model_from_bits(bits, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                             np.zeros(shape.n_layers))
    m.thresholds = loop.calibrate_thresholds(m, prompt_tokens(seed + 100, 24, shape.vocab), q,
                                             shape.max_len)
    return m


# ---------------------------------------------------------------- cache-free restatement

def _silu(z):
    return z / (1.0 + math.exp(-z))


def _rms(v):
    return [e / math.sqrt(sum(x * x for x in v) / len(v) + 1e-5) for e in v]


def _matvec(w, v):
    return [sum(w[i][k] * v[k] for k in range(len(v))) for i in range(len(w))]


def _nocache_logits(m, tokens, sparse_from):
    """Logits of every position of `tokens`, recomputed from scratch with plain loops:
    positions >= sparse_from take the sparse FFN (threshold rule), the others the dense one;
    keys and values are rounded to bf16 as the cache stores them."""
    H, Hkv, hd = m.n_heads, m.n_kv_heads, m.head_dim
    g = H // Hkv
    T = len(tokens)
    h = [list(m.embed[t]) for t in tokens]
    for layer in range(m.n_layers):
        wq, wk, wv, wo = (m.wq[layer].tolist(), m.wk[layer].tolist(), m.wv[layer].tolist(),
                          m.wo[layer].tolist())
        xn = [_rms(h[p]) for p in range(T)]
        qs = [_matvec(wq, xn[p]) for p in range(T)]
        ks = [list(loop.round_bf16(np.array(_matvec(wk, xn[p])))) for p in range(T)]
        vs = [list(loop.round_bf16(np.array(_matvec(wv, xn[p])))) for p in range(T)]
        for p in range(T):
            att = []
            for head in range(H):
                kvh = head // g
                qv = qs[p][head * hd:(head + 1) * hd]
                sc = [sum(qv[e] * ks[u][kvh * hd + e] for e in range(hd)) / math.sqrt(hd)
                      for u in range(p + 1)]
                mx = max(sc)
                w = [math.exp(s - mx) for s in sc]
                z = sum(w)
                att += [sum(w[u] * vs[u][kvh * hd + e] for u in range(p + 1)) / z for e in range(hd)]
            o = _matvec(wo, att)
            h[p] = [h[p][e] + o[e] for e in range(len(o))]
        wg, wu, wd = m.w_gate[layer].tolist(), m.w_up[layer].tolist(), m.w_down[layer].tolist()
        for p in range(T):
            xf = _rms(h[p])
            gg, uu = _matvec(wg, xf), _matvec(wu, xf)
            y = [0.0] * len(xf)
            for i in range(len(wg)):
                a = _silu(gg[i])
                if p >= sparse_from and not abs(a) > m.thresholds[layer]:
                    continue
                for e in range(len(xf)):
                    y[e] += a * uu[i] * wd[i][e]
            h[p] = [h[p][e] + y[e] for e in range(len(y))]
    return [_matvec(m.lm_head.tolist(), _rms(h[p])) for p in range(T)]


def _argmax(row):
    return max(range(len(row)), key=lambda i: (row[i], -i))


def _prob(row, tok):
    mx = max(row)
    return math.exp(row[tok] - mx) / sum(math.exp(v - mx) for v in row)


def _nocache_generate(m, prompt, n, r, periods):
    seqall = [int(t) for t in prompt]
    committed, accepts = [], []
    for _ in range(periods):
        P = len(seqall) - 1
        seq = [seqall[-1]]
        for i in range(n):
            lg = _nocache_logits(m, seqall + seq[1:], P)
            seq.append(_argmax(lg[-1]))
        lg = _nocache_logits(m, seqall + seq[1:n], len(seqall) + n)  # the full model everywhere
        j = n
        for i in range(n):
            if _prob(lg[P + i], seq[i + 1]) < r:
                j = i
                break
        new = seq[1:j + 1] + ([_argmax(lg[P + j])] if j < n else [])
        committed += new
        seqall += new
        accepts.append(j)
    return committed, accepts


def _greedy_full(m, prompt, count):
    seq = [int(t) for t in prompt]
    for _ in range(count):
        seq.append(_argmax(_nocache_logits(m, seq, len(seq) + 1)[-1]))
    return seq[len(prompt):]


# ---------------------------------------------------------------- pins

def test_round_bf16_hand_values():
    # 1 + 2^-8 lies halfway between 1 and 1 + 2^-7: ties go to the even mantissa (1.0);
    # 1 + 3 2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6: even is 1 + 2^-6.
    vals = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -30,
                     -(1.0 + 2.0 ** -8), 3.0, 0.1, -1e-3])
    want = np.array([1.0, 1.0 + 2.0 ** -6, 1.0 + 2.0 ** -7, -1.0, 3.0])
    got = loop.round_bf16(vals)
    assert np.array_equal(got[:5], want)
    # values representable in fp32 agree with the storage conversion of the input generators
    rng = np.random.default_rng(0)
    f = rng.standard_normal(10000).astype(np.float32) * np.float32(7.0)
    assert np.array_equal(loop.round_bf16(f.astype(np.float64)), widen_bf16(bf16_bits(f)))


def test_thresholds_hit_the_target_sparsity():
    m = _model()
    for q in (0.4, 0.5, 0.65):
        t = loop.calibrate_thresholds(m, prompt_tokens(103, 24, SMALL.vocab), q, SMALL.max_len)
        assert t.shape == (SMALL.n_layers,) and np.all(t > 0)
    # layer 0's FFN input only depends on the token embedding through attention; check the
    # count of values above t_0 on the calibration set directly: M - ceil(q M)
    q = 0.5
    toks = prompt_tokens(103, 24, SMALL.vocab)
    t = loop.calibrate_thresholds(m, toks, q, SMALL.max_len)
    cache = loop.new_cache(m, SMALL.max_len)
    # one dense pass, collecting layer 0's gate activations through the sparse path's sets:
    # with threshold t_0 the sparse model keeps exactly the values above it
    m2 = dataclasses.replace(m, thresholds=np.array([t[0], -1.0]))
    _, sets = loop.forward(m2, toks, cache, 0, True)
    kept = sum(len(s) for s in sets[0])
    M = len(toks) * SMALL.d_ff
    assert kept == M - math.ceil(q * M)


@pytest.mark.parametrize("seed,r", [(5, 0.3), (7, 0.5)])
def test_cached_loop_equals_cache_free_restatement(seed, r):
    m = _model(seed=seed)
    prompt = prompt_tokens(7, 5, SMALL.vocab)
    n, periods = 4, 5
    out, recs, _, pos = loop.generate(m, prompt, n, r, periods, SMALL.max_len)
    ref, accepts = _nocache_generate(m, prompt, n, r, periods)
    assert [rc.accept for rc in recs] == accepts
    assert out == ref
    assert pos == len(prompt) - 1 + len(out)
    assert loop.aal(recs) == len(out) / periods
    # a mix of outcomes, so that rollback and interleaving are both exercised
    assert 0 in accepts and n in accepts and any(0 < a < n for a in accepts)


def test_reject_everything_is_full_model_greedy_decoding():
    m = _model()
    prompt = prompt_tokens(8, 4, SMALL.vocab)
    out, recs, _, _ = loop.generate(m, prompt, 3, 1.5, 6, SMALL.max_len)
    assert [rc.accept for rc in recs] == [0] * 6
    assert out == _greedy_full(m, prompt, 6)
    assert loop.aal(recs) == 1.0


def test_dense_draft_accept_everything_is_full_model_greedy_decoding():
    m = _model()
    m.thresholds = np.full(SMALL.n_layers, -1.0)  # the sparse model keeps every neuron
    prompt = prompt_tokens(9, 4, SMALL.vocab)
    n = 4
    out, recs, _, _ = loop.generate(m, prompt, n, 0.0, 3, SMALL.max_len)
    assert [rc.accept for rc in recs] == [n] * 3
    assert [rc.corrected for rc in recs] == [-1] * 3
    assert out == _greedy_full(m, prompt, 3 * n)
    # with the drafts equal to the full model's own greedy tokens, a draft is rejected only
    # when its (maximal) probability is below r
    out2, recs2, _, _ = loop.generate(m, prompt, n, 0.5, 3, SMALL.max_len)
    for rc in recs2:
        assert rc.accept == next((i for i, qq in enumerate(rc.q) if qq < 0.5), n)
        if rc.accept < n:
            assert rc.corrected == rc.seq[rc.accept + 1]  # the full model's argmax is the draft


def test_full_pass_input_rounding_only_moves_the_full_model():
    """The bf16 rounding of the full model's FFN input changes the check's logits by about
    the rounding error and leaves the drafts' logits (sparse model, rows not yet rewritten)
    untouched."""
    m = _model()
    prompt = prompt_tokens(10, 5, SMALL.vocab)
    c1 = loop.new_cache(m, SMALL.max_len)
    c2 = loop.new_cache(m, SMALL.max_len)
    a, _ = loop.forward(m, prompt, c1, 0, False)
    b, _ = loop.forward(m, prompt, c2, 0, False, full_ffn_input_bf16=True)
    d = np.abs(a - b).max() / np.abs(a).max()
    assert 0 < d < 0.05
    s1, _ = loop.forward(m, prompt, loop.new_cache(m, SMALL.max_len), 0, True)
    s2, _ = loop.forward(m, prompt, loop.new_cache(m, SMALL.max_len), 0, True, full_ffn_input_bf16=True)
    assert np.array_equal(s1, s2)


@pytest.mark.parametrize("n", [1, 2])
def test_small_kernels(n):
    m = _model(seed=5)
    prompt = prompt_tokens(11, 3, SMALL.vocab)
    out, recs, _, pos = loop.generate(m, prompt, n, 0.3, 4, SMALL.max_len)
    ref, accepts = _nocache_generate(m, prompt, n, 0.3, 4)
    assert out == ref and [rc.accept for rc in recs] == accepts
    assert pos == len(prompt) - 1 + len(out)
