"""Oracle: the Sirius generation loop (Algorithm 1) on a small decoder with random weights.

Test infrastructure only (see the package docstring). Float64.

Algorithm 1 runs two models that share their weights and one KV cache: the sparse model
M_S drafts a chunk ("kernel") of n tokens one at a time, writing its keys and values into
the cache; the cache position is then wound back by n and the full model M_F runs the n
tokens of the chunk in one pass, rewriting the same cache rows directly; the first drafted
token whose full-model likelihood falls below the threshold r is rejected, the cache
position rolls back to just after the accepted prefix, and the full model's own token takes
the rejected token's place ("interleaving key token"). Sec. 4 ("How to correct") describes
the same procedure in prose.

The paper does not spell out the model; the readings adopted here (the design notes list
them) are:

  * a Llama-style pre-norm decoder: token embedding E; per layer an attention block
    h <- h + W_o attn(RMSNorm(h)) with grouped-query heads (query head h reads key/value
    head h // (H / Hkv)), scores q . k / sqrt(hd), no positional rotation (mechanics only),
    and an FFN block h <- h + FFN(RMSNorm(h)); final RMSNorm and an LM head W_lm; RMSNorm
    with unit weight and eps 1e-5;
  * the cache stores keys and values in bf16 (round to nearest even of the exact value);
  * M_F's FFN is the dense SwiGLU FFN; M_S's is the threshold-sparse one (the CATS rule of
    the FFN oracle, threshold t_l per layer: neuron i kept iff |SiLU(g_i)| > t_l);
  * the full model's multi-token FFN may consume its normalised input rounded to bf16
    (``full_ffn_input_bf16``), the operand format of a matrix-core pass;
  * sampling is greedy (argmax, lowest index on ties) for both the drafts and the
    corrected token -- the paper samples at temperature 0.6, but any sampler serves the
    mechanics and greedy keeps them deterministic;
  * index alignment: with s_0 the period's first input (already committed, not yet in the
    cache) at position P, draft step i feeds s_i at P + i and drafts s_{i+1}; the check
    feeds s_0 .. s_{n-1} at P .. P + n - 1, and its row i is the likelihood of s_{i+1};
    with j the first rejected row (j = n if none), the tokens s_1 .. s_j are accepted, the
    position becomes P + min(j + 1, n), and the next input is argmax of row j when j < n
    (the corrected token, committed too), else s_n.

Each period commits j + 1 tokens when j < n, n tokens when j = n; the average over periods
is the average advance length AAL of Sec. 2.2.
"""

from __future__ import annotations

import dataclasses

import numpy as np

from .ffn import widen_bf16, silu, rmsnorm
from .kv import attn_kv

NORM_EPS = 1e-5


def round_bf16(a) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even), kept as float64.

    bf16 keeps 8 significant bits: with a = m 2^e and 0.5 <= |m| < 1, the result is
    rint(256 m) / 256 * 2^e (numpy's rint rounds halves to even). Finite normal inputs.
    """
    a = np.asarray(a, dtype=np.float64)
    m, e = np.frexp(a)
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


@dataclasses.dataclass
class Model:
    """Weights of the small decoder, float64 copies of the stored bf16 values.

    embed [V, d]; wq [L, H hd, d]; wk, wv [L, Hkv hd, d]; wo [L, d, H hd];
    w_gate, w_up, w_down [L, F, d] (neuron-major); lm_head [V, d]; thresholds [L] (M_S).
    """
    n_heads: int
    n_kv_heads: int
    head_dim: int
    embed: np.ndarray
    wq: np.ndarray
    wk: np.ndarray
    wv: np.ndarray
    wo: np.ndarray
    w_gate: np.ndarray
    w_up: np.ndarray
    w_down: np.ndarray
    lm_head: np.ndarray
    thresholds: np.ndarray

    @property
    def n_layers(self) -> int:
        return self.wq.shape[0]

    @property
    def vocab(self) -> int:
        return self.embed.shape[0]


def model_from_bits(bits: dict, n_heads: int, n_kv_heads: int, head_dim: int, thresholds) -> Model:
    """Model from bf16 bit patterns (uint16 arrays keyed like the Model fields)."""
    w = {k: widen_bf16(bits[k]) for k in ("embed", "wq", "wk", "wv", "wo", "w_gate", "w_up",
                                         "w_down", "lm_head")}
    return Model(n_heads, n_kv_heads, head_dim, thresholds=np.asarray(thresholds, np.float64), **w)


def new_cache(m: Model, max_len: int):
    """Empty shared cache: per layer (keys, values) [1, max_len, Hkv, hd]."""
    shape = (1, max_len, m.n_kv_heads, m.head_dim)
    return [(np.zeros(shape), np.zeros(shape)) for _ in range(m.n_layers)]


def forward(m: Model, tokens, cache, pos: int, sparse: bool, *, active_sets=None,
            full_ffn_input_bf16: bool = False, acts=None):
    """One pass of M_S (sparse=True) or M_F over tokens at positions pos .. pos + n - 1.

    The tokens' keys and values replace the cache rows at those positions (the cache list is
    updated in place) and token i attends to rows 0 .. pos + i. active_sets, when given,
    is [layer][token] -> the neuron set M_S uses instead of its threshold rule (so a caller
    can replay another implementation's sets). Returns (logits [n, V], sets) where sets is
    [layer][token] -> the ascending neuron set used (M_S) or None (M_F). When acts is a list,
    each layer's gate activations SiLU(g) [n, d_ff] are appended to it.
    """
    toks = np.asarray(tokens, dtype=np.int64)
    n = toks.shape[0]
    H, Hkv, hd = m.n_heads, m.n_kv_heads, m.head_dim
    h = m.embed[toks].copy()  # [n, d]
    used = []
    for layer in range(m.n_layers):
        xn = rmsnorm(h, NORM_EPS)
        q = xn @ m.wq[layer].T
        k = round_bf16(xn @ m.wk[layer].T)
        v = round_bf16(xn @ m.wv[layer].T)
        kc, vc = cache[layer]
        att, kc, vc = attn_kv(q.reshape(1, n, H, hd), k.reshape(1, n, Hkv, hd),
                              v.reshape(1, n, Hkv, hd), kc, vc, np.array([pos]))
        cache[layer] = (kc, vc)
        h = h + att.reshape(n, H * hd) @ m.wo[layer].T
        xf = rmsnorm(h, NORM_EPS)
        if not sparse and full_ffn_input_bf16:
            xf = round_bf16(xf)
        g = xf @ m.w_gate[layer].T
        u = xf @ m.w_up[layer].T
        a = silu(g)
        if acts is not None:
            acts.append(a)
        hid = a * u
        if sparse:
            if active_sets is not None:
                sets = [np.asarray(active_sets[layer][i], dtype=np.int64) for i in range(n)]
            else:
                sets = [np.flatnonzero(np.abs(a[i]) > m.thresholds[layer]) for i in range(n)]
            mask = np.zeros_like(hid, dtype=bool)
            for i, s in enumerate(sets):
                mask[i, s] = True
            hid = np.where(mask, hid, 0.0)
            used.append(sets)
        else:
            used.append(None)
        h = h + hid @ m.w_down[layer]
    logits = rmsnorm(h, NORM_EPS) @ m.lm_head.T
    return logits, used


def calibrate_thresholds(m: Model, tokens, q: float, max_len: int) -> np.ndarray:
    """Per-layer thresholds of M_S for target sparsity q: M_F runs over the calibration tokens
    and t_l is the nearest-rank q-quantile of |SiLU(gate)| over every FFN input of layer l
    (the calibration rule of the FFN oracle, applied layer by layer)."""
    toks = np.asarray(tokens, dtype=np.int64)
    n = toks.shape[0]
    H, Hkv, hd = m.n_heads, m.n_kv_heads, m.head_dim
    cache = new_cache(m, max_len)
    h = m.embed[toks].copy()
    out = np.zeros(m.n_layers)
    for layer in range(m.n_layers):
        xn = rmsnorm(h, NORM_EPS)
        q_ = xn @ m.wq[layer].T
        k = round_bf16(xn @ m.wk[layer].T)
        v = round_bf16(xn @ m.wv[layer].T)
        att, _, _ = attn_kv(q_.reshape(1, n, H, hd), k.reshape(1, n, Hkv, hd),
                            v.reshape(1, n, Hkv, hd), *cache[layer], np.array([0]))
        h = h + att.reshape(n, H * hd) @ m.wo[layer].T
        xf = rmsnorm(h, NORM_EPS)
        a = np.sort(np.abs(silu(xf @ m.w_gate[layer].T)).ravel())
        out[layer] = a[int(np.ceil(q * a.size)) - 1]
        h = h + (silu(xf @ m.w_gate[layer].T) * (xf @ m.w_up[layer].T)) @ m.w_down[layer]
    return out


def _softmax_prob(row, tok: int) -> float:
    z = np.asarray(row, dtype=np.float64)
    mx = float(np.max(z))
    return float(np.exp(z[tok] - mx) / np.sum(np.exp(z - mx)))


@dataclasses.dataclass
class Period:
    """One period's record: inputs s_0 .. s_n, accept length j, corrected token (or -1),
    the committed tokens, the positions before and after, the full model's likelihoods q, the
    drafting neuron sets ([step][layer] -> set) and gate activations ([step][layer] -> row)."""
    seq: list
    accept: int
    corrected: int
    committed: list
    pos_before: int
    pos_after: int
    q: list
    draft_sets: list
    draft_acts: list


def sirius_period(m: Model, cache, pos: int, cur: int, n: int, r: float, *,
                  full_ffn_input_bf16: bool = False, follow=None) -> Period:
    """One period of Algorithm 1 (drafting, check, rollback, interleaving), greedy.

    follow, when given, replays another implementation's decisions where they are not
    decided by a margin: a callable follow(kind, i, own, margin_info) -> the decision to
    take ("draft" / "accept" / "corrected" / "sets" kinds; see the GPU parity tests). The
    plain oracle passes None and takes every decision itself.
    """
    seq = [int(cur)]
    draft_sets, draft_acts = [], []
    for i in range(n):  # M_S drafts, writing rows pos + i
        sets = follow("sets", i, None, None) if follow else None
        acts = []
        logits, used = forward(m, [seq[i]], cache, pos + i, True, active_sets=sets, acts=acts)
        draft_sets.append([u[0] for u in used])
        draft_acts.append([a[0] for a in acts])
        own = int(np.argmax(logits[0]))
        seq.append(follow("draft", i, own, logits[0]) if follow else own)
    # cache position wound back by n; M_F rewrites rows pos .. pos + n - 1 in one pass
    logits, _ = forward(m, seq[:n], cache, pos, False, full_ffn_input_bf16=full_ffn_input_bf16)
    q = [_softmax_prob(logits[i], seq[i + 1]) for i in range(n)]
    j = n
    for i in range(n):
        if q[i] < r:
            j = i
            break
    if follow:
        j = follow("accept", 0, j, q)
    if j < n:
        own = int(np.argmax(logits[j]))
        corrected = follow("corrected", j, own, logits[j]) if follow else own
        committed = seq[1:j + 1] + [corrected]
        pos_after = pos + j + 1
    else:
        corrected = -1
        committed = seq[1:n + 1]
        pos_after = pos + n
    return Period(seq, j, corrected, committed, pos, pos_after, q, draft_sets, draft_acts)


def prefill(m: Model, cache, prompt):
    """M_F over every prompt token but the last, at positions 0 .. T - 2. Returns the state
    (position T - 1, current input = the last prompt token)."""
    p = np.asarray(prompt, dtype=np.int64)
    if p.shape[0] > 1:
        forward(m, p[:-1], cache, 0, False)
    return p.shape[0] - 1, int(p[-1])


def generate(m: Model, prompt, n: int, r: float, periods: int, max_len: int, *,
             full_ffn_input_bf16: bool = False, follow_factory=None):
    """Prefill, then `periods` periods of Algorithm 1. Returns (committed tokens, the list
    of Period records, the final cache and position)."""
    cache = new_cache(m, max_len)
    pos, cur = prefill(m, cache, prompt)
    out, recs = [], []
    for p in range(periods):
        if pos + n > max_len:
            raise ValueError("the cache is full")
        follow = follow_factory(p) if follow_factory else None
        rec = sirius_period(m, cache, pos, cur, n, r, full_ffn_input_bf16=full_ffn_input_bf16,
                            follow=follow)
        out.extend(rec.committed)
        recs.append(rec)
        pos = rec.pos_after
        cur = rec.committed[-1]
    return out, recs, cache, pos


def aal(records) -> float:
    """Average advance length: committed tokens per period (Sec. 2.2)."""
    return float(np.mean([len(r.committed) for r in records]))


__all__ = ["Model", "model_from_bits", "new_cache", "forward", "sirius_period", "prefill",
           "generate", "aal", "calibrate_thresholds", "round_bf16", "Period", "NORM_EPS"]
