"""Seeded generators for the synthetic workloads.

Shapes follow the Llama-3 FFN sizes the method is evaluated on (8B:
d_model=4096, d_ff=14336; 70B: d_model=8192, d_ff=28672) plus a tiny layer
(256 x 688) small enough for the fp64 oracle to run in milliseconds.

Every generator takes an explicit integer seed and uses numpy's PCG64, so
the same call always yields the same bytes. Separate seed streams are used
for weights, decode inputs, calibration inputs, prompts and logits.

Distribution conventions (see the input recipe in the design notes):
  * "N(0, 1/d_model)" and "N(0, 2)", "N(0, 3)" are variances;
  * "N(0, 0.02)" for the 8B/70B weights is a standard deviation (the usual
    LLM initialisation scale).
"""

from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass(frozen=True)
class FFNShape:
    name: str
    d_model: int
    d_ff: int
    weight_std: float


TINY = FFNShape("tiny-256x688", 256, 688, 1.0 / 16.0)  # variance 1/256
LLAMA3_8B = FFNShape("llama3-8b-ffn", 4096, 14336, 0.02)
LLAMA3_70B = FFNShape("llama3-70b-ffn", 8192, 28672, 0.02)


@dataclasses.dataclass(frozen=True)
class VerifyShape:
    name: str
    batch: int
    k: int
    vocab: int
    logit_var: float


VERIFY_TINY = VerifyShape("verify-tiny", 1, 4, 1000, 2.0)
VERIFY_8B = VerifyShape("verify-llama3-vocab", 8, 16, 128256, 3.0)


def _rng(seed: int, stream: int) -> np.random.Generator:
    # Independent, reproducible streams: (seed, stream) -> PCG64 state.
    return np.random.default_rng(np.random.SeedSequence([int(seed) & 0xFFFFFFFF, int(stream)]))


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bfloat16 (round-to-nearest-even), returned as uint16 bit patterns.

    Storage-format conversion only. Inputs are finite.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


_STREAM_WEIGHTS = 1
_STREAM_DECODE = 2
_STREAM_CALIB = 3
_STREAM_PROMPT = 4
_STREAM_LOGITS = 5
_STREAM_TREE = 6
_STREAM_ATTN = 7


def ffn_weights(seed: int, d_model: int, d_ff: int, std: float):
    """Three neuron-major bf16 matrices (W_gate, W_up, W_down), each [d_ff, d_model] uint16.

    Row i of every matrix belongs to FFN neuron i: W_gate[i] and W_up[i] are
    the input weights of neuron i, W_down[i] its output weights.
    """
    rng = _rng(seed, _STREAM_WEIGHTS)
    out = []
    for _ in range(3):
        w = rng.standard_normal((d_ff, d_model), dtype=np.float32)
        w *= np.float32(std)
        out.append(bf16_bits(w))
    return tuple(out)


def decode_inputs(seed: int, n: int, d_model: int, std: float = 1.0) -> np.ndarray:
    """n decode activations x ~ N(0, std^2), fp32 [n, d_model]."""
    rng = _rng(seed, _STREAM_DECODE)
    x = rng.standard_normal((n, d_model), dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def calibration_inputs(seed: int, n: int, d_model: int) -> np.ndarray:
    """n calibration activations ~ N(0, 1), fp32 [n, d_model], from their own stream."""
    rng = _rng(seed, _STREAM_CALIB)
    return rng.standard_normal((n, d_model), dtype=np.float32)


def griffin_prompt(seed: int, t: int, d_model: int) -> np.ndarray:
    """Prompt activations ~ N(0, 1) stored as bf16 bits [t, d_model] uint16."""
    rng = _rng(seed, _STREAM_PROMPT)
    return bf16_bits(rng.standard_normal((t, d_model), dtype=np.float32))


def verify_inputs(seed: int, batch: int, k: int, vocab: int, logit_var: float,
                  rows: int | None = None, boost: float = 6.0,
                  calibrated: bool = False):
    """Logits [batch, rows, vocab] fp32 ~ N(0, logit_var) and drafted ids [batch, k] int32.

    rows defaults to k; rows = k + 1 adds a bonus row with no drafted token.
    The drafted token's logit in row j (j < k) is raised by U(0, boost).
    With calibrated=True the drafted logit is instead set to the row's
    largest logit plus U(0, boost), so that acceptance lengths spread over
    0..k instead of collapsing to 0 (the literal recipe gives drafted-token
    probabilities near 1e-3 at vocab 128256).
    """
    if rows is None:
        rows = k
    rng = _rng(seed, _STREAM_LOGITS)
    logits = rng.standard_normal((batch, rows, vocab), dtype=np.float32)
    logits *= np.float32(np.sqrt(logit_var))
    drafted = rng.integers(0, vocab, size=(batch, k), dtype=np.int64).astype(np.int32)
    bump = rng.uniform(0.0, boost, size=(batch, k)).astype(np.float32)
    for b in range(batch):
        for j in range(k):
            tok = drafted[b, j]
            if calibrated:
                logits[b, j, tok] = logits[b, j].max() + bump[b, j]
            else:
                logits[b, j, tok] += bump[b, j]
    return logits, drafted


def tree_build_inputs(seed: int, batch: int, wc: int, vocab: int, logit_var: float, root: bool = False):
    """Sparse-model logits at the current leaves [batch, wc, vocab] fp32 ~ N(0, logit_var) and the
    leaves' cumulative log-likelihoods [batch, wc] fp32 (None when root=True).

    The cumulative values are -Exp(scale 3) draws put in descending order per tree (the drafting
    step stores its leaves best first).
    """
    rng = _rng(seed, _STREAM_TREE)
    logits = rng.standard_normal((batch, wc, vocab), dtype=np.float32)
    logits *= np.float32(np.sqrt(logit_var))
    if root:
        return logits, None
    cum = -np.sort(rng.exponential(3.0, size=(batch, wc)), axis=1).astype(np.float32)
    return logits, cum


def tree_verify_inputs(seed: int, batch: int, k: int, w: int, vocab: int, logit_var: float,
                       bonus: bool = False, boost: float = 6.0, calibrated: bool = True):
    """A drafted tree of k steps and width w per batch entry, with full-model logits per node.

    Returns logits [batch, k*w (+ w with bonus), vocab] fp32 ~ N(0, logit_var), node tokens
    [batch, k, w] int32 uniform over the vocabulary, and parent slots [batch, k, w] int32
    uniform over [0, w) (step 0 holds -1: its parent is the root). The node's own token logit is
    raised as in verify_inputs (calibrated: the row's largest logit plus U(0, boost)).
    """
    rows = k * w + (w if bonus else 0)
    rng = _rng(seed, _STREAM_TREE)
    logits = rng.standard_normal((batch, rows, vocab), dtype=np.float32)
    logits *= np.float32(np.sqrt(logit_var))
    tokens = rng.integers(0, vocab, size=(batch, k, w), dtype=np.int64).astype(np.int32)
    parents = rng.integers(0, w, size=(batch, k, w), dtype=np.int64).astype(np.int32)
    parents[:, 0, :] = -1
    bump = rng.uniform(0.0, boost, size=(batch, k, w)).astype(np.float32)
    for b in range(batch):
        for i in range(k):
            for j in range(w):
                row, tok = i * w + j, tokens[b, i, j]
                if calibrated:
                    logits[b, row, tok] = logits[b, row].max() + bump[b, i, j]
                else:
                    logits[b, row, tok] += bump[b, i, j]
    return logits, tokens, parents


def attn_inputs(seed: int, batch: int, n: int, heads: int, kv_heads: int, head_dim: int, lmax: int):
    """One attention call's inputs: q [batch, n, heads, head_dim] fp32 ~ N(0, 1); new keys and
    values [batch, n, kv_heads, head_dim] and the caches [batch, lmax, kv_heads, head_dim] ~ N(0, 1)
    stored as bf16 bits."""
    rng = _rng(seed, _STREAM_ATTN)
    q = rng.standard_normal((batch, n, heads, head_dim), dtype=np.float32)
    kn = bf16_bits(rng.standard_normal((batch, n, kv_heads, head_dim), dtype=np.float32))
    vn = bf16_bits(rng.standard_normal((batch, n, kv_heads, head_dim), dtype=np.float32))
    kc = bf16_bits(rng.standard_normal((batch, lmax, kv_heads, head_dim), dtype=np.float32))
    vc = bf16_bits(rng.standard_normal((batch, lmax, kv_heads, head_dim), dtype=np.float32))
    return q, kn, vn, kc, vc


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """A small Llama-style decoder for the generation loop (random weights, mechanics only)."""
    name: str
    n_layers: int
    d_model: int
    d_ff: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    vocab: int
    max_len: int
    lm_std: float  # logit scale: W_lm ~ N(0, lm_std^2 / d_model)


TINY_MODEL = ModelShape("tiny-decoder", 2, 256, 688, 4, 2, 64, 1000, 256, 6.0)

_STREAM_MODEL = 8


def model_weights(seed: int, s: ModelShape) -> dict:
    """bf16 bit patterns of a random decoder: embed [V, d] ~ N(0, 1); wq [L, H hd, d],
    wk, wv [L, Hkv hd, d], w_gate, w_up, w_down [L, F, d] ~ N(0, 1/d); wo [L, d, H hd]
    ~ N(0, 1/(H hd)); lm_head [V, d] ~ N(0, lm_std^2/d)."""
    rng = _rng(seed, _STREAM_MODEL)
    d, hq, hkv = s.d_model, s.n_heads * s.head_dim, s.n_kv_heads * s.head_dim

    def draw(shape, std):
        w = rng.standard_normal(shape, dtype=np.float32)
        w *= np.float32(std)
        return bf16_bits(w)

    out = {"embed": draw((s.vocab, d), 1.0)}
    out["wq"] = draw((s.n_layers, hq, d), d ** -0.5)
    out["wk"] = draw((s.n_layers, hkv, d), d ** -0.5)
    out["wv"] = draw((s.n_layers, hkv, d), d ** -0.5)
    out["wo"] = draw((s.n_layers, d, hq), hq ** -0.5)
    for k in ("w_gate", "w_up", "w_down"):
        out[k] = draw((s.n_layers, s.d_ff, d), d ** -0.5)
    out["lm_head"] = draw((s.vocab, d), s.lm_std * d ** -0.5)
    return out


def prompt_tokens(seed: int, t: int, vocab: int) -> np.ndarray:
    """t prompt token ids uniform in [0, vocab), int32."""
    rng = _rng(seed, _STREAM_PROMPT)
    return rng.integers(0, vocab, size=t, dtype=np.int64).astype(np.int32)
