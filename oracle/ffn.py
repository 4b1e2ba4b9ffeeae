"""Oracle: SwiGLU FFN, contextual sparsity (FSparse/CATS and CSparse/Griffin), RMSNorm stack.

Test infrastructure only (see the package docstring). Float64 throughout.

Notation. One FFN layer has d_model inputs and d_ff neurons. All three
weight matrices are stored neuron-major, [d_ff, d_model]: row i of W_gate
and W_up are neuron i's input weights, row i of W_down its output weights.
For an input x (length d_model):

    g_i = W_gate[i] . x          (gate pre-activation)
    u_i = W_up[i]   . x          (up projection)
    a_i = SiLU(g_i) = g_i / (1 + exp(-g_i))
    h_i = a_i * u_i
    y   = sum_i h_i * W_down[i]  (down projection, i ascending)

The paper never writes the FFN equation or its sizes; it works with the
Llama family's SwiGLU MLP and says the MLP holds about 70% of the weights
(Sec. 2.1). Contextual sparsity keeps only neurons selected from the input
activation (Sec. 2.1):

  * fine-grained (FSparse, CATS): a new neuron set per token, chosen from the
    gate activation; the gate stays dense and only up and down are sparse
    (Sec. 3, FSparse description and its footnote);
  * coarse-grained (CSparse, Griffin): one neuron set per prompt, fixed for
    every generated token, and the whole MLP including the gate is sparse
    (Sec. 2.1; Sec. 3; Appendix A.1, contextual sparsity paragraph).
"""

from __future__ import annotations

import math

import numpy as np


def widen_bf16(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64, exactly (bf16 is the top half of an fp32)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _f64(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return widen_bf16(a)
    return a.astype(np.float64)


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU(z) = z * sigmoid(z) = z / (1 + exp(-z)), float64."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def gate_activations(x, w_gate) -> np.ndarray:
    """a = SiLU(x W_gate^T) for x [B, d_model]; returns [B, d_ff] float64."""
    x = np.atleast_2d(_f64(x))
    return silu(x @ _f64(w_gate).T)


def ffn_dense(x, w_gate, w_up, w_down) -> np.ndarray:
    """Dense SwiGLU FFN, y [B, d_model] float64 (the sparsity-0 model)."""
    x = np.atleast_2d(_f64(x))
    g = x @ _f64(w_gate).T
    u = x @ _f64(w_up).T
    h = silu(g) * u
    return h @ _f64(w_down)


def cats_active_sets(x, w_gate, t: float):
    """Per-token active neuron sets of threshold sparsity.

    A_b = { i : |SiLU(g_bi)| > t } with a strict comparison. A negative t
    keeps every neuron (sparsity 0); t = +inf keeps none. Returns a list of
    ascending int64 index arrays (one per row of x) and the gate
    activations a [B, d_ff].

    The paper's FSparse follows CATS: the neuron set is re-chosen for every
    token from the gate activation (Sec. 2.1; Sec. 3 FSparse description).
    The threshold form and its strictness are not printed in the paper; the
    reading adopted here is strict '>' on |SiLU(gate)|.
    """
    a = gate_activations(x, w_gate)
    sets = [np.flatnonzero(np.abs(a[b]) > t) for b in range(a.shape[0])]
    return sets, a


def ffn_masked(x, w_gate, w_up, w_down, active_sets) -> np.ndarray:
    """SwiGLU FFN restricted to a neuron set per row: y_b = sum_{i in A_b} h_bi W_down[i].

    Neurons outside A_b contribute exactly zero (their h is replaced by 0),
    so an A_b holding every neuron reproduces ffn_dense bit for bit.
    """
    x = np.atleast_2d(_f64(x))
    g = x @ _f64(w_gate).T
    u = x @ _f64(w_up).T
    h = silu(g) * u
    mask = np.zeros_like(h, dtype=bool)
    for b, s in enumerate(active_sets):
        mask[b, np.asarray(s, dtype=np.int64)] = True
    h = np.where(mask, h, 0.0)
    return h @ _f64(w_down)


def ffn_cats(x, w_gate, w_up, w_down, t: float):
    """Threshold-sparse FFN: returns (y [B, d_model], active sets)."""
    sets, _ = cats_active_sets(x, w_gate, t)
    return ffn_masked(x, w_gate, w_up, w_down, sets), sets


def topk_active_sets(x, w_gate, k: int):
    """Per-token top-k neuron sets: the paper's own fine-grained implementation.

    The paper replaces CATS's threshold by a top-k over the gate layer's
    activations, so that every token keeps exactly the target density, and
    implements the rest as CATS does (Sec. 3, footnote on the fine-grained
    implementation). Reading adopted: for each token, the k neurons with the
    largest |SiLU(g_bi)| (the magnitude CATS thresholds), ties to the lower
    neuron index. Returns ascending int64 index arrays (one per row of x) and
    the gate activations a [B, d_ff].
    """
    a = gate_activations(x, w_gate)
    f = a.shape[1]
    if not 1 <= k <= f:
        raise ValueError("k must lie in [1, d_ff]")
    idx = np.arange(f)
    sets = []
    for b in range(a.shape[0]):
        order = np.lexsort((idx, -np.abs(a[b])))  # primary key: larger |a|; then lower index
        sets.append(np.sort(order[:k]))
    return sets, a


def ffn_topk(x, w_gate, w_up, w_down, k: int):
    """Per-token top-k sparse FFN: returns (y [B, d_model], active sets)."""
    sets, _ = topk_active_sets(x, w_gate, k)
    return ffn_masked(x, w_gate, w_up, w_down, sets), sets


def calibrate_threshold(x_cal, w_gate, q: float) -> float:
    """Threshold t for target sparsity q from calibration inputs.

    Nearest-rank quantile of the pooled |SiLU(gate)| values: with the M
    values sorted ascending, t = v[ceil(q*M) - 1]. When no two values tie,
    exactly M - ceil(q*M) of them exceed t, so a fraction about q of the
    neurons is dropped on the calibration set. (The paper fixes sparsity
    levels, 50% by default, Sec. 3; how CATS derives its threshold is not
    printed there, so this is the plain quantile rule.)
    """
    v = np.sort(np.abs(gate_activations(x_cal, w_gate)).ravel())
    m = v.size
    rank = int(math.ceil(q * m))
    rank = min(max(rank, 1), m)
    return float(v[rank - 1])


def griffin_scores(x_prompt, w_gate, w_up, normalize_tokens: bool = False) -> np.ndarray:
    """Per-neuron prompt statistic s [d_ff] of coarse-grained sparsity.

    z_ti = SiLU(x_t . W_gate[i]) * (x_t . W_up[i]) for the T prompt tokens,
    s_i = sqrt(sum_t z_ti^2), the neuron's L2 norm over the prompt.

    The paper names Griffin as its CSparse method and says the neuron set is
    chosen from the prompt and kept for the whole generation (Sec. 2.1,
    Appendix A.1) but does not print the statistic; the per-neuron L2 norm
    over the prompt is the reading adopted. With normalize_tokens each
    token's row z_t is first scaled to unit L2 norm (a variant, off by
    default).
    """
    x = np.atleast_2d(_f64(x_prompt))
    z = silu(x @ _f64(w_gate).T) * (x @ _f64(w_up).T)
    if normalize_tokens:
        n = np.sqrt(np.sum(z * z, axis=1, keepdims=True))
        z = np.where(n > 0.0, z / np.where(n > 0.0, n, 1.0), 0.0)
    return np.sqrt(np.sum(z * z, axis=0))


def griffin_topk(scores, k: int) -> np.ndarray:
    """The k neurons with the largest score, returned in ascending index order.

    Order: larger score first; equal scores are broken toward the lower
    neuron index.
    """
    s = np.asarray(scores, dtype=np.float64)
    idx = np.arange(s.size)
    order = np.lexsort((idx, -s))  # primary key -s, secondary key index
    return np.sort(order[:k])


def condense(w, sel) -> np.ndarray:
    """Rows sel of a neuron-major matrix, copied unchanged (same dtype)."""
    return np.ascontiguousarray(np.asarray(w)[np.asarray(sel, dtype=np.int64)])


def ffn_condensed(x, w_gate_c, w_up_c, w_down_c) -> np.ndarray:
    """FFN over condensed weights: the dense FFN of the selected neurons only."""
    return ffn_dense(x, w_gate_c, w_up_c, w_down_c)


def rmsnorm(h, eps: float = 1e-5) -> np.ndarray:
    """RMSNorm with unit weight: h / sqrt(mean(h^2) + eps), per row."""
    h = np.atleast_2d(_f64(h))
    return h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + eps)


def stack_layer(h, ffn, eps: float = 1e-5) -> np.ndarray:
    """One FFN-only decoder layer: h + FFN(RMSNorm(h)); ffn maps [B, d] -> [B, d]."""
    h = np.atleast_2d(_f64(h))
    return h + ffn(rmsnorm(h, eps))
