"""Oracle: the full model's correction check of a chunk of drafted tokens.

Test infrastructure only (see the package docstring). Float64 throughout.

Algorithm 1 (Sirius): the sparse model drafts a chunk ("kernel") of tokens;
the full model then evaluates the whole chunk in one parallel pass and
yields, for each drafted position, its own likelihood q of the drafted
token. Scanning positions in order, the first position whose likelihood is
below the threshold r is the rejection point (strict '<', the scan stops
there); the cache is rolled back to it and the full model's own token is
emitted at that position (interleaving the key token). Sec. 4, "How to
correct", adds that a threshold of 0.1 with temperature 0.6 works well.

Readings adopted where the algorithm's indices are inconsistent (its
listing mixes relative and absolute cache positions and names the verify
likelihoods both q and p):

  * row j of the logits is the full model's distribution at drafted
    position j, already aligned by the caller;
  * q_j = softmax(logits[j] / temperature)[drafted_j];
  * accept_len = first j with q_j < r, else K (every token accepted);
  * the corrected token is the argmax of the raw logits of row accept_len
    (lowest index on ties) when accept_len < K; when all K are accepted it
    is the argmax of the bonus row K if the caller supplied K + 1 rows, else
    -1. The paper samples this token; the argmax is its deterministic form.
  * a drafted id outside [0, vocab) has likelihood 0 (always rejected).
"""

from __future__ import annotations

import numpy as np


def softmax_row_stats(row, temperature: float = 1.0):
    """(max of row/T, sum of exp(row/T - max), argmax of raw row) for one logit row."""
    r = np.asarray(row, dtype=np.float64)
    z = r / float(temperature)
    m = float(np.max(z))
    s = float(np.sum(np.exp(z - m)))
    amax = int(np.argmax(r))  # numpy returns the first (lowest) index of the maximum
    return m, s, amax


def verify_accept(logits, drafted, r: float, temperature: float = 1.0):
    """Acceptance length, corrected token and drafted-token likelihoods.

    logits [B, R, V] (R = K or K + 1), drafted [B, K] int.
    Returns (accept_len [B] int64, next_token [B] int64, q [B, K] float64).
    """
    lg = np.asarray(logits)
    dr = np.asarray(drafted)
    b_n, r_n, v_n = lg.shape
    k_n = dr.shape[1]
    if r_n not in (k_n, k_n + 1):
        raise ValueError("logits must hold K or K + 1 rows per batch entry")
    q = np.zeros((b_n, k_n), dtype=np.float64)
    amax = np.zeros((b_n, r_n), dtype=np.int64)
    for b in range(b_n):
        for j in range(r_n):
            m, s, am = softmax_row_stats(lg[b, j], temperature)
            amax[b, j] = am
            if j < k_n:
                tok = int(dr[b, j])
                if 0 <= tok < v_n:
                    q[b, j] = np.exp(float(lg[b, j, tok]) / float(temperature) - m) / s
    accept = np.full(b_n, k_n, dtype=np.int64)
    nxt = np.full(b_n, -1, dtype=np.int64)
    for b in range(b_n):
        for j in range(k_n):
            if q[b, j] < r:
                accept[b] = j
                break
        j = accept[b]
        if j < k_n:
            nxt[b] = amax[b, j]
        elif r_n == k_n + 1:
            nxt[b] = amax[b, k_n]
    return accept, nxt, q
