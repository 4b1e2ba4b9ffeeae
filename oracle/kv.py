"""Oracle: attention over the shared KV cache with the full model's direct rewrite, and the
rollback after the check. Test infrastructure only (see the package docstring). Float64.

Algorithm 1 and Sec. 4 ("How to correct"): the sparse and the full model share one KV cache.
The sparse model fills it one token at a time while drafting; at the check the position is
wound back by the kernel size n, the full model runs the n drafted tokens in parallel and its
keys and values are written directly over the sparse model's at the same positions; after the
first rejection j the position rolls back so that only the accepted prefix (and the position
of the corrected token) stays.

Readings adopted (the paper gives the procedure, not the attention arithmetic):

  * one attention layer of the Llama family: H query heads, Hkv key/value heads, query head h
    reads key/value head h // (H / Hkv) (grouped-query attention), head size hd, scores
    q . k / sqrt(hd), no positional rotation (the rotation is applied before the cache and is
    part of producing q and k, not of this step);
  * the n tokens of a call sit at positions p .. p + n - 1 (p = the cache position at the start
    of the call); their keys and values replace the cache rows there, and token i attends to
    cache rows 0 .. p + i (causal);
  * n = 1 is the sparse model's decode step (it writes its own row), n = kernel size is the
    full model's verification pass over the drafted chunk;
  * rollback: with accept length j (the first rejected position, j = n when all are
    accepted) the cache position becomes p + min(j + 1, n): the rows of the inputs before
    the rejected token stay valid, and the next input (the corrected token) goes to p + j + 1;
    when all n are accepted the next input is the last drafted token, at p + n.
"""

from __future__ import annotations

import math

import numpy as np

from .ffn import widen_bf16


def _f64(a):
    a = np.asarray(a)
    return widen_bf16(a) if a.dtype == np.uint16 else a.astype(np.float64)


def attn_kv(q, k_new, v_new, k_cache, v_cache, cache_pos):
    """Attention with the direct rewrite.

    q [B, n, H, hd]; k_new, v_new [B, n, Hkv, hd]; k_cache, v_cache [B, Lmax, Hkv, hd];
    cache_pos [B] (p per batch entry, p + n <= Lmax).
    Returns (out [B, n, H, hd], k_cache', v_cache') in float64; the caches are copies with rows
    p .. p + n - 1 replaced.
    """
    q = _f64(q)
    kn, vn = _f64(k_new), _f64(v_new)
    kc, vc = _f64(k_cache).copy(), _f64(v_cache).copy()
    bsz, n, h, hd = q.shape
    hkv = kn.shape[2]
    if h % hkv:
        raise ValueError("H must be a multiple of Hkv")
    g = h // hkv
    out = np.zeros((bsz, n, h, hd))
    scale = 1.0 / math.sqrt(hd)
    for b in range(bsz):
        p = int(cache_pos[b])
        if p < 0 or p + n > kc.shape[1]:
            raise ValueError("cache position out of range")
        kc[b, p:p + n] = kn[b]
        vc[b, p:p + n] = vn[b]
        for i in range(n):
            for hh in range(h):
                kvh = hh // g
                keys = kc[b, :p + i + 1, kvh]  # [p + i + 1, hd]
                s = keys @ q[b, i, hh] * scale
                w = np.exp(s - s.max())
                out[b, i, hh] = (w / w.sum()) @ vc[b, :p + i + 1, kvh]
    return out, kc, vc


def kv_rollback(cache_pos, accept_len, n: int):
    """New cache positions after the check: p + min(accept_len + 1, n)."""
    p = np.asarray(cache_pos, dtype=np.int64)
    a = np.asarray(accept_len, dtype=np.int64)
    return p + np.minimum(a + 1, n)
