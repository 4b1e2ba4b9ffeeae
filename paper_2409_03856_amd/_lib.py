"""ctypes binding of libsirius.so (the C ABI declared in include/sirius.h).

Argument marshalling only: every function here checks shapes and dtypes,
turns torch tensors into device pointers, passes torch's current HIP stream,
and calls the C entry point of the same name. All computation happens in the
library's HIP kernels; there is no fallback path. If the library has not been
built, loading it raises.
"""

from __future__ import annotations

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsirius.so")

SIRIUS_OK = 0
SIRIUS_EINVAL = -1
SIRIUS_EWORKSPACE = -2
SIRIUS_EHIP = -3

OP_FFN_DENSE = 0
OP_FFN_CATS = 1
OP_GRIFFIN_SELECT = 2
OP_FFN_CONDENSED = 3
OP_VERIFY = 4
OP_CATS_CALIBRATE = 5
OP_TREE_BUILD = 6
OP_TREE_VERIFY = 7
OP_FFN_TOPK = 8
OP_ATTN_KV = 9

_P = ctypes.c_void_p
_I = ctypes.c_int
_F = ctypes.c_float
_Z = ctypes.c_size_t

# name -> (restype, argtypes), in the order of include/sirius.h
SIGNATURES = {
    "sirius_ffn_dense": (_I, [_P, _I, _P, _P, _P, _I, _I, _F, _P, _P, _P, _Z, _P]),
    "sirius_ffn_cats": (_I, [_P, _I, _P, _P, _P, _I, _I, _F, _F, _P, _P, _P, _P, _P, _Z, _P]),
    "sirius_ffn_cats_noalloc": (_I, [_P, _I, _P, _P, _P, _I, _I, _F, _F, _P, _P, _P, _P, _P]),
    "sirius_ffn_topk": (_I, [_P, _I, _P, _P, _P, _I, _I, _I, _F, _P, _P, _P, _P, _P, _Z, _P]),
    "sirius_cats_calibrate": (_I, [_P, _I, _P, _I, _I, ctypes.c_double, _P, _P, _Z, _P]),
    "sirius_griffin_select": (_I, [_P, _I, _P, _P, _P, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _Z, _P]),
    "sirius_ffn_condensed": (_I, [_P, _I, _P, _P, _P, _I, _I, _F, _P, _P, _P, _Z, _P]),
    "sirius_verify_accept": (_I, [_P, _I, _I, _I, _I, _P, _F, _F, _P, _P, _P, _P, _Z, _P]),
    "sirius_tree_build_step": (_I, [_P, _I, _I, _I, _P, _I, _F, _P, _P, _P, _P, _Z, _P]),
    "sirius_tree_verify": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _F, _F, _P, _P, _P, _P, _P, _Z, _P]),
    "sirius_attn_kv": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _P, _Z, _P]),
    "sirius_kv_rollback": (_I, [_P, _P, _I, _I, _P]),
    "sirius_model_workspace_size": (_Z, [_P, _I]),
    "sirius_model_forward": (_I, [_P, _P, _I, _P, _I, _P, _P, _P, _P, _Z, _P]),
    "sirius_generate": (_I, [_P, _P, _P, _I, _F, _I, _P, _P, _P, _P, _Z, _P]),
    "sirius_rmsnorm": (_I, [_P, _I, _I, _F, _P, _P]),
    "sirius_fill_normal_bf16": (_I, [_P, _Z, ctypes.c_uint64, _F, _F, _P]),
    "sirius_profile_enable": (_I, [_I]),
    "sirius_profile_reset": (_I, []),
    "sirius_profile_query": (_I, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]),
    "sirius_workspace_size": (_Z, [_I, _I, _I, _I, _I, _I]),
    "sirius_last_error": (ctypes.c_char_p, []),
    "sirius_version": (ctypes.c_char_p, []),
}

_lock = threading.Lock()
_lib = None


class SiriusError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libsirius error {code}: {msg}")
        self.code = code


def lib() -> ctypes.CDLL:
    """Load libsirius.so (built in-tree); raises if it is missing."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"{LIB_PATH} is not built; run `python -m paper_2409_03856_amd.build` "
                    "(there is no CPU fallback)")
            handle = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in SIGNATURES.items():
                fn = getattr(handle, name)
                fn.restype = res
                fn.argtypes = args
            _lib = handle
    return _lib


def _check(rc: int) -> None:
    if rc != SIRIUS_OK:
        raise SiriusError(rc, lib().sirius_last_error().decode())


# ---------------------------------------------------------------- torch glue

def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _need(cond: bool, msg: str) -> None:
    if not cond:
        raise ValueError(msg)


def _dev_check(*ts):
    for t in ts:
        if t is not None:
            _need(t.is_cuda, "tensors must live on the GPU")
            _need(t.is_contiguous(), "tensors must be contiguous")


_ws_cache: dict = {}


def workspace(op: int, a: int, b: int, c: int, d: int = 0, e: int = 0, device=None):
    """Device workspace for an operation (cached per device; grows as needed)."""
    torch = _torch()
    n = int(lib().sirius_workspace_size(op, a, b, c, d, e))
    if n == 0:
        raise ValueError("invalid sizes for the workspace query")
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    key = (dev.index, op)
    buf = _ws_cache.get(key)
    if buf is None or buf.numel() < n:
        buf = torch.empty(n, dtype=torch.uint8, device=dev)
        _ws_cache[key] = buf
    return buf


def _w_dims(w_gate, w_up, w_down):
    torch = _torch()
    for w in (w_gate, w_up, w_down):
        _need(w.dtype in (torch.bfloat16, torch.int16, torch.uint16), "weights must be bf16 (or 16-bit bits)")
        _need(w.dim() == 2 and w.shape == w_gate.shape, "weights must share one [d_ff, d_model] shape")
    return int(w_gate.shape[1]), int(w_gate.shape[0])


# ---------------------------------------------------------------- entry points

def sirius_ffn_dense(x, w_gate, w_up, w_down, *, norm_eps=-1.0, resid=None, y=None, ws=None, stream=None):
    torch = _torch()
    d, f = _w_dims(w_gate, w_up, w_down)
    _need(x.dtype == torch.float32 and x.dim() == 2 and x.shape[1] == d, "x must be fp32 [B, d_model]")
    bsz = int(x.shape[0])
    if y is None:
        y = torch.empty_like(x)
    _dev_check(x, w_gate, w_up, w_down, resid, y)
    if ws is None:
        ws = workspace(OP_FFN_DENSE, max(bsz, 1), d, f, device=x.device)
    _check(lib().sirius_ffn_dense(_ptr(x), bsz, _ptr(w_gate), _ptr(w_up), _ptr(w_down), d, f,
                                  float(norm_eps), _ptr(resid), _ptr(y), _ptr(ws), ws.numel(), _stream(stream)))
    return y


def sirius_ffn_condensed(x, w_gate_c, w_up_c, w_down_c, *, norm_eps=-1.0, resid=None, y=None, ws=None,
                         stream=None):
    torch = _torch()
    d, k = _w_dims(w_gate_c, w_up_c, w_down_c)
    _need(x.dtype == torch.float32 and x.dim() == 2 and x.shape[1] == d, "x must be fp32 [B, d_model]")
    bsz = int(x.shape[0])
    if y is None:
        y = torch.empty_like(x)
    _dev_check(x, w_gate_c, w_up_c, w_down_c, resid, y)
    if ws is None:
        ws = workspace(OP_FFN_CONDENSED, max(bsz, 1), d, k, device=x.device)
    _check(lib().sirius_ffn_condensed(_ptr(x), bsz, _ptr(w_gate_c), _ptr(w_up_c), _ptr(w_down_c), d, k,
                                      float(norm_eps), _ptr(resid), _ptr(y), _ptr(ws), ws.numel(),
                                      _stream(stream)))
    return y


def sirius_ffn_cats(x, w_gate, w_up, w_down, t, *, norm_eps=-1.0, resid=None, y=None, active_idx=None,
                    active_cnt=None, want_active=True, ws=None, stream=None):
    """Returns (y, active_idx [B, d_ff] int32, active_cnt [B] int32); the lists are None when
    want_active is False and none were passed."""
    torch = _torch()
    d, f = _w_dims(w_gate, w_up, w_down)
    _need(x.dtype == torch.float32 and x.dim() == 2 and x.shape[1] == d, "x must be fp32 [B, d_model]")
    bsz = int(x.shape[0])
    if y is None:
        y = torch.empty_like(x)
    if want_active and active_idx is None:
        active_idx = torch.empty((bsz, f), dtype=torch.int32, device=x.device)
        active_cnt = torch.empty((bsz,), dtype=torch.int32, device=x.device)
    _dev_check(x, w_gate, w_up, w_down, resid, y, active_idx, active_cnt)
    if ws is None:
        ws = workspace(OP_FFN_CATS, max(bsz, 1), d, f, device=x.device)
    _check(lib().sirius_ffn_cats(_ptr(x), bsz, _ptr(w_gate), _ptr(w_up), _ptr(w_down), d, f, float(t),
                                 float(norm_eps), _ptr(resid), _ptr(y), _ptr(active_idx), _ptr(active_cnt),
                                 _ptr(ws), ws.numel(), _stream(stream)))
    return y, active_idx, active_cnt


def sirius_ffn_cats_noalloc(x, w_gate, w_up, w_down, t, *, norm_eps=-1.0, resid=None, y=None, active_idx=None,
                            active_cnt=None, want_active=True, stream=None):
    """sirius_ffn_cats on the library's fixed device scratch (no workspace). Returns (y, active_idx,
    active_cnt) as sirius_ffn_cats; pass y and the lists to allocate nothing here either."""
    torch = _torch()
    d, f = _w_dims(w_gate, w_up, w_down)
    _need(x.dtype == torch.float32 and x.dim() == 2 and x.shape[1] == d, "x must be fp32 [B, d_model]")
    bsz = int(x.shape[0])
    if y is None:
        y = torch.empty_like(x)
    if want_active and active_idx is None:
        active_idx = torch.empty((bsz, f), dtype=torch.int32, device=x.device)
        active_cnt = torch.empty((bsz,), dtype=torch.int32, device=x.device)
    _dev_check(x, w_gate, w_up, w_down, resid, y, active_idx, active_cnt)
    _check(lib().sirius_ffn_cats_noalloc(_ptr(x), bsz, _ptr(w_gate), _ptr(w_up), _ptr(w_down), d, f, float(t),
                                         float(norm_eps), _ptr(resid), _ptr(y), _ptr(active_idx),
                                         _ptr(active_cnt), _stream(stream)))
    return y, active_idx, active_cnt


def sirius_ffn_topk(x, w_gate, w_up, w_down, k, *, norm_eps=-1.0, resid=None, y=None, active_idx=None,
                    active_cnt=None, want_active=True, ws=None, stream=None):
    """Per-token top-k sparse FFN. x [B, d_model] fp32; weights bf16 [d_ff, d_model].
    Returns (y, active_idx [B, d_ff] or None, active_cnt [B] or None)."""
    torch = _torch()
    _need(x.dtype == torch.float32 and x.dim() == 2, "x must be fp32 [B, d_model]")
    d, f = _w_dims(w_gate, w_up, w_down)
    bsz = int(x.shape[0])
    _need(int(x.shape[1]) == d, "x and the weights disagree on d_model")
    dev = x.device
    if y is None:
        y = torch.empty((bsz, d), dtype=torch.float32, device=dev)
    if want_active and active_idx is None:
        active_idx = torch.empty((bsz, f), dtype=torch.int32, device=dev)
        active_cnt = torch.empty(bsz, dtype=torch.int32, device=dev)
    _dev_check(x, w_gate, w_up, w_down, resid, y, active_idx, active_cnt)
    if ws is None:
        ws = workspace(OP_FFN_TOPK, max(bsz, 1), d, f, device=dev)
    _check(lib().sirius_ffn_topk(_ptr(x), bsz, _ptr(w_gate), _ptr(w_up), _ptr(w_down), d, f, int(k),
                                 float(norm_eps), _ptr(resid), _ptr(y), _ptr(active_idx), _ptr(active_cnt),
                                 _ptr(ws), ws.numel(), _stream(stream)))
    return y, active_idx, active_cnt


def sirius_cats_calibrate(x_cal, w_gate, q, *, t_out=None, ws=None, stream=None):
    """Returns a 1-element fp32 device tensor holding the threshold."""
    torch = _torch()
    f, d = int(w_gate.shape[0]), int(w_gate.shape[1])
    _need(x_cal.dtype == torch.float32 and x_cal.dim() == 2 and x_cal.shape[1] == d, "x_cal must be fp32 [N, d]")
    n = int(x_cal.shape[0])
    if t_out is None:
        t_out = torch.empty(1, dtype=torch.float32, device=x_cal.device)
    _dev_check(x_cal, w_gate, t_out)
    if ws is None:
        ws = workspace(OP_CATS_CALIBRATE, n, d, f, device=x_cal.device)
    _check(lib().sirius_cats_calibrate(_ptr(x_cal), n, _ptr(w_gate), d, f, float(q), _ptr(t_out), _ptr(ws),
                                       ws.numel(), _stream(stream)))
    return t_out


def sirius_griffin_select(x_prompt, w_gate, w_up, w_down, k, *, normalize_tokens=False, sel_idx=None,
                          scores=None, want_scores=True, w_gate_c=None, w_up_c=None, w_down_c=None, ws=None,
                          stream=None):
    """Returns (sel_idx [k] int32, scores [d_ff] fp32 or None, w_gate_c, w_up_c, w_down_c)."""
    torch = _torch()
    d, f = _w_dims(w_gate, w_up, w_down)
    _need(x_prompt.dim() == 2 and x_prompt.shape[1] == d and x_prompt.element_size() == 2,
          "x_prompt must be bf16 [T, d_model]")
    t_n = int(x_prompt.shape[0])
    k = int(k)
    dev = x_prompt.device
    if sel_idx is None:
        sel_idx = torch.empty(k, dtype=torch.int32, device=dev)
    if want_scores and scores is None:
        scores = torch.empty(f, dtype=torch.float32, device=dev)
    if w_gate_c is None:
        w_gate_c = torch.empty((k, d), dtype=w_gate.dtype, device=dev)
        w_up_c = torch.empty((k, d), dtype=w_up.dtype, device=dev)
        w_down_c = torch.empty((k, d), dtype=w_down.dtype, device=dev)
    _dev_check(x_prompt, w_gate, w_up, w_down, sel_idx, scores, w_gate_c, w_up_c, w_down_c)
    if ws is None:
        ws = workspace(OP_GRIFFIN_SELECT, 0, d, f, t_n, device=dev)
    _check(lib().sirius_griffin_select(_ptr(x_prompt), t_n, _ptr(w_gate), _ptr(w_up), _ptr(w_down), d, f, k,
                                       1 if normalize_tokens else 0, _ptr(sel_idx), _ptr(scores), _ptr(w_gate_c),
                                       _ptr(w_up_c), _ptr(w_down_c), _ptr(ws), ws.numel(), _stream(stream)))
    return sel_idx, scores, w_gate_c, w_up_c, w_down_c


def sirius_verify_accept(logits, drafted, r, temperature=1.0, *, accept_len=None, next_token=None,
                         p_draft=None, want_p=True, ws=None, stream=None):
    """logits [B, R, V] fp32 (R = K or K + 1), drafted [B, K] int32.
    Returns (accept_len [B] int32, next_token [B] int32, p_draft [B, K] fp32 or None)."""
    torch = _torch()
    _need(logits.dtype == torch.float32 and logits.dim() == 3, "logits must be fp32 [B, R, V]")
    _need(drafted.dtype == torch.int32 and drafted.dim() == 2 and drafted.shape[0] == logits.shape[0],
          "drafted must be int32 [B, K]")
    bsz, rows, vocab = (int(s) for s in logits.shape)
    k = int(drafted.shape[1])
    dev = logits.device
    if accept_len is None:
        accept_len = torch.empty(bsz, dtype=torch.int32, device=dev)
        next_token = torch.empty(bsz, dtype=torch.int32, device=dev)
    if want_p and p_draft is None:
        p_draft = torch.empty((bsz, k), dtype=torch.float32, device=dev)
    _dev_check(logits, drafted, accept_len, next_token, p_draft)
    if ws is None:
        ws = workspace(OP_VERIFY, max(bsz, 1), 0, 0, vocab, rows, device=dev)
    _check(lib().sirius_verify_accept(_ptr(logits), bsz, k, rows, vocab, _ptr(drafted), float(r),
                                      float(temperature), _ptr(accept_len), _ptr(next_token), _ptr(p_draft),
                                      _ptr(ws), ws.numel(), _stream(stream)))
    return accept_len, next_token, p_draft


def sirius_tree_build_step(logits, width, cum_ll=None, temperature=1.0, *, tokens=None, parents=None,
                           cum_ll_out=None, ws=None, stream=None):
    """logits [B, Wc, V] fp32 at the current leaves, cum_ll [B, Wc] fp32 or None (the root).
    Returns (tokens [B, W] int32, parents [B, W] int32, cum_ll_out [B, W] fp32), best first."""
    torch = _torch()
    _need(logits.dtype == torch.float32 and logits.dim() == 3, "logits must be fp32 [B, Wc, V]")
    bsz, wc, vocab = (int(s) for s in logits.shape)
    w = int(width)
    if cum_ll is not None:
        _need(cum_ll.dtype == torch.float32 and tuple(cum_ll.shape) == (bsz, wc), "cum_ll must be fp32 [B, Wc]")
    dev = logits.device
    if tokens is None:
        tokens = torch.empty((bsz, w), dtype=torch.int32, device=dev)
        parents = torch.empty((bsz, w), dtype=torch.int32, device=dev)
        cum_ll_out = torch.empty((bsz, w), dtype=torch.float32, device=dev)
    _dev_check(logits, cum_ll, tokens, parents, cum_ll_out)
    if ws is None:
        ws = workspace(OP_TREE_BUILD, max(bsz, 1), wc, w, vocab, 0, device=dev)
    _check(lib().sirius_tree_build_step(_ptr(logits), bsz, wc, vocab, _ptr(cum_ll), w, float(temperature),
                                        _ptr(tokens), _ptr(parents), _ptr(cum_ll_out), _ptr(ws), ws.numel(),
                                        _stream(stream)))
    return tokens, parents, cum_ll_out


def sirius_tree_verify(logits, tokens, parents, r, temperature=1.0, *, bonus=False, best_leaf=None,
                       accept_len=None, next_token=None, q=None, want_q=True, ws=None, stream=None):
    """logits [B, K*W (+W with bonus), V] fp32, tokens / parents [B, K, W] int32.
    Returns (best_leaf [B], accept_len [B], next_token [B] int32, q [B, K, W] fp32 or None)."""
    torch = _torch()
    _need(tokens.dtype == torch.int32 and tokens.dim() == 3, "tokens must be int32 [B, K, W]")
    _need(parents.dtype == torch.int32 and tuple(parents.shape) == tuple(tokens.shape),
          "parents must be int32 [B, K, W]")
    bsz, k, w = (int(s) for s in tokens.shape)
    rows = k * w + (w if bonus else 0)
    _need(logits.dtype == torch.float32 and logits.dim() == 3 and tuple(logits.shape[:2]) == (bsz, rows),
          "logits must be fp32 [B, K*W (+W), V]")
    vocab = int(logits.shape[2])
    dev = logits.device
    if best_leaf is None:
        best_leaf = torch.empty(bsz, dtype=torch.int32, device=dev)
        accept_len = torch.empty(bsz, dtype=torch.int32, device=dev)
        next_token = torch.empty(bsz, dtype=torch.int32, device=dev)
    if want_q and q is None:
        q = torch.empty((bsz, k, w), dtype=torch.float32, device=dev)
    _dev_check(logits, tokens, parents, best_leaf, accept_len, next_token, q)
    if ws is None:
        ws = workspace(OP_TREE_VERIFY, max(bsz, 1), k, w, vocab, 1 if bonus else 0, device=dev)
    _check(lib().sirius_tree_verify(_ptr(logits), bsz, k, w, vocab, 1 if bonus else 0, _ptr(tokens), _ptr(parents),
                                    float(r), float(temperature), _ptr(best_leaf), _ptr(accept_len),
                                    _ptr(next_token), _ptr(q), _ptr(ws), ws.numel(), _stream(stream)))
    return best_leaf, accept_len, next_token, q


def _bits16(t):
    torch = _torch()
    _need(t.dtype in (torch.bfloat16, torch.int16, torch.uint16), "keys and values must be bf16 (or 16-bit bits)")


def sirius_attn_kv(q, k_new, v_new, k_cache, v_cache, cache_pos, *, out=None, ws=None, stream=None):
    """q [B, n, H, hd] fp32; k_new, v_new [B, n, Hkv, hd] bf16; caches [B, Lmax, Hkv, hd] bf16
    (updated in place: rows cache_pos[b] .. + n - 1 take the new keys and values);
    cache_pos [B] int32 on the GPU. Returns out [B, n, H, hd] fp32."""
    torch = _torch()
    _need(q.dtype == torch.float32 and q.dim() == 4, "q must be fp32 [B, n, H, hd]")
    bsz, n, h, hd = (int(s) for s in q.shape)
    for t in (k_new, v_new, k_cache, v_cache):
        _bits16(t)
        _need(t.dim() == 4 and int(t.shape[0]) == bsz and int(t.shape[3]) == hd, "bad key/value shape")
    hkv = int(k_new.shape[2])
    _need(tuple(k_new.shape) == (bsz, n, hkv, hd) and tuple(v_new.shape) == tuple(k_new.shape),
          "k_new, v_new must be [B, n, Hkv, hd]")
    lmax = int(k_cache.shape[1])
    _need(tuple(k_cache.shape) == (bsz, lmax, hkv, hd) and tuple(v_cache.shape) == tuple(k_cache.shape),
          "caches must be [B, Lmax, Hkv, hd]")
    _need(cache_pos.dtype == torch.int32 and tuple(cache_pos.shape) == (bsz,), "cache_pos must be int32 [B]")
    if out is None:
        out = torch.empty_like(q)
    _dev_check(q, k_new, v_new, k_cache, v_cache, cache_pos, out)
    if ws is None:
        ws = workspace(OP_ATTN_KV, max(bsz, 1), n, h * 65536 + hkv, hd, lmax, device=q.device)
    _check(lib().sirius_attn_kv(_ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(cache_pos),
                                bsz, n, h, hkv, hd, lmax, _ptr(out), _ptr(ws), ws.numel(), _stream(stream)))
    return out


def sirius_kv_rollback(cache_pos, accept_len, n, *, stream=None):
    """cache_pos[b] += min(accept_len[b] + 1, n), on the GPU."""
    torch = _torch()
    _need(cache_pos.dtype == torch.int32 and accept_len.dtype == torch.int32, "int32 tensors expected")
    _need(cache_pos.shape == accept_len.shape and cache_pos.dim() == 1, "cache_pos and accept_len must be [B]")
    _dev_check(cache_pos, accept_len)
    _check(lib().sirius_kv_rollback(_ptr(cache_pos), _ptr(accept_len), int(cache_pos.shape[0]), int(n),
                                    _stream(stream)))
    return cache_pos


def sirius_rmsnorm(h, eps=1e-5, *, out=None, stream=None):
    torch = _torch()
    _need(h.dtype == torch.float32 and h.dim() == 2, "h must be fp32 [B, d_model]")
    if out is None:
        out = torch.empty_like(h)
    _dev_check(h, out)
    _check(lib().sirius_rmsnorm(_ptr(h), int(h.shape[0]), int(h.shape[1]), float(eps), _ptr(out), _stream(stream)))
    return out


def sirius_fill_normal_bf16(out, seed, mean=0.0, std=1.0, *, stream=None):
    _dev_check(out)
    _need(out.element_size() == 2, "out must be a 16-bit (bf16) tensor")
    _check(lib().sirius_fill_normal_bf16(_ptr(out), out.numel(), int(seed) & 0xFFFFFFFFFFFFFFFF, float(mean),
                                         float(std), _stream(stream)))
    return out


def sirius_profile_enable(on: bool = True) -> None:
    _check(lib().sirius_profile_enable(1 if on else 0))


def sirius_profile_reset() -> None:
    _check(lib().sirius_profile_reset())


def sirius_profile_query(kernel: str):
    """(total milliseconds, launches) recorded for one kernel name since the last reset."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(lib().sirius_profile_query(kernel.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, int(n.value)


def sirius_workspace_size(op, a, b, c, d=0, e=0):
    return int(lib().sirius_workspace_size(op, a, b, c, d, e))


def sirius_version() -> str:
    return lib().sirius_version().decode()


# ---------------------------------------------------------------- small decoder and the loop

class _ModelC(ctypes.Structure):
    """struct sirius_model of include/sirius.h."""
    _fields_ = [(n, ctypes.c_int) for n in ("n_layers", "d_model", "d_ff", "n_heads", "n_kv_heads",
                                            "head_dim", "vocab", "max_len")] + \
               [("norm_eps", ctypes.c_float)] + \
               [(n, ctypes.c_void_p) for n in ("embed", "wq", "wk", "wv", "wo", "w_gate", "w_up",
                                               "w_down", "lm_head", "thresholds", "k_cache",
                                               "v_cache")]


class _TraceC(ctypes.Structure):
    """struct sirius_gen_trace of include/sirius.h."""
    _fields_ = [(n, ctypes.c_void_p) for n in ("drafted", "accept_len", "next_token", "q",
                                               "active_idx", "active_cnt")]


class Model:
    """A sirius_model over caller-owned device tensors (kept alive here). weights maps
    embed, wq, wk, wv, wo, w_gate, w_up, w_down, lm_head to bf16 device tensors of the
    shapes in include/sirius.h; the shared cache is allocated here (zeros)."""

    def __init__(self, weights: dict, n_heads: int, n_kv_heads: int, head_dim: int, max_len: int,
                 thresholds, norm_eps: float = 1e-5):
        torch = _torch()
        for k in ("embed", "wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "lm_head"):
            _need(k in weights, f"missing weight {k}")
            _bits16(weights[k])
            _dev_check(weights[k])
        self.weights = dict(weights)
        L, F, d = (int(x) for x in weights["w_gate"].shape)
        V = int(weights["embed"].shape[0])
        dev = weights["embed"].device
        shape = (L, max_len, n_kv_heads, head_dim)
        self.k_cache = torch.zeros(shape, dtype=torch.bfloat16, device=dev)
        self.v_cache = torch.zeros(shape, dtype=torch.bfloat16, device=dev)
        self.thresholds = (ctypes.c_float * L)(*[float(t) for t in thresholds])
        w = self.weights
        self.c = _ModelC(L, d, F, n_heads, n_kv_heads, head_dim, V, max_len, float(norm_eps),
                         *[w[k].data_ptr() for k in ("embed", "wq", "wk", "wv", "wo", "w_gate",
                                                     "w_up", "w_down", "lm_head")],
                         ctypes.cast(self.thresholds, ctypes.c_void_p).value,
                         self.k_cache.data_ptr(), self.v_cache.data_ptr())
        self.device = dev

    @property
    def ptr(self):
        return ctypes.byref(self.c)


def sirius_model_workspace_size(model: Model, max_tokens: int) -> int:
    return int(lib().sirius_model_workspace_size(model.ptr, int(max_tokens)))


def _model_ws(model: Model, n: int):
    torch = _torch()
    size = sirius_model_workspace_size(model, n)
    _need(size > 0, "invalid model or token count for the workspace query")
    return torch.empty(size, dtype=torch.uint8, device=model.device)


def sirius_model_forward(model: Model, tokens, cache_pos, sparse: bool, *, logits=None, want_active=False,
                         ws=None, stream=None):
    """tokens [n] int32, cache_pos [1] int32 (device). Returns (logits [n, V] fp32, active_idx
    [L, n, d_ff], active_cnt [L, n]) -- the lists None unless want_active (sparse only)."""
    torch = _torch()
    _need(tokens.dtype == torch.int32 and tokens.dim() == 1, "tokens must be int32 [n]")
    _need(cache_pos.dtype == torch.int32 and tuple(cache_pos.shape) == (1,), "cache_pos must be int32 [1]")
    n = int(tokens.shape[0])
    c = model.c
    if logits is None:
        logits = torch.empty((n, c.vocab), dtype=torch.float32, device=model.device)
    aidx = acnt = None
    if want_active:
        aidx = torch.empty((c.n_layers, n, c.d_ff), dtype=torch.int32, device=model.device)
        acnt = torch.empty((c.n_layers, n), dtype=torch.int32, device=model.device)
    _dev_check(tokens, cache_pos, logits, aidx, acnt)
    if ws is None:
        ws = _model_ws(model, n)
    _check(lib().sirius_model_forward(model.ptr, _ptr(tokens), n, _ptr(cache_pos), 1 if sparse else 0,
                                      _ptr(logits), _ptr(aidx), _ptr(acnt), _ptr(ws), ws.numel(),
                                      _stream(stream)))
    return logits, aidx, acnt


def sirius_generate(model: Model, seq, cache_pos, n: int, r: float, periods: int, *, out_tokens=None,
                    out_count=None, trace=False, trace_active=False, ws=None, stream=None):
    """seq [n + 1] int32 (seq[0] = the first input), cache_pos [1] int32, both on the device and
    updated. Returns (out_tokens [periods * n], out_count [1], trace dict or None); out_count is
    zeroed here unless passed in."""
    torch = _torch()
    _need(seq.dtype == torch.int32 and tuple(seq.shape) == (n + 1,), "seq must be int32 [n + 1]")
    _need(cache_pos.dtype == torch.int32 and tuple(cache_pos.shape) == (1,), "cache_pos must be int32 [1]")
    dev = model.device
    c = model.c
    if out_tokens is None:
        out_tokens = torch.full((max(periods * n, 1),), -1, dtype=torch.int32, device=dev)
    if out_count is None:
        out_count = torch.zeros((1,), dtype=torch.int32, device=dev)
    tr = None
    tc = None
    if trace or trace_active:
        tr = {"drafted": torch.full((periods, n), -1, dtype=torch.int32, device=dev),
              "accept_len": torch.full((periods,), -1, dtype=torch.int32, device=dev),
              "next_token": torch.full((periods,), -2, dtype=torch.int32, device=dev),
              "q": torch.zeros((periods, n), dtype=torch.float32, device=dev),
              "active_idx": None, "active_cnt": None}
        if trace_active:
            tr["active_idx"] = torch.empty((periods, n, c.n_layers, c.d_ff), dtype=torch.int32, device=dev)
            tr["active_cnt"] = torch.empty((periods, n, c.n_layers), dtype=torch.int32, device=dev)
        tc = _TraceC(*[None if tr[k] is None else tr[k].data_ptr()
                       for k in ("drafted", "accept_len", "next_token", "q", "active_idx", "active_cnt")])
    _dev_check(seq, cache_pos, out_tokens, out_count)
    if ws is None:
        ws = _model_ws(model, n)
    _check(lib().sirius_generate(model.ptr, _ptr(seq), _ptr(cache_pos), int(n), float(r), int(periods),
                                 _ptr(out_tokens), _ptr(out_count),
                                 None if tc is None else ctypes.byref(tc), _ptr(ws), ws.numel(),
                                 _stream(stream)))
    return out_tokens, out_count, tr
