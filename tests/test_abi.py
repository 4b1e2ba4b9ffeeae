"""The C-ABI library loads, exports every entry point of include/sirius.h, and
rejects bad arguments on the host before touching the GPU (no compute calls here)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sirius.h")

pytestmark = pytest.mark.skipif(
    not os.path.exists(os.path.join(ROOT, "paper_2409_03856_amd", "libsirius.so")),
    reason="libsirius.so not built (run __graft_entry__.build())")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sirius_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    from paper_2409_03856_amd import _lib
    return _lib.lib()


def test_every_declared_symbol_is_exported(L):
    names = _declared()
    assert len(names) >= 11
    for n in names:
        assert hasattr(L, n), n


def test_binding_covers_the_header():
    from paper_2409_03856_amd import _lib
    assert sorted(_lib.SIGNATURES) == _declared()


def test_version_and_empty_error(L):
    assert b"gfx950" in L.sirius_version()


FAKE = ctypes.c_void_p(1 << 20)  # non-null, 16-byte aligned; never dereferenced by these calls


def _err(L):
    return L.sirius_last_error().decode()


def test_ffn_argument_errors(L):
    big = 1 << 30
    # d_model not a multiple of 8
    rc = L.sirius_ffn_dense(FAKE, 1, FAKE, FAKE, FAKE, 100, 64, -1.0, None, FAKE, FAKE, big, None)
    assert rc == -1 and "d_model" in _err(L)
    # d_model above the limit, d_ff zero, negative batch, batch above the limit
    assert L.sirius_ffn_dense(FAKE, 1, FAKE, FAKE, FAKE, 16384, 64, -1.0, None, FAKE, FAKE, big, None) == -1
    assert L.sirius_ffn_dense(FAKE, 1, FAKE, FAKE, FAKE, 64, 0, -1.0, None, FAKE, FAKE, big, None) == -1
    assert L.sirius_ffn_dense(FAKE, -1, FAKE, FAKE, FAKE, 64, 64, -1.0, None, FAKE, FAKE, big, None) == -1
    assert L.sirius_ffn_dense(FAKE, 65, FAKE, FAKE, FAKE, 64, 64, -1.0, None, FAKE, FAKE, big, None) == -1
    # null and misaligned pointers
    rc = L.sirius_ffn_dense(None, 1, FAKE, FAKE, FAKE, 64, 64, -1.0, None, FAKE, FAKE, big, None)
    assert rc == -1 and "x is NULL" in _err(L)
    rc = L.sirius_ffn_dense(FAKE, 1, ctypes.c_void_p((1 << 20) + 2), FAKE, FAKE, 64, 64, -1.0, None, FAKE, FAKE,
                            big, None)
    assert rc == -1 and "aligned" in _err(L)
    # workspace too small
    rc = L.sirius_ffn_dense(FAKE, 1, FAKE, FAKE, FAKE, 64, 64, -1.0, None, FAKE, FAKE, 16, None)
    assert rc == -2 and "workspace" in _err(L)
    # an empty batch is a no-op
    assert L.sirius_ffn_dense(FAKE, 0, FAKE, FAKE, FAKE, 64, 64, -1.0, None, FAKE, FAKE, 0, None) == 0


def test_cats_argument_errors(L):
    big = 1 << 30
    nan = float("nan")
    rc = L.sirius_ffn_cats(FAKE, 1, FAKE, FAKE, FAKE, 64, 64, nan, -1.0, None, FAKE, FAKE, FAKE, FAKE, big, None)
    assert rc == -1 and "NaN" in _err(L)
    rc = L.sirius_ffn_cats(FAKE, 1, FAKE, FAKE, FAKE, 64, 64, 0.1, -1.0, None, FAKE, FAKE, None, FAKE, big, None)
    assert rc == -1 and "active_idx" in _err(L)
    rc = L.sirius_ffn_cats(FAKE, 1, FAKE, FAKE, FAKE, 64, 64, 0.1, -1.0, None, FAKE, None, None, FAKE, 8, None)
    assert rc == -2
    assert L.sirius_ffn_cats(FAKE, 0, FAKE, FAKE, FAKE, 64, 64, 0.1, -1.0, None, FAKE, None, None, FAKE, 0, None) == 0
    rc = L.sirius_cats_calibrate(FAKE, 4, FAKE, 64, 64, 0.0, FAKE, FAKE, big, None)
    assert rc == -1 and "q=" in _err(L)
    rc = L.sirius_cats_calibrate(FAKE, 0, FAKE, 64, 64, 0.5, FAKE, FAKE, big, None)
    assert rc == -1


def test_cats_noalloc_argument_errors_and_scratch_size(L):
    nan = float("nan")
    rc = L.sirius_ffn_cats_noalloc(FAKE, 1, FAKE, FAKE, FAKE, 64, 64, nan, -1.0, None, FAKE, FAKE, FAKE, None)
    assert rc == -1 and "NaN" in _err(L) and "noalloc" in _err(L)
    rc = L.sirius_ffn_cats_noalloc(None, 1, FAKE, FAKE, FAKE, 64, 64, 0.1, -1.0, None, FAKE, FAKE, FAKE, None)
    assert rc == -1 and "x is NULL" in _err(L)
    rc = L.sirius_ffn_cats_noalloc(FAKE, 1, FAKE, FAKE, FAKE, 100, 64, 0.1, -1.0, None, FAKE, None, None, None)
    assert rc == -1 and "d_model" in _err(L)
    assert L.sirius_ffn_cats_noalloc(FAKE, 0, FAKE, FAKE, FAKE, 64, 64, 0.1, -1.0, None, FAKE, None, None, None) == 0
    # the fixed scratch (96 MiB) covers every batch up to 64 at the Llama-3-8B and 70B shapes;
    # a larger call is refused on the host, before anything is enqueued
    limit = 96 << 20
    for d, f in ((4096, 14336), (8192, 28672), (256, 688)):
        for bsz in range(1, 65):
            assert 0 < L.sirius_workspace_size(1, bsz, d, f, 0, 0) <= limit, (d, f, bsz)
    assert L.sirius_workspace_size(1, 64, 8192, 65536, 0, 0) > limit
    rc = L.sirius_ffn_cats_noalloc(FAKE, 64, FAKE, FAKE, FAKE, 8192, 65536, 0.1, -1.0, None, FAKE, None, None,
                                   None)
    assert rc == -2 and "scratch" in _err(L)


def test_topk_argument_errors(L):
    big = 1 << 30
    base = [FAKE, 1, FAKE, FAKE, FAKE, 64, 100, 50, -1.0, None, FAKE, FAKE, FAKE, FAKE, big, None]

    def call(**kw):
        a = list(base)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return L.sirius_ffn_topk(*a)

    assert call(a7=0) == -1 and "k=" in _err(L)
    assert call(a7=101) == -1
    assert call(a5=100) == -1            # d_model not a multiple of 8
    assert call(a12=None) == -1          # exactly one list pointer
    assert call(a8=float("nan")) == -1   # NaN norm_eps
    assert call(a14=16) == -2            # workspace too small
    assert call(a1=0) == 0               # empty batch


def test_griffin_argument_errors(L):
    big = 1 << 30
    args = [FAKE, 8, FAKE, FAKE, FAKE, 64, 100, 50, 0, FAKE, None, FAKE, FAKE, FAKE, FAKE, big, None]
    bad_k = list(args)
    bad_k[7] = 101
    assert L.sirius_griffin_select(*bad_k) == -1 and "k=" in _err(L)
    bad_k[7] = 0
    assert L.sirius_griffin_select(*bad_k) == -1
    bad_t = list(args)
    bad_t[1] = 0
    assert L.sirius_griffin_select(*bad_t) == -1
    small = list(args)
    small[15] = 64
    assert L.sirius_griffin_select(*small) == -2


def test_verify_argument_errors(L):
    big = 1 << 30
    nan = float("nan")
    base = [FAKE, 2, 4, 4, 100, FAKE, 0.1, 1.0, FAKE, FAKE, None, FAKE, big, None]

    def call(**kw):
        a = list(base)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return L.sirius_verify_accept(*a)

    assert call(a2=0) == -1            # K < 1
    assert call(a3=6) == -1            # R not in {K, K+1}
    assert call(a4=0) == -1            # V < 1
    assert call(a6=nan) == -1          # NaN r
    assert call(a7=0.0) == -1          # temperature 0
    assert call(a7=-1.0) == -1
    assert call(a7=float("inf")) == -1
    assert call(a5=None) == -1         # drafted NULL
    assert call(a12=16) == -2          # workspace too small
    assert call(a1=20000) == -1 and "rows" in _err(L)  # B * R above the grid limit
    assert call(a1=0) == 0             # empty batch


def test_tree_build_argument_errors(L):
    big = 1 << 30
    # logits, B, Wc, V, cum_ll, W, temperature, tokens, parents, cum_out, ws, ws_bytes, stream
    base = [FAKE, 2, 4, 100, FAKE, 8, 1.0, FAKE, FAKE, ctypes.c_void_p(1 << 21), FAKE, big, None]

    def call(**kw):
        a = list(base)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return L.sirius_tree_build_step(*a)

    assert call(a1=-1) == -1           # B < 0
    assert call(a2=0) == -1            # Wc < 1
    assert call(a2=17) == -1           # Wc above 16
    assert call(a5=0) == -1            # W < 1
    assert call(a5=17) == -1           # W above 16
    assert call(a3=1, a2=7) == -1 and "candidates" in _err(L)  # Wc * V < W
    assert call(a3=0) == -1            # V < 1
    assert call(a6=0.0) == -1          # temperature
    assert call(a6=float("inf")) == -1
    assert call(a7=None) == -1         # tokens NULL
    assert call(a9=FAKE) == -1 and "alias" in _err(L)
    assert call(a11=16) == -2          # workspace too small
    assert call(a0=ctypes.c_void_p((1 << 20) + 4)) == -1 and "aligned" in _err(L)
    assert call(a1=20000) == -1 and "rows" in _err(L)  # B * Wc above the grid limit
    assert call(a4=None, a1=0) == 0    # cum_ll may be NULL
    assert call(a1=0) == 0             # empty batch


def test_tree_verify_argument_errors(L):
    big = 1 << 30
    nan = float("nan")
    # logits, B, K, W, V, bonus, tokens, parents, r, T, best, acc, next, q, ws, ws_bytes, stream
    base = [FAKE, 2, 4, 8, 100, 1, FAKE, FAKE, 0.1, 1.0, FAKE, FAKE, FAKE, None, FAKE, big, None]

    def call(**kw):
        a = list(base)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return L.sirius_tree_verify(*a)

    assert call(a1=-1) == -1           # B < 0
    assert call(a2=0) == -1            # K < 1
    assert call(a3=0) == -1            # W < 1
    assert call(a3=65) == -1           # W above 64
    assert call(a2=16, a3=64) == -1 and "rows" in _err(L)  # K*W + W > 1024
    assert call(a2=16, a3=64, a5=0, a1=0) == 0  # exactly 1024 rows, empty batch
    assert call(a4=0) == -1            # V < 1
    assert call(a8=nan) == -1          # NaN r
    assert call(a9=0.0) == -1          # temperature
    assert call(a7=None) == -1         # parents NULL
    assert call(a10=None) == -1        # best_leaf NULL
    assert call(a0=ctypes.c_void_p((1 << 20) + 4)) == -1 and "aligned" in _err(L)
    assert call(a15=16) == -2          # workspace too small
    assert call(a1=2000) == -1 and "rows" in _err(L)  # B * R above the grid limit
    assert call(a1=0) == 0             # empty batch


def test_attn_argument_errors(L):
    big = 1 << 30
    # q, k_new, v_new, k_cache, v_cache, cache_pos, B, n, H, Hkv, hd, Lmax, out, ws, ws_bytes, stream
    base = [FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 16, 32, 8, 128, 4096, FAKE, FAKE, big, None]

    def call(**kw):
        a = list(base)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return L.sirius_attn_kv(*a)

    assert call(a7=0) == -1            # n < 1
    assert call(a7=2000) == -1         # n above 1024
    assert call(a8=30) == -1 and "Hkv" in _err(L)   # H not a multiple of Hkv
    assert call(a10=100) == -1         # head_dim not a multiple of 8
    assert call(a10=256) == -1         # head_dim above 128
    assert call(a11=8) == -1           # Lmax < n
    assert call(a5=None) == -1         # cache_pos NULL
    assert call(a3=ctypes.c_void_p((1 << 20) + 8)) == -1 and "aligned" in _err(L)
    assert call(a14=16) == -2          # workspace too small
    assert call(a6=0) == 0             # empty batch
    assert L.sirius_kv_rollback(None, FAKE, 1, 16, None) == -1
    assert L.sirius_kv_rollback(FAKE, FAKE, 1, 0, None) == -1
    assert L.sirius_kv_rollback(FAKE, FAKE, 0, 16, None) == 0


def test_glue_argument_errors(L):
    assert L.sirius_rmsnorm(None, 1, 64, 1e-5, FAKE, None) == -1
    assert L.sirius_rmsnorm(FAKE, 1, 64, -1.0, FAKE, None) == -1
    assert L.sirius_rmsnorm(FAKE, 0, 64, 1e-5, FAKE, None) == 0
    assert L.sirius_fill_normal_bf16(None, 10, 1, 0.0, 1.0, None) == -1
    assert L.sirius_fill_normal_bf16(FAKE, 10, 1, 0.0, -1.0, None) == -1
    assert L.sirius_fill_normal_bf16(FAKE, 0, 1, 0.0, 1.0, None) == 0


def test_workspace_sizes(L):
    f = L.sirius_workspace_size
    assert f(99, 1, 64, 64, 0, 0) == 0
    assert f(0, 1, 100, 64, 0, 0) == 0
    s1 = f(1, 1, 4096, 14336, 0, 0)
    s4 = f(1, 4, 4096, 14336, 0, 0)
    assert 0 < s1 < (64 << 20) and 0 < s4 < (64 << 20)
    assert f(4, 8, 0, 0, 128256, 16) > 0
    assert f(4, 8, 0, 0, 128256, 2000) == 0
    g = f(2, 0, 4096, 14336, 512, 0)
    assert g >= 512 * 14336 * 4
    c = f(5, 256, 4096, 14336, 0, 0)
    assert c >= 256 * 14336 * 4
    # per-token top-k: the activation buffer and cuts come before the FFN workspace
    assert f(8, 1, 4096, 14336, 0, 0) >= 14336 * 4 + f(1, 1, 4096, 14336, 0, 0)
    assert f(8, 3, 4096, 14336, 0, 0) >= 3 * 14336 * 4 + f(1, 3, 4096, 14336, 0, 0)
    # attention: B, n, H * 65536 + Hkv, head_dim, Lmax
    assert f(9, 1, 16, 32 * 65536 + 8, 128, 4096) > 0
    assert f(9, 1, 16, 30 * 65536 + 8, 128, 4096) == 0
    assert f(9, 1, 16, 32 * 65536 + 8, 128, 8) == 0
    # tree drafting step: B, Wc, W, V
    assert f(6, 1, 8, 8, 128256, 0) > 0
    assert f(6, 1, 17, 8, 128256, 0) == 0
    assert f(6, 1, 8, 17, 128256, 0) == 0
    assert f(6, 1, 8, 8, 7, 0) > 0     # 8 leaves of 7 tokens: 56 candidates
    assert f(6, 1, 1, 8, 7, 0) == 0
    # tree verification: B, K, W, V, bonus; the rows K*W (+W) are those of a chain check
    assert f(7, 1, 16, 8, 128256, 1) == f(4, 1, 0, 0, 128256, 16 * 8 + 8)
    assert f(7, 1, 16, 64, 128256, 0) > 0
    assert f(7, 1, 16, 64, 128256, 1) == 0
    assert f(7, 1, 4, 65, 128256, 0) == 0


def _fake_model(**kw):
    from paper_2409_03856_amd._lib import _ModelC
    thr = (ctypes.c_float * 2)(0.1, 0.1)
    vals = dict(n_layers=2, d_model=256, d_ff=688, n_heads=4, n_kv_heads=2, head_dim=64, vocab=1000,
                max_len=256, norm_eps=1e-5)
    ptrs = {k: FAKE.value for k in ("embed", "wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "lm_head",
                                    "k_cache", "v_cache")}
    ptrs["thresholds"] = ctypes.cast(thr, ctypes.c_void_p).value
    vals.update(ptrs)
    vals.update(kw)
    m = _ModelC(**vals)
    m._keep = thr
    return m


def test_model_argument_errors(L):
    big = 1 << 30
    m = _fake_model()
    assert L.sirius_model_workspace_size(ctypes.byref(m), 16) > 0
    assert L.sirius_model_workspace_size(ctypes.byref(m), 0) == 0
    assert L.sirius_model_workspace_size(ctypes.byref(m), 65) == 0
    assert L.sirius_model_workspace_size(None, 16) == 0
    # model, tokens, n, cache_pos, sparse, logits, active_idx, active_cnt, ws, ws_bytes, stream
    fwd = lambda mm, n=4, ws=big, **kw: L.sirius_model_forward(
        ctypes.byref(mm), FAKE, n, FAKE, kw.get("sparse", 1), FAKE, kw.get("ai"), kw.get("ac"), FAKE, ws, None)
    assert fwd(_fake_model(d_model=100)) == -1 and "d_model" in _err(L)
    assert fwd(_fake_model(n_heads=3)) == -1 and "n_kv_heads" in _err(L)
    assert fwd(_fake_model(head_dim=256)) == -1 and "head_dim" in _err(L)
    assert fwd(_fake_model(wq=None)) == -1 and "wq" in _err(L)
    assert fwd(_fake_model(k_cache=(1 << 20) + 4)) == -1 and "aligned" in _err(L)
    assert fwd(_fake_model(thresholds=None)) == -1 and "thresholds" in _err(L)
    assert fwd(_fake_model(thresholds=None), sparse=0, ws=16) == -2  # the full model needs none
    assert fwd(m, n=0) == -1 and fwd(m, n=65) == -1
    assert fwd(m, ai=FAKE) == -1 and "both" in _err(L)
    assert fwd(m, sparse=0, ai=FAKE, ac=FAKE) == -1 and "sparse" in _err(L)
    assert fwd(m, ws=16) == -2 and "workspace" in _err(L)
    nan = (ctypes.c_float * 2)(float("nan"), 0.1)
    assert fwd(_fake_model(thresholds=ctypes.cast(nan, ctypes.c_void_p).value)) == -1 and "NaN" in _err(L)
    # model, seq, cache_pos, n, r, periods, out_tokens, out_count, trace, ws, ws_bytes, stream
    gen = lambda n=16, r=0.1, periods=4, ws=big, seq=FAKE: L.sirius_generate(
        ctypes.byref(m), seq, FAKE, n, r, periods, FAKE, FAKE, None, FAKE, ws, None)
    assert gen(n=0) == -1 and gen(n=65) == -1
    assert gen(periods=-1) == -1
    assert gen(r=float("nan")) == -1 and "r is NaN" in _err(L)
    assert gen(seq=None) == -1
    assert gen(ws=16) == -2
    assert gen(periods=0) == 0  # nothing to do
