"""GPU parity: attention over the shared KV cache with the full model's direct rewrite, and
the rollback (Algorithm 1; Sec. 4, how to correct)."""

import math

import numpy as np
import pytest

import oracle
from synth import attn_inputs, bf16_bits
from gpu_util import say, dev_bf16, dev_f32, dev_i32, host

pytestmark = pytest.mark.gpu

ATTN_TOL = 1e-4  # max-abs error / RMS of the fp64 output (fp32 scores, softmax and sums)


@pytest.fixture(scope="module")
def sr():
    import paper_2409_03856_amd as sr
    sr.lib()
    return sr


def _check_out(got, want):
    rms = float(np.sqrt(np.mean(want * want)))
    err = float(np.max(np.abs(got - want))) / rms
    assert err <= ATTN_TOL, f"max-abs error {err:.3e} x RMS"
    return err


def _run(sr, q, kn, vn, kc, vc, pos):
    Kc, Vc = dev_bf16(kc), dev_bf16(vc)
    out = sr.sirius_attn_kv(dev_f32(q), dev_bf16(kn), dev_bf16(vn), Kc, Vc, dev_i32(np.asarray(pos)))
    return host(out), host(Kc), host(Vc)


def _check_call(sr, q, kn, vn, kc, vc, pos):
    out, kc2, vc2 = _run(sr, q, kn, vn, kc, vc, pos)
    ref, rk, rv = oracle.attn_kv(q, kn, vn, kc, vc, pos)
    e = _check_out(out, ref)
    # the rewrite is a copy of bf16 rows: bit-exact, and nothing else changes
    n = q.shape[1]
    want_k, want_v = kc.copy(), vc.copy()
    for b, p in enumerate(pos):
        want_k[b, p:p + n] = kn[b]
        want_v[b, p:p + n] = vn[b]
    assert np.array_equal(kc2, want_k) and np.array_equal(vc2, want_v)
    return e


def test_hand_case(sr):
    hd = 8
    q = np.zeros((1, 1, 1, hd), np.float32)
    q[0, 0, 0, 0] = math.sqrt(8.0) * math.log(3.0)
    kc = np.zeros((1, 4, 1, hd), np.float32)
    vc = np.zeros((1, 4, 1, hd), np.float32)
    vc[0, 0, 0, 0] = 4.0
    kn = np.zeros((1, 1, 1, hd), np.float32)
    vn = np.zeros((1, 1, 1, hd), np.float32)
    kn[0, 0, 0, 0] = 1.0
    vn[0, 0, 0, 1] = 8.0
    out, _, _ = _run(sr, q, bf16_bits(kn), bf16_bits(vn), bf16_bits(kc), bf16_bits(vc), [1])
    np.testing.assert_allclose(out[0, 0, 0, :2], [1.0, 6.0], rtol=2e-6)  # weights 1/4 and 3/4


@pytest.mark.parametrize("bsz,n,h,hkv,hd,lmax,pos", [
    (2, 3, 4, 2, 16, 100, [5, 80]),       # small, two batch entries
    (1, 1, 4, 4, 8, 9, [8]),              # decode into the last row
    (3, 5, 6, 3, 24, 70, [0, 33, 65]),     # from an empty cache; ragged head size
    (1, 16, 8, 1, 64, 300, [120]),        # one key/value head shared by all
])
def test_small_shapes(sr, bsz, n, h, hkv, hd, lmax, pos):
    say(f"attn B={bsz} n={n} H={h} Hkv={hkv} hd={hd} Lmax={lmax} pos={pos}")
    q, kn, vn, kc, vc = attn_inputs(bsz * 100 + n, bsz, n, h, hkv, hd, lmax)
    _check_call(sr, q, kn, vn, kc, vc, pos)


@pytest.mark.parametrize("n,p", [(1, 2047), (16, 2000), (1, 0), (16, 4080)])
def test_llama3_8b_heads(sr, n, p):
    # 32 query heads, 8 key/value heads, head size 128, a 4096-row cache
    say(f"attn 8B heads n={n} p={p}")
    q, kn, vn, kc, vc = attn_inputs(7 + n, 1, n, 32, 8, 128, 4096)
    e = _check_call(sr, q, kn, vn, kc, vc, [p])
    say(f"  error {e:.2e} x RMS")


def test_many_rows_and_chunks(sr):
    # 64 query heads over 8 (70B grouping): 128 query rows per key/value head at n = 16 (two row
    # groups); a 20000-row cache (128-row chunks)
    say("attn 70B heads n=16 p=17000")
    q, kn, vn, kc, vc = attn_inputs(11, 1, 16, 64, 8, 128, 20000)
    _check_call(sr, q, kn, vn, kc, vc, [17000])


def test_positions_outside_the_cache_leave_it_untouched(sr):
    q, kn, vn, kc, vc = attn_inputs(13, 3, 4, 4, 2, 16, 50)
    out, kc2, vc2 = _run(sr, q, kn, vn, kc, vc, [-1, 20, 47])
    assert np.isnan(out[0]).all() and np.isnan(out[2]).all()
    ref, rk, rv = oracle.attn_kv(q[1:2], kn[1:2], vn[1:2], kc[1:2], vc[1:2], [20])
    _check_out(out[1:2], ref)
    assert np.array_equal(kc2[0], kc[0]) and np.array_equal(kc2[2], kc[2])
    assert np.array_equal(vc2[0], vc[0]) and np.array_equal(vc2[2], vc[2])


def test_rollback(sr):
    import torch
    pos = dev_i32(np.array([10, 10, 10, 10, 0], np.int32))
    acc = dev_i32(np.array([0, 5, 15, 16, 0], np.int32))
    sr.sirius_kv_rollback(pos, acc, 16)
    assert host(pos).tolist() == oracle.kv_rollback([10, 10, 10, 10, 0], [0, 5, 15, 16, 0], 16).tolist()


def test_draft_verify_rollback_episode(sr):
    """Algorithm 1 on one attention layer: the sparse model drafts n tokens one position at a
    time, the full model rewrites the n rows and attends in one pass, the position rolls back
    to the accepted prefix; twice. The GPU cache and positions must track the oracle's."""
    h, hkv, hd, lmax, n = 8, 2, 32, 200, 6
    rng = np.random.default_rng(5)
    _, _, _, kc, vc = attn_inputs(17, 1, 1, h, hkv, hd, lmax)
    Kc, Vc = dev_bf16(kc), dev_bf16(vc)
    ref_k, ref_v = oracle.widen_bf16(kc), oracle.widen_bf16(vc)
    pos = dev_i32(np.array([40], np.int32))
    p_ref = 40
    for episode, accept in enumerate((2, 6)):
        start = p_ref
        for i in range(n):  # sparse decode steps
            q = rng.standard_normal((1, 1, h, hd)).astype(np.float32)
            kn = bf16_bits(rng.standard_normal((1, 1, hkv, hd)).astype(np.float32))
            vn = bf16_bits(rng.standard_normal((1, 1, hkv, hd)).astype(np.float32))
            out = sr.sirius_attn_kv(dev_f32(q), dev_bf16(kn), dev_bf16(vn), Kc, Vc, pos)
            ref, ref_k, ref_v = oracle.attn_kv(q, kn, vn, ref_k, ref_v, [p_ref])
            _check_out(host(out), ref)
            sr.sirius_kv_rollback(pos, dev_i32(np.array([0], np.int32)), 1)  # advance by one
            p_ref += 1
        # the full model's pass over the chunk: wind back, rewrite, attend
        pos = dev_i32(np.array([start], np.int32))
        p_ref = start
        q = rng.standard_normal((1, n, h, hd)).astype(np.float32)
        kn = bf16_bits(rng.standard_normal((1, n, hkv, hd)).astype(np.float32))
        vn = bf16_bits(rng.standard_normal((1, n, hkv, hd)).astype(np.float32))
        out = sr.sirius_attn_kv(dev_f32(q), dev_bf16(kn), dev_bf16(vn), Kc, Vc, pos)
        ref, ref_k, ref_v = oracle.attn_kv(q, kn, vn, ref_k, ref_v, [p_ref])
        _check_out(host(out), ref)
        sr.sirius_kv_rollback(pos, dev_i32(np.array([accept], np.int32)), n)
        p_ref = int(oracle.kv_rollback([p_ref], [accept], n)[0])
        assert int(host(pos)[0]) == p_ref
        assert np.array_equal(oracle.widen_bf16(host(Kc)), ref_k)
        assert np.array_equal(oracle.widen_bf16(host(Vc)), ref_v)
        say(f"episode {episode}: position {p_ref}")
