"""Helpers for the GPU parity tests: upload seeded inputs, parity checks against the oracle.

Tolerances (see the design notes for their derivation):
  * active-neuron sets: bit-exact outside a guard band |(|a| - t)| <= 1e-3;
  * FFN outputs on the fp32-input paths: max-abs error <= 1e-4 x RMS of the
    oracle output (fp32 accumulation of bf16 x fp32 products); the stated
    bound of the method, 2e-2 x RMS, is asserted as well;
  * FFN outputs on the MFMA path (batch >= 8; the normalised input rounded to bf16):
    <= 1e-4 x RMS against the oracle on the rounded input (with RMSNorm plus a first-order
    allowance for inputs whose rounding is ambiguous, see check_ffn_rounded_norm), and the
    method bound against the unrounded input;
  * per-token top-k sets: exactly k neurons, bit-exact outside |(|a| - a_(k))| <= 1e-3
    (a_(k) the token's k-th largest |a|), then the output against the oracle's FFN on the
    GPU's own set;
  * acceptance lengths: bit-exact outside a guard band |q - r| <= 1e-5 r, with at most
    one excluded row (or tree) per case;
  * tree drafting step: (parent, token) pairs bit-exact at every rank whose score is more
    than 1e-5 from its neighbours' (and from the first excluded candidate's); near-tied ranks
    must hold valid, distinct pairs whose scores match the oracle's rank scores within the
    band; stored scores within 2e-5 + 2e-6 |score| (fp32 storage of an fp64 value).
"""

from __future__ import annotations

import sys

import numpy as np

import oracle

FP32_PATH_TOL = 1e-4
METHOD_TOL = 2e-2
MFMA_MIN_BATCH = 8
# The GPU's fp32 RMSNorm differs from the fp64 one by a few fp32 ulps; an element whose fp64
# value lies within this relative distance of a bf16 rounding boundary may round either way.
NORM_ROUNDING_BAND = 4e-6
CATS_BAND = 1e-3
VERIFY_BAND = 1e-5
# At most this many rows (or trees) of one parity case may be excluded for a q inside the guard
# band: a q that is systematically wrong near r would otherwise be excluded instead of caught.
MAX_BOUNDARY_ROWS = 1
TREE_SCORE_BAND = 1e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev_bf16(bits: np.ndarray):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).cuda()


def dev_f32(a: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def dev_i32(a: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def host(t) -> np.ndarray:
    import torch
    torch.cuda.synchronize()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def rounded_bf16(x) -> np.ndarray:
    """x rounded to bf16 (nearest even) and widened back: the MFMA path's input precision."""
    from synth import bf16_bits
    return oracle.widen_bf16(bf16_bits(np.asarray(x, dtype=np.float32)))


def rel_err(got, want) -> float:
    want = np.asarray(want, dtype=np.float64)
    rms = float(np.sqrt(np.mean(want * want)))
    return float(np.max(np.abs(np.asarray(got, dtype=np.float64) - want))) / max(rms, 1e-300)


def check_cats_sets(x_in, wg, t, idx, cnt, band=CATS_BAND):
    """GPU sets equal the oracle's outside the guard band. Returns (gpu_sets, boundary_count)."""
    sets_o, a = oracle.cats_active_sets(x_in, wg, t)
    gpu_sets = []
    n_boundary = 0
    for b in range(len(sets_o)):
        g = idx[b, : int(cnt[b])].astype(np.int64)
        assert np.all(np.diff(g) > 0), "active list must be strictly ascending"
        near = np.abs(np.abs(a[b]) - t) <= band
        n_boundary += int(near.sum())
        sym = np.setxor1d(g, sets_o[b])
        assert np.all(near[sym]), f"token {b}: {int((~near[sym]).sum())} set mismatches outside the band"
        gpu_sets.append(g)
    return gpu_sets, n_boundary


def check_topk_sets(x_in, wg, k, idx, cnt, band=CATS_BAND):
    """Per-token top-k sets: exactly k ascending neurons per token, equal to the oracle's outside
    the guard band around the token's k-th largest |a| (the GPU decides on fp32 activations).
    Returns (gpu_sets, boundary_count)."""
    sets_o, a = oracle.topk_active_sets(x_in, wg, k)
    gpu_sets = []
    n_boundary = 0
    for b in range(len(sets_o)):
        assert int(cnt[b]) == k, f"token {b}: {int(cnt[b])} neurons kept, expected {k}"
        g = idx[b, :k].astype(np.int64)
        assert np.all(np.diff(g) > 0), "active list must be strictly ascending"
        assert g[0] >= 0 and g[-1] < a.shape[1]
        tk = np.sort(np.abs(a[b]))[::-1][k - 1]
        near = np.abs(np.abs(a[b]) - tk) <= band
        n_boundary += int(near.sum())
        sym = np.setxor1d(g, sets_o[b])
        assert np.all(near[sym]), f"token {b}: {int((~near[sym]).sum())} set mismatches outside the band"
        gpu_sets.append(g)
    return gpu_sets, n_boundary


def check_ffn(y_gpu, y_ref, resid=None, tol=FP32_PATH_TOL):
    y_gpu = np.asarray(y_gpu, dtype=np.float64)
    if resid is not None:
        y_gpu = y_gpu - np.asarray(resid, dtype=np.float64)
    e = rel_err(y_gpu, y_ref)
    assert e <= METHOD_TOL, f"max-abs error {e:.3e} x RMS exceeds the method bound"
    assert e <= tol, f"max-abs error {e:.3e} x RMS exceeds {tol:.1e}"
    return e


def check_ffn_rounded_norm(y_gpu, xn, w_gate, w_up, w_down, sets=None, resid=None,
                           tol=FP32_PATH_TOL, band=NORM_ROUNDING_BAND):
    """Output check for the MFMA path with RMSNorm, whose gate/up input is the GPU's fp32
    normalised input rounded to bf16.

    Reference: the oracle FFN (masked to `sets` when given) on the fp64 normalised input xn
    rounded to bf16. Where xn lies within `band` (relative) of a bf16 rounding boundary the
    GPU may have rounded the other way, by one bf16 ulp. The effect of each such element k
    on the output is bounded to first order by |J[:, k]| * ulp_k, J the FFN's Jacobian at the
    reference input; the sum over the boundary elements (with a 1.5x margin for second-order
    terms) is added, per output element, to tol x RMS. Returns (max-abs error / RMS, number of
    boundary elements)."""
    from synth import bf16_bits
    xn = np.atleast_2d(np.asarray(xn, dtype=np.float64))
    widen = lambda v: oracle.widen_bf16(bf16_bits(np.asarray(v, dtype=np.float32)))
    xr = widen(xn)
    lo, hi = widen(xn * (1.0 - band)), widen(xn * (1.0 + band))
    if sets is None:
        ref = oracle.ffn_dense(xr, w_gate, w_up, w_down)
    else:
        ref = oracle.ffn_masked(xr, w_gate, w_up, w_down, sets)
    y = np.atleast_2d(np.asarray(y_gpu, dtype=np.float64))
    if resid is not None:
        y = y - np.asarray(resid, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    allow = np.zeros_like(ref)
    nb = 0
    wg64, wu64, wd64 = (oracle.widen_bf16(np.asarray(w)) for w in (w_gate, w_up, w_down))
    for b in range(xn.shape[0]):
        ks = np.flatnonzero(lo[b] != hi[b])
        if ks.size == 0:
            continue
        nb += int(ks.size)
        g, u = wg64 @ xr[b], wu64 @ xr[b]
        sg = 1.0 / (1.0 + np.exp(-g))
        dsilu = sg * (1.0 + g * (1.0 - sg))
        dh = (dsilu * u)[:, None] * wg64[:, ks] + (g * sg)[:, None] * wu64[:, ks]  # [F, |K|]
        if sets is not None:
            keep = np.zeros(g.shape[0], dtype=bool)
            keep[np.asarray(sets[b], dtype=np.int64)] = True
            dh[~keep] = 0.0
        jac = wd64.T @ dh  # [d, |K|]
        allow[b] = 1.5 * (np.abs(jac) @ np.abs(hi[b, ks] - lo[b, ks]))
    err = np.abs(y - ref)
    e = float(np.max(err)) / rms
    assert e <= METHOD_TOL, f"max-abs error {e:.3e} x RMS exceeds the method bound"
    bad = err > tol * rms + allow
    assert not np.any(bad), (f"{int(bad.sum())} outputs exceed {tol:.1e} x RMS plus the rounding "
                             f"allowance of {nb} boundary inputs (max-abs error {e:.3e} x RMS)")
    return e, nb


def verify_boundary_rows(q_oracle, acc_oracle, r, band=VERIFY_BAND):
    """Rows where some q_j (j <= accept_len) lies within the guard band of r."""
    rows = []
    for b in range(q_oracle.shape[0]):
        jmax = min(int(acc_oracle[b]), q_oracle.shape[1] - 1)
        if np.any(np.abs(q_oracle[b, : jmax + 1] - r) <= band * abs(r)):
            rows.append(b)
    return rows


def check_tree_build(logits, cum, width, tau, tok, par, out, band=TREE_SCORE_BAND):
    """Check one tree's drafting step (tokens tok, parents par, scores out, best first) against
    the oracle. Returns the number of near-tied ranks, where only validity is checked."""
    lg = np.atleast_2d(np.asarray(logits, dtype=np.float64))
    wc, v = lg.shape
    n_cand = wc * v
    tok_o, par_o, sc_o = oracle.tree_build_step(lg, cum, min(width + 1, n_cand), tau)
    ls = oracle.log_softmax(lg, tau)
    base = np.zeros(wc) if cum is None else np.asarray(cum, dtype=np.float64)
    tok = np.asarray(tok, dtype=np.int64)
    par = np.asarray(par, dtype=np.int64)
    assert tok.shape == (width,) and par.shape == (width,)
    assert ((tok >= 0) & (tok < v)).all(), tok
    assert ((par >= 0) & (par < wc)).all(), par
    assert len(set(zip(par.tolist(), tok.tolist()))) == width, "a (parent, token) pair is repeated"
    got = base[par] + ls[par, tok]
    tol = band * np.maximum(1.0, np.abs(sc_o[:width]))
    assert np.all(np.abs(got - sc_o[:width]) <= tol), (got, sc_o[:width])
    np.testing.assert_allclose(np.asarray(out, dtype=np.float64), sc_o[:width], rtol=2e-6, atol=2e-5)
    near = 0
    for j in range(width):
        lo_gap = sc_o[j - 1] - sc_o[j] if j > 0 else np.inf
        hi_gap = sc_o[j] - sc_o[j + 1] if j + 1 < len(sc_o) else np.inf
        if min(lo_gap, hi_gap) <= tol[j]:
            near += 1
            continue
        assert (par[j], tok[j]) == (par_o[j], tok_o[j]), (j, par[j], tok[j], par_o[j], tok_o[j])
    return near
