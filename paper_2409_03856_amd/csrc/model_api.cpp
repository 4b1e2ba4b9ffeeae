// C ABI of the small decoder and of the Sirius generation loop (Algorithm 1): host-side
// validation, the workspace carve, and the fixed launch sequence of a forward pass and of a
// period. Every step runs in the library's kernels; nothing here touches device data.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "sirius.h"
#include "common.h"
#include "kernels.h"

namespace {

constexpr int kMaxModelTokens = 64;  // tokens per forward pass (the FFN batch limit)

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  sirius::set_last_error(buf);
  return code;
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return SIRIUS_OK;
  return fail(SIRIUS_EHIP, "%s: HIP error %d (%s)", what, (int)e, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Workspace of a forward pass of up to nmax tokens (and of a period with n = nmax).
struct ModelLayout {
  size_t h, xn, q, kb, vb, att, logits, ints, sub, total;
};

size_t ffn_ws_any(int B, int d, int F, bool sparse) {
  return sirius::ffn_any_ws(B, d, F, sparse ? sirius::kFfnModeThreshold : sirius::kFfnModeDense);
}

ModelLayout model_layout(const sirius_model* m, int nmax) {
  const int d = m->d_model, hq = m->n_heads * m->head_dim, hkv = m->n_kv_heads * m->head_dim;
  ModelLayout L{};
  sirius::Carve c;
  L.h = c.take((size_t)nmax * d * 4);
  L.xn = c.take((size_t)nmax * d * 4);
  L.q = c.take((size_t)nmax * hq * 4);
  L.kb = c.take((size_t)nmax * hkv * 2);
  L.vb = c.take((size_t)nmax * hkv * 2);
  L.att = c.take((size_t)nmax * hq * 4);
  L.logits = c.take((size_t)nmax * m->vocab * 4);
  L.ints = c.take(64);
  size_t sub = 0;
  for (int b = 1; b <= nmax; ++b) {
    sub = std::max(sub, sirius::attn_layout(1, b, m->n_heads, m->n_kv_heads, m->head_dim,
                                            m->max_len).total);
    sub = std::max(sub, ffn_ws_any(b, d, m->d_ff, true));
    sub = std::max(sub, ffn_ws_any(b, d, m->d_ff, false));
    sub = std::max(sub, sirius::verify_layout(1, b, m->vocab).total);
  }
  L.sub = c.take(sub);
  L.total = c.off;
  return L;
}

int check_model(const char* fn, const sirius_model* m) {
  if (m == nullptr) return fail(SIRIUS_EINVAL, "%s: model is NULL", fn);
  if (m->n_layers < 1) return fail(SIRIUS_EINVAL, "%s: n_layers=%d must be >= 1", fn, m->n_layers);
  if (m->d_model < 8 || m->d_model > 8192 || m->d_model % 8 != 0)
    return fail(SIRIUS_EINVAL, "%s: d_model=%d must be a multiple of 8 in [8, 8192]", fn, m->d_model);
  if (m->d_ff < 1 || m->d_ff > 65536) return fail(SIRIUS_EINVAL, "%s: d_ff=%d outside [1, 65536]", fn, m->d_ff);
  if (m->n_heads < 1 || m->n_kv_heads < 1 || m->n_heads % m->n_kv_heads != 0)
    return fail(SIRIUS_EINVAL, "%s: n_heads=%d must be a positive multiple of n_kv_heads=%d", fn,
                m->n_heads, m->n_kv_heads);
  if (m->head_dim < 8 || m->head_dim > 128 || m->head_dim % 8 != 0)
    return fail(SIRIUS_EINVAL, "%s: head_dim=%d must be a multiple of 8 in [8, 128]", fn, m->head_dim);
  if ((long)m->n_heads * m->head_dim > 8192)
    return fail(SIRIUS_EINVAL, "%s: n_heads*head_dim above 8192", fn);
  if (m->vocab < 1 || m->vocab > (1 << 24)) return fail(SIRIUS_EINVAL, "%s: vocab=%d outside [1, 2^24]", fn, m->vocab);
  if (m->max_len < 1 || m->max_len > (1 << 20)) return fail(SIRIUS_EINVAL, "%s: max_len=%d outside [1, 2^20]", fn, m->max_len);
  if (!(m->norm_eps >= 0.f) || std::isinf(m->norm_eps)) return fail(SIRIUS_EINVAL, "%s: norm_eps must be finite and >= 0", fn);
  const void* ptrs[] = {m->embed, m->wq, m->wk, m->wv, m->wo, m->w_gate, m->w_up, m->w_down,
                        m->lm_head, m->k_cache, m->v_cache};
  const char* names[] = {"embed", "wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "lm_head",
                         "k_cache", "v_cache"};
  for (int i = 0; i < 11; ++i) {
    if (ptrs[i] == nullptr) return fail(SIRIUS_EINVAL, "%s: model.%s is NULL", fn, names[i]);
    if (!aligned16(ptrs[i])) return fail(SIRIUS_EINVAL, "%s: model.%s is not 16-byte aligned", fn, names[i]);
  }
  return SIRIUS_OK;
}

int check_thresholds(const char* fn, const sirius_model* m) {
  if (m->thresholds == nullptr) return fail(SIRIUS_EINVAL, "%s: model.thresholds is NULL", fn);
  for (int l = 0; l < m->n_layers; ++l)
    if (std::isnan(m->thresholds[l])) return fail(SIRIUS_EINVAL, "%s: thresholds[%d] is NaN", fn, l);
  return SIRIUS_OK;
}

// Per-layer strides (elements)
struct Strides {
  size_t q, kv, o, ffn, cache;
};
Strides strides(const sirius_model* m) {
  const size_t d = m->d_model, hq = (size_t)m->n_heads * m->head_dim,
               hkv = (size_t)m->n_kv_heads * m->head_dim;
  return {hq * d, hkv * d, d * hq, (size_t)m->d_ff * d, (size_t)m->max_len * hkv};
}

hipError_t ffn_any(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                   const uint16_t* wd, int d, int F, bool sparse, float t, float eps,
                   const float* resid, float* y, int32_t* aidx, int32_t* acnt, char* ws,
                   hipStream_t s) {
  return sirius::launch_ffn_any(x, B, wg, wu, wd, d, F,
                                sparse ? sirius::kFfnModeThreshold : sirius::kFfnModeDense, t, eps,
                                resid, y, aidx, acnt, ws, s);
}

// One pass over n tokens at the device-held position. Active lists (sparse only) go to
// aidx + l * a_lstride, acnt + l * c_lstride for layer l.
hipError_t forward(const sirius_model* m, const int32_t* tokens, int n, const int32_t* cache_pos,
                   bool sparse, float* logits, int32_t* aidx, size_t a_lstride, int32_t* acnt,
                   size_t c_lstride, char* ws, const ModelLayout& L, hipStream_t s) {
  const int d = m->d_model, H = m->n_heads, Hkv = m->n_kv_heads, hd = m->head_dim;
  const int hq = H * hd, hkv = Hkv * hd;
  const Strides st = strides(m);
  float* h = reinterpret_cast<float*>(ws + L.h);
  float* xn = reinterpret_cast<float*>(ws + L.xn);
  float* q = reinterpret_cast<float*>(ws + L.q);
  uint16_t* kb = reinterpret_cast<uint16_t*>(ws + L.kb);
  uint16_t* vb = reinterpret_cast<uint16_t*>(ws + L.vb);
  float* att = reinterpret_cast<float*>(ws + L.att);
  char* sub = ws + L.sub;
  hipError_t e;
  // the norm folds into the projections' launch when the rows take the vectorised norm (the
  // same sums, so the same bits); otherwise the separate norm and one launch per product
  const bool fused = (d & 3) == 0 && d <= 8192 && (reinterpret_cast<uintptr_t>(h) & 15) == 0;
  if ((e = sirius::launch_embed(tokens, n, m->embed, d, m->vocab, h, s)) != hipSuccess) return e;
  for (int l = 0; l < m->n_layers; ++l) {
    if (fused) {
      if ((e = sirius::launch_norm_qkv(h, n, d, m->norm_eps, m->wq + l * st.q, hq, m->wk + l * st.kv,
                                       m->wv + l * st.kv, hkv, q, kb, vb, s)) != hipSuccess)
        return e;
    } else {
      if ((e = sirius::launch_rmsnorm(h, n, d, m->norm_eps, xn, s)) != hipSuccess) return e;
      if ((e = sirius::launch_linear(xn, n, m->wq + l * st.q, d, hq, nullptr, q, nullptr, s)) != hipSuccess) return e;
      if ((e = sirius::launch_linear(xn, n, m->wk + l * st.kv, d, hkv, nullptr, nullptr, kb, s)) != hipSuccess) return e;
      if ((e = sirius::launch_linear(xn, n, m->wv + l * st.kv, d, hkv, nullptr, nullptr, vb, s)) != hipSuccess) return e;
    }
    const sirius::AttnLayout AL = sirius::attn_layout(1, n, H, Hkv, hd, m->max_len);
    if ((e = sirius::launch_attn_kv(q, kb, vb, m->k_cache + l * st.cache, m->v_cache + l * st.cache,
                                    cache_pos, 1, n, H, Hkv, hd, m->max_len, att, sub, AL, s)) != hipSuccess)
      return e;
    if ((e = sirius::launch_linear(att, n, m->wo + l * st.o, hq, d, h, h, nullptr, s)) != hipSuccess) return e;
    const float t = sparse ? m->thresholds[l] : 0.f;
    if ((e = ffn_any(h, n, m->w_gate + l * st.ffn, m->w_up + l * st.ffn, m->w_down + l * st.ffn, d,
                     m->d_ff, sparse, t, m->norm_eps, h, h, aidx ? aidx + l * a_lstride : nullptr,
                     acnt ? acnt + l * c_lstride : nullptr, sub, s)) != hipSuccess)
      return e;
  }
  if (fused)
    return sirius::launch_norm_qkv(h, n, d, m->norm_eps, m->lm_head, m->vocab, nullptr, nullptr, 0,
                                   logits, nullptr, nullptr, s);
  if ((e = sirius::launch_rmsnorm(h, n, d, m->norm_eps, xn, s)) != hipSuccess) return e;
  return sirius::launch_linear(xn, n, m->lm_head, d, m->vocab, nullptr, logits, nullptr, s);
}

}  // namespace

extern "C" {

size_t sirius_model_workspace_size(const sirius_model* model, int max_tokens) {
  if (model == nullptr || max_tokens < 1 || max_tokens > kMaxModelTokens) return 0;
  if (check_model("sirius_model_workspace_size", model) != SIRIUS_OK) return 0;
  return model_layout(model, max_tokens).total;
}

int sirius_model_forward(const sirius_model* model, const int32_t* tokens, int n,
                         const int32_t* cache_pos, int sparse, float* logits, int32_t* active_idx,
                         int32_t* active_cnt, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sirius_model_forward";
  int rc = check_model(fn, model);
  if (rc) return rc;
  if (n < 1 || n > kMaxModelTokens) return fail(SIRIUS_EINVAL, "%s: n=%d outside [1, %d]", fn, n, kMaxModelTokens);
  if (tokens == nullptr || cache_pos == nullptr || logits == nullptr || ws == nullptr)
    return fail(SIRIUS_EINVAL, "%s: a required pointer is NULL", fn);
  if (!aligned16(logits) || !aligned16(ws)) return fail(SIRIUS_EINVAL, "%s: logits and ws must be 16-byte aligned", fn);
  if ((active_idx == nullptr) != (active_cnt == nullptr))
    return fail(SIRIUS_EINVAL, "%s: active_idx and active_cnt must both be given or both be NULL", fn);
  if (active_idx != nullptr && !sparse)
    return fail(SIRIUS_EINVAL, "%s: active lists are only produced by the sparse model", fn);
  if (sparse && (rc = check_thresholds(fn, model))) return rc;
  if (n > model->max_len) return fail(SIRIUS_EINVAL, "%s: n=%d above max_len=%d", fn, n, model->max_len);
  const ModelLayout L = model_layout(model, n);
  if (ws_bytes < L.total)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, L.total);
  return hip_status(forward(model, tokens, n, cache_pos, sparse != 0, logits, active_idx,
                            (size_t)n * model->d_ff, active_cnt, (size_t)n, static_cast<char*>(ws),
                            L, static_cast<hipStream_t>(stream)),
                    fn);
}

int sirius_generate(const sirius_model* model, int32_t* seq, int32_t* cache_pos, int n, float r,
                    int periods, int32_t* out_tokens, int32_t* out_count,
                    const sirius_gen_trace* trace, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sirius_generate";
  int rc = check_model(fn, model);
  if (rc) return rc;
  if ((rc = check_thresholds(fn, model))) return rc;
  if (n < 1 || n > kMaxModelTokens) return fail(SIRIUS_EINVAL, "%s: n=%d outside [1, %d]", fn, n, kMaxModelTokens);
  if (n > model->max_len) return fail(SIRIUS_EINVAL, "%s: n=%d above max_len=%d", fn, n, model->max_len);
  if (periods < 0) return fail(SIRIUS_EINVAL, "%s: periods=%d < 0", fn, periods);
  if ((long)periods * n > (1L << 30)) return fail(SIRIUS_EINVAL, "%s: periods*n too large", fn);
  if (std::isnan(r)) return fail(SIRIUS_EINVAL, "%s: r is NaN", fn);
  if (seq == nullptr || cache_pos == nullptr || out_tokens == nullptr || out_count == nullptr || ws == nullptr)
    return fail(SIRIUS_EINVAL, "%s: a required pointer is NULL", fn);
  if (!aligned16(ws)) return fail(SIRIUS_EINVAL, "%s: ws must be 16-byte aligned", fn);
  if (trace != nullptr && (trace->active_idx == nullptr) != (trace->active_cnt == nullptr))
    return fail(SIRIUS_EINVAL, "%s: trace active_idx and active_cnt must both be given or both be NULL", fn);
  const ModelLayout L = model_layout(model, n);
  if (ws_bytes < L.total)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, L.total);
  if (periods == 0) return SIRIUS_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  float* logits = reinterpret_cast<float*>(w + L.logits);
  int32_t* acc = reinterpret_cast<int32_t*>(w + L.ints);
  int32_t* nxt = acc + 1;
  const int V = model->vocab, Ln = model->n_layers, F = model->d_ff;
  const int cap = periods * n;
  for (int p = 0; p < periods; ++p) {
    // drafting: the sparse model, one token at a time, rows P .. P + n - 1
    for (int i = 0; i < n; ++i) {
      int32_t* aidx = nullptr;
      int32_t* acnt = nullptr;
      if (trace != nullptr && trace->active_idx != nullptr) {
        const size_t step = (size_t)p * n + i;
        aidx = trace->active_idx + step * Ln * F;
        acnt = trace->active_cnt + step * Ln;
      }
      hipError_t e = forward(model, seq + i, 1, cache_pos, true, logits, aidx, (size_t)F, acnt, 1,
                             w, L, s);
      if (e != hipSuccess) return hip_status(e, fn);
      e = sirius::launch_draft_tail(logits, V, seq, i + 1, cache_pos, (i + 1 < n) ? 1 : 1 - n,
                                    (trace && trace->drafted) ? trace->drafted + (size_t)p * n : nullptr, s);
      if (e != hipSuccess) return hip_status(e, fn);
    }
    // the check: the full model over seq[0 .. n - 1] at P (rewriting rows P .. P + n - 1)
    hipError_t e = forward(model, seq, n, cache_pos, false, logits, nullptr, 0, nullptr, 0, w, L, s);
    if (e != hipSuccess) return hip_status(e, fn);
    e = sirius::launch_verify(logits, 1, n, n, V, seq + 1, r, 1.0f, acc, nxt,
                              (trace && trace->q) ? trace->q + (size_t)p * n : nullptr, w + L.sub,
                              sirius::verify_layout(1, n, V), s);
    if (e != hipSuccess) return hip_status(e, fn);
    e = sirius::launch_period_tail(seq, n, acc, nxt, cache_pos, out_tokens, out_count, cap,
                                   (trace && trace->accept_len) ? trace->accept_len + p : nullptr,
                                   (trace && trace->next_token) ? trace->next_token + p : nullptr, s);
    if (e != hipSuccess) return hip_status(e, fn);
  }
  return SIRIUS_OK;
}

}  // extern "C"
