// C ABI of libsirius: host-side argument validation, workspace checks and dispatch to the
// gfx950 kernels. Nothing is enqueued unless every argument check passes.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "sirius.h"
#include "kernels.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return SIRIUS_OK;
  return fail(SIRIUS_EHIP, "%s: HIP error %d (%s)", what, (int)e, hipGetErrorString(e));
}

constexpr int kMaxDModel = 8192;
constexpr int kMaxDFF = 65536;
constexpr int kMaxBatch = 64;
constexpr int kMaxVerifyRows = 1024;
constexpr int kMaxTreeBuildW = 16;   // tree width and current-leaf limit of a drafting step
constexpr int kMaxTreeVerifyW = 64;  // tree width limit of tree verification
constexpr long kMaxLogitRows = 65535;  // B * rows of a logit pass (second grid dimension)
constexpr int kMaxAttnTokens = 1024;   // tokens per attention call
constexpr int kMaxCacheLen = 1 << 20;  // cache rows per batch entry

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_ffn_dims(const char* fn, int B, int d_model, int d_ff) {
  if (B < 0 || B > kMaxBatch) return fail(SIRIUS_EINVAL, "%s: B=%d outside [0, %d]", fn, B, kMaxBatch);
  if (d_model < 8 || d_model > kMaxDModel || (d_model % 8) != 0)
    return fail(SIRIUS_EINVAL, "%s: d_model=%d must be a multiple of 8 in [8, %d]", fn, d_model, kMaxDModel);
  if (d_ff < 1 || d_ff > kMaxDFF)
    return fail(SIRIUS_EINVAL, "%s: d_ff=%d outside [1, %d]", fn, d_ff, kMaxDFF);
  return SIRIUS_OK;
}

int check_ptrs(const char* fn, std::initializer_list<std::pair<const void*, const char*>> ptrs) {
  for (auto& p : ptrs) {
    if (p.first == nullptr) return fail(SIRIUS_EINVAL, "%s: %s is NULL", fn, p.second);
    if (!aligned16(p.first)) return fail(SIRIUS_EINVAL, "%s: %s is not 16-byte aligned", fn, p.second);
  }
  return SIRIUS_OK;
}

bool dims_ok(int d_model, int d_ff) {
  return d_model >= 8 && d_model <= kMaxDModel && (d_model % 8) == 0 && d_ff >= 1 && d_ff <= kMaxDFF;
}

}  // namespace

namespace sirius {

// Input pieces of the batched MFMA path: the dense chunk/tree pass (8 or more tokens) takes x
// rounded to bf16, every other batched call the exact fp32 input as three bf16 pieces.
static int batch_px(int B, int mode) {
  return (mode == kFfnModeDense && B >= kMfmaMinBatch) ? 1 : 3;
}

// B == 1 runs the one-pass decode kernel; 2..64 tokens with d_model % 256 == 0 the batched MFMA
// kernels; other shapes the older MFMA kernels (dense, B >= 8) or the small-batch kernels in
// LDS-sized chunks.
size_t ffn_any_ws(int B, int d, int F, int mode) {
  if (B <= 1) return decode1_layout(d, F).total;
  if (batch_path_ok(B, d, F)) return batch_layout(B, d, F, batch_px(B, mode)).total;
  if (mode == kFfnModeDense && B >= kMfmaMinBatch) return mfma_layout(B, d, F).total;
  return gemv_layout(B, d, F).total;
}

hipError_t launch_ffn_any(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                          const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                          char* ws, hipStream_t s) {
  if (B == 1)
    return launch_ffn_decode1(x, wg, wu, wd, d, F, mode, t, norm_eps, resid, y, active_idx,
                              active_cnt, ws, decode1_layout(d, F), s);
  if (batch_path_ok(B, d, F))
    return launch_ffn_batch(x, B, wg, wu, wd, d, F, mode, t, norm_eps, resid, y, active_idx,
                            active_cnt, ws, batch_layout(B, d, F, batch_px(B, mode)), s);
  if (mode == kFfnModeDense && B >= kMfmaMinBatch)
    return launch_ffn_mfma(x, B, wg, wu, wd, d, F, norm_eps, resid, y, ws, mfma_layout(B, d, F), s);
  const GemvLayout L = gemv_layout(B, d, F);
  for (int b0 = 0; b0 < B; b0 += L.bc) {
    const int nb = std::min(L.bc, B - b0);
    hipError_t e = launch_ffn_gemv(
        x + (size_t)b0 * d, nb, wg, wu, wd, d, F, mode, t, norm_eps,
        resid ? resid + (size_t)b0 * d : nullptr, y + (size_t)b0 * d,
        active_idx ? active_idx + (size_t)b0 * F : nullptr, active_cnt ? active_cnt + b0 : nullptr,
        ws, L, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace sirius

namespace {

size_t gemv_ws(int B, int d, int F) { return sirius::ffn_any_ws(B, d, F, sirius::kFfnModeThreshold); }
size_t ffn_ws(int B, int d, int F) { return sirius::ffn_any_ws(B, d, F, sirius::kFfnModeDense); }

int run_ffn_gemv(const char* fn, const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                 const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                 const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt, void* ws,
                 hipStream_t s) {
  return hip_status(sirius::launch_ffn_any(x, B, wg, wu, wd, d, F, mode, t, norm_eps, resid, y,
                                           active_idx, active_cnt, static_cast<char*>(ws), s),
                    fn);
}

int ffn_dense_impl(const char* fn, const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                   const uint16_t* wd, int d, int F, float norm_eps, const float* resid, float* y,
                   void* ws, size_t ws_bytes, void* stream) {
  int rc = check_ffn_dims(fn, B, d, F);
  if (rc) return rc;
  if ((rc = check_ptrs(fn, {{x, "x"}, {wg, "w_gate"}, {wu, "w_up"}, {wd, "w_down"}, {y, "y"}, {ws, "ws"}})))
    return rc;
  if (resid != nullptr && !aligned16(resid)) return fail(SIRIUS_EINVAL, "%s: resid is not 16-byte aligned", fn);
  if (std::isnan(norm_eps)) return fail(SIRIUS_EINVAL, "%s: norm_eps is NaN", fn);
  if (B == 0) return SIRIUS_OK;
  const size_t need = ffn_ws(B, d, F);
  if (ws_bytes < need)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, need);
  return run_ffn_gemv(fn, x, B, wg, wu, wd, d, F, sirius::kFfnModeDense, 0.f, norm_eps, resid, y,
                      nullptr, nullptr, ws, static_cast<hipStream_t>(stream));
}

}  // namespace

namespace sirius {
void set_last_error(const char* msg) { g_last_error = msg; }

int ffn_cats_validate(const char* fn, const float* x, int B, const uint16_t* w_gate,
                      const uint16_t* w_up, const uint16_t* w_down, int d_model, int d_ff, float t,
                      float norm_eps, const float* resid, const float* y,
                      const int32_t* active_idx, const int32_t* active_cnt, size_t* need) {
  int rc = check_ffn_dims(fn, B, d_model, d_ff);
  if (rc) return rc;
  if ((rc = check_ptrs(fn, {{x, "x"}, {w_gate, "w_gate"}, {w_up, "w_up"}, {w_down, "w_down"}, {y, "y"}})))
    return rc;
  if (resid != nullptr && !aligned16(resid)) return fail(SIRIUS_EINVAL, "%s: resid is not 16-byte aligned", fn);
  if ((active_idx == nullptr) != (active_cnt == nullptr))
    return fail(SIRIUS_EINVAL, "%s: active_idx and active_cnt must both be given or both be NULL", fn);
  if (std::isnan(t)) return fail(SIRIUS_EINVAL, "%s: threshold t is NaN", fn);
  if (std::isnan(norm_eps)) return fail(SIRIUS_EINVAL, "%s: norm_eps is NaN", fn);
  *need = B == 0 ? 0 : gemv_ws(B, d_model, d_ff);
  return SIRIUS_OK;
}

int ffn_cats_run(const char* fn, const float* x, int B, const uint16_t* w_gate, const uint16_t* w_up,
                 const uint16_t* w_down, int d_model, int d_ff, float t, float norm_eps,
                 const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt, void* ws,
                 void* stream) {
  return run_ffn_gemv(fn, x, B, w_gate, w_up, w_down, d_model, d_ff, kFfnModeThreshold, t, norm_eps,
                      resid, y, active_idx, active_cnt, ws, static_cast<hipStream_t>(stream));
}
}  // namespace sirius

extern "C" {

const char* sirius_last_error(void) { return g_last_error.c_str(); }

const char* sirius_version(void) { return "sirius-mi355x 0.1 (gfx950)"; }

size_t sirius_workspace_size(int op, int B, int d_model, int d_ff, int T_or_V, int K_or_R) {
  switch (op) {
    case SIRIUS_OP_FFN_DENSE:
    case SIRIUS_OP_FFN_CONDENSED:
      if (B < 0 || B > kMaxBatch || !dims_ok(d_model, d_ff)) return 0;
      return ffn_ws(B, d_model, d_ff);
    case SIRIUS_OP_FFN_CATS:
      if (B < 0 || B > kMaxBatch || !dims_ok(d_model, d_ff)) return 0;
      return gemv_ws(B, d_model, d_ff);
    case SIRIUS_OP_CATS_CALIBRATE:
      if (B < 1 || !dims_ok(d_model, d_ff)) return 0;
      return (((size_t)B * d_ff * sizeof(float) + 255) & ~size_t(255)) + sirius::select_ws_bytes();
    case SIRIUS_OP_GRIFFIN_SELECT:
      if (T_or_V < 1 || !dims_ok(d_model, d_ff)) return 0;
      return sirius::griffin_layout(T_or_V, d_model, d_ff).total;
    case SIRIUS_OP_VERIFY:
      if (B < 0 || T_or_V < 1 || K_or_R < 1 || K_or_R > kMaxVerifyRows) return 0;
      return sirius::verify_layout(std::max(B, 1), K_or_R, T_or_V).total;
    case SIRIUS_OP_FFN_TOPK:
      if (B < 0 || B > kMaxBatch || !dims_ok(d_model, d_ff)) return 0;
      return sirius::topk_layout(std::max(B, 1), d_model, d_ff).total;
    case SIRIUS_OP_ATTN_KV: {
      // B, n, H, Hkv, head_dim (d_model) ... packed: B, d_model = n, d_ff = H * 65536 + Hkv,
      // T_or_V = head_dim, K_or_R = Lmax
      const int H = d_ff >> 16, Hkv = d_ff & 0xffff;
      if (B < 0 || d_model < 1 || H < 1 || Hkv < 1 || H % Hkv != 0 || T_or_V < 8 ||
          T_or_V > 128 || T_or_V % 8 != 0 || K_or_R < d_model)
        return 0;
      return sirius::attn_layout(std::max(B, 1), d_model, H, Hkv, T_or_V, K_or_R).total;
    }
    case SIRIUS_OP_TREE_BUILD:
      if (B < 0 || d_model < 1 || d_model > kMaxTreeBuildW || d_ff < 1 || d_ff > kMaxTreeBuildW ||
          T_or_V < 1 || (long)d_model * T_or_V < d_ff)
        return 0;
      return sirius::tree_build_layout(std::max(B, 1), d_model, d_ff, T_or_V).total;
    case SIRIUS_OP_TREE_VERIFY: {
      if (B < 0 || d_model < 1 || d_ff < 1 || d_ff > kMaxTreeVerifyW || T_or_V < 1) return 0;
      const long R = (long)d_model * d_ff + (K_or_R ? d_ff : 0);
      if (R > kMaxVerifyRows) return 0;
      return sirius::verify_layout(std::max(B, 1), (int)R, T_or_V).total;
    }
    default:
      return 0;
  }
}

int sirius_ffn_dense(const float* x, int B, const uint16_t* w_gate, const uint16_t* w_up,
                     const uint16_t* w_down, int d_model, int d_ff, float norm_eps,
                     const float* resid, float* y, void* ws, size_t ws_bytes, void* stream) {
  return ffn_dense_impl("sirius_ffn_dense", x, B, w_gate, w_up, w_down, d_model, d_ff, norm_eps,
                        resid, y, ws, ws_bytes, stream);
}

int sirius_ffn_condensed(const float* x, int B, const uint16_t* w_gate_c, const uint16_t* w_up_c,
                         const uint16_t* w_down_c, int d_model, int k, float norm_eps,
                         const float* resid, float* y, void* ws, size_t ws_bytes, void* stream) {
  return ffn_dense_impl("sirius_ffn_condensed", x, B, w_gate_c, w_up_c, w_down_c, d_model, k,
                        norm_eps, resid, y, ws, ws_bytes, stream);
}

int sirius_ffn_cats(const float* x, int B, const uint16_t* w_gate, const uint16_t* w_up,
                    const uint16_t* w_down, int d_model, int d_ff, float t, float norm_eps,
                    const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                    void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sirius_ffn_cats";
  size_t need = 0;
  int rc = sirius::ffn_cats_validate(fn, x, B, w_gate, w_up, w_down, d_model, d_ff, t, norm_eps,
                                     resid, y, active_idx, active_cnt, &need);
  if (rc) return rc;
  if (ws == nullptr) return fail(SIRIUS_EINVAL, "%s: ws is NULL", fn);
  if (!aligned16(ws)) return fail(SIRIUS_EINVAL, "%s: ws is not 16-byte aligned", fn);
  if (B == 0) return SIRIUS_OK;
  if (ws_bytes < need)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, need);
  return sirius::ffn_cats_run(fn, x, B, w_gate, w_up, w_down, d_model, d_ff, t, norm_eps, resid, y,
                              active_idx, active_cnt, ws, stream);
}

int sirius_ffn_topk(const float* x, int B, const uint16_t* w_gate, const uint16_t* w_up,
                    const uint16_t* w_down, int d_model, int d_ff, int k, float norm_eps,
                    const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                    void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sirius_ffn_topk";
  int rc = check_ffn_dims(fn, B, d_model, d_ff);
  if (rc) return rc;
  if ((rc = check_ptrs(fn, {{x, "x"}, {w_gate, "w_gate"}, {w_up, "w_up"}, {w_down, "w_down"}, {y, "y"}, {ws, "ws"}})))
    return rc;
  if (resid != nullptr && !aligned16(resid)) return fail(SIRIUS_EINVAL, "%s: resid is not 16-byte aligned", fn);
  if ((active_idx == nullptr) != (active_cnt == nullptr))
    return fail(SIRIUS_EINVAL, "%s: active_idx and active_cnt must both be given or both be NULL", fn);
  if (k < 1 || k > d_ff) return fail(SIRIUS_EINVAL, "%s: k=%d outside [1, d_ff=%d]", fn, k, d_ff);
  if (std::isnan(norm_eps)) return fail(SIRIUS_EINVAL, "%s: norm_eps is NaN", fn);
  if (B == 0) return SIRIUS_OK;
  const sirius::TopkLayout L = sirius::topk_layout(B, d_model, d_ff);
  if (ws_bytes < L.total)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, L.total);
  return hip_status(sirius::launch_ffn_topk(x, B, w_gate, w_up, w_down, d_model, d_ff, k, norm_eps,
                                            resid, y, active_idx, active_cnt,
                                            static_cast<char*>(ws), L,
                                            static_cast<hipStream_t>(stream)),
                    fn);
}

int sirius_cats_calibrate(const float* x_cal, int N, const uint16_t* w_gate, int d_model, int d_ff,
                          double q, float* t_out, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sirius_cats_calibrate";
  if (N < 1) return fail(SIRIUS_EINVAL, "%s: N=%d must be >= 1", fn, N);
  int rc = check_ffn_dims(fn, 1, d_model, d_ff);
  if (rc) return rc;
  if ((rc = check_ptrs(fn, {{x_cal, "x_cal"}, {w_gate, "w_gate"}, {ws, "ws"}}))) return rc;
  if (t_out == nullptr) return fail(SIRIUS_EINVAL, "%s: t_out is NULL", fn);
  if (!(q > 0.0 && q <= 1.0)) return fail(SIRIUS_EINVAL, "%s: q=%g outside (0, 1]", fn, q);
  const size_t M = (size_t)N * d_ff;
  if (M > (size_t)INT32_MAX) return fail(SIRIUS_EINVAL, "%s: N*d_ff too large", fn);
  const size_t need = sirius_workspace_size(SIRIUS_OP_CATS_CALIBRATE, N, d_model, d_ff, 0, 0);
  if (ws_bytes < need)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, need);
  // nearest rank r = ceil(q*M) (1-based, ascending) == the (M - r + 1)-th largest
  long long r = (long long)std::ceil(q * (double)M);
  r = std::min<long long>(std::max<long long>(r, 1), (long long)M);
  const int k = (int)((long long)M - r + 1);
  hipStream_t s = static_cast<hipStream_t>(stream);
  float* absact = static_cast<float*>(ws);
  char* sel_ws = static_cast<char*>(ws) + ((M * sizeof(float) + 255) & ~size_t(255));
  hipError_t e = sirius::launch_gate_absact(x_cal, N, w_gate, d_model, d_ff, absact, s);
  if (e != hipSuccess) return hip_status(e, fn);
  return hip_status(sirius::launch_select_kth_largest(absact, (int)M, k, t_out, sel_ws, s), fn);
}

int sirius_griffin_select(const uint16_t* x_prompt, int T, const uint16_t* w_gate,
                          const uint16_t* w_up, const uint16_t* w_down, int d_model, int d_ff,
                          int k, int normalize_tokens, int32_t* sel_idx, float* scores,
                          uint16_t* w_gate_c, uint16_t* w_up_c, uint16_t* w_down_c, void* ws,
                          size_t ws_bytes, void* stream) {
  const char* fn = "sirius_griffin_select";
  if (T < 1) return fail(SIRIUS_EINVAL, "%s: T=%d must be >= 1", fn, T);
  int rc = check_ffn_dims(fn, 1, d_model, d_ff);
  if (rc) return rc;
  if (k < 1 || k > d_ff) return fail(SIRIUS_EINVAL, "%s: k=%d outside [1, d_ff=%d]", fn, k, d_ff);
  if ((rc = check_ptrs(fn, {{x_prompt, "x_prompt"}, {w_gate, "w_gate"}, {w_up, "w_up"}, {w_down, "w_down"},
                            {sel_idx, "sel_idx"}, {w_gate_c, "w_gate_c"}, {w_up_c, "w_up_c"},
                            {w_down_c, "w_down_c"}, {ws, "ws"}})))
    return rc;
  if ((size_t)T * d_ff > (size_t)INT32_MAX) return fail(SIRIUS_EINVAL, "%s: T*d_ff too large", fn);
  const sirius::GriffinLayout L = sirius::griffin_layout(T, d_model, d_ff);
  if (ws_bytes < L.total)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, L.total);
  return hip_status(sirius::launch_griffin(x_prompt, T, w_gate, w_up, w_down, d_model, d_ff, k,
                                           normalize_tokens ? 1 : 0, sel_idx, scores, w_gate_c,
                                           w_up_c, w_down_c, static_cast<char*>(ws), L,
                                           static_cast<hipStream_t>(stream)),
                    fn);
}

int sirius_verify_accept(const float* logits, int B, int K, int R, int V, const int32_t* drafted,
                         float r, float temperature, int32_t* accept_len, int32_t* next_token,
                         float* p_draft, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sirius_verify_accept";
  if (B < 0) return fail(SIRIUS_EINVAL, "%s: B=%d < 0", fn, B);
  if (K < 1) return fail(SIRIUS_EINVAL, "%s: K=%d must be >= 1", fn, K);
  if (R != K && R != K + 1) return fail(SIRIUS_EINVAL, "%s: R=%d must be K or K+1 (K=%d)", fn, R, K);
  if (R > kMaxVerifyRows) return fail(SIRIUS_EINVAL, "%s: R=%d above %d", fn, R, kMaxVerifyRows);
  if (V < 1) return fail(SIRIUS_EINVAL, "%s: V=%d must be >= 1", fn, V);
  if (std::isnan(r)) return fail(SIRIUS_EINVAL, "%s: r is NaN", fn);
  if (!(temperature > 0.f) || std::isinf(temperature))
    return fail(SIRIUS_EINVAL, "%s: temperature=%g must be finite and > 0", fn, (double)temperature);
  if (logits == nullptr || drafted == nullptr || accept_len == nullptr || next_token == nullptr || ws == nullptr)
    return fail(SIRIUS_EINVAL, "%s: a required pointer is NULL", fn);
  if (!aligned16(logits)) return fail(SIRIUS_EINVAL, "%s: logits is not 16-byte aligned", fn);
  if (B == 0) return SIRIUS_OK;
  if ((long)B * R > kMaxLogitRows)
    return fail(SIRIUS_EINVAL, "%s: B*R=%ld rows above %ld", fn, (long)B * R, kMaxLogitRows);
  if ((size_t)B * R * V > ((size_t)1 << 40)) return fail(SIRIUS_EINVAL, "%s: logits too large", fn);
  const sirius::VerifyLayout L = sirius::verify_layout(B, R, V);
  if (ws_bytes < L.total)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, L.total);
  return hip_status(sirius::launch_verify(logits, B, K, R, V, drafted, r, temperature, accept_len,
                                          next_token, p_draft, static_cast<char*>(ws), L,
                                          static_cast<hipStream_t>(stream)),
                    fn);
}

int sirius_tree_build_step(const float* logits, int B, int Wc, int V, const float* cum_ll, int W,
                           float temperature, int32_t* tokens, int32_t* parents,
                           float* cum_ll_out, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sirius_tree_build_step";
  if (B < 0) return fail(SIRIUS_EINVAL, "%s: B=%d < 0", fn, B);
  if (Wc < 1 || Wc > kMaxTreeBuildW)
    return fail(SIRIUS_EINVAL, "%s: Wc=%d outside [1, %d]", fn, Wc, kMaxTreeBuildW);
  if (W < 1 || W > kMaxTreeBuildW)
    return fail(SIRIUS_EINVAL, "%s: W=%d outside [1, %d]", fn, W, kMaxTreeBuildW);
  if (V < 1 || (long)Wc * V < W)
    return fail(SIRIUS_EINVAL, "%s: Wc*V=%ld candidates below W=%d", fn, (long)Wc * V, W);
  if (!(temperature > 0.f) || std::isinf(temperature))
    return fail(SIRIUS_EINVAL, "%s: temperature=%g must be finite and > 0", fn, (double)temperature);
  if (logits == nullptr || tokens == nullptr || parents == nullptr || cum_ll_out == nullptr ||
      ws == nullptr)
    return fail(SIRIUS_EINVAL, "%s: a required pointer is NULL", fn);
  if (cum_ll != nullptr && cum_ll == cum_ll_out)
    return fail(SIRIUS_EINVAL, "%s: cum_ll_out aliases cum_ll", fn);
  if (!aligned16(logits)) return fail(SIRIUS_EINVAL, "%s: logits is not 16-byte aligned", fn);
  if (B == 0) return SIRIUS_OK;
  if ((long)B * Wc > kMaxLogitRows)
    return fail(SIRIUS_EINVAL, "%s: B*Wc=%ld rows above %ld", fn, (long)B * Wc, kMaxLogitRows);
  if ((size_t)B * Wc * V > ((size_t)1 << 40)) return fail(SIRIUS_EINVAL, "%s: logits too large", fn);
  const sirius::TreeBuildLayout L = sirius::tree_build_layout(B, Wc, W, V);
  if (ws_bytes < L.total)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, L.total);
  return hip_status(sirius::launch_tree_build(logits, B, Wc, V, cum_ll, W, temperature, tokens,
                                              parents, cum_ll_out, static_cast<char*>(ws), L,
                                              static_cast<hipStream_t>(stream)),
                    fn);
}

int sirius_tree_verify(const float* logits, int B, int K, int W, int V, int bonus,
                       const int32_t* tokens, const int32_t* parents, float r, float temperature,
                       int32_t* best_leaf, int32_t* accept_len, int32_t* next_token, float* q,
                       void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sirius_tree_verify";
  if (B < 0) return fail(SIRIUS_EINVAL, "%s: B=%d < 0", fn, B);
  if (K < 1) return fail(SIRIUS_EINVAL, "%s: K=%d must be >= 1", fn, K);
  if (W < 1 || W > kMaxTreeVerifyW)
    return fail(SIRIUS_EINVAL, "%s: W=%d outside [1, %d]", fn, W, kMaxTreeVerifyW);
  const long R = (long)K * W + (bonus ? W : 0);
  if (R > kMaxVerifyRows)
    return fail(SIRIUS_EINVAL, "%s: K*W%s = %ld rows above %d", fn, bonus ? "+W" : "", R,
                kMaxVerifyRows);
  if (V < 1) return fail(SIRIUS_EINVAL, "%s: V=%d must be >= 1", fn, V);
  if (std::isnan(r)) return fail(SIRIUS_EINVAL, "%s: r is NaN", fn);
  if (!(temperature > 0.f) || std::isinf(temperature))
    return fail(SIRIUS_EINVAL, "%s: temperature=%g must be finite and > 0", fn, (double)temperature);
  if (logits == nullptr || tokens == nullptr || parents == nullptr || best_leaf == nullptr ||
      accept_len == nullptr || next_token == nullptr || ws == nullptr)
    return fail(SIRIUS_EINVAL, "%s: a required pointer is NULL", fn);
  if (!aligned16(logits)) return fail(SIRIUS_EINVAL, "%s: logits is not 16-byte aligned", fn);
  if (B == 0) return SIRIUS_OK;
  if ((long)B * R > kMaxLogitRows)
    return fail(SIRIUS_EINVAL, "%s: B*R=%ld rows above %ld", fn, (long)B * R, kMaxLogitRows);
  if ((size_t)B * R * V > ((size_t)1 << 40)) return fail(SIRIUS_EINVAL, "%s: logits too large", fn);
  const sirius::VerifyLayout L = sirius::verify_layout(B, (int)R, V);
  if (ws_bytes < L.total)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, L.total);
  return hip_status(sirius::launch_tree_verify(logits, B, K, W, V, bonus ? 1 : 0, tokens, parents,
                                               r, temperature, best_leaf, accept_len, next_token, q,
                                               static_cast<char*>(ws), L,
                                               static_cast<hipStream_t>(stream)),
                    fn);
}

int sirius_attn_kv(const float* q, const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache,
                   uint16_t* v_cache, const int32_t* cache_pos, int B, int n, int H, int Hkv,
                   int head_dim, int Lmax, float* out, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sirius_attn_kv";
  if (B < 0 || B > kMaxLogitRows) return fail(SIRIUS_EINVAL, "%s: B=%d outside [0, %ld]", fn, B, kMaxLogitRows);
  if (n < 1 || n > kMaxAttnTokens) return fail(SIRIUS_EINVAL, "%s: n=%d outside [1, %d]", fn, n, kMaxAttnTokens);
  if (H < 1 || Hkv < 1 || H % Hkv != 0)
    return fail(SIRIUS_EINVAL, "%s: H=%d must be a positive multiple of Hkv=%d", fn, H, Hkv);
  if (head_dim < 8 || head_dim > 128 || head_dim % 8 != 0)
    return fail(SIRIUS_EINVAL, "%s: head_dim=%d must be a multiple of 8 in [8, 128]", fn, head_dim);
  if (Lmax < n || Lmax > kMaxCacheLen)
    return fail(SIRIUS_EINVAL, "%s: Lmax=%d outside [n, %d]", fn, Lmax, kMaxCacheLen);
  const long rows = (long)(H / Hkv) * n;
  if ((long)Hkv * ((rows + 63) / 64) > kMaxLogitRows)
    return fail(SIRIUS_EINVAL, "%s: too many query rows per call", fn);
  int rc;
  if ((rc = check_ptrs(fn, {{q, "q"}, {k_new, "k_new"}, {v_new, "v_new"}, {k_cache, "k_cache"},
                            {v_cache, "v_cache"}, {out, "out"}, {ws, "ws"}})))
    return rc;
  if (cache_pos == nullptr) return fail(SIRIUS_EINVAL, "%s: cache_pos is NULL", fn);
  if (B == 0) return SIRIUS_OK;
  const sirius::AttnLayout L = sirius::attn_layout(B, n, H, Hkv, head_dim, Lmax);
  if (ws_bytes < L.total)
    return fail(SIRIUS_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, L.total);
  return hip_status(sirius::launch_attn_kv(q, k_new, v_new, k_cache, v_cache, cache_pos, B, n, H,
                                           Hkv, head_dim, Lmax, out, static_cast<char*>(ws), L,
                                           static_cast<hipStream_t>(stream)),
                    fn);
}

int sirius_kv_rollback(int32_t* cache_pos, const int32_t* accept_len, int B, int n, void* stream) {
  const char* fn = "sirius_kv_rollback";
  if (cache_pos == nullptr || accept_len == nullptr) return fail(SIRIUS_EINVAL, "%s: NULL pointer", fn);
  if (B < 0 || n < 1) return fail(SIRIUS_EINVAL, "%s: bad sizes B=%d n=%d", fn, B, n);
  if (B == 0) return SIRIUS_OK;
  return hip_status(sirius::launch_kv_rollback(cache_pos, accept_len, B, n,
                                               static_cast<hipStream_t>(stream)),
                    fn);
}

int sirius_rmsnorm(const float* h, int B, int d_model, float eps, float* out, void* stream) {
  const char* fn = "sirius_rmsnorm";
  if (h == nullptr || out == nullptr) return fail(SIRIUS_EINVAL, "%s: NULL pointer", fn);
  if (B < 0 || d_model < 1) return fail(SIRIUS_EINVAL, "%s: bad sizes B=%d d_model=%d", fn, B, d_model);
  if (!(eps >= 0.f)) return fail(SIRIUS_EINVAL, "%s: eps must be >= 0", fn);
  if (B == 0) return SIRIUS_OK;
  return hip_status(sirius::launch_rmsnorm(h, B, d_model, eps, out, static_cast<hipStream_t>(stream)), fn);
}

int sirius_fill_normal_bf16(uint16_t* out, size_t n, uint64_t seed, float mean, float std,
                            void* stream) {
  const char* fn = "sirius_fill_normal_bf16";
  if (out == nullptr) return fail(SIRIUS_EINVAL, "%s: out is NULL", fn);
  if (!(std >= 0.f) || std::isinf(std) || !std::isfinite(mean))
    return fail(SIRIUS_EINVAL, "%s: need finite mean and std >= 0", fn);
  if (n == 0) return SIRIUS_OK;
  return hip_status(sirius::launch_fill_normal_bf16(out, n, seed, mean, std, static_cast<hipStream_t>(stream)), fn);
}

}  // extern "C"
