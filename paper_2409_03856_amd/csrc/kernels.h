// Internal launchers of libsirius (not part of the C ABI). Every launcher
// only enqueues kernels on `stream`; the C-ABI layer validates arguments
// before calling any of them.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sirius {

// The calling thread's message for sirius_last_error (the C-ABI files set it on failure).
void set_last_error(const char* msg);

// sirius_ffn_cats in two halves, shared by the entry points that differ only in where the
// workspace comes from. ffn_cats_validate checks every argument but the workspace (and sets the
// error message on failure) and stores the workspace bytes the call needs in *need (0 for an
// empty batch); ffn_cats_run enqueues the call on a workspace of at least that size.
int ffn_cats_validate(const char* fn, const float* x, int B, const uint16_t* w_gate,
                      const uint16_t* w_up, const uint16_t* w_down, int d_model, int d_ff, float t,
                      float norm_eps, const float* resid, const float* y,
                      const int32_t* active_idx, const int32_t* active_cnt, size_t* need);
int ffn_cats_run(const char* fn, const float* x, int B, const uint16_t* w_gate, const uint16_t* w_up,
                 const uint16_t* w_down, int d_model, int d_ff, float t, float norm_eps,
                 const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt, void* ws,
                 void* stream);

// FFN selection modes of the small-batch and batch-1 launchers
constexpr int kFfnModeDense = 0;      // every neuron (dense and condensed)
constexpr int kFfnModeThreshold = 1;  // |SiLU(gate)| > t per token
constexpr int kFfnModeTopK = 2;       // the top-k key cut per token (stored activations)

// ---- small-batch FFN (gate GEMV + SiLU + threshold + compaction, sparse down, reduce)
struct GemvLayout {
  int bc;       // batch rows handled per pass (x staged in LDS needs bc*d*4 <= 64 KiB)
  int ntiles;   // gate row segments (one per gate workgroup)
  int rmax;     // rows per segment at most
  int cs, gr;   // down-projection grid: 512-column slices x row ranges
  size_t uidx, h, ucnt, bidx, bcnt, part, total;  // workspace byte offsets / size
};
GemvLayout gemv_layout(int B, int d, int F);

// mode: kFfnMode*. x/y/resid/active_* (and act [B][F], cut [B] for top-k) already offset
// to the chunk; B <= layout.bc.
hipError_t launch_ffn_gemv(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                           const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                           char* ws, const GemvLayout& L, hipStream_t stream,
                           const float* act = nullptr, const unsigned long long* cut = nullptr);

// Signed gate activations SiLU(W_gate xn) for N inputs into act [N, F] (top-k first pass);
// xn = RMSNorm(x) when norm_eps >= 0.
hipError_t launch_gate_act(const float* x, int N, const uint16_t* wg, int d, int F,
                           float norm_eps, float* act, hipStream_t stream);

// Gate activations |SiLU(W_gate x)| for N inputs into absact [N, F] (calibration).
hipError_t launch_gate_absact(const float* x, int N, const uint16_t* wg, int d, int F,
                              float* absact, hipStream_t stream);

// Row-split down projection over compacted neuron lists: nseg segments of up to rmax rows
// (uidx[seg*rmax + k], count ucnt[seg]), h values at hbuf[slot*hstride + b] for b < B <= 16,
// partial sums into part[gr][B][d].
hipError_t launch_down(int B, int d, int nseg, int rmax, int gr, const uint16_t* wd,
                       const int32_t* uidx, const float* hbuf, int hstride, const int32_t* ucnt,
                       float* part, hipStream_t stream);
// y[b] = sum_r part[r][b] (+ resid[b]) in a fixed order. With active_idx, B * 16 more
// workgroups concatenate token b's per-segment lists bidx[b][seg][0 .. bcnt[b][seg]) (nseg
// segments of rmax slots, nseg <= 2048) into active_idx[b][*] and write active_cnt[b].
hipError_t launch_reduce(const float* part, int gr, int B, int d, const float* resid, float* y,
                         hipStream_t stream, int F = 0, int nseg = 0, int rmax = 0,
                         const int32_t* bidx = nullptr, const int32_t* bcnt = nullptr,
                         int32_t* active_idx = nullptr, int32_t* active_cnt = nullptr);

// ---- batch-1 decode: gate, threshold, compaction, kept up rows and kept down rows of one
// row segment per 1024-thread workgroup, then launch_reduce over the segment partials
struct Decode1Layout {
  int nseg, rmax;
  size_t uidx, ucnt, part, total;
};
// Batch-1 gate pass of per-token top-k: the signed activations SiLU(W_gate x) of one token
// (x RMS-normalised when norm_eps >= 0) into act [F], by the decode kernel's gate phase.
hipError_t launch_decode1_act(const float* x, const uint16_t* wg, int d, int F, float norm_eps,
                              float* act, hipStream_t stream);
Decode1Layout decode1_layout(int d, int F);
hipError_t launch_ffn_decode1(const float* x, const uint16_t* wg, const uint16_t* wu,
                              const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                              const float* resid, float* y, int32_t* active_idx,
                              int32_t* active_cnt, char* ws, const Decode1Layout& L,
                              hipStream_t stream, const float* act = nullptr,
                              const unsigned long long* cut = nullptr);

// ---- per-token top-k FSparse: gate pass, key cut per token, then the keyed FFN pass
struct TopkLayout {
  size_t act, cut, ffn, total;  // act [B][F] fp32, cut [B] u64, then the FFN workspace
};
TopkLayout topk_layout(int B, int d, int F);
hipError_t launch_ffn_topk(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, int d, int F, int k, float norm_eps,
                           const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                           char* ws, const TopkLayout& L, hipStream_t stream);

// ---- multi-token FFN on MFMA (B >= kMfmaMinBatch)
constexpr int kMfmaMinBatch = 8;
struct MfmaLayout {
  int mpad;          // batch padded to the MFMA M tile
  int ntiles, f16;   // neuron tiles of 16, d_ff rounded up to 16
  int cs, gr;        // down grid: 64-column tiles x neuron ranges
  int nchunk;        // 64-neuron chunks of the down product
  size_t xb, hhi, hlo, part, total;  // workspace byte offsets / size
};
MfmaLayout mfma_layout(int B, int d, int F);
hipError_t launch_ffn_mfma(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, int d, int F, float norm_eps, const float* resid,
                           float* y, char* ws, const MfmaLayout& L, hipStream_t stream);

// ---- batched FFN on MFMA rings (2 <= B <= 64, d_model % 256 == 0): dense / condensed with the
// input as px bf16 pieces (1: rounded to bf16; 3: exact fp32), per-token threshold or top-k
// sparsity (three pieces) reading up and down rows of the tokens' union only
struct BatchLayout {
  int mpad, px;      // tokens padded to whole 16-token tiles; input pieces
  int nseg, np;      // gate/up segments and neurons per segment (<= 56)
  int sp;            // positions per segment in the segment layout (16, 32 or 64)
  int hs;            // h row stride: nseg * sp rounded up to whole 64-position down blocks
  int nblocks, gr;   // 64-position down blocks and down ranges
  size_t xp, hhi, hlo, uidx, ucnt, bidx, bcnt, part, total;  // workspace offsets / size
};
bool batch_path_ok(int B, int d, int F);
// One FFN call of any batch (dense or threshold mode): the decode kernel at B = 1, the batched
// kernels above when the shape allows them, else the older MFMA (dense, B >= 8) or small-batch
// kernels. Shared by the C entry points and the model's forward pass.
size_t ffn_any_ws(int B, int d, int F, int mode);
hipError_t launch_ffn_any(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                          const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                          char* ws, hipStream_t s);
// sparse: the segment layout (per-segment union blocks), used by every call with px = 3
BatchLayout batch_layout(int B, int d, int F, int px);
// mode: kFfnMode*; with active_idx (sparse modes) the per-token kept lists are written; top-k
// takes the activations act [B][F] and the per-token cut keys (launch_cut).
hipError_t launch_ffn_batch(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                            const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                            const float* resid, float* y, int32_t* active_idx,
                            int32_t* active_cnt, char* ws, const BatchLayout& L,
                            hipStream_t stream, const float* act = nullptr,
                            const unsigned long long* cut = nullptr);
// Top-k gate pass of a batch: act [B][F] = SiLU(W_gate xn) from the exact (three-piece) input;
// L = batch_layout(B, d, F, 3, true).
hipError_t launch_batch_act(const float* x, int B, const uint16_t* wg, int d, int F,
                            float norm_eps, float* act, char* ws, const BatchLayout& L,
                            hipStream_t stream);

// ---- radix select of the k-th largest non-negative float (ties resolved by index)
hipError_t launch_select_kth_largest(const float* v, int n, int k, float* out_value,
                                     char* ws, hipStream_t stream);
size_t select_ws_bytes();

// ---- Griffin
struct GriffinLayout {
  size_t z, rownorm, part, scores, total;  // z is used by the normalised variant only
};
GriffinLayout griffin_layout(int T, int d, int F);
hipError_t launch_griffin(const uint16_t* xp, int T, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, int d, int F, int k, int normalize,
                          int32_t* sel, float* scores_out, uint16_t* wgc, uint16_t* wuc,
                          uint16_t* wdc, char* ws, const GriffinLayout& L, hipStream_t stream);

// ---- verify
struct VerifyLayout {
  int splits;
  size_t part, total;
};
VerifyLayout verify_layout(int B, int R, int V);
hipError_t launch_verify(const float* logits, int B, int K, int R, int V, const int32_t* drafted,
                         float r, float temperature, int32_t* accept_len, int32_t* next_token,
                         float* p_draft, char* ws, const VerifyLayout& L, hipStream_t stream);

// Tree verification: rows [b][i * W + w] (i < K) are the nodes of step i, then W bonus rows
// if bonus != 0; tokens/parents [B][K][W]; q [B][K][W] or null. Needs R = K * W (+ W) <= 1024
// and W <= 64; L = verify_layout(B, R, V).
hipError_t launch_tree_verify(const float* logits, int B, int K, int W, int V, int bonus,
                              const int32_t* tokens, const int32_t* parents, float r,
                              float temperature, int32_t* best_leaf, int32_t* accept_len,
                              int32_t* next_token, float* q, char* ws, const VerifyLayout& L,
                              hipStream_t stream);

// ---- tree drafting step: the W best (leaf, token) expansions of each of B trees
struct TreeBuildLayout {
  int splits;                // segments per leaf row
  size_t rm, rs, rk, total;  // workspace byte offsets / size
};
TreeBuildLayout tree_build_layout(int B, int Wc, int W, int V);
// logits [B][Wc][V] (16-byte aligned), cum_ll [B][Wc] or null (all 0); outputs [B][W].
// 1 <= Wc, W <= 16.
hipError_t launch_tree_build(const float* logits, int B, int Wc, int V, const float* cum_ll, int W,
                             float temperature, int32_t* tokens, int32_t* parents,
                             float* cum_out, char* ws, const TreeBuildLayout& L,
                             hipStream_t stream);

// ---- attention over the shared KV cache with the direct rewrite, and the rollback
struct AttnLayout {
  int rgroups, chunk, nsplit;    // query-row groups per kv head, positions per chunk, chunks
  size_t pm, pl, po, total;      // per-chunk partials: max, sum, output
};
AttnLayout attn_layout(int B, int n, int H, int Hkv, int hd, int Lmax);
// q [B][n][H][hd] fp32; k_new, v_new [B][n][Hkv][hd] bf16; caches [B][Lmax][Hkv][hd] bf16;
// cache_pos [B] on the device; out [B][n][H][hd]. hd % 8 == 0, hd <= 128, H % Hkv == 0.
hipError_t launch_attn_kv(const float* q, const uint16_t* k_new, const uint16_t* v_new,
                          uint16_t* k_cache, uint16_t* v_cache, const int32_t* cache_pos, int B,
                          int n, int H, int Hkv, int hd, int Lmax, float* out, char* ws,
                          const AttnLayout& L, hipStream_t stream);
hipError_t launch_kv_rollback(int32_t* cache_pos, const int32_t* accept_len, int B, int n,
                              hipStream_t stream);

// ---- small decoder and the generation loop (model.hip)
// h[i] = E[tokens[i]] widened to fp32 (0 for an id outside [0, V)); d % 8 == 0.
hipError_t launch_embed(const int32_t* tokens, int n, const uint16_t* E, int d, int V, float* out,
                        hipStream_t s);
// y[i][j] = x[i] . W[j] (+ resid[i][j]) for i < n, j < N; W [N][K] bf16; K % 8 == 0 and
// K <= 16384. With y_bf16 the rows are written as bf16 instead (resid and y unused).
// RMSNorm (unit weight, bit for bit rmsnorm_vec_kernel's result) of n rows of x [n][K] as they
// are staged, then q = xn Wq^T [n][Nq] fp32 and, for Nkv > 0, k = xn Wk^T, v = xn Wv^T [n][Nkv]
// bf16 in one launch per 16 rows. K % 8 == 0, K <= 8192, 16-byte aligned rows.
hipError_t launch_norm_qkv(const float* x, int n, int K, float eps, const uint16_t* Wq, int Nq,
                           const uint16_t* Wk, const uint16_t* Wv, int Nkv, float* yq,
                           uint16_t* yk, uint16_t* yv, hipStream_t s);
hipError_t launch_linear(const float* x, int n, const uint16_t* W, int K, int N,
                         const float* resid, float* y, uint16_t* y_bf16, hipStream_t s);
// seq[slot] = argmax of the V logits (lowest index on ties); cache_pos[0] += pos_delta;
// trace_drafted[slot - 1] = the token when given.
hipError_t launch_draft_tail(const float* logits, int V, int32_t* seq, int slot,
                             int32_t* cache_pos, int pos_delta, int32_t* trace_drafted,
                             hipStream_t s);
// After the check of an n-token chunk seq[0 .. n - 1] (drafts seq[1 .. n]): cache_pos +=
// min(j + 1, n); out[count ..] += seq[1 .. j] and the corrected token when j < n (at most
// out_cap entries in all); seq[0] = the next period's first input.
hipError_t launch_period_tail(int32_t* seq, int n, const int32_t* accept_len,
                              const int32_t* next_token, int32_t* cache_pos, int32_t* out,
                              int32_t* out_count, int out_cap, int32_t* tr_accept,
                              int32_t* tr_next, hipStream_t s);

// ---- glue
hipError_t launch_rmsnorm(const float* h, int B, int d, float eps, float* out, hipStream_t stream);
hipError_t launch_fill_normal_bf16(uint16_t* out, size_t n, uint64_t seed, float mean, float std,
                                   hipStream_t stream);

}  // namespace sirius
