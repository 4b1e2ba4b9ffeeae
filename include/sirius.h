/*
 * sirius.h -- C ABI of the MI355X (gfx950) library for the hot path of
 * Sirius, "Contextual Sparsity with Correction for Efficient LLMs"
 * (arXiv 2409.03856).
 *
 * The path has two halves:
 *   1. the contextual-sparse SwiGLU FFN decode step the sparse model runs on
 *      every token (Sec. 2.1: fine-grained per-token sparsity, FSparse, after
 *      CATS; coarse-grained prompt-fixed sparsity, CSparse, after Griffin);
 *   2. the full model's correction check of a chunk of drafted tokens
 *      (Algorithm 1; Sec. 4 "How to correct"): likelihood of each drafted
 *      token, first rejection below a threshold, the full model's own token
 *      at that position.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensor arguments are DEVICE pointers owned by the caller, contiguous,
 *    row-major. The library never frees or retains them.
 *  - Weights are bfloat16 passed as uint16_t bit patterns. All three FFN
 *    matrices are NEURON-MAJOR [d_ff, d_model]: row i of W_gate and W_up are
 *    neuron i's input weights, row i of W_down its output weights. Rows
 *    must be 16-byte aligned (d_model % 8 == 0 and 16-byte aligned bases).
 *  - Activations x, y, residuals are fp32 [B, d_model]. Accumulation is fp32.
 *  - `stream` is a hipStream_t (NULL = the default stream). Every call only
 *    enqueues work on that stream and returns; nothing synchronizes.
 *  - `ws` is a caller-owned device workspace of at least
 *    sirius_workspace_size(op, ...) bytes, 256-byte aligned. Its contents on
 *    entry are ignored; calls that share one workspace must be ordered on
 *    one stream.
 *  - Return value: SIRIUS_OK (0) on success, else a negative code. Arguments
 *    are validated on the host BEFORE anything is enqueued, so a failing
 *    call has launched nothing. sirius_last_error() returns a message for
 *    the calling thread's most recent failure.
 *  - B == 0 (empty batch) is a valid no-op that returns SIRIUS_OK.
 *  - Limits of this library: 8 <= d_model <= 8192, 1 <= d_ff <= 65536,
 *    B <= 64 for the FFN entry points.
 */
#ifndef SIRIUS_H
#define SIRIUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SIRIUS_OK 0
#define SIRIUS_EINVAL (-1)    /* null pointer, bad size, bad scalar */
#define SIRIUS_EWORKSPACE (-2) /* ws_bytes smaller than sirius_workspace_size() */
#define SIRIUS_EHIP (-3)      /* the HIP runtime refused a launch */

/* Operation codes for sirius_workspace_size(). */
#define SIRIUS_OP_FFN_DENSE 0
#define SIRIUS_OP_FFN_CATS 1
#define SIRIUS_OP_GRIFFIN_SELECT 2
#define SIRIUS_OP_FFN_CONDENSED 3
#define SIRIUS_OP_VERIFY 4
#define SIRIUS_OP_CATS_CALIBRATE 5
#define SIRIUS_OP_TREE_BUILD 6
#define SIRIUS_OP_TREE_VERIFY 7
#define SIRIUS_OP_FFN_TOPK 8
#define SIRIUS_OP_ATTN_KV 9

/*
 * Dense SwiGLU FFN (the full model, sparsity 0):
 *   y[b] = resid[b] + sum_i SiLU(W_gate[i].xn[b]) * (W_up[i].xn[b]) * W_down[i]
 * where xn = RMSNorm(x) with unit weight when norm_eps >= 0, else xn = x.
 * The FFN form is the Llama SwiGLU MLP the paper sparsifies (Sec. 2.1);
 * the full model's parallel pass over a drafted chunk (Algorithm 1, Sec.
 * 2.2) is this call with B = chunk length.
 *   x      [B, d_model] fp32 input (read only).
 *   resid  [B, d_model] fp32 added to the output, or NULL. May alias y.
 *   y      [B, d_model] fp32 output. May alias resid, must not alias x
 *          unless resid == x == y (in-place residual layer).
 * Precision by batch: B = 1 keeps xn and h in fp32 (bf16 weights times
 * fp32 values, fp32 sums). For 2 <= B <= 64 with d_model % 256 == 0, and
 * for B >= 8 at other shapes, both products run on MFMA and accumulate in
 * fp32; the down product takes h as a pair of bf16 values (hi = bf16(h),
 * lo = bf16(h - hi): about 16 significant bits). The gate and up products
 * take xn rounded to bf16 when B >= 8, and for B < 8 xn split exactly into
 * three bf16 pieces (hi + mid + lo = xn), so their products equal the fp32
 * ones. At d_model % 256 != 0, B < 8 keeps xn and h in fp32.
 * Errors: SIRIUS_EINVAL for null pointers (resid may be NULL), d_model not
 * a multiple of 8 or outside [8, 8192], d_ff < 1, B < 0 or B > 64.
 */
int sirius_ffn_dense(const float* x, int B, const uint16_t* w_gate, const uint16_t* w_up,
                     const uint16_t* w_down, int d_model, int d_ff, float norm_eps,
                     const float* resid, float* y, void* ws, size_t ws_bytes, void* stream);

/*
 * Fine-grained (per-token) contextual sparsity, FSparse after CATS
 * (Sec. 2.1; Sec. 3 FSparse description: the gate stays dense, up and down
 * are sparse). For each token b:
 *   a_bi = SiLU(W_gate[i].xn[b]);  A_b = { i : |a_bi| > t }  (strict;
 *   t < 0 keeps every neuron, t = +inf none)
 *   y[b] = resid[b] + sum_{i in A_b} a_bi * (W_up[i].xn[b]) * W_down[i]
 * Only rows of W_up and W_down in the union of the A_b are read.
 *   active_idx [B, d_ff] int32 out: A_b in ascending order in
 *              active_idx[b*d_ff .. b*d_ff + active_cnt[b]); the rest of the
 *              row is left untouched. May be NULL together with active_cnt.
 *   active_cnt [B] int32 out: |A_b|.
 * The gate dot products, SiLU and the comparison are fp32 from the fp32
 * input (x is never rounded to bf16 here), for every B; so are the up
 * products. For 2 <= B <= 64 with d_model % 256 == 0 the down product
 * takes h as a bf16 hi/lo pair, as in sirius_ffn_dense; B = 1 and other
 * shapes keep h in fp32.
 * Errors: as sirius_ffn_dense, plus SIRIUS_EINVAL for NaN t or for exactly
 * one of active_idx / active_cnt being NULL.
 */
int sirius_ffn_cats(const float* x, int B, const uint16_t* w_gate, const uint16_t* w_up,
                    const uint16_t* w_down, int d_model, int d_ff, float t, float norm_eps,
                    const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * sirius_ffn_cats without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc). Same
 * arguments, semantics and results as sirius_ffn_cats (bit for bit: the same kernels run); the
 * workspace is a fixed device array of SIRIUS_NOALLOC_SCRATCH_BYTES that the library holds on
 * every GPU it runs on until the process ends. The call allocates nothing: no hipMalloc, no
 * hipFree, no events (per-kernel timing is not recorded for it).
 * All calls on one GPU share that GPU's array: calls that overlap on one GPU (from two streams
 * or two threads) race and must be ordered by the caller. The array's contents carry over from
 * call to call; the kernels read only what the same call wrote.
 * Errors: as sirius_ffn_cats, plus SIRIUS_EWORKSPACE when the call would need more than
 * SIRIUS_NOALLOC_SCRATCH_BYTES, 96 MiB (sirius_workspace_size(SIRIUS_OP_FFN_CATS, ...) tells;
 * every batch up to 64 at the Llama-3-8B FFN shape, 4096 x 14336, and at the 70B shape,
 * 8192 x 28672, fits), SIRIUS_EHIP when the array's device address cannot be obtained, and
 * SIRIUS_EINVAL for a device index of 64 or more.
 */
#define SIRIUS_NOALLOC_SCRATCH_BYTES ((size_t)96 << 20)
int sirius_ffn_cats_noalloc(const float* x, int B, const uint16_t* w_gate, const uint16_t* w_up,
                            const uint16_t* w_down, int d_model, int d_ff, float t, float norm_eps,
                            const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                            void* stream);

/*
 * Per-token top-k sparse FFN, the paper's own fine-grained (FSparse)
 * implementation (Sec. 3, footnote on the fine-grained implementation): in
 * place of CATS's threshold, every token keeps exactly the k neurons of
 * largest |SiLU(W_gate[i].xn)| (ties to the lower neuron index); the gate is
 * read whole, W_up and W_down only for the kept neurons:
 *   y[b] = resid[b] + sum_{i in A_b} SiLU(W_gate[i].xn[b]) (W_up[i].xn[b]) W_down[i]
 * with xn as for sirius_ffn_dense. The gate activations are computed in
 * fp32 (bf16 weights x fp32 inputs), the selection is taken on those values;
 * the up and down products have the precision of sirius_ffn_cats.
 *   x, resid, y   as for sirius_ffn_cats.
 *   active_idx    [B, d_ff] int32 out: row b starts with the ascending A_b
 *                 (k entries), or NULL (then active_cnt must be NULL too).
 *   active_cnt    [B] int32 out: k, or NULL.
 * Errors: as for sirius_ffn_cats, and SIRIUS_EINVAL for k outside [1, d_ff].
 */
int sirius_ffn_topk(const float* x, int B, const uint16_t* w_gate, const uint16_t* w_up,
                    const uint16_t* w_down, int d_model, int d_ff, int k, float norm_eps,
                    const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * Threshold calibration for sirius_ffn_cats: the nearest-rank q-quantile of
 * the pooled |SiLU(W_gate[i].x_cal[n])| over N calibration inputs and all
 * d_ff neurons (with the M = N*d_ff values sorted ascending, the value at
 * rank ceil(q*M)). Dropping values <= t then removes a fraction q on the
 * calibration set. The paper fixes FSparse sparsity levels (50% by
 * default, Sec. 3) without printing how CATS sets its threshold; this is
 * the plain quantile rule.
 *   x_cal [N, d_model] fp32; t_out: ONE float in device memory. q is a double
 *   so that ceil(q*M) is the exact nearest rank (a float q such as 0.4f
 *   would move the rank by one when q*M is an integer).
 * Errors: SIRIUS_EINVAL for null pointers, N < 1, q outside (0, 1].
 */
int sirius_cats_calibrate(const float* x_cal, int N, const uint16_t* w_gate, int d_model,
                          int d_ff, double q, float* t_out, void* ws, size_t ws_bytes,
                          void* stream);

/*
 * Coarse-grained (prompt-fixed) contextual sparsity, CSparse after Griffin
 * (Sec. 2.1; Appendix A.1): one neuron set per prompt, used for every
 * generated token, sparsifying the whole MLP including the gate.
 *   z_ti = SiLU(x_t.W_gate[i]) * (x_t.W_up[i])   over the T prompt tokens
 *   s_i  = sqrt(sum_t z_ti^2)                     (normalize_tokens = 0)
 *   s_i  = sqrt(sum_t (z_ti / ||z_t||)^2)          (normalize_tokens = 1)
 * keeps the k neurons of largest s (equal scores: lower index first) and
 * copies their rows of all three matrices into the condensed matrices.
 *   x_prompt [T, d_model] bf16 bits; products are exact and accumulate in
 *            fp32 on MFMA; z in fp32 with SiLU through the hardware exp2
 *            and reciprocal (each within about 1 ulp), squares summed in
 *            fp64.
 *   sel_idx  [k] int32 out, ascending.
 *   scores   [d_ff] fp32 out (s), or NULL.
 *   w_*_c    [k, d_model] bf16 out: row j = row sel_idx[j] of w_*.
 * Errors: SIRIUS_EINVAL for null pointers (scores may be NULL), T < 1,
 * k < 1 or k > d_ff, d_model/d_ff limits as above.
 */
int sirius_griffin_select(const uint16_t* x_prompt, int T, const uint16_t* w_gate,
                          const uint16_t* w_up, const uint16_t* w_down, int d_model, int d_ff,
                          int k, int normalize_tokens, int32_t* sel_idx, float* scores,
                          uint16_t* w_gate_c, uint16_t* w_up_c, uint16_t* w_down_c, void* ws,
                          size_t ws_bytes, void* stream);

/*
 * Decode with condensed weights (the CSparse model's FFN): the dense SwiGLU
 * FFN over the k selected neurons. Same arguments and rules as
 * sirius_ffn_dense with d_ff = k.
 */
int sirius_ffn_condensed(const float* x, int B, const uint16_t* w_gate_c, const uint16_t* w_up_c,
                         const uint16_t* w_down_c, int d_model, int k, float norm_eps,
                         const float* resid, float* y, void* ws, size_t ws_bytes, void* stream);

/*
 * Correction check of a drafted chunk (Algorithm 1; Sec. 4 "How to
 * correct"). Row j of logits is the full model's distribution at drafted
 * position j (the caller aligns rows to drafted tokens):
 *   q_bj = softmax(logits[b, j, :] / temperature)[drafted[b, j]]
 *          (0 when drafted[b, j] is outside [0, V))
 *   accept_len[b] = first j with q_bj < r (strict), else K
 *   next_token[b] = argmax_v logits[b, accept_len[b], v]  if accept_len < K
 *                 = argmax_v logits[b, K, v]              if all accepted and R == K+1
 *                 = -1                                    otherwise
 * Argmax is over the raw logits; ties go to the lowest index. The paper
 * samples the corrected token; the argmax is its deterministic form.
 *   logits  [B, R, V] fp32, R = K (no bonus row) or K + 1.
 *   drafted [B, K] int32.
 *   p_draft [B, K] fp32 out (q), or NULL.
 * Errors: SIRIUS_EINVAL for null pointers (p_draft may be NULL), K < 1,
 * V < 1, R not in {K, K+1}, B * R > 65535, NaN r, temperature not > 0.
 */
int sirius_verify_accept(const float* logits, int B, int K, int R, int V, const int32_t* drafted,
                         float r, float temperature, int32_t* accept_len, int32_t* next_token,
                         float* p_draft, void* ws, size_t ws_bytes, void* stream);

/*
 * One pruned expansion step of the drafted tree (Sec. 4, hardware-friendly
 * tree building): the sparse model drafts a tree that keeps W leaves per
 * step, ranked by the cumulative log-likelihood of their paths, so that the
 * tree has a fixed shape. For each of B trees, every (leaf w, token v) pair
 * is scored
 *   score = cum_ll[b, w] + log softmax(logits[b, w] / temperature)[v]
 * and the W largest are kept, best first; ties go to the lower leaf slot,
 * then the lower token id. The root step is Wc = 1 with cum_ll = NULL (0).
 *   logits     [B, Wc, V] fp32 (sparse-model logits at the current leaves),
 *              16-byte aligned.
 *   cum_ll     [B, Wc] fp32 cumulative log-likelihoods, or NULL (all 0).
 *   tokens     [B, W] int32 out: the new leaves' tokens.
 *   parents    [B, W] int32 out: their parent slots in [0, Wc).
 *   cum_ll_out [B, W] fp32 out: their scores. May not alias cum_ll.
 * Softmax sums accumulate in fp64, scores are formed in fp64 and stored as
 * fp32.
 * Errors: SIRIUS_EINVAL for null pointers (cum_ll may be NULL), B < 0,
 * Wc or W outside [1, 16], B * Wc > 65535, V < 1 or Wc * V < W,
 * temperature not finite and > 0.
 */
int sirius_tree_build_step(const float* logits, int B, int Wc, int V, const float* cum_ll, int W,
                           float temperature, int32_t* tokens, int32_t* parents,
                           float* cum_ll_out, void* ws, size_t ws_bytes, void* stream);

/*
 * Verification of B drafted trees of K steps and width W in one pass of the
 * full model (Sec. 4, hardware-friendly tree building; the acceptance test
 * is the one of sirius_verify_accept, Algorithm 1). Node (i, w) carries the
 * token tokens[b, i, w] and the full model's logits for that position at
 * row i * W + w; parents[b, i, w] (i >= 1) is the slot of its parent in
 * step i - 1 (parents[b, 0, *] is ignored). With bonus != 0, rows K * W + w
 * hold the logits after leaf w. With q_iw = softmax(L_iw / temperature)
 * [token] (0 for a token outside [0, V)), leaf w's advance is the first
 * step on its root path whose node has q < r (strict), else K.
 *   best_leaf[b]  = the leaf with the longest advance (lowest slot on ties)
 *   accept_len[b] = its advance
 *   next_token[b] = argmax of the raw logits at its rejected node, or of its
 *                   bonus row when all K are accepted, else -1.
 *   logits  [B, R, V] fp32, R = K * W (+ W with bonus), 16-byte aligned.
 *   tokens, parents [B, K, W] int32. A parent slot outside [0, W) is read
 *                   as slot 0.
 *   q       [B, K, W] fp32 out, or NULL.
 * With W = 1 this is sirius_verify_accept with R = K (+ 1).
 * Errors: SIRIUS_EINVAL for null pointers (q may be NULL), B < 0, K < 1,
 * W outside [1, 64], R > 1024, B * R > 65535, V < 1, NaN r, temperature not
 * finite and > 0.
 */
int sirius_tree_verify(const float* logits, int B, int K, int W, int V, int bonus,
                       const int32_t* tokens, const int32_t* parents, float r, float temperature,
                       int32_t* best_leaf, int32_t* accept_len, int32_t* next_token, float* q,
                       void* ws, size_t ws_bytes, void* stream);

/*
 * One attention layer over the KV cache shared by the sparse and the full
 * model, with the full model's direct rewrite (Algorithm 1; Sec. 4, how to
 * correct): the n tokens of batch entry b sit at positions p .. p + n - 1,
 * p = cache_pos[b]; their keys and values k_new, v_new are written into the
 * cache rows there (replacing what the sparse model wrote while drafting),
 * and token i attends causally to cache rows 0 .. p + i:
 *   out[b,i,h] = sum_j softmax_j(q[b,i,h] . K[b,j,h/G] / sqrt(head_dim)) V[b,j,h/G]
 * over j <= p + i, G = H / Hkv (grouped-query attention). n = 1 is the
 * sparse model's decode step; n = the kernel size is the full model's
 * verification pass over the drafted chunk. Scores, softmax and the weighted
 * sum run in fp32 on the stored bf16 keys and values.
 *   q          [B, n, H, head_dim] fp32 (any positional rotation applied).
 *   k_new, v_new [B, n, Hkv, head_dim] bf16.
 *   k_cache, v_cache [B, Lmax, Hkv, head_dim] bf16, updated in place.
 *   cache_pos  [B] int32 on the device, read only. An entry with p < 0 or
 *              p + n > Lmax leaves the cache untouched and gets NaN outputs.
 *   out        [B, n, H, head_dim] fp32.
 * All arrays 16-byte aligned. Errors: SIRIUS_EINVAL for null pointers, B
 * outside [0, 65535], n outside [1, 1024], H not a positive multiple of Hkv,
 * head_dim not a multiple of 8 in [8, 128], Lmax outside [n, 2^20].
 */
int sirius_attn_kv(const float* q, const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache,
                   uint16_t* v_cache, const int32_t* cache_pos, int B, int n, int H, int Hkv,
                   int head_dim, int Lmax, float* out, void* ws, size_t ws_bytes, void* stream);

/*
 * Rollback after the check (Algorithm 1): with the first rejected position
 * accept_len[b] of a chunk of n (n when all are accepted), the cache
 * position moves past the inputs that stay valid:
 *   cache_pos[b] += min(accept_len[b] + 1, n)
 * (cache_pos holding the chunk's start p, as passed to the verification
 * pass). Rows past the new position are simply overwritten later. Runs on
 * the device: no synchronisation with the host.
 * Errors: SIRIUS_EINVAL for null pointers, B < 0, n < 1.
 */
int sirius_kv_rollback(int32_t* cache_pos, const int32_t* accept_len, int B, int n, void* stream);

/*
 * A small Llama-style decoder whose sparse model M_S and full model M_F share
 * the weights and one KV cache (Algorithm 1). Every pointer but thresholds is
 * a device pointer, 16-byte aligned; weights are bf16 bit patterns:
 *   embed    [vocab, d_model]
 *   wq       [n_layers, n_heads * head_dim, d_model]
 *   wk, wv   [n_layers, n_kv_heads * head_dim, d_model]
 *   wo       [n_layers, d_model, n_heads * head_dim]
 *   w_gate, w_up, w_down [n_layers, d_ff, d_model] (neuron-major)
 *   lm_head  [vocab, d_model]
 *   k_cache, v_cache [n_layers, max_len, n_kv_heads, head_dim], the shared
 *            cache, updated in place
 *   thresholds HOST [n_layers]: M_S keeps FFN neuron i of layer l iff
 *            |SiLU(gate_i)| > thresholds[l] (a negative value keeps all).
 * Per layer: h += W_o attn(RMSNorm(h)) (grouped-query attention over the
 * cache, as sirius_attn_kv, no positional rotation) and h += FFN(RMSNorm(h))
 * (M_F: the dense FFN of sirius_ffn_dense, M_S: the threshold-sparse FFN of
 * sirius_ffn_cats); logits = W_lm RMSNorm(h). RMSNorm has unit weight and
 * epsilon norm_eps. Keys and values enter the cache as bf16 (round to
 * nearest even); every product accumulates in fp32. Limits: d_model and
 * n_heads * head_dim multiples of 8 up to 8192, head_dim a multiple of 8 up
 * to 128, n_heads a multiple of n_kv_heads, d_ff <= 65536, vocab <= 2^24,
 * max_len <= 2^20.
 */
typedef struct sirius_model {
  int n_layers, d_model, d_ff, n_heads, n_kv_heads, head_dim, vocab, max_len;
  float norm_eps;
  const uint16_t* embed;
  const uint16_t* wq;
  const uint16_t* wk;
  const uint16_t* wv;
  const uint16_t* wo;
  const uint16_t* w_gate;
  const uint16_t* w_up;
  const uint16_t* w_down;
  const uint16_t* lm_head;
  const float* thresholds;
  uint16_t* k_cache;
  uint16_t* v_cache;
} sirius_model;

/* Workspace bytes of sirius_model_forward with up to max_tokens tokens and of
 * sirius_generate with kernel size n = max_tokens (1 <= max_tokens <= 64);
 * 0 for an invalid model. */
size_t sirius_model_workspace_size(const sirius_model* model, int max_tokens);

/*
 * One pass of M_S (sparse != 0) or M_F over n tokens (device [n] int32; an id
 * outside [0, vocab) embeds as zeros) at positions p .. p + n - 1, p =
 * cache_pos[0] on the device (read only): the tokens' keys and values replace
 * those cache rows in every layer and token i attends to rows 0 .. p + i.
 *   logits      [n, vocab] fp32.
 *   active_idx  [n_layers, n, d_ff] int32 and active_cnt [n_layers, n], or
 *               both NULL (sparse only): the kept neurons of every token and
 *               layer, ascending.
 * The full model's FFN at n >= 8 runs on MFMA with its normalised input
 * rounded to bf16 (as sirius_ffn_dense). With p + n > max_len the attention
 * leaves the cache untouched and the logits are NaN.
 * Errors: SIRIUS_EINVAL for an invalid model, n outside [1, min(64, max_len)],
 * null pointers, a NaN threshold (sparse); SIRIUS_EWORKSPACE.
 */
int sirius_model_forward(const sirius_model* model, const int32_t* tokens, int n,
                         const int32_t* cache_pos, int sparse, float* logits, int32_t* active_idx,
                         int32_t* active_cnt, void* ws, size_t ws_bytes, void* stream);

/* Optional per-period records of sirius_generate (device pointers, each may be
 * NULL; active_idx and active_cnt go together). */
typedef struct sirius_gen_trace {
  int32_t* drafted;     /* [periods, n]: M_S's drafts */
  int32_t* accept_len;  /* [periods]: the first rejected draft, n if none */
  int32_t* next_token;  /* [periods]: the corrected token, -1 if none */
  float* q;             /* [periods, n]: M_F's likelihood of each draft */
  int32_t* active_idx;  /* [periods, n, n_layers, d_ff]: M_S's kept neurons per draft step */
  int32_t* active_cnt;  /* [periods, n, n_layers] */
} sirius_gen_trace;

/*
 * `periods` periods of the Sirius loop (Algorithm 1) with kernel size n,
 * greedy drafting and greedy correction, all on the device:
 *   drafting  M_S runs seq[i] at position P + i and drafts seq[i + 1] =
 *             argmax of its logits (lowest index on ties), for i < n; P =
 *             cache_pos[0] at the period's start;
 *   check     the position winds back to P and M_F runs seq[0 .. n - 1] in
 *             one pass, rewriting cache rows P .. P + n - 1; row i's softmax
 *             gives the likelihood q_i of seq[i + 1]; j = the first i with
 *             q_i < r, else n (sirius_verify_accept);
 *   rollback  cache_pos[0] = P + min(j + 1, n) (sirius_kv_rollback);
 *   interleave seq[1 .. j] and, when j < n, the corrected token argmax of
 *             row j are appended to out_tokens at out_count[0] (which is
 *             advanced); seq[0] becomes the corrected token, or seq[n].
 * seq [n + 1] int32 on the device: seq[0] holds the first input (the last
 * committed token, not yet in the cache) on entry and the next one on
 * return. cache_pos [1], out_count [1] int32 on the device; out_tokens has
 * room for periods * n tokens (never written past that). The caller keeps
 * cache_pos[0] + periods * n <= max_len. Nothing synchronises with the host:
 * the committed count is read from out_count afterwards.
 * Errors: as sirius_model_forward, plus n outside [1, 64], periods < 0, r NaN.
 */
int sirius_generate(const sirius_model* model, int32_t* seq, int32_t* cache_pos, int n, float r,
                    int periods, int32_t* out_tokens, int32_t* out_count,
                    const sirius_gen_trace* trace, void* ws, size_t ws_bytes, void* stream);

/*
 * RMSNorm with unit weight, the layer-stack glue around the FFN:
 *   out[b] = h[b] / sqrt(mean(h[b]^2) + eps). out may alias h.
 * Errors: SIRIUS_EINVAL for null pointers, d_model < 1, eps < 0.
 */
int sirius_rmsnorm(const float* h, int B, int d_model, float eps, float* out, void* stream);

/*
 * Seeded N(mean, std^2) bf16 fill, for building large synthetic weight
 * stacks directly in HBM. Counter-based (Philox4x32-10, Salmon et al., SC
 * 2011) with a Box-Muller transform: element e depends only on (seed, e).
 * Errors: SIRIUS_EINVAL for a null pointer or std < 0.
 */
int sirius_fill_normal_bf16(uint16_t* out, size_t n, uint64_t seed, float mean, float std,
                            void* stream);

/*
 * Per-kernel timing, for measurement. While enabled, each kernel the library
 * launches carries a pair of HIP events on its own dispatch (hipExtLaunchKernel):
 * the elapsed time between them is the kernel's execution time, as a kernel
 * trace reports it (where one name covers several launches of one call, from
 * the first one's start to the last one's end). sirius_profile_query waits for
 * the events of one kernel name and returns the summed duration in
 * milliseconds and the number of launches (0 and 0 for an unknown name).
 * Kernel names: "cats_decode", "cats_reduce", "dense_decode", "dense_reduce",
 * "topk_decode", "topk_reduce" (batch 1); "batch_prep", "batch_gate_up",
 * "batch_seg_gate_up", "batch_cats_up", "batch_topk_prep", "batch_topk_gate",
 * "batch_topk_up", "batch_down", "batch_reduce" (2..64 tokens with d_model a
 * multiple of 256); "cats_gate", "cats_down", "dense_gate", "dense_down",
 * "topk_up", "topk_down" (small batches at other shapes); "ffn_mfma_prep",
 * "ffn_mfma_gate_up", "ffn_mfma_down", "ffn_mfma_reduce" (8 or more tokens
 * at other shapes); "embed", "norm_qkv", "linear", "draft_tail",
 * "period_tail" (the small decoder);
 * "calib_gate", "select_init", "select_hist", "select_pick"; "topk_gate",
 * "topk_cut"; "verify_stats", "verify_scan", "tree_stats", "tree_scan",
 * "tree_topw", "tree_select"; "griffin_z", "griffin_rownorm", "griffin_score",
 * "griffin_topk", "condense"; "rmsnorm", "fill_normal"; "attn_partial",
 * "attn_combine", "kv_rollback".
 * sirius_profile_reset drops every record (it waits for pending events).
 * Errors: SIRIUS_EINVAL for NULL arguments, SIRIUS_EHIP if an event fails.
 */
int sirius_profile_enable(int on);
int sirius_profile_reset(void);
int sirius_profile_query(const char* kernel, double* total_ms, int64_t* launches);

/* Workspace bytes needed by an operation (SIRIUS_OP_*). Arguments:
 *   FFN_DENSE / FFN_CATS / FFN_CONDENSED / FFN_TOPK: B, d_model, d_ff (= k for
 *     the condensed layer), unused, unused
 *   CATS_CALIBRATE: N, d_model, d_ff, unused, unused
 *   GRIFFIN_SELECT: unused, d_model, d_ff, T, unused
 *   VERIFY: B, unused, unused, V, R (rows per batch entry)
 *   TREE_BUILD: B, Wc, W, V, unused
 *   TREE_VERIFY: B, K, W, V, bonus
 *   ATTN_KV: B, n, H * 65536 + Hkv, head_dim, Lmax
 * Returns 0 for an unknown op or invalid sizes. */
size_t sirius_workspace_size(int op, int B, int d_model, int d_ff, int T_or_V, int K_or_R);

/* Message for the calling thread's most recent failure ("" if none). */
const char* sirius_last_error(void);

/* Library version string. */
const char* sirius_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SIRIUS_H */
