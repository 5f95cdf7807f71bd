/*
 * sc.h - C ABI of the SparseCoder hot path on MI355X (gfx950).
 *
 * SparseCoder (arXiv 2310.07109) prunes tokens layer by layer inside an encoder
 * whose self-attention is a sliding window plus global tokens.  Per layer the
 * library computes, on one GPU:
 *
 *   sc_window_attention   banded Q.K^T, masked softmax and P.V for the sliding
 *                         window (Sec. 4.2.1, Fig. 4) plus the global tokens'
 *                         dense rows and columns (Sec. 3.2.1 "Global attention",
 *                         Fig. 3b-c; Sec. 5.5), and the per-query partial sums
 *                         of the attention probabilities each key receives;
 *   sc_ltp_score          the importance score of every token: probabilities
 *                         accumulated down its column after the row softmax
 *                         (Sec. 1, Fig. 1 caption; Sec. 3.3), i.e. the sum over
 *                         the band's sub-diagonal plus the global strips
 *                         (Sec. 5.5), averaged over heads and valid queries;
 *   sc_ltp_prune_compact  the binarised mask (keep iff score > threshold,
 *                         Sec. 4.2.2 step 2) and hard pruning: surviving tokens
 *                         are compacted into a shorter sequence (Sec. 4.2.2
 *                         step 3) for the next layer;
 *   sc_topk_prune_compact the same compaction with a top-k rule instead of the
 *                         threshold (a variant in the family of cascade token
 *                         pruning the paper cites in Sec. 3.3);
 *   sc_ltp_soft_mask      the soft mask of LTP's training phase (Sec. 4.2.2
 *                         step 1) and sc_ltp_soft_backward, the gradients of
 *                         q, k, v and the threshold through it;
 *   sc_encoder_stack      the full encoder stack: the layers above with a GELU
 *                         feed-forward block and a window per layer;
 *   sc_encoder_attn_stack the attention-only encoder stack (QKV projection,
 *                         the three steps above, output projection, residual
 *                         and LayerNorm) over several layers, each layer on the
 *                         previous layer's surviving tokens (Sec. 4.2, Fig. 5).
 *
 * Conventions shared by every entry point
 *   - Tensor pointers are DEVICE pointers owned by the caller; the library never
 *     allocates device memory.  Scratch memory comes from `workspace`, whose
 *     size is returned by the matching *_workspace_size() call (may be 0, in
 *     which case workspace may be NULL).
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     All work is enqueued asynchronously on it; nothing synchronises.  Calls
 *     on different streams may overlap when each has its own outputs and
 *     workspace (the library keeps no state between calls, apart from
 *     sc_window_attention_noalloc's device array and the benchmark events of
 *     sc_profile_window_kernel); e.g. a batch split into two halves on two
 *     streams gives the single call's results.
 *   - Arguments are validated on the host before anything is enqueued.  On any
 *     error nothing is enqueued and a negative sc_status is returned.
 *     Device-resident arguments (valid_len, global_pos) cannot be checked on
 *     the host: values outside their documented range are clamped or ignored
 *     by the kernels (memory-safe), with unspecified numerical results.
 *     sc_validate_desc checks them on the device; the debug build of the
 *     library (libsc_debug.so) does so before every call and refuses it.
 *   - Activations are token-major: [B, n, H, d] with d contiguous, so one token
 *     of one sequence is one contiguous row of H*d elements.
 *   - Sequence b holds valid_len[b] real tokens followed by padding.  Padding
 *     tokens are neither queries nor keys; their outputs are zero.
 */
#ifndef SC_H_
#define SC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t sc_status;
#define SC_OK 0
#define SC_EINVAL (-1)        /* invalid argument (null pointer, bad size, aliasing) */
#define SC_EUNSUPPORTED (-2)  /* valid but not implemented (e.g. head dim != 64)     */
#define SC_EWORKSPACE (-3)    /* workspace missing or smaller than required           */
#define SC_EHIP (-4)          /* a HIP runtime call failed (launch error)              */
#define SC_ENOSCRATCH (-5)    /* sc_window_attention_noalloc: the problem's workspace  */
                              /* exceeds SC_NOALLOC_SCRATCH_BYTES                       */

/* Size of the static device workspace of sc_window_attention_noalloc. */
#define SC_NOALLOC_SCRATCH_BYTES (16u << 20)

#define SC_F32 0   /* float32 storage and arithmetic                               */
#define SC_BF16 1  /* bfloat16 storage, float32 accumulation                        */

#define SC_SCORE_FROM_PARTIALS 0   /* sc_ltp_score reads sc_window_attention's partials */
#define SC_SCORE_FROM_BAND_PROBS 1 /* sc_ltp_score reads the band-stored probabilities   */

/*
 * Geometry of one attention layer over a padded batch.
 *   B, n        batch size and padded length; B >= 1, n >= 1.
 *   H, d        heads and head dimension; H >= 1, d must be 64.
 *   window      full window width w >= 0: query i attends to key j when
 *               |i - j| <= floor(w / 2) (both valid).  The paper states the
 *               window both as i-w..i+w (Sec. 4.2.1) and as a band stored as
 *               n x (2w - 1) (Sec. 5.5); this ABI takes w as the full width.
 *   G           global-token slots per sequence, 0 <= G <= n.
 *   global_pos  device int32 [B, G]: positions of the global tokens of each
 *               sequence, ascending and distinct, each < valid_len[b];
 *               -1 marks an unused slot.  May be NULL when G == 0.
 *   valid_len   device int32 [B]: 0 <= valid_len[b] <= n.
 *   softmax_scale  alpha >= 0 applied to Q.K^T before the softmax (finite).
 *   dtype       SC_F32 or SC_BF16 for q, k, v and outputs.
 * Sizes the kernels cannot index return SC_EUNSUPPORTED: one sequence's rows
 * of q, k or v (n * H * d elements; for sc_encoder_attn_stack its fused q|k|v
 * rows, 3 * n * H * d) must span less than 4 GiB, and each launch grid must
 * have fewer than 2^31 workgroups.
 */
typedef struct sc_attn_desc {
  int32_t B, n, H, d;
  int32_t window;
  int32_t G;
  const int32_t *global_pos;
  const int32_t *valid_len;
  float softmax_scale;
  int32_t dtype;
  /* 0: the bidirectional attention above; 1: causal variant (the decoder
   * direction the paper's Sec. 7.2 names as future work): N(i) also requires
   * j <= i, for the band and the global rows and columns alike.  Causal needs
   * SC_BF16 and no band_probs output (else SC_EUNSUPPORTED); other values are
   * SC_EINVAL. */
  int32_t causal;
} sc_attn_desc;

/* Human-readable text for a status code (static storage). */
const char *sc_status_str(sc_status s);

/* Bytes of the score partials written by sc_window_attention and read by
 * sc_ltp_score(SC_SCORE_FROM_PARTIALS); 0 on an invalid descriptor.  The layout
 * is private to the library: per (sequence, head) the band column sums of the
 * non-global keys, the column sums of the global keys per 512-query range, and
 * the column sums over the global query rows. */
size_t sc_score_partials_size(const sc_attn_desc *desc);

/* Bytes of the band-stored probabilities (paper layout, Sec. 5.5 / Fig. 3d),
 * three float32 arrays back to back, r = min(floor(w/2), n - 1):
 *   band [B, H, n, 2r+1]: entry (i, j) = P[i][i - r + j] when query i and key
 *        i - r + j are valid and neither is global, else 0 (the local part);
 *   gcol [B, H, n, G]: P[i][global_pos[b,s]] for valid non-global queries i and
 *        used slots s, else 0 (the global columns);
 *   grow [B, H, G, n]: P[global_pos[b,s]][k] for used slots s and valid keys k,
 *        else 0 (the global rows).
 * A token's score is its band sub-diagonal plus its global column and its
 * entries of the global rows.  0 on an invalid descriptor. */
size_t sc_band_probs_size(const sc_attn_desc *desc);

size_t sc_window_attention_workspace_size(const sc_attn_desc *desc);

/*
 * Sliding-window + global sparse attention of one layer (Sec. 4.2.1, Sec. 3.2.1,
 * Sec. 5.5): for every valid query i of sequence b and head h,
 *   N(i) = { j < L : |i - j| <= r  or  i global  or  j global },  r = floor(w/2)
 *   out[b,i,h,:] = sum_{j in N(i)} softmax_j(alpha * q_i . k_j) * v_j
 *   lse[b,h,i]   = log sum_{j in N(i)} exp(alpha * q_i . k_j)   (natural log)
 * Padding queries get out = 0 and lse = -inf.
 *   q, k, v     [B, n, H, d] in desc->dtype (read only).
 *   out         [B, n, H, d] in desc->dtype; must not overlap q, k or v.
 *   lse         float32 [B, H, n], or NULL.
 *   score_partials  float32 buffer of sc_score_partials_size() bytes, or NULL
 *               (skips the second pass that sums exact probabilities).
 *   band_probs  float32 buffer of sc_band_probs_size() bytes, or NULL; when set
 *               every probability is also stored in the paper's band layout.
 * Softmax is computed in float32 (exp2 of log2-scaled logits, running max);
 * in bf16 mode P is rounded to bf16 for the P.V product only.
 */
sc_status sc_window_attention(const sc_attn_desc *desc, const void *q, const void *k, const void *v, void *out,
                              float *lse, float *score_partials, float *band_probs, void *workspace,
                              size_t ws_bytes, void *stream);

/* Workspace of sc_ltp_score: 0 for SC_SCORE_FROM_PARTIALS; for
 * SC_SCORE_FROM_BAND_PROBS, sc_score_partials_size(desc) bytes (the band layout
 * is reduced to the same partials) plus one float per (sequence, head, block of
 * 128 rows, key the block reaches, rounded up to 256 keys).  0 on an invalid
 * descriptor. */
size_t sc_ltp_score_workspace_size(const sc_attn_desc *desc, int32_t mode);

/*
 * Importance score of every token (Sec. 1 Fig. 1; Sec. 3.3; Sec. 5.5):
 *   scores[b,k] = 1/(H * L_b) * sum_h sum_{i < L_b} P_h[i][k]   for k < L_b,
 *   scores[b,k] = 0                                              for k >= L_b,
 * so the scores of one sequence sum to one.  Deterministic: fixed-order sums,
 * no atomics.
 *   mode  SC_SCORE_FROM_PARTIALS: src = score_partials of sc_window_attention
 *         with the same desc; SC_SCORE_FROM_BAND_PROBS: src = band_probs.
 *   scores  float32 [B, n].
 *   workspace  device, sc_ltp_score_workspace_size(desc, mode) bytes (may be
 *         NULL when that is 0); must not overlap src or scores.
 * Errors: SC_EINVAL (null src or scores, bad mode, overlaps), SC_EWORKSPACE.
 */
sc_status sc_ltp_score(const sc_attn_desc *desc, int32_t mode, const float *src, float *scores, void *workspace,
                       size_t ws_bytes, void *stream);

size_t sc_ltp_prune_compact_workspace_size(const sc_attn_desc *desc);

/*
 * Binarised mask and hard pruning of one layer (Sec. 4.2.2 steps 2-3):
 *   keep(b,k) = k < L_b and (scores[b,k] > threshold  or  (keep_global and k global))
 * compared in float32, strictly.  Surviving tokens keep their order.
 *   scores          float32 [B, n] (e.g. from sc_ltp_score).
 *   n_tensors       0..4 tensors to compact, each [B, n, row_bytes[t]] bytes.
 *   src, dst        HOST arrays of n_tensors device pointers; dst row j of
 *                   sequence b = src row keep_idx[b,j] for j < new_len[b]; dst
 *                   rows at or beyond new_len are left untouched.  src[t] and
 *                   dst[t] must not overlap.
 *   row_bytes       HOST array of n_tensors row sizes in bytes (> 0).
 *   keep_idx        int32 [B, n]: input position of the j-th survivor, -1 beyond.
 *   new_len         int32 [B]: survivors per sequence.
 *   new_global_pos  int32 [B, G]: surviving global tokens renumbered into the
 *                   compacted sequence, ascending, -1 padded; may be NULL.
 *   orig_idx_in     int32 [B, n] or NULL (identity): original positions of the
 *                   layer's input tokens.
 *   orig_idx_out    int32 [B, n] or NULL: orig_idx_in[keep_idx], -1 beyond
 *                   new_len.  Must not overlap orig_idx_in.
 */
sc_status sc_ltp_prune_compact(const sc_attn_desc *desc, const float *scores, float threshold, int32_t keep_global,
                               int32_t n_tensors, const void *const *src, void *const *dst, const int64_t *row_bytes,
                               int32_t *keep_idx, int32_t *new_len, int32_t *new_global_pos,
                               const int32_t *orig_idx_in, int32_t *orig_idx_out, void *workspace, size_t ws_bytes,
                               void *stream);

/*
 * Top-k pruning, an alternative selection rule to the threshold above (the
 * paper's Sec. 3.3 places LTP among token-pruning methods, some of which keep a
 * fixed fraction of the tokens by rank).  Per sequence b, the candidates are the
 * valid tokens k < L_b, except the global ones when keep_global is set (those
 * are always kept); with C_b candidates,
 *   K_b = ceil(keep_ratio * C_b)   (computed in double; 0 <= K_b <= C_b)
 * candidates are kept: those with the K_b largest scores, where equal scores
 * (compared in float32) go to the lower index.  Survivors keep their order.
 *   keep_ratio      in [0, 1] (else SC_EINVAL; NaN included).
 * Every other argument, output, overlap rule, error and the workspace (same
 * size as sc_ltp_prune_compact_workspace_size) are as for
 * sc_ltp_prune_compact.
 */
sc_status sc_topk_prune_compact(const sc_attn_desc *desc, const float *scores, float keep_ratio, int32_t keep_global,
                                int32_t n_tensors, const void *const *src, void *const *dst, const int64_t *row_bytes,
                                int32_t *keep_idx, int32_t *new_len, int32_t *new_global_pos,
                                const int32_t *orig_idx_in, int32_t *orig_idx_out, void *workspace, size_t ws_bytes,
                                void *stream);

/*
 * LTP soft pruning, the training form of the pruning (Sec. 4.2.2 step 1: the
 * model and the per-layer thresholds are trained through a soft mask, which
 * is binarised afterwards).  The paper describes the mask in words only; the
 * form here is the one of the Learned Token Pruning method it adopts:
 *   mask[b,k] = sigmoid((scores[b,k] - theta) / temperature)  for k < L_b,
 *               except 1 for global tokens when keep_global is set,
 *   mask[b,k] = 0 for k >= L_b,
 *   y[b,k,:,:] = bf16(mask[b,k] * out[b,k,:,:]).
 * As temperature goes to 0 the mask becomes the binarised mask of
 * sc_ltp_prune_compact.
 *   scores      float32 [B, n] (sc_ltp_score).
 *   out         bf16 [B, n, H, d] (sc_window_attention's output).
 *   mask        float32 [B, n], written.   y  bf16 [B, n, H, d], written.
 * desc->dtype must be SC_BF16 and causal 0 (else SC_EUNSUPPORTED); theta
 * finite and temperature > 0 (else SC_EINVAL).  y must not overlap out.
 */
sc_status sc_ltp_soft_mask(const sc_attn_desc *desc, const float *scores, float theta, float temperature,
                           int32_t keep_global, const void *out, float *mask, void *y, void *stream);

size_t sc_ltp_soft_backward_workspace_size(const sc_attn_desc *desc);

/*
 * Backward of the soft-pruned layer y = mask * attention(q, k, v), with the
 * mask computed from the layer's own importance scores (the sigmoid above of
 * s_k = (1 / (H L)) sum_h sum_q P_h[q][k]).  Given dy = dL/dy and optionally
 * dmask = dL/dmask (e.g. a regulariser on the kept fraction), it writes
 *   dq, dk, dv  bf16 [B, n, H, d]: dL/dq, dL/dk, dL/dv through the attention
 *               output and through the scores (0 on padding rows);
 *   dtheta      one float32 (device): dL/dtheta.
 * Inputs: q, k, v, out bf16 [B, n, H, d] and lse float32 [B, H, n] of the
 * forward sc_window_attention (same desc), mask float32 [B, n] of
 * sc_ltp_soft_mask, dy bf16 [B, n, H, d], dmask float32 [B, n] or NULL, and
 * the temperature and keep_global of the forward.  Probabilities are
 * recomputed from q, k and lse in float32; products run on bf16 MFMA with
 * float32 accumulation; dL/dmask is accumulated in float32.  Deterministic
 * (fixed-order sums, no atomics).  desc->dtype must be SC_BF16 and causal 0
 * (else SC_EUNSUPPORTED).  Outputs must not overlap each other, the inputs
 * or the workspace.
 */
sc_status sc_ltp_soft_backward(const sc_attn_desc *desc, const void *q, const void *k, const void *v,
                               const void *out, const float *lse, const float *mask, float temperature,
                               int32_t keep_global, const void *dy, const float *dmask, void *dq, void *dk,
                               void *dv, float *dtheta, void *workspace, size_t ws_bytes, void *stream);

size_t sc_encoder_attn_stack_workspace_size(const sc_attn_desc *desc, int32_t n_layers);

/*
 * Attention-only encoder stack of n_layers RoBERTa-shaped layers without FFN
 * (Sec. 4.2, Fig. 5; pruning after each layer, Sec. 4.2.2):
 *   qkv = bf16(x . Wqkv[l])                 Wqkv [D, 3D] row-major, columns q|k|v,
 *                                            each head-major (head h = cols h*d..)
 *   O   = bf16(sc_window_attention(q,k,v))   with the layer's current lengths
 *   keep, compaction as sc_ltp_prune_compact with thresholds[l]
 *   x   = bf16(LayerNorm(x + O . Wo[l]))     on the survivors; Wo [D, D];
 *                                            LayerNorm gamma 1, beta 0, eps ln_eps
 * desc gives the layer-0 geometry (dtype must be SC_BF16, causal 0, D = H*d,
 * B <= 8192: the products pack the surviving rows of all sequences, larger
 * batches return SC_EUNSUPPORTED); lengths and global positions shrink on the
 * device from layer to layer, with no host synchronisation.
 *   x_in            bf16 [B, n, D]; x_out bf16 [B, n, D] (survivors first).
 *   Wqkv, Wo        HOST arrays of n_layers device pointers (bf16).
 *   thresholds      HOST float [n_layers].
 *   final_len       int32 [B]; orig_idx int32 [B, n] (input position of each
 *                   surviving row, -1 beyond final_len); kept_per_layer int32
 *                   [n_layers, B] (sequence length after each layer's pruning).
 */
sc_status sc_encoder_attn_stack(const sc_attn_desc *desc, int32_t n_layers, const void *x_in,
                                const void *const *Wqkv, const void *const *Wo, const float *thresholds,
                                int32_t keep_global, float ln_eps, void *x_out, int32_t *final_len,
                                int32_t *orig_idx, int32_t *kept_per_layer, void *workspace, size_t ws_bytes,
                                void *stream);

size_t sc_encoder_stack_workspace_size(const sc_attn_desc *desc, int32_t n_layers, int32_t ffn_dim);

/*
 * Full encoder stack: every layer as in sc_encoder_attn_stack, followed by the
 * feed-forward block of a RoBERTa-shaped post-LN layer (Sec. 4.2, Fig. 5), with
 * a window per layer (Sec. 7.1 names small windows in lower layers and large
 * ones in higher layers):
 *   x1  = bf16(LayerNorm(x + O . Wo[l]))          on the survivors
 *   h   = bf16(GELU(x1 . W1[l]))                   W1 [D, ffn_dim]; GELU exact,
 *                                                   v * Phi(v)
 *   x   = bf16(LayerNorm(x1 + h . W2[l]))          W2 [ffn_dim, D]
 * No biases; LayerNorm gamma 1, beta 0, eps ln_eps.
 *   windows         HOST int32 [n_layers], each >= 0, or NULL (desc->window in
 *                   every layer).
 *   W1, W2          HOST arrays of n_layers device pointers (bf16), non-NULL.
 *   ffn_dim         > 0 and a multiple of 8 (3072 for RoBERTa-base).
 * Everything else (arguments, outputs, errors) as for sc_encoder_attn_stack;
 * the workspace is sc_encoder_stack_workspace_size(desc, n_layers, ffn_dim).
 */
sc_status sc_encoder_stack(const sc_attn_desc *desc, int32_t n_layers, const int32_t *windows, const void *x_in,
                           const void *const *Wqkv, const void *const *Wo, const void *const *W1,
                           const void *const *W2, int32_t ffn_dim, const float *thresholds, int32_t keep_global,
                           float ln_eps, void *x_out, int32_t *final_len, int32_t *orig_idx, int32_t *kept_per_layer,
                           void *workspace, size_t ws_bytes, void *stream);

/*
 * sc_window_attention_noalloc: sc_window_attention for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same computation, outputs and
 * argument rules, without the workspace arguments.  The workspace is a static
 * device array of SC_NOALLOC_SCRATCH_BYTES (16 MiB) that every GPU the library
 * runs on holds until the process ends; the call itself allocates nothing
 * (no hipMalloc, no allocating library routine, no benchmark events).
 *   stream  must belong to the current device (else SC_EINVAL).
 * Errors: as sc_window_attention (no SC_EWORKSPACE); SC_ENOSCRATCH when
 * sc_window_attention_workspace_size(desc) exceeds SC_NOALLOC_SCRATCH_BYTES
 * (nothing is enqueued).  Every call on a GPU shares that GPU's array and the
 * array keeps the last call's contents (nothing in it needs to start at zero):
 * calls that overlap on one GPU (on different streams, or from different host
 * threads without ordering) race on it and must be serialised by the caller.
 */
sc_status sc_window_attention_noalloc(const sc_attn_desc *desc, const void *q, const void *k, const void *v,
                                      void *out, float *lse, float *score_partials, float *band_probs,
                                      void *stream);

/*
 * Checks the device-resident parts of a descriptor, which the host cannot
 * read and the kernels clamp or ignore when out of range: for callers that
 * want such inputs reported rather than computed on (and the library's debug
 * build, below).  Enqueues on `stream` the setting of *err (a device int32
 * owned by the caller) to the OR of the SC_VALID_* bits of the violations
 * found, 0 when valid_len and global_pos are as sc_attn_desc documents them;
 * the value is there once the enqueued work completes.  Capture-safe (no
 * memset node).  Errors: those of the descriptor's host-side check, and
 * SC_EINVAL for a null err.
 *
 * Debug build.  paper_2310_07109_amd/libsc_debug.so is the same library built
 * with SC_DEBUG: every entry point that takes a descriptor first runs this
 * check and waits for it, returning SC_EINVAL (nothing else enqueued) when a
 * bit is set, and waits for its own work before returning, reporting a failed
 * launch or execution as SC_EHIP.  It synchronises the stream, so it is not
 * capture-safe; its results are the release library's.
 */
#define SC_VALID_LEN 1              /* a valid_len[b] outside [0, n]                      */
#define SC_VALID_POS_RANGE 2        /* a global position below -1 or >= its valid_len[b]  */
#define SC_VALID_POS_ORDER 4        /* used global positions not strictly ascending       */
#define SC_VALID_POS_UNUSED_FIRST 8 /* a used slot after an unused (-1) one               */
sc_status sc_validate_desc(const sc_attn_desc *desc, int32_t *err, void *stream);

/*
 * Kernel timing for benchmarks.  While enabled, every window-attention call
 * (sc_window_attention, and each layer of the stacks) records three hipEvents
 * on the caller's stream: before its first launch (softmax and P.V), between
 * the launches, and after its second launch (the exact-probability column
 * sums).  sc_profile_window_kernel_read() waits for the recorded events and
 * writes, for the first min(capacity, *calls) calls in call order, the time of
 * launch 1 to fwd_ms[i] and of launch 2 to cols_ms[i], in milliseconds (host
 * arrays owned by the caller); *calls receives the number of calls recorded.
 * It then clears the record; enabling with a non-zero argument clears it too.
 * Errors: SC_EINVAL for a null `calls`, a negative capacity or null arrays
 * with a positive capacity; SC_EHIP if an event failed.  Not thread-safe; at
 * most 4096 calls are recorded.
 */
sc_status sc_profile_window_kernel(int32_t enable);
sc_status sc_profile_window_kernel_read(double *fwd_ms, double *cols_ms, int64_t capacity, int64_t *calls);

#ifdef __cplusplus
}
#endif
#endif /* SC_H_ */
