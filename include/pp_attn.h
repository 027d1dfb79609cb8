/*
 * pp_attn.h -- C ABI of the preference-packing hot path for AMD MI355X (gfx950).
 *
 * Preference packing (Sec. 3.2 of "Preference Packing: Efficient Preference
 * Optimization for Large Language Models") writes one prompt once and then its
 * K ranked responses one after another in a single row; a causal mask lets every
 * response see the whole prompt and its own earlier tokens but never another
 * response, and position IDs keep each token's unpacked position.  The library
 * computes, on one GPU:
 *
 *   pp_attn_fwd     masked attention forward over packed rows  (Sec. 3.2)
 *   pp_attn_bwd     its gradients dQ, dK, dV                   (Sec. 3.2)
 *   pp_seq_logprob  per-response summed token log-probs        (Sec. 2.1, Sec. 3.2)
 *   pp_seq_logprob_bwd  their gradient with respect to the logits (all rows,
 *                   or only the rows that predict a response token)
 *   pp_rm_scores    reward-model head on each response's last token (Sec. 2.1)
 *   pp_rm_scores_bwd    its gradients
 *   pp_dpo_loss     ranked-pair DPO / Bradley-Terry loss        (Sec. 2.1)
 *   pp_rope, pp_attn_fwd_rope, pp_attn_bwd_rope
 *                   rotary position embedding on the packed position IDs
 *                   (Sec. 3.2), alone or fused into attention
 *   pp_plan_create, pp_attn_fwd_planned, pp_attn_bwd_planned
 *                   the same attention on a plan built once per packed batch
 *                   and reused (e.g. by every layer of a model)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  Every pointer named "dev" is device memory owned by the caller;
 *   every pointer named "host" is host memory read before the call returns.
 *   The library allocates no device memory; it keeps a small ring of pinned host
 *   staging buffers for plan metadata, freed when the library is unloaded.
 *   Tensor arguments of the attention and rotary entry points (q, k, v, o, dout,
 *   dq, dk, dv, q_rot, k_rot, x, y) must be 16-byte aligned, lse 4-byte aligned
 *   (rows move in 16-byte vectors); a misaligned pointer is rejected with
 *   PP_ERR_INVALID_ARGUMENT.  Workspaces (`ws`) must be 256-byte aligned, and
 *   are rejected the same way otherwise.  Allocations from hipMalloc or torch
 *   qualify.
 * Streams.  All device work is enqueued on `hip_stream` (a hipStream_t; NULL
 *   means the null stream) in call order; no entry point synchronises the device.
 * Errors.  Arguments are validated on the host before anything is enqueued; a
 *   failed validation returns an error code and enqueues nothing.  A HIP error
 *   while enqueuing returns PP_ERR_HIP.  No entry point throws or aborts.
 *   pp_last_error() returns a human-readable message for the last failure on the
 *   calling thread.
 * Concurrency.  Calls may be made from several host threads; calls that share a
 *   workspace must be ordered on one stream.
 *
 * The packed layout (pp_pack_desc)
 * --------------------------------
 * B rows are concatenated on one flat token axis of sumT = row_start[B] tokens.
 * Row b spans [row_start[b], row_start[b+1]) (its capacity T_b).  Its prompt is
 * the first P_b = prompt_len[b] tokens; response k (0 <= k < K_b = num_resp[b])
 * is [resp_off[b*max_resp+k], + resp_len[b*max_resp+k]) relative to the row
 * start.  Responses are contiguous: resp_off[b,0] = P_b and resp_off[b,k+1] =
 * resp_off[b,k] + resp_len[b,k] ("sequentially pack", Sec. 1 and Sec. 3.2), and
 * P_b + sum_k resp_len[b,k] <= T_b.  Tokens after that are padding: their
 * attention output, LSE and gradients are written as 0.  Responses are in the
 * paper's ranking order: a larger index is preferred (Sec. 3.1).
 *
 * Mask (Sec. 3.2; Figure 1 is described only by its caption): query i sees key
 * j iff j <= i, neither is padding, and j is a prompt token or lies in the same
 * response as i.  q-head h reads kv-head h / (hq / hkv).
 *
 * Tensor layouts (row-major, contiguous):
 *   q, o, dout, dq      [sumT, hq,  head_dim]
 *   k, v, dk, dv        [sumT, hkv, head_dim]
 *   lse                 [hq, sumT] float, natural log of the softmax denominator
 *   logits              [sumT, vocab]: row t holds the next-token logits produced
 *                       at packed position t
 *   tokens              [sumT] int32 packed input ids
 */
#ifndef PP_ATTN_H
#define PP_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum pp_status {
  PP_OK = 0,
  PP_ERR_INVALID_ARGUMENT = 1,  /* null pointer, bad count or size, no loss pair */
  PP_ERR_BAD_LAYOUT = 2,        /* descriptor violates the packed layout above */
  PP_ERR_UNSUPPORTED = 3,       /* valid but not implemented (e.g. head_dim)  */
  PP_ERR_WORKSPACE_TOO_SMALL = 4,
  PP_ERR_HIP = 5,               /* a HIP runtime call failed */
  /* range markers, not statuses: they make every int32 a valid value of the
     type, so an out-of-range value from a caller is defined behaviour */
  PP_STATUS_RANGE_MIN_ = -0x7fffffff - 1,
  PP_STATUS_RANGE_MAX_ = 0x7fffffff
} pp_status;

typedef enum pp_dtype {
  PP_BF16 = 0,  /* bfloat16 */
  PP_FP32 = 1,  /* float; attention inputs are rounded to bf16 (nearest even) */
  /* range markers (see pp_status): any other value is rejected with
     PP_ERR_INVALID_ARGUMENT */
  PP_DTYPE_RANGE_MIN_ = -0x7fffffff - 1,
  PP_DTYPE_RANGE_MAX_ = 0x7fffffff
} pp_dtype;

/* Host description of a packed batch; see "The packed layout" above. */
typedef struct pp_pack_desc {
  int32_t num_rows;          /* B >= 1 */
  int32_t max_resp;          /* K_max >= 0: stride of resp_off / resp_len */
  const int32_t* row_start;  /* host [B+1], row_start[0] = 0, non-decreasing */
  const int32_t* prompt_len; /* host [B], P_b >= 0 */
  const int32_t* num_resp;   /* host [B], 0 <= K_b <= K_max */
  const int32_t* resp_off;   /* host [B*K_max], row-relative */
  const int32_t* resp_len;   /* host [B*K_max], >= 0 */
} pp_pack_desc;

/* Device workspace (bytes) that each entry point needs for this batch.
 * Any output pointer may be NULL.  dtype is the attention input dtype (fp32
 * inputs need room for their bf16 copies).  vocab is used only for logprob and
 * may be 0.  hq, hkv and head_dim are validated as for pp_attn_fwd when fwd or
 * bwd is requested.  bwd is the workspace of pp_attn_bwd / pp_attn_bwd_rope in
 * their default (recompute) mode; pp_bwd_stored_ds_workspace_size gives the
 * larger one of the stored-dS mode.  logprob serves both pp_seq_logprob and
 * pp_seq_logprob_bwd.  loss is the workspace of pp_dpo_loss for this batch's B. */
pp_status pp_workspace_size(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                            int vocab, size_t* fwd, size_t* bwd, size_t* logprob, size_t* loss);

/* Forward packed attention (Sec. 3.2): for every non-padding query i and head h
 *   O[i,h]   = sum_j softmax_j(scale * q[i,h] . k[j,g]) v[j,g] over the keys j
 *              that query i sees, g = h / (hq/hkv);
 *   lse[h,i] = ln sum_j exp(scale * q[i,h] . k[j,g]).
 * Padding queries get O = 0 and lse = 0.
 * dtype: PP_BF16 or PP_FP32 for q, k, v and o (fp32 inputs are rounded to bf16,
 * nearest even, into the workspace first; products accumulate in fp32).
 * head_dim in {64, 128}; hq % hkv == 0.
 * scale <= 0 selects 1/sqrt(head_dim).
 * Errors: PP_ERR_UNSUPPORTED for another head_dim; PP_ERR_INVALID_ARGUMENT for
 * null or misaligned pointers or bad head counts; PP_ERR_BAD_LAYOUT for a bad descriptor;
 * PP_ERR_WORKSPACE_TOO_SMALL if ws_bytes is below pp_workspace_size's fwd. */
pp_status pp_attn_fwd(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                      float scale, const void* q, const void* k, const void* v, void* o,
                      float* lse, void* ws, size_t ws_bytes, void* hip_stream);

/* Backward of pp_attn_fwd: gradients of sum(dout * O) (Sec. 3.2).
 *   dV[j,g] = sum_{h in g} sum_i P_ij dO[i,h]
 *   dS_ij   = P_ij (dO[i,h] . v[j,g] - dO[i,h] . O[i,h])
 *   dQ[i,h] = scale sum_j dS_ij k[j,g]
 *   dK[j,g] = scale sum_{h in g} sum_i dS_ij q[i,h]
 * The gradient of a prompt key gathers the contributions of the prompt's own
 * queries and of every response's queries (the prompt is stored once).
 * o and lse are the outputs of pp_attn_fwd on the same inputs.  dq, dk, dv have
 * the input dtype; padding rows are written as 0.  The result is deterministic
 * (no atomics).  Errors as pp_attn_fwd.
 *
 * Workspace and mode: with ws_bytes >= pp_workspace_size's bwd the dQ pass
 * recomputes S and dP (scratch linear in the tokens, as Sec. 3.2.1's memory
 * argument assumes).  With ws_bytes >= pp_bwd_stored_ds_workspace_size's bwd
 * the key-major pass also stores dS (bf16, one value per query-key pair of
 * every 32 x 32 block with a visible pair, per query head) at the end of the
 * workspace and the dQ pass reads it back instead, so S, P and dP are computed
 * once.  Both modes round dS to bf16 before the products that use it; they agree
 * to fp32 rounding.  Below pp_workspace_size's bwd: PP_ERR_WORKSPACE_TOO_SMALL. */
pp_status pp_attn_bwd(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                      float scale, const void* q, const void* k, const void* v, const void* o,
                      const float* lse, const void* dout, void* dq, void* dk, void* dv, void* ws,
                      size_t ws_bytes, void* hip_stream);

/* pp_attn_fwd for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  Same
 * kernels, same plan and bit-identical results as pp_attn_fwd with dtype
 * PP_BF16 (q, k, v, o are bf16; fp32 inputs would need workspace room for their
 * bf16 copies and are not offered here), but no workspace argument: the plan's
 * metadata is copied (hipMemcpyAsync from host memory, on hip_stream) into a
 * static device array of PP_NOALLOC_SCRATCH_BYTES that the library holds on
 * every device it runs on until the process ends.  The call allocates no
 * device memory and no pinned host memory (host-side planning uses ordinary
 * heap memory).  Every call on a device reuses that device's array, whose
 * contents are those of the last call: calls that overlap on one device (other
 * streams, or unordered host threads) race; calls ordered on one stream do not.
 * Errors as pp_attn_fwd; PP_ERR_WORKSPACE_TOO_SMALL when the pack's plan needs
 * more than PP_NOALLOC_SCRATCH_BYTES (pp_workspace_size's fwd for PP_BF16 is
 * the amount; about 4 bytes per token twice plus the tile lists, so roughly up
 * to 400K tokens), before anything is enqueued. */
#define PP_NOALLOC_SCRATCH_BYTES ((size_t)4 << 20)
pp_status pp_attn_fwd_noalloc(const pp_pack_desc* desc, int hq, int hkv, int head_dim, float scale,
                              const void* q, const void* k, const void* v, void* o, float* lse,
                              void* hip_stream);

/* Rotary position embedding on the packed position IDs.  Sec. 3.2 requires that
 * every packed token keep the position it has in its unpacked sequence: prompt
 * token t has position t, token j of a response has P_b + j (so every response
 * continues from the end of the shared prompt), padding has 0 -- the
 * position_ids of pp_pack_export.  The embedding is the half-split rotary form
 * of the Llama / Qwen models: for j < head_dim/2 the pair (x_j, x_{j+head_dim/2})
 * of a token at position p is rotated by the angle p * rope_base^(-2j/head_dim),
 *   y_j = x_j cos - x_{j+d/2} sin,   y_{j+d/2} = x_{j+d/2} cos + x_j sin.
 * inverse != 0 applies the transpose (the rotation by the negative angle), which
 * is also the map that carries a gradient back through the embedding.  Angles
 * are formed and reduced to [-pi, pi] in fp64, sines and cosines and the
 * rotation are fp32, bf16 outputs are rounded to nearest even.
 * x, y: dev [sumT, heads, head_dim] in dtype; y may equal x (in place).
 * head_dim a multiple of 8 in [8, 1024] (PP_ERR_UNSUPPORTED otherwise);
 * rope_base finite and > 0 (PP_ERR_INVALID_ARGUMENT otherwise).
 * ws_bytes >= pp_rope_workspace_size's bytes (positions and frequencies). */
pp_status pp_rope_workspace_size(const pp_pack_desc* desc, int head_dim, size_t* bytes);
pp_status pp_rope(const pp_pack_desc* desc, pp_dtype dtype, int heads, int head_dim, float rope_base,
                  int inverse, const void* x, void* y, void* ws, size_t ws_bytes, void* hip_stream);

/* pp_attn_fwd of rotated queries and keys (the rotation of pp_rope): q and k are
 * the un-rotated inputs.  k is rotated once into k_rot (dev [sumT, hkv,
 * head_dim], dtype, required); each query row is rotated in registers inside the
 * attention kernel right after it is loaded, and written to q_rot (dev [sumT,
 * hq, head_dim], dtype) when q_rot is not NULL.  For PP_FP32 the queries are
 * rounded to bf16 before they are rotated, as for attention.  o and lse are those
 * of pp_attn_fwd(rope(q), rope(k), v).  Workspace: pp_workspace_size's fwd.
 * Errors as pp_attn_fwd, plus PP_ERR_INVALID_ARGUMENT for a bad rope_base or a
 * NULL k_rot. */
pp_status pp_attn_fwd_rope(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                           float scale, float rope_base, const void* q, const void* k, const void* v,
                           void* o, float* lse, void* q_rot, void* k_rot, void* ws, size_t ws_bytes,
                           void* hip_stream);

/* Backward of pp_attn_fwd_rope: takes the rotated q_rot and k_rot (as written by
 * pp_attn_fwd_rope), v, o, lse and dout, and writes dq and dk with respect to
 * the UN-rotated q and k -- the dQ and dK/dV kernels rotate their gradient rows
 * back (the inverse rotation) just before storing them -- and dv.  Otherwise as
 * pp_attn_bwd (deterministic; workspace pp_workspace_size's bwd). */
pp_status pp_attn_bwd_rope(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                           float scale, float rope_base, const void* q_rot, const void* k_rot,
                           const void* v, const void* o, const float* lse, const void* dout, void* dq,
                           void* dk, void* dv, void* ws, size_t ws_bytes, void* hip_stream);

/* Reusable plans (the Plan step of the packed path, Sec. 3.2).  Every pp_attn_*
 * call above plans the pack on the host and copies the plan's metadata into its
 * workspace before its kernels run.  A model applies attention to the same
 * packed batch in every layer, so the plan can be built once per batch instead:
 *
 *   pp_plan_workspace_size(desc, ...)           -> bytes for the plan's workspace
 *   pp_plan_create(desc, ..., ws, stream, &pl)  plans on the host and enqueues one
 *                                               copy of the forward and backward
 *                                               metadata into ws on stream
 *   pp_attn_fwd_planned(pl, ...) / pp_attn_bwd_planned(pl, ...)
 *                                               enqueue kernels only, any number
 *                                               of times (e.g. once per layer)
 *   pp_plan_destroy(pl)                         frees the host record
 *
 * The planned calls compute exactly what pp_attn_fwd / pp_attn_bwd (or, with a
 * rope_base, pp_attn_fwd_rope / pp_attn_bwd_rope) compute for the same pack and
 * arguments.  Ownership: the plan (host memory, freed by pp_plan_destroy) refers
 * to ws, which stays the caller's; ws must outlive the plan and must not be
 * written by anything else while the plan is in use.  The planned calls also
 * use ws as scratch (delta, fp32 casts, dS), so calls on one plan must be ordered
 * on one stream, after the stream that pp_plan_create used (or synchronised
 * with it).  pp_plan_create copies the descriptor: the caller may free or
 * change it afterwards.  A plan is bound to the dtype, head counts, head_dim and
 * rope_base it was made with. */
typedef struct pp_plan pp_plan;

/* Workspace bytes of a plan for this pack and shape (forward and backward
 * metadata and the backward's scratch, for the recompute backward).  Errors as
 * pp_attn_fwd. */
pp_status pp_plan_workspace_size(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                                 size_t* bytes);

/* The larger workspaces that select the backward's stored-dS mode (see
 * pp_attn_bwd): *bwd for pp_attn_bwd / pp_attn_bwd_rope, *plan for
 * pp_plan_create (a plan made with at least this many bytes stores dS).
 * Either pointer may be NULL.  Errors as pp_attn_fwd, plus PP_ERR_UNSUPPORTED
 * when the batch has 2^31 or more stored tiles per head. */
pp_status pp_bwd_stored_ds_workspace_size(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                                          size_t* bwd, size_t* plan);

/* Builds a plan and enqueues its metadata copy into ws (dev, ws_bytes >=
 * pp_plan_workspace_size's bytes, or >= pp_bwd_stored_ds_workspace_size's plan
 * for the stored-dS backward) on hip_stream.  rope_base (host, may be NULL)
 * selects the rotary variants.  *plan receives the handle, or NULL on error.
 * Errors as pp_attn_fwd, plus PP_ERR_INVALID_ARGUMENT for a NULL plan pointer
 * or a bad rope_base. */
pp_status pp_plan_create(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                         const float* rope_base, void* ws, size_t ws_bytes, void* hip_stream, pp_plan** plan);

/* Frees a plan's host record (NULL is accepted).  Does not touch ws. */
pp_status pp_plan_destroy(pp_plan* plan);

/* pp_attn_fwd (or pp_attn_fwd_rope when the plan has a rope_base; q_rot may be
 * NULL, k_rot is required then and ignored otherwise) on a plan.  Tensor
 * arguments, scale and errors as there; PP_ERR_INVALID_ARGUMENT for a NULL plan. */
pp_status pp_attn_fwd_planned(const pp_plan* plan, float scale, const void* q, const void* k, const void* v,
                              void* o, float* lse, void* q_rot, void* k_rot, void* hip_stream);

/* pp_attn_bwd (or pp_attn_bwd_rope, with q, k the rotated ones) on a plan. */
pp_status pp_attn_bwd_planned(const pp_plan* plan, float scale, const void* q, const void* k, const void* v,
                              const void* o, const float* lse, const void* dout, void* dq, void* dk, void* dv,
                              void* hip_stream);

/* Per-response sequence log-probabilities (Sec. 2.1 scores, Sec. 3.2 layout).
 * Token j of response k of row b sits at row-relative position t = o_bk + j; it
 * is predicted by the logits at position P_b - 1 when j = 0 (the last prompt
 * token, shared by all K responses) and at t - 1 otherwise, with label
 * tokens[t].  Its log-prob is logit[label] - ln sum_v exp(logit[v]), computed in
 * fp32.  seq_logp[b*K_max+k] (dev, float) = sum over the response's tokens, in
 * token order; empty responses and slots k >= K_b get 0.  tok_logp (dev, float
 * [sumT], may be NULL) receives each response token's log-prob at its own
 * position and 0 at every other position.  A label outside [0, vocab) makes that
 * response's sum NaN.  Only the logit rows that predict a response token are
 * read.  logits_dtype: PP_BF16 or PP_FP32.
 * Errors: PP_ERR_BAD_LAYOUT also when a row has P_b = 0 and a non-empty response
 * (its first token has no predicting position). */
pp_status pp_seq_logprob(const pp_pack_desc* desc, pp_dtype logits_dtype, int vocab,
                         const void* logits, const int32_t* tokens, float* seq_logp,
                         float* tok_logp, void* ws, size_t ws_bytes, void* hip_stream);

/* Backward of pp_seq_logprob: the gradient of sum_{b,k} dseq[b*K_max+k] *
 * seq_logp[b*K_max+k] with respect to the logits (Sec. 2.1 scores; dseq is
 * typically pp_dpo_loss's dlogp_pol).  Every response token adds
 * dseq[b,k] * (onehot(label) - softmax(row)) to the logit row that predicts it
 * (the same rows as pp_seq_logprob, so the last prompt row gathers the first
 * token of every response); every other row of dlogits is written as 0.  A
 * label outside [0, vocab) makes its predicting row NaN.
 * logits (dev [sumT, vocab], logits_dtype), tokens (dev int32 [sumT]), dseq (dev
 * float [B*K_max]); dlogits (dev [sumT, vocab], logits_dtype) is overwritten.
 * Softmax and products are computed in fp32; bf16 outputs are rounded to
 * nearest even.  ws_bytes >= pp_workspace_size's logprob.
 * Errors: as pp_seq_logprob; PP_ERR_UNSUPPORTED when max_resp > 256. */
pp_status pp_seq_logprob_bwd(const pp_pack_desc* desc, pp_dtype logits_dtype, int vocab,
                             const void* logits, const int32_t* tokens, const float* dseq,
                             void* dlogits, void* ws, size_t ws_bytes, void* hip_stream);

/* pp_seq_logprob_bwd restricted to the logit rows that predict a response token
 * (Sec. 2.1 scores over the Sec. 3.2 layout): only those rows -- a row's last
 * prompt position once (it predicts the first token of every response), then
 * for each response k its positions o_bk .. o_bk + L_bk - 2 -- are written,
 * back to back in that order (rows of the batch in order), so the gradient of a
 * batch costs one read and one write of each such row instead of a write of all
 * sumT rows.  pp_logprob_row_count gives their number n (host only).
 * dlogits_rows: dev [n, vocab] in logits_dtype; row i is the gradient of the
 * flat logit row row_index[i] (dev int32 [n], strictly increasing, may be NULL)
 * and equals that row of pp_seq_logprob_bwd's output bit for bit; every other
 * row of the dense gradient is 0.  Arguments and errors as pp_seq_logprob_bwd
 * (ws_bytes >= pp_workspace_size's logprob). */
pp_status pp_logprob_row_count(const pp_pack_desc* desc, int64_t* n_rows);
pp_status pp_seq_logprob_bwd_rows(const pp_pack_desc* desc, pp_dtype logits_dtype, int vocab,
                                  const void* logits, const int32_t* tokens, const float* dseq,
                                  void* dlogits_rows, int32_t* row_index, void* ws, size_t ws_bytes,
                                  void* hip_stream);

/* Reward-model head (Sec. 2.1: the reward model maps a token sequence to a
 * scalar).  The score of the sequence (prompt b, response k) is
 *   scores[b*K_max+k] = w . hidden[row] + bias,
 * with row the last token of that unpacked sequence in the packed layout:
 * row_start[b] + o_bk + L_bk - 1, or row_start[b] + P_b - 1 when the response
 * is empty (a prompt token sees only the prompt, Sec. 3.2, so its hidden state
 * is the unpacked one).  Slots k >= K_b and sequences without any token get 0.
 * hidden (dev [sumT, hidden_dim], dtype), w (dev [hidden_dim], dtype), scores
 * (dev float [B*K_max]); dot products accumulate in fp32.  The scores go to
 * pp_dpo_loss with logp_ref = NULL for the Bradley-Terry loss.
 * ws_bytes >= pp_rm_workspace_size's bytes. */
pp_status pp_rm_workspace_size(const pp_pack_desc* desc, size_t* bytes);
pp_status pp_rm_scores(const pp_pack_desc* desc, pp_dtype dtype, int hidden_dim, const void* hidden,
                       const void* w, float bias, float* scores, void* ws, size_t ws_bytes,
                       void* hip_stream);

/* Backward of pp_rm_scores for dscores = dL/dscores (dev float [B*K_max]):
 *   dhidden[row] = (sum of dscores over the slots scored at row) * w, and 0 on
 *                  every other row (dev [sumT, hidden_dim], dtype, overwritten);
 *   dw           = sum over scored slots of dscores * hidden[row] (dev float
 *                  [hidden_dim], summed in slot order: deterministic);
 *   *dbias       = sum of dscores over scored slots (dev float; may be NULL).
 * Errors as pp_rm_scores. */
pp_status pp_rm_scores_bwd(const pp_pack_desc* desc, pp_dtype dtype, int hidden_dim, const void* hidden,
                           const void* w, const float* dscores, void* dhidden, float* dw, float* dbias,
                           void* ws, size_t ws_bytes, void* hip_stream);

/* Ranked-pair DPO / Bradley-Terry loss (Sec. 2.1, extended to K > 2).
 * z_k = beta (logp_pol[b,k] - logp_ref[b,k]), or beta logp_pol[b,k] when
 * logp_ref is NULL (reward-model scores).  For every pair a > c of row b's first
 * K_b slots (slot a preferred, Sec. 3.1) the term is softplus(-(z_a - z_c)) =
 * -ln sigmoid(z_a - z_c).  row_loss[b] = mean over the row's K_b(K_b-1)/2 pairs
 * (0 for rows with K_b < 2); *loss = mean of row_loss over rows with K_b >= 2;
 * dlogp_pol[b,k] = d(*loss)/d(logp_pol[b,k]).
 * num_resp is host [B]; logp_pol, logp_ref, loss, row_loss, dlogp_pol are dev
 * float; row_loss and dlogp_pol may be NULL.  ws_bytes >= pp_workspace_size's
 * loss.  PP_ERR_INVALID_ARGUMENT when no row has two responses. */
pp_status pp_dpo_loss(int32_t num_rows, int32_t max_resp, const int32_t* num_resp,
                      const float* logp_pol, const float* logp_ref, float beta, float* loss,
                      float* row_loss, float* dlogp_pol, void* ws, size_t ws_bytes,
                      void* hip_stream);

/* Host-only export of the planner's integer view of a batch (no GPU needed):
 *   position_ids[sumT]  prompt token t -> t, response token j -> P_b + j,
 *                       padding -> 0 (Sec. 3.2: original positions kept);
 *   segment_ids[sumT]   0 prompt, k+1 response k, -1 padding;
 *   tile_class          for every row, its ceil(T_b/block_q) x ceil(T_b/block_k)
 *                       grid of mask tiles, row-major, rows concatenated:
 *                       0 EMPTY (no visible pair), 1 PARTIAL, 2 FULL (every pair
 *                       of the tile, clipped to the row, visible).
 * Any output may be NULL.  tile_class_len must be at least the total grid size
 * when tile_class is not NULL (PP_ERR_INVALID_ARGUMENT otherwise). */
pp_status pp_pack_export(const pp_pack_desc* desc, int block_q, int block_k, int32_t* position_ids,
                         int32_t* segment_ids, uint8_t* tile_class, size_t tile_class_len);

/* Cost and memory accounting of a packed batch against the unpacked layout
 * that repeats each prompt once per response (host only, no GPU needed).
 * "Unpacked" is the K_b sequences (prompt_b, response_bk) of every row;
 * "padded" pads all of them to the longest one.  Rows with K_b = 0 count as
 * their prompt alone on both sides. */
typedef struct pp_pack_stats_t {
  int64_t tokens_packed;      /* sum_b (P_b + sum_k L_bk)                          */
  int64_t tokens_unpacked;    /* sum_b sum_k (P_b + L_bk)                          */
  int64_t tokens_padded;      /* (number of unpacked sequences) x (longest one)    */
  int64_t pairs_packed;       /* visible (query, key) pairs of the packed mask     */
  int64_t pairs_unpacked;     /* causal pairs of the unpacked sequences            */
  int64_t pairs_padded;       /* causal pairs of the padded sequences, padding incl. */
  int64_t pairs_dense_packed; /* causal pairs of each packed row taken whole: the
                                 work of a kernel that cannot skip the blocks that
                                 hide one response from another                   */
  double eq1_cost_ratio;      /* sum_b (P_b + sum_k L_bk)^2 / sum_b K_b (P_b + max_k L_bk)^2,
                                 the cost model of Sec. 3.2.1 summed over rows     */
  double eq1_memory_ratio;    /* the same with first powers (Sec. 3.2.1, linear-
                                 memory attention)                                 */
  int32_t rows_eq1_cheaper;   /* rows that satisfy Eq. (1)                          */
  int32_t rows_with_responses;    /* rows with K_b >= 1                                 */
} pp_pack_stats_t;
pp_status pp_pack_stats(const pp_pack_desc* desc, pp_pack_stats_t* out);

/* Number of tile_class entries pp_pack_export writes for (block_q, block_k). */
pp_status pp_tile_class_len(const pp_pack_desc* desc, int block_q, int block_k, size_t* len);

/* Kernel timing for measurement.  While enabled, each kernel launch of this
 * library is bracketed by two hipEvents recorded on its own stream.
 * pp_timing_count returns how many distinct kernels were timed since the last
 * reset; pp_timing_get waits for their events and returns, for entry idx, the
 * kernel's name (static string), its total elapsed milliseconds and its launch
 * count. */
pp_status pp_timing_enable(int on);
/* Restricts timing to the launches named in `names`, a comma-separated list of
 * the names pp_timing_get reports (e.g. "pp_logprob_rows,pp_attn_fwd"); NULL or
 * "" times every launch again.  The list is copied.  Launches left out get no
 * events, so the work around them runs as it would untimed. */
pp_status pp_timing_select(const char* names);
pp_status pp_timing_reset(void);
int pp_timing_count(void);
pp_status pp_timing_get(int idx, const char** name, double* total_ms, int64_t* launches);

const char* pp_status_string(pp_status status);
const char* pp_last_error(void);
/* ABI version: major * 10000 + minor * 100 + patch. */
int pp_version(void);
/* Identity of the sources this library was built from: the hex sha256 over the
 * library's source files and this header (names and contents), fixed at build
 * time, so a caller can tell a library built from other sources.  Static string. */
const char* pp_build_id(void);

#ifdef __cplusplus
}
#endif

#endif /* PP_ATTN_H */
