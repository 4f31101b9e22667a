/*
 * alr.h -- C ABI of the anchor-branched greedy-rollout library (gfx950 / MI355X).
 *
 * The library computes, for a fixed corpus and a set of anchor positions, the
 * target model's greedy continuation of every anchor's prefix, one draft block
 * long: Eq. 3 of Sec. 3.2 ("Labels from the target's rollout").  The structure
 * is the one App. A ("Training Configuration", "Rollout implementation")
 * describes.  alr_prefill runs the decoder once over each corpus sequence and
 * keeps its keys and values as a cache that every anchor of that sequence
 * reads.  alr_rollout then advances all anchors by one token per step, as one
 * batch.  At each step an anchor's query is normalised in one softmax over two
 * key sets: the cached corpus entries at positions up to the anchor, and the
 * entries its own earlier rollout steps produced.  The second set lives in a
 * buffer private to the anchor, so no corpus entry is duplicated per anchor.
 * The next-token distribution comes from the final RMSNorm and the output
 * head; the greedy pick is the lowest id among equal maxima; the residual
 * stream after chosen layers is returned as features.
 *
 * Slot convention.  Slot s (0 <= s < block) of anchor a sits at position a+s.
 * Its input token is the corpus token x_a for s = 0 and the token fed after
 * slot s-1 otherwise.  It outputs log p(. | x_{<=a}, y_1..y_s) over the whole
 * vocabulary (the paper's label for draft slot k = s+1), its greedy token
 * y_{s+1}, and the outputs of the feature layers at position a+s.
 *
 * Model.  Llama-style decoder: per layer h += Wo Attn(RoPE(Wq n1), RoPE(Wk n1),
 * Wv n1) with n1 = RMSNorm(h), then h += Wd (SiLU(Wg n2) * Wu n2) with
 * n2 = RMSNorm(h); RMSNorm(x) = x g / sqrt(mean(x^2) + eps); grouped-query
 * attention maps query head j to key/value head j / (n_heads/n_kv_heads);
 * scores are scaled by 1/sqrt(head_dim); RoPE rotates the pairs
 * (i, i + head_dim/2) by pos * rope_base^(-2i/head_dim).
 *
 * Precision.  ALR_F32: all storage and arithmetic in fp32.  ALR_BF16: weights
 * and GEMM operands (RMSNorm outputs, q/k after RoPE, v, attention output,
 * SwiGLU output) are bf16; accumulation, residual stream, softmax statistics
 * and logits are fp32.  Log-probabilities and features are always returned in
 * fp32.
 *
 * Operand sizes (ALR_BF16).  The GEMM kernels address their operands with
 * 32-bit byte offsets, so every activation operand, max(max_tokens,
 * max_anchors) rows of max(d_model, d_ffn, n_heads*head_dim) bf16 values, and
 * every weight matrix (vocab x d_model, 2*d_ffn x d_model, ...) must be smaller
 * than 4 GiB; otherwise alr_create returns ALR_E_UNSUPPORTED and
 * alr_workspace_bytes returns 0.
 *
 * Memory and ownership.  All device memory is owned by the caller: weights,
 * inputs, outputs and one workspace whose size alr_workspace_bytes() gives.
 * The library allocates no device memory (its code object holds the fixed
 * scratch array of alr_rollout_topk_noalloc; opt-in rollout graphs hold the
 * runtime's resources, see alr_set_rollout_graphs).  alr_create copies (repacks) the
 * weights into the workspace, so the weight buffers may be freed after it
 * returns.  The shared key/value cache lives in the workspace and stays valid
 * until the next alr_prefill on the same context.
 *
 * Execution.  Every compute call only enqueues work on the given stream and
 * returns; results are valid once the stream has been synchronised.  A context
 * is not thread-safe: use one context per host thread and stream.  Errors are
 * reported through the return code; nothing is thrown across the ABI.  All
 * argument checks happen on the host before anything is enqueued, so a call
 * that returns an error has launched nothing.  alr_last_error() gives a
 * message for the last failing call on a context.
 */
#ifndef ALR_H
#define ALR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ALR_OK = 0,
  ALR_E_INVALID_ARG = 1,  /* null pointer, non-positive count, bad config field  */
  ALR_E_OUT_OF_RANGE = 2, /* anchor, sequence, token or position outside bounds  */
  ALR_E_WORKSPACE = 3,    /* workspace smaller than alr_workspace_bytes() says   */
  ALR_E_STATE = 4,        /* rollout before any prefill                           */
  ALR_E_UNSUPPORTED = 5,  /* shape the kernels do not handle (see alr_config)     */
  ALR_E_HIP = 6           /* HIP runtime error; alr_last_error() has its text     */
} alr_status;

typedef enum { ALR_F32 = 0, ALR_BF16 = 1 } alr_dtype;

#define ALR_MAX_FEAT 8

/* Model shape.  Requirements checked by every entry point:
 *   n_layers >= 0; d_model, d_ffn, n_heads*head_dim and n_kv_heads*head_dim are
 *   multiples of 64; head_dim is even and <= 256; n_heads % n_kv_heads == 0;
 *   (n_heads*head_dim/2) and (n_kv_heads*head_dim/2) are multiples of 32;
 *   vocab is a multiple of 64; 0 <= feat_layers[i] < n_layers;
 *   max_pos >= 1 bounds every position a slot may reach (a + block - 1), on
 *   every position axis.
 *   mrope_sections: multimodal RoPE (App. A, "Rollout implementation": the
 *   three M-RoPE axes advance together).  The head_dim/2 rotary frequencies
 *   are split into consecutive runs of mrope_sections[0], [1], [2] driven by the
 *   t, h and w positions of a token; all zero = plain RoPE on one position
 *   axis.  Otherwise each >= 0 and their sum == head_dim / 2. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
  float rms_eps, rope_base;
  int32_t dtype;   /* alr_dtype */
  int32_t max_pos;
  int32_t n_feat;  /* 0 .. ALR_MAX_FEAT */
  int32_t feat_layers[ALR_MAX_FEAT];
  int32_t mrope_sections[3];
} alr_config;

/* Device pointers to the weights, element type given by alr_config.dtype
 * (float for ALR_F32, bf16 bit patterns for ALR_BF16), row-major, [out, in]
 * layout of a linear map y = W x.  The per-layer fields are HOST arrays of
 * n_layers DEVICE pointers.  Shapes: tok_embed and lm_head [vocab, d_model];
 * final_norm, attn_norm[l], ffn_norm[l] [d_model]; wq [n_heads*head_dim,
 * d_model]; wk, wv [n_kv_heads*head_dim, d_model]; wo [d_model,
 * n_heads*head_dim]; w_gate, w_up [d_ffn, d_model]; w_down [d_model, d_ffn]. */
typedef struct {
  const void* tok_embed;
  const void* final_norm;
  const void* lm_head;
  const void* const* attn_norm;
  const void* const* wq;
  const void* const* wk;
  const void* const* wv;
  const void* const* wo;
  const void* const* ffn_norm;
  const void* const* w_gate;
  const void* const* w_up;
  const void* const* w_down;
} alr_weights;

typedef struct alr_ctx alr_ctx;
typedef void* alr_stream; /* a hipStream_t; NULL is the null stream */

/* Capacity limits a context is created for. */
typedef struct {
  int32_t max_tokens;  /* total corpus tokens over all sequences of one prefill */
  int32_t max_seqs;    /* sequences per prefill                                 */
  int32_t max_anchors; /* anchors per rollout                                    */
  int32_t max_block;   /* slots per anchor (block)                               */
} alr_limits;

/* Bytes of device workspace a context with this config and these limits needs.
 * Returns 0 if the config or limits are invalid or a GEMM operand would reach
 * 4 GiB (see "Operand sizes").  Host only, no GPU needed. */
size_t alr_workspace_bytes(const alr_config* cfg, const alr_limits* lim);

/* Validate cfg (host only, no GPU needed).  On failure writes a message into
 * msg (if msg_len > 0) and returns the status alr_create would return. */
alr_status alr_check_config(const alr_config* cfg, char* msg, size_t msg_len);

/* Validate a rollout request against a prefill of n_seq sequences of lengths
 * seq_len[] (host arrays) and the limits (host only, no GPU needed).  Same
 * checks and status codes as alr_rollout. */
alr_status alr_check_rollout(const alr_config* cfg, const alr_limits* lim, int32_t n_seq,
                             const int32_t* seq_len, int32_t n_anchor,
                             const int32_t* anchor_seq, const int32_t* anchor_pos,
                             int32_t block, char* msg, size_t msg_len);

/* Create a context.  workspace: device buffer of ws_bytes >= alr_workspace_bytes
 * (256-byte aligned); the weights are repacked into it on `stream`.  On success
 * *out receives the context.  Synchronises `stream` before returning. */
alr_status alr_create(const alr_config* cfg, const alr_weights* w, const alr_limits* lim,
                      void* workspace, size_t ws_bytes, alr_stream stream, alr_ctx** out);

/* Forward pass over n_seq corpus sequences (the shared prefix of every anchor).
 *   seq_len    HOST [n_seq], each >= 1 and <= max_pos; sum <= max_tokens.
 *   tokens     DEVICE int32 [sum seq_len], sequences concatenated; ids < vocab.
 *   embeds     DEVICE [sum seq_len, d_model] in the weight dtype, or NULL: rows
 *              used instead of the token embedding where embed_mask is nonzero.
 *   embed_mask DEVICE uint8 [sum seq_len], or NULL (both or neither).
 *   feats_out  DEVICE fp32 [sum seq_len, n_feat, d_model] or NULL: residual
 *              stream after each feature layer at every corpus position.
 * Token ids are not range-checked on the device: ids outside [0, vocab) give
 * undefined results, so the caller must validate them. */
alr_status alr_prefill(alr_ctx* ctx, int32_t n_seq, const int32_t* seq_len,
                       const int32_t* tokens, const void* embeds,
                       const uint8_t* embed_mask, float* feats_out, alr_stream stream);

/* alr_prefill with explicit token positions (RoPE / M-RoPE).
 *   positions  HOST int32 [sum seq_len][3]: (t, h, w) position of every corpus
 *              token, each in [0, max_pos); or NULL for the token's index in its
 *              sequence on every axis (then identical to alr_prefill).  With
 *              plain RoPE (mrope_sections all zero) only the t column is used.
 * A rollout slot s of an anchor sits at the anchor token's position plus s on
 * every axis, so each axis value + block - 1 must stay below max_pos (checked
 * by the rollout calls).  Other arguments and checks as in alr_prefill. */
alr_status alr_prefill_positions(alr_ctx* ctx, int32_t n_seq, const int32_t* seq_len,
                                 const int32_t* tokens, const int32_t* positions,
                                 const void* embeds, const uint8_t* embed_mask, float* feats_out,
                                 alr_stream stream);

/* Greedy rollout of `block` slots from every anchor of the last prefill.
 *   n_anchor   in [1, max_anchors] and block in [1, max_block]; an empty
 *              request is ALR_E_INVALID_ARG (nothing is launched).
 *   anchor_seq, anchor_pos  HOST int32 [n_anchor]: sequence index and position;
 *              0 <= anchor_pos < seq_len[anchor_seq]; anchor_pos + block - 1 <
 *              max_pos.  Any order; duplicates allowed (identical outputs).
 *   forced     DEVICE int32 [n_anchor, block] or NULL: where forced[i,s] >= 0 it
 *              is fed to slot s+1 instead of the greedy token (column block-1
 *              is ignored); values must be < vocab.
 *   tokens_out DEVICE int32 [n_anchor, block]: greedy token of every slot.
 *   logprobs_out DEVICE fp32 [n_anchor, block, vocab]: log-softmax of each slot.
 *   feats_out  DEVICE fp32 [n_anchor, block, n_feat, d_model] or NULL.
 * Outputs are in the caller's anchor order. */
alr_status alr_rollout(alr_ctx* ctx, int32_t n_anchor, const int32_t* anchor_seq,
                       const int32_t* anchor_pos, int32_t block, const int32_t* forced,
                       int32_t* tokens_out, float* logprobs_out, float* feats_out,
                       alr_stream stream);

/* Number of most probable tokens a label keeps (the paper's distillation
 * loss: top 8 probabilities plus one bucket for the remaining mass). */
#define ALR_TOPK 8

/* Greedy rollout with labels in the paper's loss format (Sec. 3.1, Eq. 1; App.
 * A, the loss row of the training table and "Rollout implementation": the 8
 * most probable tokens of each slot plus the remaining mass).  Arguments as in
 * alr_rollout, plus:
 *   top_ids_out  DEVICE int32 [n_anchor, block, ALR_TOPK]: token ids ranked by
 *                decreasing probability, equal probabilities by increasing id
 *                (entry 0 is the greedy token).
 *   top_logp_out DEVICE fp32 [n_anchor, block, ALR_TOPK]: their log-probs.
 *   tail_out     DEVICE fp32 [n_anchor, block]: probability summed over every
 *                other token (summed directly, not as 1 - top mass).
 *   logprobs_out DEVICE fp32 [n_anchor, block, vocab] or NULL: the full
 *                log-softmax as in alr_rollout.  When NULL the logits of each
 *                step go to workspace rows and only the compact labels (4 +
 *                68 bytes per slot) reach the caller.
 * Tokens, features and the top-8 labels are identical whether or not the full
 * log-probs are requested.  Same checks and status codes as alr_rollout. */
alr_status alr_rollout_topk(alr_ctx* ctx, int32_t n_anchor, const int32_t* anchor_seq,
                            const int32_t* anchor_pos, int32_t block, const int32_t* forced,
                            int32_t* tokens_out, int32_t* top_ids_out, float* top_logp_out,
                            float* tail_out, float* logprobs_out, float* feats_out,
                            alr_stream stream);

/* Bytes of the fixed device array behind alr_rollout_topk_noalloc (64 MiB). */
#define ALR_NOALLOC_SCRATCH_BYTES (64u << 20)

/* alr_rollout_topk for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same arguments, checks and results as alr_rollout_topk with
 * logprobs_out = NULL, but the per-step scratch -- each step's fp32 logit rows
 * [n_anchor, vocab] and their per-64-column log-sum-exp partials [n_anchor,
 * vocab/64] of 8 bytes -- lives in a fixed array of ALR_NOALLOC_SCRATCH_BYTES
 * that the library holds on every device it runs on until the process ends
 * (its address is looked up once per device by alr_create), not in the
 * context's workspace.  The call allocates nothing and frees nothing.
 *   Limit: 256-byte-aligned n_anchor * vocab * 4 plus n_anchor * (vocab/64) * 8
 *   must fit in the array (at most 126 anchors at vocab 128256, 508 at 32000);
 *   larger requests return ALR_E_WORKSPACE before anything is enqueued.
 * Every entry of the scratch a call reads is first written by that call, so
 * nothing needs clearing between calls.  All calls on one device share the one
 * array: calls whose execution overlaps on a device (other streams, other
 * contexts, other threads) race on it and must be serialised by the caller. */
alr_status alr_rollout_topk_noalloc(alr_ctx* ctx, int32_t n_anchor, const int32_t* anchor_seq,
                                    const int32_t* anchor_pos, int32_t block,
                                    const int32_t* forced, int32_t* tokens_out,
                                    int32_t* top_ids_out, float* top_logp_out, float* tail_out,
                                    float* feats_out, alr_stream stream);

/* Rollout launch graphs.  A launch mechanism, not an operation of the method:
 * results are bit-identical with graphs on or off.  Off by default (then
 * nothing is allocated after alr_create).  When turned on, alr_rollout and
 * alr_rollout_topk record their kernel launches (one per layer step, thousands
 * per call) into a HIP graph the first time a combination of n_anchor, block,
 * the size of the decode attention work list, `forced`, `feats_out` and every
 * output pointer is seen, and replay that graph for later calls with the same
 * combination.  Anchors, positions and attention plans are uploaded by every
 * call before its graph runs, so the anchors themselves may differ between
 * replays, and a new prefill leaves the graphs valid.  The graphs run on a
 * stream of the context's own that first waits for the work already on the
 * caller's `stream`; later work on `stream` waits for the graph.  Up to 4
 * graphs are kept per context (the least recently used is dropped, after the
 * context's stream has drained); the first call of a combination costs the
 * recording and instantiation on the host.
 * Not used by alr_rollout_topk_noalloc (instantiation allocates), while a
 * launch site of the rollout is being timed (alr_profile_start with a rollout
 * or output-head site), or when `stream` is itself being captured (the
 * launches then go into the caller's own graph).
 *   enable: 1 on (the first time, creates the context's stream and two events;
 *           each recorded graph holds the runtime's resources for its
 *           instantiation until it is dropped), 0 off (drops the cached graphs).
 * Errors: ALR_E_INVALID_ARG for a NULL ctx or another value of enable; ALR_E_HIP
 * if the stream or events cannot be created (graphs stay off). */
alr_status alr_set_rollout_graphs(alr_ctx* ctx, int32_t enable);

/* Fixed-corpus distillation labels and erase gates (Sec. 3.1: the KD labels
 * pi_{a,k} = p_T(. | x_{<a+k}), and Eq. 2, the survival gate with its hard
 * variant), read from the last prefill's final normalised rows through the
 * output head.  Index s = 0 .. block-1 of anchor a is the paper's slot k = s+1
 * at position a+s; it is valid while a + s <= seq_len - 1.
 *   anchor_seq, anchor_pos  HOST int32 [n_anchor] as in alr_rollout
 *              (anchor_pos + block - 1 < max_pos; slots past the sequence end
 *              are reported invalid, not rejected).
 *   argmax_out   DEVICE int32 [n_anchor, block]: greedy token of the label
 *                (ties -> lower id), -1 for an invalid index.
 *   top_ids_out, top_logp_out, tail_out: as in alr_rollout_topk, or all NULL;
 *                invalid indices get ids -1, log-probs -inf, tail 0.
 *   logprobs_out DEVICE fp32 [n_anchor, block, vocab] or NULL (rows of -inf
 *                at invalid indices).  At least one label form must be given.
 *   corpus_logp_out DEVICE fp32 [n_anchor, block]: log p_T(x_{a+s+1} |
 *                x_{<=a+s}); nan when a+s+1 is past the end or holds a given
 *                input row (alr_prefill's embeds) instead of a token.
 *   gate_soft_out DEVICE fp32 [n_anchor, block]: g = exp(sum over earlier
 *                indices of corpus_logp); 1 at index 0; 0 at invalid indices
 *                and after an undefined factor.
 *   gate_hard_out DEVICE fp32 [n_anchor, block]: product over earlier indices
 *                of [argmax == corpus token], same conventions.
 * Outputs are in the caller's anchor order.  Same host checks as
 * alr_rollout. */
alr_status alr_corpus_labels(alr_ctx* ctx, int32_t n_anchor, const int32_t* anchor_seq,
                             const int32_t* anchor_pos, int32_t block, int32_t* argmax_out,
                             int32_t* top_ids_out, float* top_logp_out, float* tail_out,
                             float* logprobs_out, float* corpus_logp_out, float* gate_soft_out,
                             float* gate_hard_out, alr_stream stream);

/* Secondary blocks of in-rollout anchors (Sec. 3.2, Eq. 4), gathered from the
 * outputs of alr_rollout_topk over n_primary primary blocks of `block` slots
 * (no target computation).  Secondary q sits at offset j = sec_offset[q] of
 * primary p = sec_primary[q] (HOST arrays [n_secondary]; 0 <= p < n_primary,
 * 1 <= j <= block-1; the paper draws j uniformly from 2 .. K-1 with K =
 * block-1).  Inputs tokens [n_primary, block], top_ids/top_logp
 * [n_primary, block, ALR_TOPK], tail [n_primary, block] are DEVICE arrays.
 *   token0_out  DEVICE int32 [n_secondary]: slot-0 token y*_j = tokens[p, j-1];
 *               the block's slot 0 sits at position anchor_pos[p] + j and its
 *               context is the prefix up to the anchor plus the primary's
 *               rollout positions 1 .. j-1 (their features are the primary's
 *               feature rows 1 .. j-1).
 *   top_ids_out, top_logp_out [n_secondary, block, ALR_TOPK], tail_out
 *               [n_secondary, block]: index s' holds the primary's labels at
 *               index j + s' (paper slot j + k with k = s'+1) while j + s' <=
 *               block-1, else ids -1, log-probs -inf, tail 0.
 *   weight_out  DEVICE fp32 [n_secondary, block]: w_k = exp(-(k-1)/gamma)
 *               where j + k <= block-1 and the primary had not ended before
 *               the inherited slot (no eos_id among tokens[p, 0 .. j+s'-1];
 *               eos_id < 0: no early end), else 0 (unsupervised tail).
 * gamma > 0.  n_secondary = 0 is a no-op. */
alr_status alr_ira_assemble(alr_ctx* ctx, int32_t n_primary, int32_t block,
                            const int32_t* tokens, const int32_t* top_ids, const float* top_logp,
                            const float* tail, int32_t n_secondary, const int32_t* sec_primary,
                            const int32_t* sec_offset, float gamma, int32_t eos_id,
                            int32_t* token0_out, int32_t* top_ids_out, float* top_logp_out,
                            float* tail_out, float* weight_out, alr_stream stream);

/* Slot weights of ALR blocks (Eq. 1 envelope; Sec. 3.2: slots that follow an
 * early end of the rollout are masked): weight_out[i, s] = exp(-s / gamma)
 * while no token equal to eos_id occurs in tokens[i, 0 .. s-1] (the tokens fed
 * before index s), else 0.  eos_id < 0: no early end.  tokens DEVICE int32
 * [n, block] (e.g. alr_rollout's tokens_out), weight_out DEVICE fp32 [n, block];
 * n >= 0, block >= 1, gamma > 0. */
alr_status alr_slot_weights(alr_ctx* ctx, int32_t n, int32_t block, const int32_t* tokens,
                            int32_t eos_id, float gamma, float* weight_out, alr_stream stream);

/* Message of the last failing call on ctx ("" if none); ctx may be NULL, then
 * the message of the last failing alr_create in this thread is returned. */
const char* alr_last_error(const alr_ctx* ctx);

/* Static name of a status code. */
const char* alr_status_string(alr_status st);

/* Destroy a context (host memory only; the workspace stays the caller's). */
void alr_destroy(alr_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* ALR_H */
