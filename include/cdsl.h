/*
 * cdsl.h -- C ABI of the CDSL lookahead-step library for MI355X (gfx950).
 *
 * One lookahead step of constrained decoding with speculative lookaheads
 * (Nakshatri et al., "Constrained Decoding with Speculative Lookaheads"):
 *
 *   cdsl_prefill   prompt forward of both decoders, first beam heads
 *   cdsl_rollout   the draft model extends each of the k beam heads by d
 *                  greedy tokens (Sec. 3.2.1; Alg. 1, drafting loop)
 *   cdsl_verify    the target model scores all k*d lookahead tokens in one
 *                  tree-masked forward pass; per-token log-probs, target
 *                  argmax, hard-rejection counts and beam scores
 *                  (Sec. 3.2.2; Alg. 1, verification and rejection loops)
 *   cdsl_reward_*  the task reward R per beam (Sec. 3.2.2, validation by R;
 *                  Sec. 4.1 concept counting; a linear head stands in for the
 *                  semantic reward model)
 *   cdsl_select    the beam maximising score + alpha * reward (Alg. 2, the
 *                  reward argmax; alpha = +inf is exactly that rule)
 *   cdsl_commit    emits the selected beam's head plus its accepted tokens
 *                  (S1 action of Sec. 3.2.3, no bonus token), makes them part
 *                  of the shared prefix and produces the next beam heads
 *   cdsl_rollout_keep, cdsl_verify_soft, cdsl_commit_soft
 *                  the same step with speculative sampling's soft rejection
 *                  (Sec. 3.2.2) in place of the argmax test
 *   cdsl_draft_prefix, cdsl_verify_prefix(_soft), cdsl_reward_keywords_prefix,
 *   cdsl_commit_prefix
 *                  one iteration of the paper's Alg. 1 itself: d draft
 *                  tokens from the prefix (no beam head), their verification
 *                  p_1..p_d, the reward of the accepted tokens and the commit
 *                  of x_1..x_n
 *   cdsl_rollout_with, cdsl_reward_keywords_upto, cdsl_controller_states,
 *   cdsl_select_first, cdsl_commit_heads
 *                  the rest of Alg. 1 (the state decision between S1..S4 and
 *                  the one-token actions of Step-1 / Step-2) and its
 *                  baselines CDLH (target-rolled lookaheads) and CDLH-appx.
 *                  (draft-rolled, unverified)
 *
 * Conventions
 *   - Every call returns CDSL_OK (0) or a negative CDSL_E* code; the message
 *     of the last failure is available from cdsl_last_error(ctx).  No C++
 *     exception crosses this boundary.  Arguments are checked on the host
 *     before anything is launched; a call that fails that check has launched
 *     nothing.  The commits check the selected beams (and acceptance counts)
 *     on the device first: a commit that fails with EINVAL or ERANGE leaves
 *     the prefix, its generated tokens and next_beams as they were.
 *   - A context that was destroyed, or a prefix handle that was freed, is
 *     refused with CDSL_ESTATE by every call that takes it (the library
 *     keeps a registry of live handles).
 *   - Token ids must lie in [0, V).  Ids that reach the device (prompt
 *     tokens, lookaheads passed to a verification) are checked there: an id
 *     outside the range is read as a clamped id and makes the next call that
 *     synchronises (cdsl_prefill, the commits) fail with CDSL_EINVAL before
 *     it changes anything; the log-probs gathered at such an id are NaN.
 *   - Pointer arguments are DEVICE pointers unless the name ends in _host.
 *     They are owned by the caller and only read/written during the call
 *     (device work is ordered on the context's stream).
 *   - Calls are asynchronous on the stream given to cdsl_init, except
 *     cdsl_commit, cdsl_commit_soft and cdsl_commit_heads, which
 *     synchronise that stream once (they must learn how many tokens each
 *     prompt emitted to manage the KV blocks).
 *   - Shapes are row-major, innermost last.  Token ids are int32 in [0, V).
 *   - Nothing is allocated after cdsl_init except by cdsl_prefill (the
 *     prefix handle's bookkeeping; KV blocks come from the pool sized at
 *     init).  A context is not thread-safe.
 */
#ifndef CDSL_H
#define CDSL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  CDSL_OK = 0,
  CDSL_EINVAL = -1,   /* bad argument (shape, pointer, value)            */
  CDSL_ERANGE = -2,   /* beyond the limits given at init                 */
  CDSL_ENOMEM = -3,   /* device memory or KV pool exhausted              */
  CDSL_EDEVICE = -4,  /* a HIP runtime call failed                       */
  CDSL_ESTATE = -5    /* call out of order (e.g. verify before rollout)  */
};

enum { CDSL_F32 = 0, CDSL_BF16 = 1 };

/* Shape of one Llama-style decoder: pre-norm RMSNorm, rotary embedding
 * (rotate-half pairing, 0-based positions), grouped-query attention,
 * SwiGLU MLP, no biases, untied LM head.  head_dim = d_model / n_heads and
 * must be 32, 64 or 128 (64 or 128 for CDSL_BF16); d_model <= 8192. */
typedef struct cdsl_model_config {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t ffn_dim;
  int32_t vocab;
  float rope_theta;
  float rms_eps;
  int32_t dtype;      /* CDSL_F32 or CDSL_BF16: the weight type.  Activations
                         and KV values are fp32 either way (CDSL_BF16 keeps
                         them as bf16 hi + lo pairs where MFMAs read them). */
} cdsl_model_config;

/* Weights of one decoder, device pointers in the dtype of cfg (norm gains
 * are always fp32).  Matrices are [out_features, in_features] row-major.
 * layer_ptrs points to a HOST array of n_layers * 9 device pointers, per
 * layer in this order:
 *   attn_norm[D], wq[H*hd, D], wk[Hkv*hd, D], wv[Hkv*hd, D], wo[D, H*hd],
 *   mlp_norm[D], w_gate[F, D], w_up[F, D], w_down[D, F]
 * Ownership: tok_emb, lm_head, the norm gains, wo and w_down are BORROWED --
 * the kernels read them in place, so the caller keeps them alive and
 * unchanged until cdsl_destroy; every weight pointer must be 16-byte aligned
 * (CDSL_EINVAL otherwise).  wq/wk/wv and w_gate/w_up are re-packed at
 * cdsl_init into library-owned copies (q/k/v concatenated into one matrix,
 * gate/up interleaved in groups of 16 rows, so each fused projection reads
 * one contiguous weight); the caller's wq, wk, wv, w_gate and w_up are not
 * referenced after cdsl_init returns. */
typedef struct cdsl_model {
  cdsl_model_config cfg;
  const void* tok_emb;              /* [V, D]   */
  const void* final_norm;           /* [D] fp32 */
  const void* lm_head;              /* [V, D]   */
  const void* const* layer_ptrs;    /* host array, n_layers * 9 entries */
} cdsl_model;

/* Capacity limits; every later call is checked against them. */
typedef struct cdsl_limits {
  int32_t max_batch;     /* prompts per prefix handle                    */
  int32_t max_ctx;       /* prompt + generated tokens per prompt         */
  int32_t max_k;         /* beams (<= 16)                                */
  int32_t max_d;         /* lookahead depth (<= 32)                      */
  int32_t max_prompt;    /* longest prompt passed to cdsl_prefill        */
  int32_t max_prefixes;  /* prefix handles alive at once                 */
} cdsl_limits;

typedef struct cdsl_ctx cdsl_ctx;
typedef struct cdsl_prefix cdsl_prefix;

/* Create a context for a draft/target pair (same vocabulary and dtype, as
 * speculative decoding requires models of one family, Sec. 4.2).  stream is
 * a hipStream_t (NULL = the default stream).  Allocates the re-packed
 * q/k/v and gate/up weights, the paged KV pools of both models, the rotary
 * tables and all workspaces; the other weights are borrowed (see
 * cdsl_model).  Errors: EINVAL (shapes, vocab or dtype mismatch, a weight
 * pointer not 16-byte aligned), ENOMEM (also a KV pool beyond the free
 * device memory, refused before it is allocated), EDEVICE. */
int cdsl_init(const cdsl_model* draft, const cdsl_model* target,
              const cdsl_limits* limits, void* stream, cdsl_ctx** out);

/* Prompt forward of both models over tokens[B, L] (device int32), writing
 * the shared-prefix KV blocks of a new prefix handle (*out, library-owned,
 * released by cdsl_free_prefix).  Writes the first beam heads: beams[B, k]
 * = the k most likely next tokens of the target (log-prob descending, token
 * id ascending on ties) and head_lp[B, k] their log-probs (fp32) -- the
 * top-k candidates of the lookahead-heuristic algorithm (Sec. 2.1 and the
 * appendix algorithm; Step-2 of Sec. 3.2.3 takes the same set).
 * Synchronises the context stream.  Errors: EINVAL (also a prompt token
 * outside [0, V); no handle is created), ERANGE (B, L or k beyond limits),
 * ENOMEM (KV pool). */
int cdsl_prefill(cdsl_ctx* ctx, const int32_t* tokens, int32_t B, int32_t L,
                 int32_t k, cdsl_prefix** out, int32_t* beams, float* head_lp);

/* Draft rollout.  For every prompt b and beam i, feeds the head
 * beams[b, i] and then its own greedy outputs to the draft model for d
 * steps: lookaheads[b, i, 0] = beams[b, i] and lookaheads[b, i, j] =
 * argmax of the draft at step j (lowest id on ties), j = 1..d.
 * lookaheads is [B, k, d+1] int32.  All beams of a prompt read that
 * prompt's prefix KV blocks once; each beam writes its own suffix blocks.
 * Errors: EINVAL, ERANGE (k, d). */
int cdsl_rollout(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* beams,
                 int32_t k, int32_t d, int32_t* lookaheads);

/* cdsl_rollout with a choice of roller: 0 = the draft model (as
 * cdsl_rollout), 1 = the target model.  The target rolls the lookaheads of
 * the lookahead-heuristic baseline (CDLH: Sec. 2.1 and the appendix
 * algorithm, lookaheads generated by M_p); the draft rolls those of its
 * approximate variant (CDLH-appx., Sec. 3.1).  Same layout, ordering and
 * errors as cdsl_rollout, plus EINVAL for another roller. */
int cdsl_rollout_with(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* beams,
                      int32_t k, int32_t d, int32_t roller, int32_t* lookaheads);

/* Target verification of lookaheads[B, k, d+1] (any values, not only those
 * of the last rollout: the call depends on its arguments and the prefix
 * only).  Feeds rows (i, j) = lookaheads[b, i, j], j = 0..d-1, at positions
 * L_b + j in ONE forward pass; row (i, j) attends to the whole prefix and to
 * rows (i, 0..j) of its own beam.  Outputs (device):
 *   logprobs[B,k,d]       log p_j(x_{i,j}) where p_j is row (i, j-1)'s
 *                         distribution and x_{i,j} = lookaheads[b, i, j]
 *   target_argmax[B,k,d]  argmax of row (i, j-1) (lowest id on ties)
 *   n_accept[B,k]         leading j with target_argmax == x (hard rejection)
 *   scores[B,k]           head_lp[b, i] + sum_j logprobs[b, i, j]
 *   row_topk_ids[B,k,d,k], row_topk_lp[B,k,d,k]  top-k of every fed row
 *   hidden[B,k,D]         fp32 final-normed hidden state of row (i, d-1),
 *                         or NULL if not wanted
 * Errors: EINVAL, ERANGE. */
int cdsl_verify(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                int32_t k, int32_t d, const float* head_lp, float* logprobs,
                int32_t* target_argmax, int32_t* n_accept, float* scores,
                int32_t* row_topk_ids, float* row_topk_lp, float* hidden);

/* cdsl_verify with a top-k width kk (1..max_k) that differs from the beam
 * count: row_topk_ids / row_topk_lp are [B, k, d, kk].  The paper's Alg. 1
 * drafts one sequence (k = 1) but its Step-2 needs the k best target tokens
 * after the accepted ones (Sec. 3.2.3).  cdsl_verify is kk = k.  Errors as
 * cdsl_verify, plus ERANGE for kk. */
int cdsl_verify_kk(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                   int32_t k, int32_t d, int32_t kk, const float* head_lp,
                   float* logprobs, int32_t* target_argmax, int32_t* n_accept,
                   float* scores, int32_t* row_topk_ids, float* row_topk_lp,
                   float* hidden);

/* Keyword reward: for every beam, the number of distinct keywords of
 * keywords[b, 0..n_kw) that occur in generated-so-far + lookaheads[b, i,
 * 0..d] (the prompt is not searched).  With normalize != 0 the count is
 * divided by the number of distinct keywords (concept coverage, Sec. 4.1).
 * reward is [B, k] fp32.  Errors: EINVAL. */
int cdsl_reward_keywords(cdsl_ctx* ctx, cdsl_prefix* prefix,
                         const int32_t* lookaheads, int32_t k, int32_t d,
                         const int32_t* keywords, int32_t n_kw, int32_t normalize,
                         float* reward);

/* cdsl_reward_keywords over a shorter window: generated-so-far + the head
 * of beam i + its first upto[b, i] lookahead tokens (clamped to 0..d);
 * upto [B, k] int32 on the device, or NULL for all d.  With upto = the
 * verify's n_accept this is the reward of the accepted tokens, R(x_1..x_n)
 * in the rejection step of the paper's Alg. 1 (Sec. 3.2.2-3.2.3).  Errors
 * as cdsl_reward_keywords. */
int cdsl_reward_keywords_upto(cdsl_ctx* ctx, cdsl_prefix* prefix,
                              const int32_t* lookaheads, int32_t k, int32_t d,
                              const int32_t* upto, const int32_t* keywords,
                              int32_t n_kw, int32_t normalize, float* reward);

/* Linear reward head: reward[b, i] = dot(w, hidden[b, i, :]), hidden as
 * written by cdsl_verify, w [D] fp32.  Errors: EINVAL. */
int cdsl_reward_linear(cdsl_ctx* ctx, const float* hidden, const float* w,
                       int32_t B, int32_t k, int32_t D, float* reward);

/* beam[b] = argmax_i (scores[b, i] + alpha * reward[b, i]), lowest i on
 * ties; alpha = +INFINITY selects on the reward alone.  A NaN score or
 * reward makes beam[b] = -1, which cdsl_commit reports as EINVAL. */
int cdsl_select(cdsl_ctx* ctx, const float* scores, const float* reward,
                float alpha, int32_t B, int32_t k, int32_t* beam);

/* Speculative sampling (soft rejection, Sec. 3.2.2) replaces the argmax
 * test of the verification.  The three calls below are used in place of
 * cdsl_rollout, cdsl_verify and cdsl_commit (reward and selection are
 * unchanged); the draft and the target must share one vocabulary V. */

/* cdsl_rollout that also keeps the draft's logits of every draft pass:
 * draft_logits[B, k, d, V] (fp32, device, caller-owned, B*k*d*V*4 bytes;
 * entry (b, i, j) is q_{j+1} of beam i, the distribution its token
 * x_{i,j+1} was drawn from).  The buffer must stay untouched until the
 * matching cdsl_verify_soft.  Errors as cdsl_rollout; ERANGE if d * V
 * exceeds 2^31 - 1. */
int cdsl_rollout_keep(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* beams,
                      int32_t k, int32_t d, int32_t* lookaheads,
                      float* draft_logits);

/* cdsl_verify_kk with speculative sampling's test (kk: top-k width of the
 * row_topk outputs and of the next heads; kk = k for the beam step, k = 1
 * with kk = the beam count for the controller): x_{i,j} is kept while
 * u[b, i, j-1] <= min(1, p_j(x_{i,j}) / q_j(x_{i,j})), and n_accept counts
 * the kept tokens before the first rejection.  u and v are [B, k, d]
 * uniforms in [0, 1) supplied by the caller (the method's random numbers
 * are inputs).  Outputs, beyond those of cdsl_verify (row_topk_ids and
 * row_topk_lp are [B, k, d, kk]):
 *   draft_lp[B, k, d]  log q_j(x_{i,j})
 *   res_ids[B, k, d]   for every fed row, the draw at v from the normalised
 *                      max(0, p_j - q_j) (token ids in ascending order;
 *                      argmax p_j if p_j <= q_j everywhere)
 *   res_lp[B, k, d]    log p_j of that draw.
 * draft_logits must be the buffer of the last cdsl_rollout_keep on this
 * prefix with the same k and d (ESTATE otherwise).  Errors as cdsl_verify;
 * EINVAL if the two models' vocabularies differ. */
int cdsl_verify_soft(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                     int32_t k, int32_t d, int32_t kk, const float* head_lp,
                     const float* draft_logits, const float* u, const float* v,
                     float* logprobs, float* draft_lp, int32_t* target_argmax,
                     int32_t* n_accept, float* scores, int32_t* row_topk_ids,
                     float* row_topk_lp, int32_t* res_ids, float* res_lp,
                     float* hidden);

/* cdsl_commit after cdsl_verify_soft (same k, d, kk).  Emits
 * [c_i*, x_i*,1..n] as cdsl_commit does (no bonus token).  When n < d, the
 * next heads ([B, kk]) are the residual draw res_ids[b, i*, n] (head_lp
 * res_lp) followed by the kk - 1 best tokens of that row's top-kk without
 * it; when n = d they are the target's top-kk after the catch-up, as in
 * cdsl_commit.  Errors as
 * cdsl_commit; ESTATE if the last verification was not soft or used
 * another kk (and cdsl_commit / cdsl_commit_kk return ESTATE after a soft
 * one). */
int cdsl_commit_soft(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                     const int32_t* beam, const int32_t* n_accept,
                     const int32_t* row_topk_ids, const float* row_topk_lp,
                     const int32_t* res_ids, const float* res_lp, int32_t k,
                     int32_t d, int32_t kk, int32_t* emitted_host,
                     int32_t* n_emit_host, int32_t* next_beams,
                     float* next_head_lp);

/* ---- Alg. 1 itself: a lookahead drafted from the prefix (no beam head) ----
 * These calls take one lookahead per prompt (k = 1), laid out [B, d+1]:
 * column 0 is the last token of the prefix (the prompt's last token until
 * something has been generated) and columns 1..d are x_1..x_d. */

/* Alg. 1, drafting loop: x_j = argmax q_j with q_1 = M_q(pfx) and q_j =
 * M_q(pfx + x_1..x_{j-1}) (greedy, lowest id on ties), j = 1..d.  Writes
 * lookaheads[B, d+1] (column 0 as above).  The first of the d draft passes
 * re-feeds the prefix's last token into the lookahead's first suffix slot,
 * so q_1 comes from a pass like the others.  draft_logits: NULL, or [B, d, V]
 * fp32 caller-owned that receives q_1..q_d (for cdsl_verify_prefix_soft;
 * keep it untouched until then).  Errors as cdsl_rollout. */
int cdsl_draft_prefix(cdsl_ctx* ctx, cdsl_prefix* prefix, int32_t d,
                      int32_t* lookaheads, float* draft_logits);

/* Alg. 1, verification (hard rejection): one target pass over the d fed
 * rows [lookaheads[b, 0], x_1..x_{d-1}] at positions L_b - 1 .. L_b + d - 2,
 * so row j-1 gives p_j = M_p(pfx + x_1..x_{j-1}), j = 1..d (p_1 = M_p(pfx)).
 * Outputs (device): logprobs[B, d] = log p_j(x_j), target_argmax[B, d] =
 * argmax p_j, n_accept[B] = the leading j with argmax p_j = x_j (the
 * rejection loop), scores[B] = sum_j logprobs, row_topk_ids / row_topk_lp
 * [B, d, kk] the top-kk of p_1..p_d (row n's are the candidates of Step-2
 * after n accepted tokens).  lookaheads[b, 0] must be the prefix's last
 * token, as cdsl_draft_prefix writes it.  Errors as cdsl_verify_kk. */
int cdsl_verify_prefix(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                       int32_t d, int32_t kk, float* logprobs, int32_t* target_argmax,
                       int32_t* n_accept, float* scores, int32_t* row_topk_ids,
                       float* row_topk_lp);

/* cdsl_verify_prefix with speculative sampling's test in the rejection loop
 * (Sec. 3.2.2; the paper plugs it into Alg. 1's rejection lines): x_j is
 * kept while u[b, j-1] <= min(1, p_j(x_j) / q_j(x_j)), with q_j from the
 * draft_logits of the matching cdsl_draft_prefix.  u, v: [B, d] uniforms in
 * [0, 1).  Also writes draft_lp[B, d] = log q_j(x_j) and, per row, the draw
 * at v from the normalised max(0, p_j - q_j) (res_ids, res_lp [B, d]).
 * Errors as cdsl_verify_soft. */
int cdsl_verify_prefix_soft(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                            int32_t d, int32_t kk, const float* draft_logits,
                            const float* u, const float* v, float* logprobs,
                            float* draft_lp, int32_t* target_argmax, int32_t* n_accept,
                            float* scores, int32_t* row_topk_ids, float* row_topk_lp,
                            int32_t* res_ids, float* res_lp);

/* Alg. 1's reward of the accepted tokens, r = R(x_1..x_n) with the
 * generated-so-far tokens in front (the prompt is not searched): the number
 * (normalize: fraction) of distinct keywords present in generated-so-far +
 * lookaheads[b, 1..upto[b]] (upto [B] device int32, clamped to 0..d; NULL:
 * all d).  reward [B] fp32.  Errors as cdsl_reward_keywords. */
int cdsl_reward_keywords_prefix(cdsl_ctx* ctx, cdsl_prefix* prefix,
                                const int32_t* lookaheads, int32_t d, const int32_t* upto,
                                const int32_t* keywords, int32_t n_kw, int32_t normalize,
                                float* reward);

/* Commit of an Alg. 1 iteration's accepted tokens: emits O = [x_1..x_n],
 * n = n_accept[b] in [0, d] (emitted_host [B, d], n_emit_host [B] = n; n =
 * 0 emits nothing), as every state of Alg. 1 does before its own action.
 * The KV of x_1..x_n becomes part of the prefix (both models; when n = d,
 * x_d is fed through both models as one appended row).  next_beams /
 * next_head_lp [B, kk] receive the target's top-kk after O: row n of the
 * verification when n < d, the appended row when n = d.  Synchronises the
 * context stream once.  Errors: EINVAL (n_accept out of range), ERANGE,
 * ENOMEM, ESTATE (no cdsl_draft_prefix + cdsl_verify_prefix(_soft) with
 * this d and kk since the last commit). */
int cdsl_commit_prefix(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                       const int32_t* n_accept, int32_t d, int32_t kk,
                       const int32_t* row_topk_ids, const float* row_topk_lp,
                       int32_t* emitted_host, int32_t* n_emit_host,
                       int32_t* next_beams, float* next_head_lp);

/* Reward-only selection with Step-1 of the controller (Sec. 3.2.3, S2/S3
 * with b = 1): beam[b] = 0 when reward[b, 0] >= first_at[b] (head 0 is the
 * target's greedy token), otherwise argmax_i reward[b, i] with the lowest i
 * on ties.  first_at[b] = NaN disables the rule for prompt b (plain Alg. 2
 * argmax, as CDLH-appx. in Step-2).  reward is [B, k], first_at [B], beam
 * [B], all device.  A NaN reward makes beam[b] = -1 (reported by the next
 * commit as EINVAL).  Errors: EINVAL for null pointers or B, k <= 0. */
int cdsl_select_first(cdsl_ctx* ctx, const float* reward, const float* first_at,
                      int32_t B, int32_t k, int32_t* beam);

/* The controller's state per prompt after an Alg. 1 lookahead (Sec. 3.2.3,
 * Alg. 1 decision between S1..S4): a = n_accept[b] / d compared in float64
 * with a_t, r = reward[b] (the accepted window's reward, float32 widened to
 * float64) with r_t.  state[b] = 1 (S1: a >= a_t and r >= r_t), 2 (S2/S3:
 * a < a_t) or 4 (S4: a >= a_t, r < r_t).  first_at[b] = r_t for state 2
 * when b = 1 (the input cdsl_select_first takes for Step-1), NaN otherwise.
 * n_accept and reward are [B] (the outputs of cdsl_verify_prefix and
 * cdsl_reward_keywords_prefix), state and first_at [B]; all device.  Errors:
 * EINVAL for null pointers, B or d <= 0, b not in {0, 1}, NaN thresholds. */
int cdsl_controller_states(cdsl_ctx* ctx, const int32_t* n_accept, const float* reward,
                           int32_t B, int32_t d, double a_t, double r_t, int32_t b,
                           int32_t* state, float* first_at);

/* Commit the selected beams.  Emits, per prompt, O = [c_i*, x_i*,1..n]
 * with n = n_accept[b, i*]: emitted_host[b, 0..n] and n_emit_host[b] = n+1
 * (host buffers, [B, d+1] and [B]).  The beam's KV for those tokens becomes
 * part of the prefix (both models); if n == d the last token is fed through
 * both models so the prefix is complete.  next_beams[B, k] / next_head_lp
 * receive the next beam heads (top-k of the target after O).  Synchronises
 * the context stream once.  Errors: EINVAL (beam -1 / out of range),
 * ERANGE (max_ctx exceeded), ENOMEM, ESTATE (no verify since the last
 * commit). */
int cdsl_commit(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                const int32_t* beam, const int32_t* n_accept,
                const int32_t* row_topk_ids, const float* row_topk_lp,
                int32_t k, int32_t d, int32_t* emitted_host,
                int32_t* n_emit_host, int32_t* next_beams, float* next_head_lp);

/* cdsl_commit after cdsl_verify_kk: row_topk_* are [B, k, d, kk] and
 * next_beams / next_head_lp [B, kk].  cdsl_commit is kk = k.  Errors as
 * cdsl_commit; ESTATE also when the last verify used another kk. */
int cdsl_commit_kk(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                   const int32_t* beam, const int32_t* n_accept,
                   const int32_t* row_topk_ids, const float* row_topk_lp,
                   int32_t k, int32_t d, int32_t kk, int32_t* emitted_host,
                   int32_t* n_emit_host, int32_t* next_beams, float* next_head_lp);

/* Head-only commit: after a rollout (no verification needed), prompt b with
 * mask_host[b] != 0 (mask_host NULL: every prompt) emits the head of beam
 * beam[b], c = lookaheads[b, beam[b], 0], and nothing else: one token
 * generated by lookahead-heuristic decoding (CDLH / CDLH-appx., Sec. 2.1,
 * 3.1 and the appendix algorithm; also the single token of the S2/S3/S4
 * branches of Sec. 3.2.3).  The token is fed through both models at the end
 * of the prefix; the rolled suffixes are dropped.  emitted_host[b] is the
 * token or -1 (host, [B]); next_beams / next_head_lp [B, kk] of emitting
 * prompts receive the top-kk of the target after it, the other prompts'
 * rows are left as they are.  Synchronises the context stream once.
 * Errors: EINVAL (beam -1 or out of range for an emitting prompt), ERANGE
 * (max_ctx, kk), ENOMEM, ESTATE (no rollout with this k and d since the
 * last commit). */
int cdsl_commit_heads(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* lookaheads,
                      const int32_t* beam, int32_t k, int32_t d, int32_t kk,
                      const int32_t* mask_host, int32_t* emitted_host,
                      int32_t* next_beams, float* next_head_lp);

/* Append one given token per selected prompt: prompt b with mask_host[b]
 * != 0 (mask_host NULL: every prompt) emits tokens[b] (device [B] int32),
 * which is added to its generated tokens and fed through both models as
 * one appended row; next_beams / next_head_lp [B, kk] of emitting prompts
 * receive the target's top-kk after it, the other rows are left as they
 * are.  emitted_host[b] is the token or -1.  This is the move of Alg. 1's
 * Step-1 (Sec. 3.2.3): M_p's greedy token after the accepted ones, taken
 * tentatively while its draft lookahead is scored.  Synchronises the
 * context stream once.  Errors: EINVAL (a selected token outside [0, V):
 * nothing is appended), ERANGE (max_ctx, kk), ENOMEM. */
int cdsl_append(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* tokens,
                const int32_t* mask_host, int32_t kk, int32_t* emitted_host,
                int32_t* next_beams, float* next_head_lp);

/* Withdraw the last count_host[b] generated tokens of prompt b (host [B];
 * 0 leaves a prompt as it is): Step-1 drops its tentative M_p tokens when
 * none of their lookaheads reaches the reward threshold (Sec. 3.2.3).  The
 * prefix is shortened (its KV past the new end is ignored and later
 * overwritten) and the tokens leave the generated sequence the rewards
 * read.  The caller's beam heads are not recomputed: keep those of the
 * shorter prefix.  Errors: EINVAL (more than the generated tokens). */
int cdsl_withdraw(cdsl_ctx* ctx, cdsl_prefix* prefix, const int32_t* count_host);

/* Current length (prompt + emitted) of every prompt: lengths_host[B]. */
int cdsl_prefix_lengths(cdsl_ctx* ctx, const cdsl_prefix* prefix,
                        int32_t* lengths_host);

/* Per-kernel-class timing, for measurement.  While enabled, every launch
 * is bracketed by a pair of HIP events on the context stream and its
 * algorithmic work is added to its class: flops (2*M*N*K for a projection,
 * 4*hd per visible (query, key) pair for attention) and bytes (each operand
 * read once, each output written once; for attention the prefix KV of a
 * prompt counts once for all its beams).  cdsl_profile_enable(ctx, 1)
 * resets the totals; cdsl_profile_read synchronises the stream and returns
 * the totals since then.  Disabled (the default), no events are recorded. */
enum {
  CDSL_K_GEMM_DENSE = 0,   /* bf16 MFMA projection, > 128 rows          */
  CDSL_K_GEMM_SKINNY = 1,  /* bf16 MFMA projection, <= 128 rows (decode) */
  CDSL_K_ATTENTION = 2,    /* paged shared-prefix / tree attention       */
  CDSL_K_ATTN_COMBINE = 3, /* merge of key-split partials                */
  CDSL_K_LOGIT_ROWS = 4,   /* log-softmax + gather + argmax + top-k      */
  CDSL_K_ROWWISE = 5,      /* embedding, RMSNorm, rotary + KV write      */
  CDSL_K_STEP = 6,         /* scores, rewards, select, commit, promote   */
  CDSL_K_GEMM_F32 = 7,     /* fp32 projection                            */
  CDSL_K_SPLITK_REDUCE = 8,/* sum of split-K partials + epilogue         */
  CDSL_K_CLASSES = 9
};
typedef struct cdsl_kernel_stats {
  int64_t launches[CDSL_K_CLASSES];
  double ms[CDSL_K_CLASSES];
  double flops[CDSL_K_CLASSES];
  double bytes[CDSL_K_CLASSES];
} cdsl_kernel_stats;
int cdsl_profile_enable(cdsl_ctx* ctx, int32_t enable);
int cdsl_profile_read(cdsl_ctx* ctx, cdsl_kernel_stats* out);

int cdsl_free_prefix(cdsl_ctx* ctx, cdsl_prefix* prefix);
/* NULL is accepted; a context already destroyed gives ESTATE. */
int cdsl_destroy(cdsl_ctx* ctx);
const char* cdsl_last_error(const cdsl_ctx* ctx);   /* never NULL */

#ifdef __cplusplus
}
#endif
#endif /* CDSL_H */
