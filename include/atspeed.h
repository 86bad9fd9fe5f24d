/*
 * atspeed.h — C ABI of the MI355X (gfx950) speculative-decoding verify path of
 * AtSpeed (arXiv 2410.05165): top-K generative recommendation with a draft model
 * and a target LLM.
 *
 * Problem statement (task formulation, Sec. 2): given a user's history x, the
 * target model returns the top-K item identifiers (L codebook tokens each) by
 * constrained beam search.  Speculative decoding drafts gamma beam-search levels
 * of width N with a small model (Eq. 1) and verifies all of them with ONE target
 * forward over the tree of drafted beams (tree-based attention, Sec. 3.3),
 * followed by strict top-K verification (Algorithm 1) or relaxed sampling
 * verification (Sec. 3.2, Algorithm 2).
 *
 * Conventions shared by every call
 *   - "dev" pointers are device (HBM) pointers, "host" pointers are host memory.
 *   - The caller owns every buffer (weights, workspace, inputs, outputs); they
 *     must outlive the context.  The library allocates no device memory.
 *   - All device work is enqueued on config.stream (a hipStream_t; NULL = the
 *     default stream).  Calls that return host-visible results synchronise that
 *     stream before returning; this is stated per call.
 *   - Every call returns a status; no C++ exception crosses the ABI.  Argument
 *     errors are detected on the host before any launch and leave the context
 *     unchanged.  The message of the last error of the calling thread is
 *     returned by atspeed_last_error().
 *   - Token ids: item code c at item level l (0-based) is token
 *     item_base + codebook*l + c.  Items are fixed-length: L tokens.
 *   - A context is bound to one stream and is not thread-safe.
 */
#ifndef ATSPEED_H
#define ATSPEED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ATSPEED_API __attribute__((visibility("default")))

typedef enum {
  ATSPEED_OK = 0,
  ATSPEED_E_INVALID = 1,    /* bad argument (null pointer, value out of range, invalid tree)   */
  ATSPEED_E_SHAPE = 2,      /* shapes inconsistent with the configuration                      */
  ATSPEED_E_WORKSPACE = 3,  /* workspace too small or misaligned                               */
  ATSPEED_E_DEVICE = 4,     /* a HIP call failed (message holds the HIP error string)          */
  ATSPEED_E_STATE = 5       /* call out of order (e.g. verify before prefill)                  */
} atspeed_status;

typedef enum {
  ATSPEED_STRICT = 0,         /* Algorithm 1: accept level j iff TopK(p_j) is a subset of the drafted level */
  ATSPEED_RELAXED_EXACT = 1,  /* Sec. 3.2 with K i.i.d. slots per level (the with-replacement reading)       */
  ATSPEED_RELAXED_PAPER = 2   /* Algorithm 2 reading: N distinct drafts, K accepted kept, residual resample  */
} atspeed_mode;

typedef enum { ATSPEED_FP32 = 0, ATSPEED_BF16 = 1 } atspeed_dtype;

/* LLaMA-style decoder dimensions.  d_model % n_heads == 0 and d_model <= 8192;
 * bf16: d_head 64 or 128, d_model % 256 == 0, d_ffn % 128 == 0;
 * fp32: d_head 32, 64 or 128, d_model and d_ffn multiples of 16.
 * Violations make atspeed_create return ATSPEED_E_SHAPE. */
typedef struct {
  int32_t n_layers, d_model, n_heads, d_ffn, vocab, item_base;
} atspeed_model_dims;

typedef struct {
  atspeed_model_dims target, draft;
  int32_t L;            /* item identifier length (tokens per item), 1..4          */
  int32_t codebook;     /* codes per level, <= 256                                  */
  int32_t K;            /* target beam size (recommended items)                     */
  int32_t N;            /* draft beam size, N >= K                                  */
  int32_t gamma;        /* drafted levels per speculative step, >= 1                */
  int32_t max_batch;    /* users per call, 1..1024                                  */
  int32_t max_prefix;   /* prefix (history) tokens per user; max_batch x max(max_prefix,
                           K*(L-1) + gamma*N) x max(d_model, d_ffn, L*codebook) must stay
                           below 2^31 (ATSPEED_E_SHAPE otherwise)                    */
  int32_t mode;         /* atspeed_mode                                             */
  float temperature;    /* sampling temperature of the relaxed modes (> 0)          */
  uint64_t seed;        /* Philox key of the relaxed modes                          */
  int32_t dtype;        /* atspeed_dtype of weights, activations and KV caches      */
  int32_t sd_start_level; /* atspeed_decode_topk schedule: 0 speculates from t = 0, as
                           Algorithm 1 does; 1 first takes level 1 from the prefill's
                           root log-probs (a verify with no drafted levels, no forward)
                           and speculates from t = 1, so no drafted level 1 is wasted.
                           The lists are the same either way.  Strict mode only:
                           with a relaxed mode, 1 makes create (and
                           workspace_bytes) return ATSPEED_E_INVALID.             */
  int32_t reuse_tree_kv; /* atspeed_decode_topk: 1 keeps the target's per-layer K/V and
                           log-probs of every forwarded tree node until the next
                           verify of the same call, which takes the nodes it shares
                           with the previous tree (same depth and path: the Y_t
                           paths and accepted levels) from there and forwards only
                           the others.  A node's K/V depends only on the prefix and
                           its path, so the lists are the same either way.  Costs
                           2 x target n_layers x max_batch x (K*(L-1) + gamma*N) x
                           d_model K/V elements (plus two log-prob buffers) of
                           workspace instead of one layer's.  atspeed_verify
                           itself always forwards the whole tree.  0: off.      */
  void* stream;         /* hipStream_t                                              */
} atspeed_config;

/* Model weights (device, caller-owned).  Matrices are row-major [out, in] in the
 * configured dtype (bf16 or fp32); norm gains are fp32 [d_model].
 *   tok_emb       [vocab, d_model]
 *   layers        host array of n_layers*9 device pointers, per layer in order:
 *                 attn_norm, wq, wk, wv, wo ([d,d]), ffn_norm, w_gate, w_up ([f,d]), w_down ([d,f])
 *   final_norm    [d_model]
 *   lm_head_item  [L*codebook, d_model]: the output-head rows of the item tokens
 *                 (item_base .. item_base + L*codebook - 1); no other row is read. */
typedef struct {
  const void* tok_emb;
  const void* const* layers;
  const float* final_norm;
  const void* lm_head_item;
} atspeed_weights;

/* Item catalog (host): n_items distinct identifiers, codes[i*L + l] in [0, codebook). */
typedef struct {
  int32_t n_items;
  const int32_t* codes;
} atspeed_catalog;

/* Tree of drafted beams (device, structure of arrays, one row of max_nodes slots
 * per user).  Nodes of a user are level-ordered (depth never decreases with the
 * slot index); a node's parent has a smaller slot; parent = -1 for depth-1 nodes.
 * A verify tree must contain the paths of the current target beams Y_t (depths
 * 1..t) and the drafted levels t+1..t+J (tree-based attention, Sec. 3.3; the
 * flattened sequence of its appendix is the slot order). */
typedef struct {
  int32_t max_nodes;
  int32_t* n_nodes;   /* [B]             */
  int32_t* token;     /* [B, max_nodes]  item-token ids                          */
  int32_t* parent;    /* [B, max_nodes]  parent slot or -1                       */
  int32_t* depth;     /* [B, max_nodes]  1..L                                    */
  float* q_score;     /* [B, max_nodes]  draft cumulative log-prob (relaxed modes) */
} atspeed_tree;

/* Per-call statistics (host).  Arrays are caller-provided; NULL skips them. */
typedef struct {
  int32_t n_steps;     /* speculative steps run                                  */
  int32_t* accepted;   /* [L, max_batch]: accepted levels per step, -1 once done */
  int32_t* t_after;    /* [L, max_batch]: item level reached after each step     */
  double ms_prefill, ms_draft, ms_verify;  /* stream time per stage (HIP events) */
  int64_t rows_target; /* target tree rows forwarded over all verify steps       */
} atspeed_stats;

/* Kernel classes timed by atspeed_get_timing. */
enum {
  ATSPEED_K_QKV = 0,     /* q/k/v projection + rotary + KV scatter (bf16 MFMA GEMM) */
  ATSPEED_K_O = 1,       /* attention output projection + residual                  */
  ATSPEED_K_GU = 2,      /* gate/up projection + SiLU * up                           */
  ATSPEED_K_DOWN = 3,    /* down projection + residual                               */
  ATSPEED_K_LMHEAD = 4,  /* item rows of the output head                             */
  ATSPEED_K_ATTN = 5,    /* tree / prefill attention                                 */
  ATSPEED_K_ROW = 6,     /* embedding, RMSNorm, log-softmax                          */
  ATSPEED_K_SELECT = 7,  /* tree planning, TopK selection, acceptance                */
  ATSPEED_K_COUNT = 8
};

/* Stream time per kernel class, from HIP events recorded between consecutive
 * launches on the context's stream while timing is enabled.  gflop: algorithmic
 * GFLOP of the bracketed GEMM launches of the target model (2 x rows x n x k with
 * the rows the launch forwards; the draft's launches, sized by a bound of their
 * rows, and the non-GEMM classes count 0). */
typedef struct {
  double ms[ATSPEED_K_COUNT];
  int64_t launches[ATSPEED_K_COUNT];
  double gflop[ATSPEED_K_COUNT];
} atspeed_kernel_times;

typedef struct atspeed_ctx atspeed_ctx;

/* Bytes of device workspace a context needs for this configuration and catalog. */
ATSPEED_API atspeed_status atspeed_workspace_bytes(const atspeed_config* cfg, const atspeed_catalog* cat, size_t* bytes);

/* Create a context.  Builds the item trie on the host from the catalog and copies
 * it, the rotary tables and the zeroed state into the workspace (256-byte aligned,
 * >= atspeed_workspace_bytes).  Synchronises the stream.  draft may be NULL, then
 * atspeed_draft and atspeed_decode_topk return ATSPEED_E_STATE. */
ATSPEED_API atspeed_status atspeed_create(const atspeed_config* cfg, const atspeed_weights* target,
                              const atspeed_weights* draft, const atspeed_catalog* cat,
                              void* workspace_dev, size_t ws_bytes, atspeed_ctx** out);
ATSPEED_API void atspeed_destroy(atspeed_ctx* ctx);
ATSPEED_API const char* atspeed_last_error(void);

/* Prefill of the users' histories x (task formulation, Sec. 2): the prefilling
 * stage that the appendix case study separates from decoding (its time is the
 * same with and without speculative decoding), which every verify's tree
 * attention then reads (Sec. 3.3).  One causal forward of the target (and draft)
 * over B prefixes of P tokens each (prefix_dev [B, P] int32, device), filling the
 * prefix KV caches and
 * the root log-probs (logits at the last prefix position).  Positions that all
 * users share with user 0 (a common prompt; found on the device, one read-back)
 * are forwarded once and their K/V copied to the other users: the results are
 * those of forwarding every position.  Resets every user to
 * item level t = 0 with the empty beam.  root_logits_dev (nullable): [B, L*codebook]
 * fp32 item logits of the target at the last prefix position.  Asynchronous. */
ATSPEED_API atspeed_status atspeed_prefill(atspeed_ctx* ctx, int32_t B, int32_t P, const int32_t* prefix_dev,
                               float* root_logits_dev);

/* Draft (Eq. 1): from each user's current target beams Y_t, run J = min(gamma, L-t)
 * levels of draft beam search of width N over trie-valid codes and write the
 * verify tree (Y_t paths + drafted levels) into the context's tree.  Users with
 * t = L get an empty tree.  Asynchronous. */
ATSPEED_API atspeed_status atspeed_draft(atspeed_ctx* ctx);

/* The context's own tree (device pointers inside the workspace).  A caller may
 * overwrite its contents to verify a tree of its own. */
ATSPEED_API atspeed_status atspeed_get_tree(atspeed_ctx* ctx, atspeed_tree* out);

/* Verify: ONE target forward over every tree node of depth < L (tree attention on
 * the prefix KV cache plus each node's ancestors), log-softmax over the item
 * tokens, cumulative log-probs, trie-constrained TopK and acceptance (strict:
 * Algorithm 1; relaxed: Algorithm 2 per the configured mode).  Updates the state
 * (t, beams, scores).  accepted_dev / t_after_dev: [B] int32 (device, nullable).
 * logits_dev (nullable): [B, max_nodes, L*codebook] fp32 target item logits of
 * every forwarded node by slot.  Synchronises the stream once, after tree
 * planning and before the forward (reads back the validity word and the row
 * counts that size the forward's launches): ATSPEED_E_INVALID if the tree is
 * malformed (no forward runs; state unchanged).  The
 * tree is validated on the device before the forward: n_nodes within 0..max_nodes,
 * level order, depths 1..L, each parent an earlier node one level up (-1 at depth
 * 1), tokens the item tokens of their level, every path in the catalog, and (t > 0)
 * every beam of Y_t a node of depth t.  A user whose tree fails any check forwards
 * no rows, so a malformed tree never sends a kernel outside its buffers. */
ATSPEED_API atspeed_status atspeed_verify(atspeed_ctx* ctx, int32_t* accepted_dev, int32_t* t_after_dev,
                              float* logits_dev);

/* Forward only: target item logits of every tree node of depth < L (the first
 * part of atspeed_verify), written to logits_dev [B, max_nodes, L*codebook].
 * Synchronises the stream. */
ATSPEED_API atspeed_status atspeed_tree_logits(atspeed_ctx* ctx, float* logits_dev);

/* Accept only: the selection and acceptance part of atspeed_verify on caller
 * logits (logits_dev [B, max_nodes, L*codebook] fp32 by slot; root logits
 * [B, L*codebook] fp32).  Updates the state like atspeed_verify. */
ATSPEED_API atspeed_status atspeed_accept(atspeed_ctx* ctx, const float* logits_dev, const float* root_logits_dev,
                              int32_t* accepted_dev, int32_t* t_after_dev);

/* Allocation-free accept, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, checks and results as atspeed_accept, but the buffers that call
 * takes from the workspace for its own use -- the log-prob rows of the caller's
 * logits, the selection keys, the relaxed modes' candidate buffers and the
 * tree-validation word -- live in a static device array of 64 MiB that the
 * library holds on each GPU until the process ends (its address is taken at
 * atspeed_create, on the context's device).  Needs 4*(B*max_nodes + B)*L*codebook
 * + 8*B*N*codebook bytes (+ 20*B*N*codebook in a relaxed mode, plus alignment);
 * a prefilled batch that needs more returns ATSPEED_E_WORKSPACE before any launch.
 * Every call on a GPU shares that GPU's array and finds the last call's contents
 * there (each call writes what it reads): calls that overlap on one GPU, from
 * any context or stream, race.  No allocating call is made.  Synchronises the
 * stream. */
ATSPEED_API atspeed_status atspeed_accept_noalloc(atspeed_ctx* ctx, const float* logits_dev,
                                                  const float* root_logits_dev, int32_t* accepted_dev,
                                                  int32_t* t_after_dev);

/* Whole decode: prefill, then draft/verify steps until every user holds L-token
 * items (Algorithm 1 / 2 repeated; the schedule options sd_start_level and
 * reuse_tree_kv of the config change the work, not the lists).  items_dev
 * [B, K, L] int32 codes (strict: best first; relaxed modes: in code order),
 * scores_dev [B, K] fp32 cumulative target
 * log-probs, n_items_dev [B] number of valid lists (< K when the catalog has
 * fewer candidates, or in the relaxed modes when a rejected level's residual
 * distribution max(0, p - q) has fewer candidates than the draws it owes).
 * stats_host (nullable): steps, per-step accepted levels and levels reached,
 * stage times and target tree rows forwarded.  Synchronises once per step. */
ATSPEED_API atspeed_status atspeed_decode_topk(atspeed_ctx* ctx, int32_t B, int32_t P, const int32_t* prefix_dev,
                                   int32_t* items_dev, float* scores_dev, int32_t* n_items_dev,
                                   atspeed_stats* stats_host);

/* Target-only constrained beam search (task formulation, Sec. 2): the standard
 * inference that speculative decoding accelerates, and the baseline of the
 * paper's walltime speedup WS@K (Sec. 4.1).  Prefill of the target alone (the
 * draft's caches are left stale: atspeed_draft and atspeed_align_data need
 * atspeed_prefill again), then L levels, each a verify of the tree of the Y_t
 * paths with no drafted level -- one target forward (with reuse_tree_kv, only
 * the new level's nodes: the earlier levels' K/V is carried) and the target's
 * TopK of the next level, strict whatever the configured mode.  Outputs as
 * atspeed_decode_topk (the same lists as its strict decode).  step_items_dev
 * [B, K*L, L], step_lens_dev [B, K*L], step_n_dev [B] (all nullable, given
 * together): every level's beams in level order (codes past a beam's length
 * zero) -- the multi-step data of draft alignment, whose last rows are the
 * final lists.  Synchronises once per level. */
ATSPEED_API atspeed_status atspeed_target_search(atspeed_ctx* ctx, int32_t B, int32_t P, const int32_t* prefix_dev,
                                                 int32_t* items_dev, float* scores_dev, int32_t* n_items_dev,
                                                 int32_t* step_items_dev, int32_t* step_lens_dev,
                                                 int32_t* step_n_dev);

/* Mixture beam search: the training sequences D' of AtSpeed-S (Sec. 3.1) for a
 * mixing weight lambda in [0, 1] -- constrained beam search of width K whose
 * token distribution is (1 - lambda) q + lambda p (the draft's and the target's
 * item distributions), a sequence scored by the sum of the log of the mixture
 * over its tokens.  Prefill of both models, then L levels, each a forward of
 * the target and of the draft over the tree of the Y_t paths (with
 * reuse_tree_kv the target carries the earlier levels' K/V) and the strict
 * TopK of the next level under the mixture.  lambda = 1 gives bitwise the
 * lists and beams of atspeed_target_search.  Outputs as atspeed_target_search
 * (scores: cumulative log-mixture).  Leaves the draft's root log-probs mixed:
 * atspeed_draft and atspeed_align_data need atspeed_prefill again.
 * ATSPEED_E_INVALID for lambda outside [0, 1]; ATSPEED_E_STATE without a
 * draft.  Synchronises once per level. */
ATSPEED_API atspeed_status atspeed_mixed_search(atspeed_ctx* ctx, float lambda, int32_t B, int32_t P,
                                                const int32_t* prefix_dev, int32_t* items_dev, float* scores_dev,
                                                int32_t* n_items_dev, int32_t* step_items_dev,
                                                int32_t* step_lens_dev, int32_t* step_n_dev);

/* Log-probabilities a verify step consumes (parity and inspection access).
 * model 0: the target's log p(. | x, path) of every node the last verify (or
 * tree_logits) forwarded; model 1: the draft's log q(. | x, path) of every node
 * the last draft forwarded (the Y_t paths and the drafted levels below the
 * deepest); both normalised over the L*codebook item-token columns (Sec. 3.1,
 * constrained generation; p_j and q_j of Algorithms 1 and 2).  lp_dev
 * [B, max_nodes, L*codebook] fp32 by tree slot (rows of nodes that were not
 * forwarded are undefined), root_dev [B, L*codebook] fp32 at the last prefix
 * position; both device, caller-owned, B = the prefilled batch.  Synchronises
 * the stream.  ATSPEED_E_STATE before prefill, or model 1 without a draft. */
ATSPEED_API atspeed_status atspeed_logprobs(atspeed_ctx* ctx, int32_t model, float* lp_dev, float* root_dev);

/* Draft alignment: training of the draft's item head on the overall objectives
 * of AtSpeed-S (Sec. 3.1, Eq. 5: alpha L_Align-S + (1 - alpha) L_Rec, for strict
 * top-K verification) and AtSpeed-R (Sec. 3.2: alpha L_Align-R + (1 - alpha)
 * L_Rec, for relaxed sampling verification), with AdamW (the optimizer of the
 * paper's implementation details).
 *
 * A batch is the prefilled users with up to S training sequences each: for D'
 * of Sec. 3.1 with lambda = 1, the target's top-K lists (atspeed_decode_topk in
 * strict mode) -- the last beam-search step's sequences -- or, for the
 * multi-step data the paper also evaluates, the target's K beams of every
 * beam-search step (lengths 1..L; atspeed_target_search), or for lambda < 1
 * those of the mixture (atspeed_mixed_search).  The last sequence of a user must be a whole
 * item: it is the K-th sequence of the p_K term.  The contexts are each user's
 * root and every distinct proper prefix of its sequences; for a context c with
 * draft and target item distributions q, p and V_c the K trie-valid codes of
 * the next level with the largest q (ties: smaller code):
 *   AtSpeed-S: l(c) = sum_{v in V_c} q(v) (log p_K - log p(v)), the reverse KL
 *     over V_c minus the density regulariser, p_K the target's probability of
 *     the last sequence's code at that level given its own prefix;
 *   AtSpeed-R: l(c) = TVD of p and q, both truncated to V_c and renormalised;
 *   L_Rec: -sum over the sequences through c of log q(next code) (the NLL of the
 *     training sequences: the recommender's loss, whose dataset labels
 *     synthetic histories do not have).
 * Every sequence y adds 1 / (|y| B) to the weight of each of its contexts; the
 * loss is the weighted sum.  The gradient holds V_c fixed.
 *
 * Buffers (device, caller-owned, fp32):
 *   ctx_weight, label_weight [B, max_nodes] (a node's weight as a context and
 *   as the label of its parent context), root_weight [B], log_pK [B, L],
 *   lp_target [B, max_nodes, L*codebook], root_target [B, L*codebook]:
 *     the batch, written by atspeed_align_data and read by atspeed_align_step;
 *   master, adam_m, adam_v, grad [L*codebook, d_model of the draft]: the head's
 *     fp32 master copy (the caller initialises it to the head's values), the
 *     AdamW moments (zero before step 1) and the last step's gradient dL/dW.
 *   hidden_out (nullable) [B * (1 + max_nodes), d_model of the draft]: the
 *     final-normed hidden states the gradient used, roots at rows [0, B), each
 *     context at row B + its tree slot (other rows untouched). */
typedef struct {
  int32_t mode;          /* 0: AtSpeed-S, 1: AtSpeed-R                              */
  float alpha;           /* alignment strength in [0, 1] (1: L_Align alone)         */
  float* ctx_weight;
  float* label_weight;
  float* root_weight;
  float* log_pK;
  float* lp_target;
  float* root_target;
  float* master;
  float* adam_m;
  float* adam_v;
  float* grad;
  float* hidden_out;
  float lr, beta1, beta2, eps, weight_decay;  /* AdamW (decoupled decay: w -= lr wd w) */
  int32_t step;          /* 1-based step number (bias correction)                   */
} atspeed_align_args;

/* Builds the context tree of the prefilled batch from items_dev [B, S, L] int32
 * codes (each user's sequences, a whole item last), lens_dev [B, S] (nullable:
 * every length L) and n_items_dev [B] (1..S) into the context's tree, level
 * ordered, leaves of depth L included (read it with atspeed_get_tree; every
 * distinct prefix must fit max_nodes: the K beams of each of the L steps do),
 * forwards the target over the contexts and writes the batch buffers of args.
 * Resets every user to t = 0.  ATSPEED_E_INVALID (nothing written but the
 * tree) if a sequence prefix is not in the catalog, a count or a length is out
 * of range, a user's last sequence is shorter than L or the prefixes overflow
 * max_nodes; ATSPEED_E_STATE before prefill or without a draft.  Synchronises
 * the stream. */
ATSPEED_API atspeed_status atspeed_align_data(atspeed_ctx* ctx, int32_t S, const int32_t* items_dev,
                                              const int32_t* lens_dev, const int32_t* n_items_dev,
                                              const atspeed_align_args* args);

/* One training step on the batch of the last atspeed_align_data: the draft's
 * forward over the contexts (its prefix caches are the last prefill's), its root
 * log-probs with the current head, the losses and their gradient, dL/dW of the
 * item head into args.grad, and one AdamW step on args.master whose result,
 * rounded to the configured dtype, overwrites the draft's lm_head_item (the
 * caller's weights).  loss_host (nullable): the loss before the update.  The
 * draft's log-probs of this step are readable with atspeed_logprobs (model 1).
 * ATSPEED_E_STATE unless atspeed_align_data ran after the last prefill or
 * draft.  Synchronises the stream. */
ATSPEED_API atspeed_status atspeed_align_step(atspeed_ctx* ctx, const atspeed_align_args* args, double* loss_host);

/* State access (host arrays; synchronise the stream).  t [B]; nbeams [B];
 * paths [B, K, L] codes (entries past depth t undefined); scores [B, K] fp32. */
ATSPEED_API atspeed_status atspeed_get_state(atspeed_ctx* ctx, int32_t B, int32_t* t, int32_t* nbeams,
                                 int32_t* paths, float* scores);
ATSPEED_API atspeed_status atspeed_set_state(atspeed_ctx* ctx, int32_t B, const int32_t* t, const int32_t* nbeams,
                                 const int32_t* paths, const float* scores);

/* Residual-stream and activation capture (instrumentation for kernel-by-kernel
 * parity tests; the decoder block is the LLaMA block of the implementation
 * details, Sec. 4.1, with tree-based attention, Sec. 3.3).  Arms a coming
 * forward of the target (model 0: in atspeed_prefill, atspeed_tree_logits,
 * atspeed_verify or a decode) or of the draft (model 1: in atspeed_prefill or
 * atspeed_draft, which forwards the paths of the current beams, then each
 * drafted level's nodes but the last) -- the one after the next `skip`
 * forwards of that model -- to copy, on the context's stream, the values of its
 * forwarded rows at every rounding point of the block (R = max_rows; widths are
 * that model's):
 *   x_dev   (device, fp32, [2 n_layers + 1][R][d_model]): index 2l is layer l's
 *           input residual, 2l + 1 the residual after its attention sublayer,
 *           2 n_layers the residual after the last layer (not written by a
 *           prefill, whose final norm runs on each user's last row only);
 *   act_dev (device, bf16 bit patterns, may be null; bf16 models only): per
 *           layer l at element offset l R (6 d_model + d_ffn), six [R][d_model]
 *           arrays -- the normalised input of q/k/v, q and k after RoPE, v, the
 *           attention output, the normalised input of gate/up -- then SiLU(gate)
 *           * up as [R][d_ffn]; after the layers (offset n_layers R (6 d_model +
 *           d_ffn)) the final norm's output [R][d_model] (not written by a
 *           prefill);
 *   plan_dev (device, [3 R + 1] int32): each row's user, position and tree
 *           slot (u * max_nodes + node; -1 for a prefix row) as three arrays of
 *           R, then the forward's row count.
 * Rows past R are not copied (check the row count).  The capture disarms itself
 * after that forward; all three pointers null disarms it at once.
 * ATSPEED_E_INVALID for a model other than 0 or 1, skip < 0, a null x_dev or
 * plan_dev with the others set, max_rows <= 0, or act_dev with an fp32 model;
 * ATSPEED_E_STATE for model 1 without a draft.  Adds device copies to the
 * forward; buffers are caller-owned. */
ATSPEED_API atspeed_status atspeed_capture_hidden(atspeed_ctx* ctx, int32_t model, int32_t skip, float* x_dev,
                                                  void* act_dev, int32_t* plan_dev, int32_t max_rows);

/* Kernel timing (instrumentation for measurement).  enable is a bit mask of the
 * kernel classes to time (bit ATSPEED_K_x; ATSPEED_TIME_ALL for every class),
 * optionally or-ed with ATSPEED_TIME_TARGET_ONLY:
 * a HIP event is recorded on the context's stream before each launch of a
 * selected class and before the launch that follows it, and the totals are
 * cleared; 0 stops.  Each event adds a little stream time, so timing only the
 * classes of interest perturbs a measurement least.  atspeed_get_timing
 * synchronises the stream, folds the recorded intervals into out (totals since
 * enabling). */
#define ATSPEED_TIME_ALL ((1 << ATSPEED_K_COUNT) - 1)
#define ATSPEED_TIME_TARGET_ONLY (1 << 16)  /* with a class mask: the draft model's launches are not bracketed */
ATSPEED_API atspeed_status atspeed_set_timing(atspeed_ctx* ctx, int32_t enable);
ATSPEED_API atspeed_status atspeed_get_timing(atspeed_ctx* ctx, atspeed_kernel_times* out);

#ifdef __cplusplus
}
#endif
#endif /* ATSPEED_H */
