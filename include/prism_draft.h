/*
 * prism_draft.h — C ABI of the PRISM drafting hot path on MI355X (gfx950).
 *
 * PRISM (Parametrically Refactoring Inference for Speculative sampling draft
 * Models) drafts K tokens with a drafter made of a frozen token embedding E,
 * a frozen LM head, and M processing modules (a fusion FC plus one
 * transformer layer each).  A surjection f_map sends draft step k to module
 * f_map(k); the KV cache is shared by every module.  (Paper Sec. 3.2, the
 * architecture paragraph, Table 2 and "Draft with PRISM".)
 *
 * One forward pass of step k, for each of R rows:
 *   u      = W_fc[s] . [E(x) ; f]          f = target feature (step 1) or the
 *                                           draft's previous hidden state
 *   a      = RMSNorm(u; g1[s])
 *   q,k,v  = W_q,k,v[s] a ; RoPE(q, k; position)    k, v -> KV cache slot
 *   o      = softmax(q K^T / sqrt(d)) V over the visible slots (GQA)
 *   r1     = u + W_o[s] o
 *   h      = r1 + W_down[s] (SiLU(W_gate[s] m) * W_up[s] m),  m = RMSNorm(r1; g2[s])
 *   logits = LM_head . RMSNorm(h; g_final)            -> top-k / argmax
 *
 * Conventions for every call:
 *   - Pointers named d_* are DEVICE pointers owned by the caller, who keeps
 *     them alive until the work enqueued on `stream` has completed.  Other
 *     pointers are host pointers, read before the call returns.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   - Every call returns a prism_status (0 = OK, < 0 = error) and never
 *     throws or prints.  Arguments are validated synchronously; the message
 *     of the last error is available from prism_last_error().  Work is
 *     enqueued asynchronously on `stream` unless stated otherwise.
 *   - Matrices are row-major.  "dtype" below is the context's storage type
 *     (prism_config.dtype): fp32 or bf16 (bit patterns in uint16).
 *   - Content that only the device sees (token ids, block-table entries,
 *     context lengths) is bounds-checked by the kernels: an out-of-range
 *     value skips the access and raises a flag that
 *     prism_device_status() reports.  So is a NaN that reaches the logits
 *     (from a feature row or a weight): the call still completes, and the
 *     flag is reported as PRISM_ERR_NONFINITE.
 *   - Device memory: prism_create allocates the workspace, and
 *     prism_draft_load_shared / prism_draft_load_params allocate the weight
 *     arena (and the embedding tables, below) on their first call for a
 *     tensor group.  Drafting and verification calls allocate nothing.
 *   - One context is used by one host thread at a time.  Results are
 *     bit-identical across repeated calls with the same inputs.
 */
#ifndef PRISM_DRAFT_H
#define PRISM_DRAFT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PRISM_OK = 0,
  PRISM_ERR_INVALID_ARG = -1,   /* null pointer, value out of range          */
  PRISM_ERR_SHAPE = -2,         /* shape not supported by the kernels         */
  PRISM_ERR_NOT_LOADED = -3,    /* weights of a referenced set not loaded     */
  PRISM_ERR_UNSUPPORTED = -4,   /* f_map asks one set for two feature widths  */
  PRISM_ERR_OUT_OF_MEMORY = -5, /* device allocation failed                   */
  PRISM_ERR_HIP = -6,           /* a HIP runtime call failed                  */
  PRISM_ERR_CAPACITY = -7,      /* KV block table / pool too small (device)   */
  PRISM_ERR_NONFINITE = -8      /* NaN logits or tree scores (device)         */
} prism_status;

typedef enum { PRISM_F32 = 0, PRISM_BF16 = 1 } prism_dtype;

typedef struct prism_ctx prism_ctx; /* opaque */

/* Model shape and capacity; fixed for the lifetime of a context. */
typedef struct {
  int32_t hidden;        /* H                                                */
  int32_t n_q_heads;     /* query heads                                      */
  int32_t n_kv_heads;    /* KV heads; n_q_heads % n_kv_heads == 0 (GQA)      */
  int32_t head_dim;      /* d; even, 32 <= d <= 256, multiple of 8           */
  int32_t ffn;           /* I, SwiGLU width                                  */
  int32_t vocab;         /* V                                                */
  int32_t n_sets;        /* M processing modules                             */
  int32_t max_steps;     /* largest K (chain) or depth D (tree), <= 63       */
  int32_t feat_width;    /* F_t, target feature width at step 1              */
  float rope_theta;      /* RoPE base                                        */
  float rms_eps;         /* RMSNorm epsilon                                  */
  int32_t dtype;         /* prism_dtype of weights, E, features and KV       */
  int32_t kv_block_size; /* slots per KV block                               */
  int32_t max_batch;     /* sequences per call                               */
  int32_t max_blocks_per_seq; /* columns of the block table                  */
  int32_t tree_width;    /* w (0 = no tree calls)                            */
  int32_t tree_nodes;    /* v output nodes of a tree call, <= 64             */
  int32_t max_new_rows;  /* largest total of new accepted tokens in one
                            prism_draft_chain_catchup call (0 = no such
                            calls), <= 4096                                 */
} prism_config;
/* Kernel tiling requires: H, n_q_heads*d, I multiples of 32 (bf16) or 16
 * (fp32); H + F_t likewise; rows per pass (max_batch, or max_batch*w for
 * trees) <= 64.  prism_create returns PRISM_ERR_SHAPE otherwise. */

/* Weights of one processing module, as device tensors in the context dtype.
 * Layouts follow y = W x with W row-major [out, in].  The call copies them
 * into the context's own step-indexed arena, so they may be freed after
 * prism_draft_load_params returns. */
typedef struct {
  const void *d_w_fc;   /* [H, H + feat_width]  input order [E(x) ; feature] */
  const void *d_g1;     /* [H]   input RMSNorm gain                          */
  const void *d_w_q;    /* [n_q_heads*d, H]                                  */
  const void *d_w_k;    /* [n_kv_heads*d, H]                                 */
  const void *d_w_v;    /* [n_kv_heads*d, H]                                 */
  const void *d_w_o;    /* [H, n_q_heads*d]                                  */
  const void *d_g2;     /* [H]   post-attention RMSNorm gain                 */
  const void *d_w_gate; /* [I, H]                                            */
  const void *d_w_up;   /* [I, H]                                            */
  const void *d_w_down; /* [H, I]                                            */
  int32_t feat_width;   /* F_s: F_t for a set that serves step 1, else H     */
} prism_param_set;

/* A batch of sequences and their paged draft KV cache (caller-owned, as in
 * a serving engine).  Slot t of sequence b lives in physical block
 * d_block_table[b*max_blocks_per_seq + t/kv_block_size] at offset
 * t % kv_block_size.  Pools are [n_pool_blocks, n_kv_heads, kv_block_size, d]
 * in the context dtype; slots 0..L_b-1 hold the prior context (K already
 * rotated).  Drafting writes slots from L_b on; rejected drafts are
 * discarded by simply not advancing L_b (paper Sec. 2, speculative
 * decoding: KV of rejected candidates is dropped). */
typedef struct {
  int32_t batch;               /* B <= max_batch                            */
  const int32_t *d_tokens;     /* [B] last accepted token per sequence      */
  const void *d_features;      /* [B, feat_width] target hidden state (dtype) */
  const int32_t *d_ctx_lens;   /* [B] prior context length L_b              */
  void *d_k_pool;              /* KV pools, see above                       */
  void *d_v_pool;
  const int32_t *d_block_table;/* [B, max_blocks_per_seq]                   */
  int32_t n_pool_blocks;       /* physical blocks in each pool              */
} prism_batch;

/* The tokens accepted since the last drafting call, for a chain whose first
 * step is the drafter's prefill over all of them (paper Sec. 3.2, "Draft
 * with PRISM": every accepted token x_i is fused with the target's hidden
 * state h_{i-1} and the fused sequence runs through module f_map(1) in one
 * pass).  Sequence b owns rows d_offsets[b] .. d_offsets[b+1]-1 (n_b >= 1
 * rows, the last one is its newest token), which take positions and KV slots
 * L_b .. L_b + n_b - 1 after its prior context L_b = d_ctx_lens[b]. */
typedef struct {
  int32_t total_rows;          /* T = sum of n_b, 1..max_new_rows (host)    */
  const int32_t *d_offsets;    /* [B + 1] row offsets, d_offsets[0] = 0,
                                  d_offsets[B] = T, increasing             */
  const int32_t *d_tokens;     /* [T] accepted tokens, sequence by sequence */
  const void *d_features;      /* [T, feat_width] target hidden states of
                                  those tokens (dtype)                      */
} prism_catchup;

/* One forward pass on R explicit rows (the general entry point). */
typedef struct {
  int32_t rows;                /* R, 1..max rows                            */
  const int32_t *d_tokens;     /* [R] input token of each row               */
  const void *d_feat;          /* feature rows, width F_s of the step's set */
  int32_t feat_dtype;          /* prism_dtype of d_feat (fp32 for hidden)   */
  const int32_t *d_feat_rows;  /* [R] row of d_feat used by row r; NULL = r */
  const int32_t *d_seq;        /* [R] sequence (index into kv arrays)       */
  const int32_t *d_pos;        /* [R] RoPE position                         */
  const int32_t *d_slot;       /* [R] KV slot this row writes               */
  const uint64_t *d_tree_bits; /* [R] visible draft slots: bit j = slot
                                  L_seq + j, plus slots 0..L_seq-1.
                                  NULL = causal: slots 0..slot[r]          */
  const prism_batch *kv;       /* ctx lens, pools, block table; d_seq values
                                  must lie in 0..kv->batch-1; tokens and
                                  features of *kv are not used            */
  int32_t topk;                /* 1..max(1, tree_width)                     */
  float *d_hidden_out;         /* [R, H] fp32 hidden state h                */
  int32_t *d_topk_ids;         /* [R, topk] ids, by (logit desc, id asc)    */
  float *d_topk_logp;          /* [R, topk] log-softmax values, or NULL     */
  float *d_logits;             /* [R, V] fp32 logits, or NULL               */
} prism_step_io;

/* Output of a tree call.  Final arrays are [B, v]; nodes are ordered by
 * (cumulative log-prob desc, creation order asc); the root is not a node. */
typedef struct {
  int32_t *d_tokens;    /* [B, v]                                          */
  int32_t *d_parent;    /* [B, v] index of the parent node, -1 = the root  */
  int32_t *d_depth;     /* [B, v] 1..D                                     */
  float *d_score;       /* [B, v] cumulative log-probability               */
  uint64_t *d_mask;     /* [B, v] bit j: node j is the node or an ancestor */
  /* optional (NULL to skip): every candidate and every pass */
  int32_t *d_cand_tokens; /* [B, C], C = w + (D-1) w^2, creation order     */
  int32_t *d_cand_parent; /* [B, C] candidate index of the parent, -1 root  */
  float *d_cand_score;    /* [B, C]                                         */
  int32_t *d_frontier;    /* [B, D-1, w] candidate index of each expanded node */
  float *d_logits;        /* [D, B, w, V] logits of each pass (root at r=0) */
} prism_tree_out;

/* Create a context on the current HIP device: validates the shape and
 * allocates the workspace.  *out receives the context (NULL on error). */
prism_status prism_create(const prism_config *cfg, prism_ctx **out);

/* Release every device resource of the context.  NULL is accepted. */
void prism_destroy(prism_ctx *ctx);

/* Message of the last failed call on ctx (empty if none); valid until the
 * next call on ctx.  With ctx == NULL: the last failure of a call that takes
 * no context (prism_create, prism_verify_chain_static). */
const char *prism_last_error(const prism_ctx *ctx);

/* Load the frozen shared tensors (paper Table 2: E and LM_head are frozen
 * and shared by every module) and the final RMSNorm gain:
 * d_embed [V, H], d_lm_head [V, H], d_final_norm [H], all in the context
 * dtype.  Copies and repacks them; synchronizes `stream` before returning.
 * Rebuilds the embedding tables of the sets already loaded (see
 * prism_draft_load_params). */
prism_status prism_draft_load_shared(prism_ctx *ctx, const void *d_embed,
                                     const void *d_lm_head,
                                     const void *d_final_norm, void *stream);

/* Load parameter set `set` (0..M-1), the weights of processing module
 * set+1 (paper Sec. 3.2: M modules, each a fusion FC and a transformer
 * layer).  Copies and repacks into the step-indexed arena; synchronizes
 * `stream`.  Allocates that set's arena slot on first use.  In every bf16
 * context whose H is a multiple of 64 the slot also holds the set's
 * embedding table, W_fc[:, :H] E[v] for every token v in fp32: V * H * 4
 * bytes per set (2.1 GB at V = 128256, H = 4096; 4.2 GB at H = 8192), on
 * top of the set's weights.  Every pass, whatever its row count, then reads
 * one table row per row instead of the FC's embedding columns.  The table is
 * built here once the shared tensors are loaded. */
prism_status prism_draft_load_params(prism_ctx *ctx, int32_t set,
                                     const prism_param_set *params,
                                     void *stream);

/* Set the surjection f_map (paper Table 2) from draft steps to sets:
 * f_map[k-1] is the 0-based set of step k, k = 1..K.  Host array.  Default:
 * the identity (step k uses set k-1).  A set may serve several steps. */
prism_status prism_set_step_map(prism_ctx *ctx, const int32_t *f_map,
                                int32_t K);

/* One forward pass of draft step k (1-based; set f_map(k)) on explicit rows
 * (paper Sec. 3.2: one pass of the module assigned to step k). */
prism_status prism_draft_step(prism_ctx *ctx, int32_t k,
                              const prism_step_io *io, void *stream);

/* Greedy K-step chain (paper Sec. 3.2, "Draft with PRISM"): step 1 fuses
 * E(token) with the target feature at position L_b; step k >= 2 fuses
 * E(x_{k-1}) with h_{k-2} at position L_b + k - 1; x_k = argmax (ties to the
 * lowest id).  Writes KV slots L_b .. L_b+K-1.  Captured once per shape and
 * buffer set in a HIP graph, then replayed.
 *   d_out_tokens [B, K] int32 drafted tokens
 *   d_out_logits [B, K, V] fp32 or NULL
 *   d_out_hidden [B, K, H] fp32 or NULL */
prism_status prism_draft_chain(prism_ctx *ctx, const prism_batch *batch,
                               int32_t K, int32_t *d_out_tokens,
                               float *d_out_logits, float *d_out_hidden,
                               void *stream);

/* K-step chain with stochastic drafting (paper Sec. 2: draft tokens are
 * drawn from p_draft and verified by a rejection rule on the ratio
 * p_target / p_draft; Sec. 3.2: PRISM works with stochastic sampling; the T =
 * 1 rows of Tables 4-5).  Steps, positions and KV slots as in
 * prism_draft_chain; x_k is drawn from softmax(logits / temperature) by
 * inverse CDF in token-id order: the smallest id whose cumulative
 * probability exceeds u = d_uniforms[b*K + k-1].  The caller draws the
 * uniforms (so a call is reproducible); values are clamped to [0, 1].
 *   temperature   > 0 (finite 1/temperature)
 *   d_uniforms    [B, K] fp32
 *   d_out_tokens  [B, K] int32 drawn tokens
 *   d_out_logp    [B, K] fp32 log p_draft(x_k) of the drawn tokens, or NULL
 *   d_out_logits  [B, K, V] fp32 raw logits, or NULL
 *   d_out_hidden  [B, K, H] fp32, or NULL */
prism_status prism_draft_chain_sample(prism_ctx *ctx, const prism_batch *batch,
                                      int32_t K, float temperature,
                                      const float *d_uniforms,
                                      int32_t *d_out_tokens, float *d_out_logp,
                                      float *d_out_logits, float *d_out_hidden,
                                      void *stream);

/* Greedy K-step chain whose first step catches up on several accepted
 * tokens per sequence (paper Sec. 3.2: the prefill over S_acc with H_base,
 * then h_0 = the last row's output and x_1 = argmax LM_head(h_0)).  Step 1
 * writes KV slots L_b .. L_b + n_b - 1 (each new row attends causally to the
 * prior context and the new rows up to itself); step k >= 2 runs at position
 * L_b + n_b + k - 2.  Writes KV slots L_b .. L_b + n_b + K - 2.  The tokens
 * and features of *batch are not used; catchup->d_offsets must describe
 * batch->batch sequences (a malformed table raises PRISM_ERR_INVALID_ARG in
 * prism_device_status and leaves the outputs unspecified).  Outputs as in
 * prism_draft_chain; d_out_logits and d_out_hidden hold the last row's
 * values for step 1.  Requires max_new_rows >= total_rows.  The fusion FC
 * and QKV of the accepted rows run in chunks of up to 64 rows (a row's KV
 * depends on no other row, and the attention runs once every chunk has
 * written its KV), so a call may take more rows than one pass. */
prism_status prism_draft_chain_catchup(prism_ctx *ctx, const prism_batch *batch,
                                       const prism_catchup *catchup, int32_t K,
                                       int32_t *d_out_tokens, float *d_out_logits,
                                       float *d_out_hidden, void *stream);

/* Dynamic draft tree of `depth` passes and width w (paper Sec. 2, tree
 * draft-and-verify with a tree attention mask; Sec. 3.2: PRISM works with
 * tree drafts; Sec. 4.3: depth / width / verified-node topology).  Pass d
 * (0-based) uses set f_map(d+1) at position L_b + d.  The root pass yields
 * w depth-1 candidates; each later pass expands the w best nodes of the
 * previous depth (by cumulative log-prob), attending to the prior context,
 * the root and its ancestors only, and each expanded node contributes its w
 * most likely children.  Output: the best v = tree_nodes candidates.  Writes
 * KV slots L_b .. L_b + (depth-1) w. */
prism_status prism_draft_tree(prism_ctx *ctx, const prism_batch *batch,
                              int32_t depth, const prism_tree_out *out,
                              void *stream);

/* Target-side scoring of draft trees (paper Sec. 2: the target model scores
 * every candidate of a draft tree in one forward pass under a tree attention
 * mask; the logits then go to prism_verify_tree).  ctx holds the scoring
 * model in the layer structure of this library (one transformer layer with
 * its own weights, the set of step 1, its own frozen embedding, LM head and
 * KV cache).  For sequence b (prior context L_b = batch->d_ctx_lens[b] in the
 * scoring model's cache):
 *   row 0      the root, batch->d_tokens[b], at position and KV slot L_b;
 *   row 1 + j  tree node j, d_tokens[b*n_nodes + j], at position
 *              L_b + d_depth[b*n_nodes + j] and slot L_b + 1 + j, attending to
 *              the prior context, the root and the nodes of
 *              d_mask[b*n_nodes + j] (its ancestors and itself);
 * every row fuses batch->d_features row b.  d_tokens, d_depth and d_mask are
 * [B, n_nodes] as prism_draft_tree writes them (node order: every parent
 * before its children).  Writes d_logits [B, n_nodes + 1, V] fp32 (row 0:
 * the token after the root; row 1 + j: after node j) and the KV slots
 * L_b .. L_b + n_nodes.  The rows run in tree order: bf16 contexts take
 * passes of whole trees, up to 256 rows each; fp32 contexts take passes of
 * up to max_batch * max(1, tree_width) rows (at most 64).  n_nodes <= 63.  A
 * depth outside 1..n_nodes, or a mask without the node's own bit or naming a
 * later node, is clamped and raises PRISM_ERR_INVALID_ARG in
 * prism_device_status. */
prism_status prism_score_tree(prism_ctx *ctx, const prism_batch *batch, int32_t n_nodes,
                              const int32_t *d_tokens, const int32_t *d_depth,
                              const uint64_t *d_mask, float *d_logits, void *stream);

/* Verification of drafted chains (paper Sec. 2, speculative decoding): the
 * target model has scored the K drafts of each sequence in one pass, giving
 * logits row i for the token after i drafts (i = 0..K).  Greedy
 * (temperature == 0): drafts are kept while each equals the arg-max of its
 * target row (ties to the lowest id); the next token is the arg-max of the
 * row after the last kept draft.  Sampled (temperature > 0): draft i is kept
 * when r_i < min(1, p_target(x_i) / p_draft(x_i)) with p = softmax(logits /
 * T) of the target row and of the draft's own row; at the first rejection
 * the next token is drawn from max(0, p_target - p_draft) at that position,
 * and when all K are kept it is drawn from p_target of row K (draws by
 * inverse CDF in token-id order with u = r_K).  Vocabulary V of the context.
 *   d_target_logits [B, K+1, V] fp32      d_draft_logits [B, K, V] fp32
 *                                         (sampled only, else NULL)
 *   d_draft_tokens  [B, K] int32          d_uniforms [B, K+1] fp32
 *                                         (sampled only, else NULL)
 *   d_n_accepted    [B] int32 kept drafts 0..K
 *   d_next_token    [B] int32 the token that follows them
 * B <= max_batch, K <= max_steps.  A draft id outside 0..V-1 is not kept and
 * raises PRISM_ERR_INVALID_ARG in prism_device_status. */
prism_status prism_verify_chain(prism_ctx *ctx, int32_t batch, int32_t K, float temperature,
                                const float *d_target_logits, const float *d_draft_logits,
                                const int32_t *d_draft_tokens, const float *d_uniforms,
                                int32_t *d_n_accepted, int32_t *d_next_token, void *stream);

/* prism_verify_chain for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same verification and kernels, with no context and no
 * allocation.  The statistics of the logits rows live in a fixed device
 * array of the library, one copy per GPU (1 MiB + 256 B, held until the
 * process ends), whose address is resolved once per device (by
 * prism_create, or by the first call on that device).  vocab is V (a
 * multiple of 16); batch * (K + 1) rows, plus batch * K when sampled, may
 * not exceed 8192 (PRISM_ERR_SHAPE otherwise); K <= 63.  Other arguments,
 * outputs and draws are those of prism_verify_chain.  Every call on one GPU
 * shares that array: calls that overlap on one GPU (other streams, other
 * threads) race and must be serialised by the caller.  An out-of-range draft
 * id is not kept, as in prism_verify_chain, but raises no flag (there is no
 * context to report it).  Errors: prism_last_error(NULL). */
prism_status prism_verify_chain_static(int32_t vocab, int32_t batch, int32_t K,
                                       float temperature, const float *d_target_logits,
                                       const float *d_draft_logits,
                                       const int32_t *d_draft_tokens, const float *d_uniforms,
                                       int32_t *d_n_accepted, int32_t *d_next_token,
                                       void *stream);

/* Greedy verification of a draft tree (paper Sec. 2, tree verification
 * under a tree attention mask): target logits row 0 is for the token after
 * the root (the last accepted token), row 1+j for the token after node j.
 * Starting at the root, the child whose token is the arg-max of the current
 * position's row is kept (the first in node order if several), until no
 * child matches.  Nodes as prism_draft_tree outputs them (parent -1 = the
 * root).
 *   d_target_logits [B, n_nodes+1, V] fp32
 *   d_tokens, d_parent [B, n_nodes] int32
 *   d_n_accepted [B]; d_path [B, n_nodes] kept node indices in depth order,
 *   then -1; d_next_token [B] the arg-max after the last kept node.
 * B <= max_batch, n_nodes <= 64. */
prism_status prism_verify_tree(prism_ctx *ctx, int32_t batch, int32_t n_nodes,
                               const float *d_target_logits, const int32_t *d_tokens,
                               const int32_t *d_parent, int32_t *d_n_accepted,
                               int32_t *d_path, int32_t *d_next_token, void *stream);

/* Synchronize `stream` and report device-side flags raised since the last
 * call, the first that applies of: PRISM_ERR_NONFINITE (a row whose logits
 * are all NaN, or a NaN tree score: the tokens of such a row are
 * unspecified and may lie outside 0..V-1; other rows are unaffected),
 * PRISM_ERR_INVALID_ARG (malformed catch-up offsets or tree-scoring rows),
 * PRISM_ERR_CAPACITY
 * (block table / pool / slot out of range), PRISM_ERR_INVALID_ARG (token id
 * out of range), else PRISM_OK.  Clears the flags. */
prism_status prism_device_status(prism_ctx *ctx, void *stream);

/* Measurement support (not part of the drafting computation).  With
 * what != 0, drafting calls launch their kernels directly on `stream`
 * instead of replaying a graph, and record a pair of HIP events on that
 * stream around every launch of the classes selected by the bits of `what`:
 * PRISM_PROFILE_LMHEAD each LM-head launch, PRISM_PROFILE_PRODUCTS each
 * other weight product (fusion FC, QKV, O, gate/up, down; a K-split
 * product with its finish pass), PRISM_PROFILE_PASSES each whole forward
 * pass (a chain step, a tree level; the catch-up prefill with its front).
 * At most 8 pairs per pass are kept.  what = 0 turns profiling off.
 * prism_profile_read() waits for the event pairs of the last drafting call
 * and returns their summed milliseconds and their number;
 * prism_profile_pairs() writes the milliseconds of each pair, in launch
 * order, to ms[0 .. min(cap, count) - 1] and their number to *count. */
enum { PRISM_PROFILE_LMHEAD = 1, PRISM_PROFILE_PRODUCTS = 2, PRISM_PROFILE_PASSES = 4 };
prism_status prism_profile_enable(prism_ctx *ctx, int32_t what);
prism_status prism_profile_read(prism_ctx *ctx, float *total_ms, int32_t *count);
prism_status prism_profile_pairs(prism_ctx *ctx, float *ms, int32_t cap, int32_t *count);

/* Captured-graph cache of a context.  Chain and tree calls capture one HIP
 * graph per distinct (call kind, shape, buffer pointers, step map) and
 * replay it; at most *capacity graphs are kept, and capturing one more
 * first destroys the least recently used (after a device-wide
 * synchronization, since it may still be running).  Writes the number held
 * and the capacity. */
prism_status prism_graph_cache(const prism_ctx *ctx, int32_t *n_graphs, int32_t *capacity);

#ifdef __cplusplus
}
#endif

#endif /* PRISM_DRAFT_H */
