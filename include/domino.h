/*
 * domino.h — C ABI of the MI355X (gfx950) Domino drafting library.
 *
 * The library runs one speculative-decoding draft step of the Domino method
 * ("Domino: Decoupling Causal Modeling from Autoregressive Drafting in
 * Speculative Decoding"): a parallel draft backbone over the masked block
 * (Sec. 4.1.1), the frozen LM head giving base logits (Sec. 4.1.1, base-logit
 * equation), the Domino head's GRU causal encoder and low-rank logit-space
 * correction rolled out over the block (Sec. 4.1.2, Fig. 3), construction of
 * a draft tree from the per-position top-beta tokens, and greedy acceptance of
 * the longest valid prefix plus a bonus token (Sec. 3.1).
 *
 * Conventions for every call:
 *  - Pointers named as device memory must be device pointers (hipMalloc or a
 *    torch CUDA tensor); the caller owns all of them.  Host-side arguments are
 *    the config/weight structs and scalar sizes.
 *  - `stream` is a hipStream_t (NULL = the default stream).  The draft, tree
 *    and acceptance calls only enqueue work and return; they never allocate
 *    and never synchronise.
 *  - Return codes cover argument validation (done before any HIP call) and
 *    launch errors.  Conditions only visible on the device (a token id out of
 *    range, a context length above max_ctx, a malformed tree) are clamped so
 *    that no access leaves its buffer, and are recorded in an error word at
 *    the start of the workspace, read with domino_workspace_error().
 *  - domino_last_error() returns a thread-local message for the last failure.
 *  - No C++ exception crosses this boundary.  A model handle may be used from
 *    several streams, but calls that share one workspace must not overlap.
 *  - Storage type: DOMINO_BF16 stores weights and KV caches as bfloat16,
 *    DOMINO_F32 as float; all arithmetic is fp32 (bf16 operands are exact in
 *    fp32; activations feeding bf16 matrix cores are split into a high and a
 *    low bf16 part so products keep fp32 accuracy).
 */
#ifndef DOMINO_H
#define DOMINO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DOMINO_OK = 0,
  DOMINO_ERR_INVALID_ARG = -1,  /* a NULL pointer, a size out of range, shapes that disagree */
  DOMINO_ERR_WORKSPACE = -2,    /* workspace NULL or smaller than the *_workspace_bytes query */
  DOMINO_ERR_UNSUPPORTED = -3,  /* a shape this build does not handle (message says which) */
  DOMINO_ERR_HIP = -4,          /* a HIP runtime call failed (message carries hipGetErrorString) */
  DOMINO_ERR_DEVICE = -5        /* returned by domino_workspace_error when the error word is set */
} domino_status;

typedef enum { DOMINO_F32 = 0, DOMINO_BF16 = 1 } domino_dtype;

/* Bits of the device error word (domino_workspace_error). */
enum {
  DOMINO_DEV_BAD_TOKEN = 1,       /* an anchor / forced / tree token id outside [0, vocab) (clamped) */
  DOMINO_DEV_BAD_CTX_LEN = 2,     /* ctx_lens[b] outside [n_new, max_ctx] (clamped) */
  DOMINO_DEV_BAD_TREE = 4,        /* a node_parent entry that is not an earlier node (ignored) */
  DOMINO_DEV_BARRIER_TIMEOUT = 8  /* a bounded cross-workgroup wait of the rollout exceeded its spin bound */
};

/*
 * Model shape.  `block` is B = 16 in the paper (anchor + B-1 draft positions,
 * Sec. 4.1.1 and Sec. 5.1); gru_hidden d_s = 1024 and rank r = 256 (Sec. 4.1.2,
 * Sec. 5.1).  Layers follow the Qwen3 layout: pre-RMSNorm, per-head q/k
 * RMSNorm, rotate-half RoPE, grouped-query attention, SwiGLU, no biases.
 * Limits of this build: head_dim in {64, 128}; hidden, ffn, gru_hidden and
 * n_q_heads*head_dim multiples of 32; gru_hidden at most 2048 (bf16) or 1024
 * (f32); rank 256 (bf16) or 128/256 (f32); n_q_heads a multiple of
 * n_kv_heads with (n_q_heads/n_kv_heads)*block <= 128; block in [2, 64];
 * mask_token_id in [0, vocab).  domino_model_create also builds the table
 * G = embed * gru_w_ih^T ([vocab, 3*gru_hidden] fp32) used by the rollout.
 * ctx_fuse_layers k in [0, 8]: with k > 0 a projected context row is the
 * concatenation of k target layers' hidden states ([k*hidden]), fused to
 * width hidden by the weight ctx_fc before each layer's K/V projections (the
 * context features C_t of Sec. 4.1.1; the paper states no formula for them:
 * k = 5 at the Qwen3-8B shape is the ~84M map its +5.3% parameter figure of
 * Sec. 1 implies).  k = 0: rows are hidden wide and used as they are.
 * domino_target_create ignores it.
 */
typedef struct {
  int32_t hidden, n_layers, n_q_heads, n_kv_heads, head_dim, ffn, vocab;
  int32_t block, gru_hidden, rank, mask_token_id;
  float rms_eps, rope_theta;
  domino_dtype dtype;
  int32_t ctx_fuse_layers;
} domino_config;

/*
 * Weights: device pointers in the config's storage type, row-major [out, in].
 * Per-layer fields are HOST arrays of n_layers device pointers.
 *   embed [V, d] (shared frozen target embedding), lm_head [V, d] (shared
 *   frozen target LM head), final_norm [d];
 *   per layer: attn_norm [d], wq [nq*dh, d], wk [nkv*dh, d], wv [nkv*dh, d],
 *   q_norm [dh], k_norm [dh], wo [d, nq*dh], ffn_norm [d],
 *   w_gate [ffn, d], w_up [ffn, d], w_down [d, ffn];
 *   GRU (reset-after form, gate order r, z, n): gru_w_ih [3ds, d],
 *   gru_w_hh [3ds, ds], gru_b_ih [3ds], gru_b_hh [3ds];
 *   correction: w1 [r, d + ds] with columns [H | S], w2 [V, r];
 *   context fusion (only when ctx_fuse_layers k > 0, else ignored):
 *   ctx_fc [d, k*d], its column block i acting on the i-th concatenated layer.
 * domino_model_create copies every matrix into its own device memory in a
 * matrix-core tile order; it keeps borrowing embed, the norm gains and the
 * GRU biases, which the caller keeps alive until domino_model_destroy.
 */
typedef struct {
  const void *embed, *lm_head, *final_norm;
  const void *const *attn_norm, *const *wq, *const *wk, *const *wv, *const *q_norm,
      *const *k_norm, *const *wo, *const *ffn_norm, *const *w_gate, *const *w_up, *const *w_down;
  const void *gru_w_ih, *gru_w_hh, *gru_b_ih, *gru_b_hh;
  const void *w1, *w2;
  const void *ctx_fc;
} domino_weights;

/* Optional per-step debug outputs (device fp32; any field may be NULL).
 *   hidden       [bs, B-1, d]   post-final-norm H_j (the LM-head input)
 *   base_logits  [bs, B-1, V]   L_base_j
 *   final_logits [bs, B-1, V]   L_j = L_base_j + dL_j
 *   states       [bs, B-1, ds]  S_{j-1}, the GRU state used at position j */
typedef struct {
  float *hidden, *base_logits, *final_logits, *states;
} domino_debug;

typedef struct domino_model *domino_model_t;

/* Validate the config, pack the weights (blocking: runs on the default stream
 * and synchronises).  On success *out owns device memory freed by destroy. */
domino_status domino_model_create(const domino_config *cfg, const domino_weights *w,
                                  domino_model_t *out);
void domino_model_destroy(domino_model_t m);

/* Bytes of workspace domino_draft_step needs for `batch` rows, caches of
 * `max_ctx` positions, up to `max_new` projected context rows and top-`branch`
 * outputs.  Returns 0 for invalid arguments. */
size_t domino_workspace_bytes(domino_model_t m, int32_t batch, int32_t max_ctx, int32_t max_new,
                              int32_t branch);

/* Thread-local text of the last error (never NULL). */
const char *domino_last_error(void);

/*
 * One draft step (Sec. 4.1.1 block construction, backbone and LM head;
 * Sec. 4.1.2 causal encoder and correction; Fig. 3 sequential rollout).
 *  batch           rows, in [1, 64]
 *  anchor_ids      device int32 [batch]: x_t, the last verified token
 *  ctx_lens        device int32 [batch]: context length n_b (RoPE positions of
 *                  the block are n_b .. n_b+B-1), in [n_new, max_ctx]
 *  ctx_k, ctx_v    device [n_layers][batch][max_ctx][n_kv][d_h] in the storage
 *                  type; K is post k-norm and RoPE.  Read-only unless n_new > 0.
 *  ctx_hidden_new  optional device fp32 [batch][n_new][w] target hidden states,
 *                  w = k*d with ctx_fuse_layers k > 0 (fused by ctx_fc first),
 *                  else d; when given, row i is projected with each layer's
 *                  W_k (k-norm, RoPE) and W_v and written at position
 *                  n_b - n_new + i.
 *  branch          beta in [1, 8]: entries kept per position
 *  forced_tokens   optional device int32 [batch][B-1]: teacher forcing — the
 *                  token fed to the causal encoder after position j is
 *                  forced[b][j-1] instead of the top-1 draft token
 *  topk_ids        device int32 [batch][B-1][branch], order (value desc, id asc)
 *  topk_vals       device fp32  [batch][B-1][branch]: final logits L_j
 *  debug           optional (NULL when timed)
 *  workspace       device, >= domino_workspace_bytes(m, batch, max_ctx, n_new, branch)
 */
domino_status domino_draft_step(domino_model_t m, int32_t batch, const int32_t *anchor_ids,
                                const int32_t *ctx_lens, void *ctx_k, void *ctx_v, int32_t max_ctx,
                                const void *ctx_hidden_new, int32_t n_new, int32_t branch,
                                const int32_t *forced_tokens, int32_t *topk_ids, float *topk_vals,
                                const domino_debug *debug, void *workspace, size_t workspace_bytes,
                                void *stream);

/*
 * One draft step with temperature sampling (Fig. 3: each draft token is drawn
 * from the final logits l_i + c_i; here from softmax((l_i + c_i) / T)), branch 1.
 * Same arguments as domino_draft_step except:
 *  temperature     T > 0 (finite)
 *  seed            64-bit key of the Philox-4x32-10 draws (Salmon et al., SC
 *                  2011): the token at depth j of row b is
 *                  argmax_v (L_j[v] / T + g), g = -log(-log u) of the word
 *                  (seed; counter v/4, j, b, stream 0; word v%4), u = (floor(
 *                  word / 2^9) + 1/2) / 2^23 — a draw from softmax(L_j / T);
 *                  the same step with the same seed draws the same tokens
 *  topk_ids        device int32 [batch][B-1][1]: the drawn tokens (fed back to
 *                  the causal encoder unless forced_tokens is given)
 *  topk_vals       device fp32 [batch][B-1][1]: the drawn tokens' final logits
 *  final_logits    device fp32 [batch][B-1][vocab], required: L_j, which
 *                  domino_verify_sample needs as the draft distributions
 *  debug           optional; its final_logits field is ignored
 *  workspace       >= domino_workspace_bytes(m, batch, max_ctx, n_new, 1)
 */
domino_status domino_draft_step_sampled(domino_model_t m, int32_t batch, const int32_t *anchor_ids,
                                        const int32_t *ctx_lens, void *ctx_k, void *ctx_v, int32_t max_ctx,
                                        const void *ctx_hidden_new, int32_t n_new, float temperature,
                                        uint64_t seed, const int32_t *forced_tokens, int32_t *topk_ids,
                                        float *topk_vals, float *final_logits, const domino_debug *debug,
                                        void *workspace, size_t workspace_bytes, void *stream);

/* Bytes of workspace domino_train_forward needs (0 for invalid arguments). */
size_t domino_train_workspace_bytes(domino_model_t m, int32_t batch, int32_t max_ctx, int32_t max_new);

/*
 * Teacher-forced training forward and the base-anchored curriculum loss
 * (Sec. 4.2).  The block goes through the backbone and LM head as in
 * domino_draft_step; the causal encoder is fed the ground-truth tokens (the
 * anchor, then labels[b][0 .. B-3]), and for every draft position k = 0..B-2
 *   CE_base[b][k]  = -log softmax(L_base)[labels[b][k]]
 *   CE_final[b][k] = -log softmax(L_base + W2 u)[labels[b][k]]
 * (NaN logits count as -inf).  With w_k = exp(-k / gamma):
 *   L_base  = sum_{b,k} w_k CE_base  / (batch * sum_k w_k), likewise L_final,
 *   loss    = (1 - lambda) L_final + lambda L_base.
 * The corrected logits are reduced on chip; they reach memory only through
 * debug->final_logits.  Deterministic: no floating-point atomics.
 * Same arguments as domino_draft_step except:
 *  labels          device int32 [batch][B-1]: ground-truth tokens of the draft
 *                  positions; a label outside [0, vocab) sets DOMINO_DEV_BAD_TOKEN
 *                  and gives NaN CEs
 *  lambda          curriculum weight in [0, 1] (annealed 1 -> 0 by the caller)
 *  gamma           position decay, positive and finite
 *  loss            device fp32 [3]: total, L_base, L_final
 *  ce              optional device fp32 [2][batch][B-1]: CE_base, then CE_final
 *  debug           optional; hidden, base_logits, final_logits (L_base + W2 u)
 *                  and states as in domino_draft_step
 *  workspace       >= domino_train_workspace_bytes(m, batch, max_ctx, n_new)
 */
domino_status domino_train_forward(domino_model_t m, int32_t batch, const int32_t *anchor_ids,
                                   const int32_t *ctx_lens, void *ctx_k, void *ctx_v, int32_t max_ctx,
                                   const void *ctx_hidden_new, int32_t n_new, const int32_t *labels,
                                   float lambda, float gamma, float *loss, float *ce,
                                   const domino_debug *debug, void *workspace, size_t workspace_bytes,
                                   void *stream);

/*
 * Target decoder for the verify side of a speculative cycle (Sec. 3.1: the
 * target scores every drafted candidate in one forward pass).  Same config and
 * weight structs as the drafter; the Domino-head fields (gru_*, w1, w2,
 * gru_hidden, rank) are ignored and may be NULL / 0, and `block` is unused
 * (the node count is given per call).  Layers, embedding and LM head are
 * packed as for the drafter; the handle only serves domino_target_* calls.
 */
domino_status domino_target_create(const domino_config *cfg, const domino_weights *w, domino_model_t *out);

/* Workspace for domino_target_verify (0 for invalid or unsupported arguments). */
size_t domino_target_workspace_bytes(domino_model_t target, int32_t batch, int32_t n_nodes, int32_t max_ctx);

/*
 * Tree-verify forward: target logits of every node of the draft trees.
 * Node i of batch row b (the arrays domino_build_tree writes) holds token
 * node_token[b][i] at RoPE position node_pos[b][i]; in every layer it attends to
 * the cached context positions [0, ctx_lens[b]) and to the nodes k with
 * ancestor_mask[b][i][k] != 0 (its root-to-node path; the diagonal always
 * counts), so each node is scored as plain causal decoding of its path would
 * score it.  Every node's K (post k-norm and RoPE) and V are also written into
 * the cache at position ctx_lens[b] + i of every layer, for domino_target_commit.
 *  n_nodes         N + 1 in [1, 64], and at most the largest block the
 *                  attention supports: (n_q_heads / n_kv_heads) * n_nodes <= 128
 *                  after rounding n_nodes up to a supported size
 *                  (DOMINO_ERR_UNSUPPORTED otherwise)
 *  node_token, node_pos  device int32 [batch][n_nodes]; ancestor_mask device
 *                  uint8 [batch][n_nodes][n_nodes]
 *  ctx_lens        device int32 [batch]; ctx_lens[b] + n_nodes <= max_ctx (else
 *                  DOMINO_DEV_BAD_CTX_LEN and the node K/V are not stored)
 *  ctx_k, ctx_v    device [n_layers][batch][max_ctx][n_kv][d_h] storage type
 *  logits          device [batch][n_nodes][vocab], fp32 or bf16 (RNE): row i is
 *                  the target's next-token logits after node i's token
 *  workspace       >= domino_target_workspace_bytes(target, batch, n_nodes, max_ctx)
 */
domino_status domino_target_verify(domino_model_t target, int32_t batch, int32_t n_nodes, const int32_t *node_token,
                                   const int32_t *node_pos, const uint8_t *ancestor_mask, const int32_t *ctx_lens,
                                   void *ctx_k, void *ctx_v, int32_t max_ctx, void *logits, domino_dtype logits_dtype,
                                   void *workspace, size_t workspace_bytes, void *stream);

/*
 * Cache commit after acceptance: node 0 (the anchor, already at ctx_lens[b])
 * and the accepted path (accepted_nodes[b][0 .. accept_len[b]-1], as
 * domino_verify_accept writes them) become positions ctx_lens[b] ..
 * ctx_lens[b] + accept_len[b] of every layer's cache; new_ctx_lens[b] =
 * ctx_lens[b] + 1 + accept_len[b].  The node at depth d must have id >= d
 * (breadth-first order) and be < n_nodes, else DOMINO_DEV_BAD_TREE and the row
 * is left unchanged (new_ctx_lens[b] = ctx_lens[b]).
 *  max_depth       B - 1: the row stride of accepted_nodes, in [1, 63]
 *  new_ctx_lens    device int32 [batch], must not alias ctx_lens
 *  workspace       the verify workspace (its error word)
 */
domino_status domino_target_commit(domino_model_t target, int32_t batch, int32_t n_nodes, int32_t max_depth,
                                   const int32_t *ctx_lens, const int32_t *accept_len, const int32_t *accepted_nodes,
                                   void *ctx_k, void *ctx_v, int32_t max_ctx, int32_t *new_ctx_lens, void *workspace,
                                   void *stream);

/*
 * Draft tree from the per-position top-beta tokens (spine-and-leaves, BFS
 * order).  The paper names tree construction as one cost of a draft step (the
 * caption of Fig. 1, beside Draft, LM Head and DHead) without defining the
 * tree, and runs Domino itself as a single block (Table 1), which is the
 * branch = 1 chain below.  The shape for branch > 1 is this library's reading:
 * the branch top-ranked tokens of every depth, only the rank-0 token having
 * children.  Node 0 is the anchor (parent -1, depth 0, position n_b); node
 * 1 + (d-1)*branch + rho holds topk_ids[b][d-1][rho] at depth d, position
 * n_b + d, with parent 0 for d = 1 and 1 + (d-2)*branch (the rank-0 node one
 * level up) otherwise.  ancestor_mask[b][i][k] = 1 iff k is i or an ancestor
 * of i.  N + 1 = 1 + depth*branch nodes per row.
 *  depth in [1, 63], branch in [1, 8]; topk_ids device int32 [batch][depth][branch];
 *  anchor_ids, ctx_lens device int32 [batch]; node_* device int32 [batch][N+1];
 *  ancestor_mask device uint8 [batch][N+1][N+1] or NULL.
 */
domino_status domino_build_tree(int32_t batch, int32_t depth, int32_t branch,
                                const int32_t *topk_ids, const int32_t *anchor_ids,
                                const int32_t *ctx_lens, int32_t *node_token, int32_t *node_parent,
                                int32_t *node_depth, int32_t *node_pos, uint8_t *ancestor_mask,
                                void *stream);

/* Workspace bytes for domino_verify_accept. */
size_t domino_verify_workspace_bytes(int32_t batch, int32_t n_nodes, int32_t vocab);

/*
 * Greedy acceptance (Sec. 3.1).  R_m = argmax_v target_logits[b][m][v] under
 * (value desc, id asc), NaN as -inf.  From the root, while some child c of the
 * current node has node_token[c] == R_cur, accept c and move to it; the bonus
 * token is R at the last accepted node, so tau = accept_len + 1 in [1, B].
 * Any tree works (node_parent[c] < c for c > 0, node_parent[0] = -1); only rows
 * of nodes with children, plus the final node's row, are read.
 *  n_nodes in [1, 1024]; block B in [2, 64] bounds the walk at B-1 steps;
 *  target_logits device [batch][n_nodes][vocab] fp32 or bf16;
 *  accept_len device int32 [batch]; accepted_nodes device int32 [batch][B-1]
 *  (-1 padded); out_tokens device int32 [batch][B] (accepted tokens then the
 *  bonus, -1 padded).
 */
domino_status domino_verify_accept(int32_t batch, int32_t n_nodes, int32_t vocab, int32_t block,
                                   const int32_t *node_token, const int32_t *node_parent,
                                   const void *target_logits, domino_dtype logits_dtype,
                                   int32_t *accept_len, int32_t *accepted_nodes,
                                   int32_t *out_tokens, void *workspace, size_t workspace_bytes,
                                   void *stream);

/*
 * Greedy acceptance exactly as domino_verify_accept, for callers that cannot
 * allocate or hand over a workspace (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation).  It calls no allocating
 * routine: its argmax partials live in a fixed device array of
 * DOMINO_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends.  batch * n_nodes * ceil(vocab / 4096) * 8 bytes must
 * fit in it (e.g. batch 32 x 61 nodes at vocab 151936: 593 KB), else
 * DOMINO_ERR_UNSUPPORTED before any launch.  Every call on a GPU shares that
 * GPU's array, so calls that overlap on one GPU (other streams, other threads)
 * race and must be serialised by the caller.
 *  error_word  device int32 [1]: cleared by the call's first kernel, then
 *              DOMINO_DEV_BAD_TREE if a node_parent entry is not an earlier node
 *  other arguments as domino_verify_accept
 */
#define DOMINO_NOALLOC_SCRATCH_BYTES (4u << 20)
domino_status domino_verify_accept_noalloc(int32_t batch, int32_t n_nodes, int32_t vocab, int32_t block,
                                           const int32_t *node_token, const int32_t *node_parent,
                                           const void *target_logits, domino_dtype logits_dtype,
                                           int32_t *accept_len, int32_t *accepted_nodes, int32_t *out_tokens,
                                           int32_t *error_word, void *stream);

/* Workspace bytes for domino_verify_sample. */
size_t domino_verify_sample_workspace_bytes(int32_t batch, int32_t block, int32_t vocab);

/*
 * Speculative-sampling verification of a drafted chain at temperature T
 * (Sec. 3.1, the standard speculative verification rule), branch 1.
 * For depth j = 1..B-1, p_j = softmax(target_logits[b][j-1] / T) (row m is the
 * target's distribution after node m) and q_j = softmax(draft_logits[b][j-1] /
 * T).  Draft token x_j = node_token[b][j] is accepted iff u_j q_j(x_j) <
 * p_j(x_j), i.e. with probability min(1, p_j(x_j) / q_j(x_j)), u_j the uniform
 * of (seed; counter 0, j, b, stream 1; word 0).  At the first rejection j the
 * bonus token is a draw from max(0, p_j - q_j) (normalised); if all B-1 are
 * accepted, from p_B; draws are argmax_v (log w_v + g_v) over w_v > 0 with g
 * from (seed; counter v/4, j, b, stream 2; word v%4).  NaN logits count as
 * -inf.  tau = accept_len + 1 in [1, B].
 *  block B in [2, 64]; node_token device int32 [batch][B] (node 0 the anchor,
 *  node j the draft token at depth j); target_logits device [batch][B][vocab]
 *  fp32 or bf16; draft_logits device fp32 [batch][B-1][vocab] (the
 *  final_logits of domino_draft_step_sampled); accept_len device int32
 *  [batch]; accepted_nodes device int32 [batch][B-1] (node indices, -1
 *  padded); out_tokens device int32 [batch][B] (accepted tokens then the
 *  bonus, -1 padded).  An out-of-range draft token sets DOMINO_DEV_BAD_TOKEN
 *  and counts as rejected.
 */
domino_status domino_verify_sample(int32_t batch, int32_t block, int32_t vocab, const int32_t *node_token,
                                   const void *target_logits, domino_dtype logits_dtype,
                                   const float *draft_logits, float temperature, uint64_t seed,
                                   int32_t *accept_len, int32_t *accepted_nodes, int32_t *out_tokens,
                                   void *workspace, size_t workspace_bytes, void *stream);

/* Philox-4x32-10 (Salmon et al., SC 2011) of n explicit counters: counters
 * device uint32 [n][4], key = (key lo, key hi) 32-bit words, out device uint32
 * [n][4].  The generator behind the sampled calls, for callers and tests that
 * need the same draws. */
domino_status domino_philox4x32_10(const uint32_t *counters, uint64_t key, uint32_t *out, int32_t n,
                                   void *stream);

/* Copy the device error word at the start of a draft or verify workspace to
 * *out (synchronises `stream`).  Returns DOMINO_ERR_DEVICE when it is set. */
domino_status domino_workspace_error(const void *workspace, void *stream, int32_t *out);

/* Clear the error word (stream-ordered). */
domino_status domino_workspace_clear_error(void *workspace, void *stream);

/*
 * Per-kernel-class timing for benchmarks: while enabled for a class, the
 * draft step brackets that class's launches with HIP events on its stream.
 * domino_profile_read synchronises and returns the summed milliseconds and
 * the number of launches timed since the last reset.  Classes that currently
 * have no launches of their own (EMBED: the embedding gather is part of the
 * first NORM launch; W1H: W1's H half shares the LMHEAD launch) read back zero
 * launches.  CTXPROJ times the context fusion (ctx_fc) of appended rows; their
 * K/V projections ride in the QKV launches.
 */
enum {
  DOMINO_KC_EMBED = 0, DOMINO_KC_NORM, DOMINO_KC_QKV, DOMINO_KC_ROPE, DOMINO_KC_ATTN,
  DOMINO_KC_WO, DOMINO_KC_GATEUP, DOMINO_KC_DOWN, DOMINO_KC_LMHEAD, DOMINO_KC_W1H,
  DOMINO_KC_HEADLOOP, DOMINO_KC_CTXPROJ, DOMINO_KC_TRAINLOSS, DOMINO_KC_COUNT
};
domino_status domino_profile_enable(domino_model_t m, uint32_t class_mask);
domino_status domino_profile_read(domino_model_t m, int32_t kernel_class, double *total_ms,
                                  int32_t *launches);
domino_status domino_profile_reset(domino_model_t m);

/*
 * Test hook for the failure path of the persistent rollout (greedy or sampled
 * drafting with bf16 weights, rank 256 and up to four batch rows, one launch
 * per pair of rows): the number
 * of polls a cross-workgroup wait may make before it gives up, raising
 * DOMINO_DEV_BARRIER_TIMEOUT in the error word and letting every workgroup
 * leave (the step's outputs are then undefined); 0 makes every wait give up at
 * once.  A negative value restores the default (2^22 polls, seconds).  Applies
 * to the model's later draft steps.
 */
domino_status domino_debug_set_poll_limit(domino_model_t m, int32_t polls);

/*
 * Which execution paths the model's last draft step (greedy, sampled or
 * training forward) launched, as DOMINO_PATH_* bits, so that tests can check
 * that a shape took the path they mean to cover.  Recorded on the host at
 * launch time; 0 before the first step.
 */
enum {
  DOMINO_PATH_PERSISTENT_ROLLOUT = 1  /* the whole rollout as one persistent launch */
};
domino_status domino_debug_last_paths(domino_model_t m, uint32_t *paths);

#ifdef __cplusplus
}
#endif
#endif /* DOMINO_H */
