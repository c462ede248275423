// Launch interfaces between the host C-ABI (api.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dk {

// Most column groups a residual epilogue (and so a deferred RMSNorm) covers.
constexpr int kNormGroups = 64;

// EPI_STORE: outputs (or K-split partials) stored; EPI_SWIGLU: silu(gate) * up
// of interleaved (gate, up) tile pairs; EPI_RESID: K-split partials, then the
// residual update with the next RMSNorm's statistics (GemmArgs res_*)
enum { EPI_STORE = 0, EPI_SWIGLU = 2, EPI_RESID = 3 };

struct GemmArgs {
  const void *P;   // packed weights
  int KS;          // k-steps per packed tile
  int tile0;       // first packed tile of this launch
  int ntiles;      // packed tiles computed by this launch
  int N;           // valid output columns
  const float *X;  // activations fp32 [M][ldx]
  int ldx, M, K;
  float *Y;        // output fp32 [M][ldy]; K-split ky writes Y + ky*ysplit
  int ldy;
  size_t ysplit;
  int ksplit;
  void *xf = nullptr;  // wide kernel: scratch for the activations' hi/lo fragment planes
                       // (gemm_wide_scratch_bytes(M, K) bytes)
  // Deferred RMSNorm of the activations (skinny kernel): X holds x * gain and
  // every output row m is scaled by rsqrt(sum_g rs_ssq[g][m] / rs_d + rs_eps),
  // the per-row sums of squares left by the producing projection's EPI_RESID.
  const float *rs_ssq = nullptr;
  int rs_ng = 0, rs_d = 0;
  float rs_eps = 0.f;
  // EPI_RESID (skinny kernel, K split over workgroups): each split's partial
  // goes out to the device coherence point and the last split of a column group
  // to arrive (res_tickets[group], zero at launch) adds the partials in split
  // order to res_in, writes the sum to res_out and, times res_gain, to res_xg,
  // and the sum's squares over the group's columns to res_ssq[group][m].
  const float *res_in = nullptr;
  float *res_out = nullptr, *res_xg = nullptr, *res_ssq = nullptr;
  const void *res_gain = nullptr;
  unsigned *res_tickets = nullptr;
};

struct GemmPlan {
  int MT, WPT, groups, mgroups, ksplit;
  int kcm;  // k-steps per staged chunk (16/MT, or 8/MT for finer K splits)
  int nw;   // waves (= tiles) per workgroup: 8 or 6
  int pgrid;  // > 0: that many workgroups loop over the groups (one pipeline across groups)
  int wide = 0;  // 1: the wide-activation kernel (gemm_wide.hip) runs this plan
};

// max_split = 1: one workgroup covers all of K (direct output); otherwise K
// may be split up to max_split ways into partial outputs.
GemmPlan plan_gemm(int ntiles, int KS, int M, int epi, int n_cu, int max_split);
void launch_gemm(bool bf16, int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st);
// Wide activations (bf16 weights; more rows than the skinny kernel's 64 per
// m-group): the activations are first split into hi/lo bf16 fragment planes
// (in a.xf), then workgroup tiles of 256 columns x 256 rows multiply them with
// the same packed weights; K-split partials as above.
GemmPlan plan_gemm_wide(int ntiles, int KS, int M, int epi, int n_cu, int max_split);
// false (nothing launched) when the arguments break the kernel's assumptions
// (K not 32 KS, no rows, no fragment scratch)
bool launch_gemm_wide(int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st);
size_t gemm_wide_scratch_bytes(int M, int K);
// above this many rows a bf16 GEMM whose K is a multiple of 32 runs the wide kernel
constexpr int kSkinnyMaxRows = 64;
void launch_pack(bool bf16, const void *W, int N, int K, int ldw, void *P, int NT, int KS,
                 int tile_mul, int tile_off, hipStream_t st);
inline int kstep_of(bool bf16) { return bf16 ? 32 : 16; }

// ---- backbone pieces (backbone.hip)
struct Dims {
  int bs, B, d, nq, nkv, dh, ffn, V, ds, r, mask_id;
  float eps, theta;
  bool bf16;
  const double *inv_freq;  // device [dh/2]: theta^(-2i/dh), fp64
};

void launch_embed_block(const Dims &D, const void *embed, const int32_t *anchor, float *X,
                        int32_t *err, hipStream_t st);
// x_out[map(row)] = x[map(row)] + sum of np partials (pstride floats apart),
// y[row] = rmsnorm(x_out[map(row)]) * gain; with skip_anchor, output row i
// reads input row i + i/(B-1) + 1 (the draft rows of each block).  x_out
// (null: not written) must not alias x.
// With `embed` given, x rows are first set to the embedding rows of the masked
// block ([anchor, MASK, ...]) before the (empty) partial sum.
// With `tokens` given (and `embed`), row i's token is tokens[i] instead.
// With `hdr` given (and `embed`, no skip_anchor), the launch also zeroes
// hdr[0 .. hdr_words) (the step's workspace header; hdr[0] is `err`) before
// any error of its own is raised.
void launch_add_norm(const Dims &D, const float *x, float *x_out, int ldx, const float *parts, int np, size_t pstride,
                     const void *gain, float *y, int ldy, int rows, int width, bool skip_anchor,
                     const void *embed, const int32_t *anchor, int32_t *err, hipStream_t st,
                     const int32_t *tokens = nullptr, uint32_t *hdr = nullptr, int hdr_words = 0);
// q/k RMSNorm + RoPE on the QKV projection (sum of np partials); writes
// Q [M][nq][dh], Kb/Vb [M][nkv][dh].  The projection's rows M + b*n_new + i
// (n_new appended context rows per batch row) have their K (k-norm, RoPE at
// n_b - n_new + i) and V stored into this layer's cache ck/cv.
// With pos_rows, block row m is rotated at pos_rows[m] instead of n_b + j; the
// first n_store rows of each block also store their K/V into the cache at n_b + j.
void launch_qk_norm_rope(const Dims &D, const float *qkv, int np, size_t pstride, const void *q_norm,
                         const void *k_norm, const int32_t *ctx_lens, int max_ctx, float *Q, float *Kb,
                         float *Vb, int n_new, void *ck, void *cv, int32_t *err, hipStream_t st,
                         const int32_t *pos_rows = nullptr, int n_store = 0);
int attn_nchunks(int max_ctx, int B);
// amask (optional, [bs][B][B] bytes, B a multiple of 4 and at most 64): block
// query j sees block key k only where amask[b][j][k] is set.
void launch_attention(const Dims &D, const float *Q, const float *Kb, const float *Vb,
                      const void *ck, const void *cv, const int32_t *ctx_lens, int max_ctx,
                      float *part, float *O, int32_t *err, hipStream_t st, const uint8_t *amask = nullptr);
size_t attn_part_floats(const Dims &D, int max_ctx);
bool attn_supported(int nq, int nkv, int B);

// ---- Domino head rollout (head.hip)
constexpr uint32_t kDefaultPollLimit = 1u << 22;  // polls a rollout wait makes before it gives up
// Spacing of the persistent rollout's exchange slots, in 64-bit words: one
// slot per 64-byte sector.  Every workgroup polls every slot; packed eight to
// a sector, the polls of all workgroups queue on a handful of sectors and an
// all-to-all round takes about 2.5 us, against about 1.6 us at this spacing.
constexpr int kSlotStride = 8;

struct HeadArgs {
  Dims D;
  int beta;
  const float *gtab;     // [V][3ds] = E W_ih^T + b_ih (built at model creation)
  const void *w_hh;      // [3ds][ds]
  const float *bhh;      // b_hh in fp32 [3ds] (b_ih is folded into gtab)
  const void *w1;        // [r][d+ds]; the S half starts at column d
  const void *w2p;       // W2 packed (tile-major, KS = r / KSTEP)
  const float *P;        // [bs][B-1] rows of stride ldp: W1[:, :d] H_j
  int ldp;
  const float *Lbase;    // [bs][B-1] rows of stride ldl: L_base_j
  int ldl;
  const int32_t *anchor; // [bs]
  const int32_t *forced; // [bs][B-1] or null
  int32_t *topk_ids;     // [bs][B-1][beta]
  float *topk_vals;
  float *final_logits;   // optional [bs][B-1][V]
  float *states;         // optional [bs][B-1][ds]
  float *hbuf;           // [2][bs][ds] states by parity of the position
  float *ghbuf;          // [2][bs][3ds] W_hh S by parity (fused small-batch path)
  float *ubuf;           // u of batch row b, position j at ubuf + b*u_ld + (j-1)*u_pos
  int u_ld, u_pos;       // (r, 0) while drafting; (r(B-1), r) keeps every position's u
  int skip_u;            // state recurrence only (states to `states`); u is formed by the caller
  float *pval;           // [B-1][bs][GC][beta] per-workgroup top-beta lists
  int32_t *pid;
  unsigned long long *best;  // [B-1][bs][8] best (value, id) keys per position, zeroed per step
  // temperature sampling (branch 1): the selection key is L / T + Gumbel noise
  // (Philox stream RNG_DRAFT); praw [B-1][bs][GC] keeps each workgroup's chosen
  // token's raw final logit for topk_vals
  int sample;
  float inv_temp;
  uint32_t seed_lo, seed_hi;
  float *praw;
  int32_t *err;
  int GC;                // workgroups of the logits kernel
  // persistent rollout exchange (workspace header, zeroed at every step):
  // u slots [bs][r] and per-workgroup best-key slots [bs][GC], each a 64-bit
  // word tagged with the position, kSlotStride words apart; abort flag of its
  // bounded waits
  unsigned long long *uslot, *kslot;
  unsigned *abort_flag;
  unsigned poll_limit;  // polls a wait makes before it gives up
  // batches above kHeadFusedBatch: W_hh S and W1[:, d:] S run as K-split
  // GEMMs over packed copies of the two matrices (partials in hpart:
  // [kHeadMaxSplit][bs][3ds], then [kHeadMaxSplit][bs][r])
  const void *whh_p, *w1s_p;
  int whh_NT, whh_KS, w1s_NT, w1s_KS;
  float *hpart;
  int n_cu;
  int row0 = 0;  // batch row of this launch's first row (the Philox stream's row index)
};
constexpr int kHeadFusedBatch = 8;  // batches up to this run the fused state kernel
constexpr int kHeadMaxSplit = 16;
inline size_t head_part_floats(const Dims &D) {
  return D.bs > kHeadFusedBatch ? (size_t)kHeadMaxSplit * D.bs * (3 * D.ds + D.r) : 0;
}
int head_logits_grid(const Dims &D);
int head_best_slots();
hipError_t launch_head(const HeadArgs &h, hipStream_t st);
// The persistent rollout where the shapes allow it (bf16, r = 256, batch <= 4,
// branch 1, a grid that fits the device at one workgroup per CU, vocabulary
// < 2^18): one launch per pair of batch rows; returns false (nothing launched)
// otherwise.
bool launch_head_persistent(const HeadArgs &h, int n_cu, hipStream_t st);
// the state recurrence of every position, teacher-forced (no logits): u into
// ubuf as above, or with skip_u only the states into `states`
hipError_t launch_head_states(const HeadArgs &h, hipStream_t st);

// ---- teacher-forced training loss (train.hip)
struct TrainArgs {
  int V, r, Mr, depth;    // Mr = bs (B-1) rows, row b (B-1) + k
  const void *w2p;        // W2 packed
  const float *P;         // [Mr] rows of stride ldp: W1[:, :d] H
  int ldp;
  const float *Y;         // [Mr][r]: W1[:, d:] S (u = SiLU(P + Y), formed while staging)
  const float *Lbase;     // [Mr] rows of stride ldl
  int ldl;
  const int32_t *labels;  // [Mr]
  float *part;            // [Mr][GC][4] per-workgroup (max, sum exp) of base and final logits
  float *lab;             // [2][Mr] label logits (base, final)
  float *ce;              // [2][Mr] cross-entropies (base, final)
  float *loss;            // [3] total, base, final
  float *final_logits;    // optional [Mr][V]
  float lambda, gamma;
  int32_t *err;
};
int train_ce_grid(int V, int r, bool bf16);
hipError_t launch_train_loss(const TrainArgs &t, bool bf16, hipStream_t st);

// ---- target verify forward: input preparation, output copy, cache commit (target.hip)
void launch_target_prep(int bs, int nn, int Bp, int V, const int32_t *tok, const int32_t *pos, const uint8_t *mask,
                        int32_t *tok_p, int32_t *pos_p, uint8_t *mask_p, int32_t *err, hipStream_t st);
void launch_target_out(int bs, int nn, int Bp, int V, const float *lg, int ldl, void *out, bool out_bf16,
                       hipStream_t st);
void launch_target_commit(bool bf16, int L, int bs, int nn, int max_depth, const int32_t *ctx_lens,
                          const int32_t *accept_len, const int32_t *accepted_nodes, void *ck, void *cv, int max_ctx,
                          int width, int32_t *new_lens, int32_t *err, hipStream_t st);

// ---- tree and acceptance (tree.hip)
void launch_build_tree(int bs, int depth, int beta, const int32_t *topk, const int32_t *anchor,
                       const int32_t *ctx_lens, int32_t *tok, int32_t *par, int32_t *dep,
                       int32_t *pos, uint8_t *mask, hipStream_t st);
size_t accept_ws_bytes(int bs, int nn, int V);
void launch_accept(int bs, int nn, int V, int B, const int32_t *tok, const int32_t *par,
                   const void *logits, bool bf16, int32_t *acc_len, int32_t *acc_nodes,
                   int32_t *out_tok, void *ws, hipStream_t st);
// the same launches with the argmax partials (accept_part_entries values pv and
// as many ids pi) and the error word (cleared by the first launch) given apart
size_t accept_part_entries(int bs, int nn, int V);
void launch_accept_parts(int bs, int nn, int V, int B, const int32_t *tok, const int32_t *par,
                         const void *logits, bool bf16, int32_t *acc_len, int32_t *acc_nodes,
                         int32_t *out_tok, float *pv, int32_t *pi, int32_t *err, hipStream_t st);

// ---- temperature sampling: speculative-sampling verification (sample.hip)
size_t vs_ws_bytes(int bs, int B, int V);
void launch_verify_sample(int bs, int B, int V, const int32_t *node_token, const void *target, bool bf16,
                          const float *draft, float temperature, uint64_t seed, int32_t *accept_len,
                          int32_t *accepted_nodes, int32_t *out_tokens, void *ws, hipStream_t st);
void launch_philox_words(const uint32_t *ctr, uint64_t key, uint32_t *out, int n, hipStream_t st);

// misc
void launch_to_f32(const void *src, bool bf16, float *dst, size_t n, hipStream_t st);
// Y[r][n] += bias[n] for r < rows, n < N (row stride N)
void launch_add_row_bias(float *Y, size_t rows, int N, const void *bias, bool bf16, hipStream_t st);
void launch_fill_u32(uint32_t *p, size_t n, uint32_t v, hipStream_t st);
// y[r][c] = sum of np K-split partial outputs parts[p*pstride + r*width + c]
// (width, pstride and ldy multiples of 4; y must not alias parts)
void launch_sum_parts(const float *parts, int np, size_t pstride, int rows, int width, float *y, int ldy,
                      hipStream_t st);

}  // namespace dk
