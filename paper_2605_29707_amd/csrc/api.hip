// Host side of the C ABI declared in include/domino.h: argument validation
// (always before any HIP call), weight packing at model creation, workspace
// planning and the launch sequence of one draft step.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/domino.h"
#include "kernels.h"

using namespace dk;

namespace {

thread_local std::string g_err = "";

domino_status fail(domino_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define HIP_TRY(expr)                                                                           \
  do {                                                                                          \
    hipError_t e_ = (expr);                                                                     \
    if (e_ != hipSuccess) return fail(DOMINO_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

struct Packed {
  size_t off;
  int NT, KS;
};

}  // namespace

struct domino_model {
  domino_config cfg;
  Dims D;  // bs filled per call
  bool bf16;
  int n_cu;
  int esz;
  // borrowed
  const void *embed, *final_norm;
  std::vector<const void *> attn_norm, q_norm, k_norm, ffn_norm;
  // owned
  void *mem = nullptr;
  size_t mem_bytes = 0;
  std::vector<Packed> qkv, wo, gateup, down;
  bool has_head = true;  // false: a target decoder (layers, embedding, LM head only)
  bool persistent = true;  // DOMINO_ROLLOUT=loop selects the launch-pair rollout everywhere
  uint32_t poll_limit = kDefaultPollLimit;  // persistent rollout: polls a wait makes before it gives up
  uint32_t last_paths = 0;  // DOMINO_PATH_* bits of the last draft step
  Packed lm, w2, w1s;
  int fuse_k = 0;  // context fusion: appended rows are fuse_k*d wide, fused by fc
  Packed fc;
  Packed whh;  // W_hh packed, for the state GEMM of batches above kHeadFusedBatch
  // training forward: the state recurrence runs on a second stream beside the backbone
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  size_t gtab_off, w_hh_off, w1_off, bhh_off, freq_off;
  // profiling
  uint32_t prof_mask = 0;
  struct Ev {
    std::vector<hipEvent_t> a, b;
    int used = 0;
  } ev[DOMINO_KC_COUNT];

  const void *at(size_t off) const { return (const char *)mem + off; }
};

namespace {

int kstep(const domino_model *m) { return m->bf16 ? 32 : 16; }

void prof_begin(domino_model *m, int cls, hipStream_t st) {
  if (!(m->prof_mask & (1u << cls))) return;
  auto &e = m->ev[cls];
  if (e.used >= (int)e.a.size()) return;
  (void)hipEventRecord(e.a[e.used], st);
}
void prof_end(domino_model *m, int cls, hipStream_t st) {
  if (!(m->prof_mask & (1u << cls))) return;
  auto &e = m->ev[cls];
  if (e.used >= (int)e.a.size()) return;
  (void)hipEventRecord(e.b[e.used], st);
  e.used++;
}

domino_status check_config(const domino_config *c, bool with_head = true) {
  if (!c) return fail(DOMINO_ERR_INVALID_ARG, "config is NULL");
  if (c->hidden <= 0 || c->n_layers <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->ffn <= 0 || c->vocab <= 1 || (with_head && (c->gru_hidden <= 0 || c->rank <= 0)))
    return fail(DOMINO_ERR_INVALID_ARG, "config sizes must be positive");
  if (c->block < 2 || c->block > 64) return fail(DOMINO_ERR_INVALID_ARG, "block must be in [2, 64]");
  if (c->mask_token_id < 0 || c->mask_token_id >= c->vocab)
    return fail(DOMINO_ERR_INVALID_ARG, "mask_token_id must be in [0, vocab)");
  if (c->dtype != DOMINO_F32 && c->dtype != DOMINO_BF16) return fail(DOMINO_ERR_INVALID_ARG, "bad dtype");
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f)) return fail(DOMINO_ERR_INVALID_ARG, "bad eps/theta");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(DOMINO_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c->n_q_heads % c->n_kv_heads) return fail(DOMINO_ERR_UNSUPPORTED, "n_q_heads must be a multiple of n_kv_heads");
  const int ks = c->dtype == DOMINO_BF16 ? 32 : 16;
  if (c->hidden % 32 || c->ffn % 32 || (c->n_q_heads * c->head_dim) % 32)
    return fail(DOMINO_ERR_UNSUPPORTED, "hidden, ffn and n_q_heads*head_dim must be multiples of 32");
  if (c->hidden > 8192) return fail(DOMINO_ERR_UNSUPPORTED, "hidden must be at most 8192");
  if (!with_head) return DOMINO_OK;
  if (c->ctx_fuse_layers < 0 || c->ctx_fuse_layers > 8)
    return fail(DOMINO_ERR_INVALID_ARG, "ctx_fuse_layers must be in [0, 8]");  // a target decoder: the node count is checked per call
  if (c->gru_hidden % 32) return fail(DOMINO_ERR_UNSUPPORTED, "gru_hidden must be a multiple of 32");
  if (c->rank % ks || c->rank > 16 * ks)
    return fail(DOMINO_ERR_UNSUPPORTED, "rank must be a multiple of %d and at most %d", ks, 16 * ks);
  if (!attn_supported(c->n_q_heads, c->n_kv_heads, c->block))
    return fail(DOMINO_ERR_UNSUPPORTED, "(n_q_heads/n_kv_heads)*block must be 32, 64 or 128");
  const int epl = c->dtype == DOMINO_BF16 ? 8 : 4;
  if (c->gru_hidden > 256 * epl) return fail(DOMINO_ERR_UNSUPPORTED, "gru_hidden must be at most %d", 256 * epl);
  if (c->dtype == DOMINO_BF16 ? c->rank != 256 : (c->rank != 128 && c->rank != 256))
    return fail(DOMINO_ERR_UNSUPPORTED, "rank must be 256 (bf16) or 128/256 (f32)");
  return DOMINO_OK;
}

Dims make_dims(const domino_model *m, int bs) {
  Dims D = m->D;
  D.bs = bs;
  return D;
}

// ---- workspace layout of the draft step
struct WsLayout {
  size_t err, best, slots, hdr_words, X, X2, A, FC, HP, QKV, Q, Kb, Vb, attn, O, WOp, F, DNp, H, LP, hbuf, ghbuf, ubuf, pval, pid,
      praw, XF, total;
  // residual-epilogue tickets (in the cleared header) and row sums of squares
  // of the deferred RMSNorms; 0: this layout has none
  size_t tickets = 0, SSQ = 0;
  int GC, ldl;
};


struct Plans {
  GemmPlan qkv, wo, gateup, down, lm;
  GemmPlan fc;  // context fusion of the appended rows (fc.ksplit = 0: none)
};

constexpr int kMaxSplit = 16;

// bf16 projections of more than kSkinnyMaxRows rows (K a multiple of 32, as
// the config checks make every K here) run the wide-activation kernel;
// everything else the skinny weight-streaming kernel
GemmPlan plan_proj(const domino_model *m, const Packed &pk, int M, int epi, int max_split) {
  if (m->bf16 && M > kSkinnyMaxRows) return plan_gemm_wide(pk.NT, pk.KS, M, epi, m->n_cu, max_split);
  return plan_gemm(pk.NT, pk.KS, M, epi, m->n_cu, max_split);
}
// false when a wide plan's arguments were refused (nothing launched)
bool launch_proj(const domino_model *m, int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  if (p.wide) return launch_gemm_wide(epi, a, p, st);  // a.K == a.KS * 32, a.xf set
  launch_gemm(m->bf16, epi, a, p, st);
  return true;
}

// Fragment scratch of the wide projections of a layout: the most rows any of
// them has times the widest K among them (0 when every plan is skinny)
size_t wide_scratch(const domino_model *m, const Plans &p, int rows, int train_rows) {
  const Dims &D = m->D;
  const bool wide = p.qkv.wide || p.wo.wide || p.gateup.wide || p.down.wide || p.lm.wide || p.fc.wide;
  const int kmax = std::max({D.d, D.nq * D.dh, D.ffn, std::max(m->fuse_k, 1) * D.d, D.ds});
  size_t b = wide ? gemm_wide_scratch_bytes(rows, kmax) : 0;
  if (train_rows > 0 && m->bf16 && train_rows > kSkinnyMaxRows)
    b = std::max(b, gemm_wide_scratch_bytes(train_rows, D.ds));
  return b;
}

// Plans for M block rows, Mlm LM-head rows and Ma QKV rows (block rows, then
// appended context rows)
Plans make_plans_rows(const domino_model *m, int M, int Mlm, int Ma) {
  Plans p;
  // projections whose consumer is elementwise write K-split partial outputs
  p.qkv = plan_proj(m, m->qkv[0], Ma, EPI_STORE, kMaxSplit);
  p.wo = plan_proj(m, m->wo[0], M, EPI_STORE, kMaxSplit);
  p.gateup = plan_proj(m, m->gateup[0], M, EPI_SWIGLU, 1);
  p.down = plan_proj(m, m->down[0], M, EPI_STORE, kMaxSplit);
  p.lm = plan_proj(m, m->lm, Mlm, EPI_STORE, 1);
  p.fc = GemmPlan();
  p.fc.ksplit = 0;
  return p;
}

Plans make_plans(const domino_model *m, int bs, int max_new) {
  const Dims &D = m->D;
  // QKV also projects the appended context rows (rows M .. M + bs*max_new - 1)
  Plans p = make_plans_rows(m, bs * D.B, bs * (D.B - 1), bs * D.B + bs * max_new);
  // the fusion's K-split partials are summed into those rows of the QKV input
  if (m->fuse_k > 0 && max_new > 0) p.fc = plan_proj(m, m->fc, bs * max_new, EPI_STORE, kMaxSplit);
  return p;
}

bool layout(const domino_model *m, int bs, int max_ctx, int max_new, int beta, WsLayout &w) {
  Dims D = make_dims(m, bs);
  const int M = bs * D.B, Mh = bs * (D.B - 1);
  const Plans p = make_plans(m, bs, max_new);
  w.GC = head_logits_grid(D);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  w.err = take(256);
  w.best = take((size_t)(D.B - 1) * bs * head_best_slots() * 8);
  w.slots = take((size_t)bs * (D.r + w.GC) * 8 * kSlotStride);  // persistent rollout: u and key slots
  w.tickets = take((size_t)2 * m->cfg.n_layers * kNormGroups * 4);
  w.hdr_words = o / 4;  // error word (+ rollout abort flag), best keys, slots, tickets: cleared at every step
  const int qkvw = (D.nq + 2 * D.nkv) * D.dh;
  w.X = take((size_t)M * D.d * 4);
  w.X2 = take((size_t)M * D.d * 4);
  const int Ma = M + bs * max_new;  // block rows, then the appended context rows
  w.A = take((size_t)Ma * D.d * 4);
  w.FC = take((size_t)p.fc.ksplit * bs * max_new * D.d * 4);
  w.HP = take(head_part_floats(D) * 4);  // state GEMM partials (batches above kHeadFusedBatch)
  w.QKV = take((size_t)p.qkv.ksplit * Ma * qkvw * 4);
  w.Q = take((size_t)M * D.nq * D.dh * 4);
  w.Kb = take((size_t)M * D.nkv * D.dh * 4);
  w.Vb = take((size_t)M * D.nkv * D.dh * 4);
  w.attn = take(attn_part_floats(D, max_ctx) * 4);
  w.O = take((size_t)M * D.nq * D.dh * 4);
  w.WOp = take((size_t)p.wo.ksplit * M * D.d * 4);
  w.F = take((size_t)M * D.ffn * 4);
  w.DNp = take((size_t)p.down.ksplit * M * D.d * 4);
  w.SSQ = take((size_t)kNormGroups * M * 4);
  w.H = take((size_t)Mh * D.d * 4);
  w.ldl = m->lm.NT * 16;
  w.LP = take((size_t)Mh * w.ldl * 4);  // [L_base | pad | P] per draft row
  w.hbuf = take((size_t)2 * bs * D.ds * 4);
  w.ghbuf = take((size_t)2 * bs * 3 * D.ds * 4);
  w.ubuf = take((size_t)bs * D.r * 4);
  w.pval = take((size_t)(D.B - 1) * bs * w.GC * beta * 4);
  w.pid = take((size_t)(D.B - 1) * bs * w.GC * beta * 4);
  w.praw = take((size_t)(D.B - 1) * bs * w.GC * 4);
  w.XF = take(wide_scratch(m, p, Ma, bs * (D.B - 1)));  // also the training forward's W1 S-half rows
  w.total = o;
  return true;
}

// Rows per batch row of a verify forward: the smallest block size the
// attention supports ((n_q / n_kv) * Bp in {32, 64, 128}, Bp a multiple of 4,
// at most 64) that holds n_nodes; 0 if none does.
int target_block(const domino_model *m, int nn) {
  const int G = m->D.nq / m->D.nkv;
  for (int R = 32; R <= 128; R *= 2)
    if (R % G == 0) {
      const int Bp = R / G;
      if (Bp >= nn && Bp % 4 == 0 && Bp <= 64) return Bp;
    }
  return 0;
}

struct TargetLayout {
  WsLayout w;
  size_t tok, pos, mask, total;
  int Bp;
};

bool target_layout(const domino_model *m, int bs, int nn, int max_ctx, TargetLayout &t) {
  t.Bp = target_block(m, nn);
  if (!t.Bp) return false;
  Dims D = make_dims(m, bs);
  D.B = t.Bp;
  const int M = bs * t.Bp;
  const Plans p = make_plans_rows(m, M, M, M);
  WsLayout &w = t.w;
  w = WsLayout();
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  w.err = take(256);
  w.hdr_words = o / 4;
  const int qkvw = (D.nq + 2 * D.nkv) * D.dh;
  w.X = take((size_t)M * D.d * 4);
  w.X2 = take((size_t)M * D.d * 4);
  w.A = take((size_t)M * D.d * 4);
  w.QKV = take((size_t)p.qkv.ksplit * M * qkvw * 4);
  w.Q = take((size_t)M * D.nq * D.dh * 4);
  w.Kb = take((size_t)M * D.nkv * D.dh * 4);
  w.Vb = take((size_t)M * D.nkv * D.dh * 4);
  w.attn = take(attn_part_floats(D, max_ctx) * 4);
  w.O = take((size_t)M * D.nq * D.dh * 4);
  w.WOp = take((size_t)p.wo.ksplit * M * D.d * 4);
  w.F = take((size_t)M * D.ffn * 4);
  w.DNp = take((size_t)p.down.ksplit * M * D.d * 4);
  w.H = take((size_t)M * D.d * 4);
  w.ldl = m->lm.NT * 16;
  w.LP = take((size_t)M * w.ldl * 4);
  w.XF = take(wide_scratch(m, p, M, 0));
  t.tok = take((size_t)M * 4);
  t.pos = take((size_t)M * 4);
  t.mask = take((size_t)bs * t.Bp * t.Bp);
  t.total = w.total = o;
  return true;
}

GemmArgs gemm_args(const void *P, const Packed &pk, int tile0, int ntiles, int N, const float *X, int ldx,
                   int M, int K, float *Y, int ldy, const GemmPlan &pl) {
  GemmArgs a;
  a.P = P;
  a.KS = pk.KS;
  a.tile0 = tile0;
  a.ntiles = ntiles;
  a.N = N;
  a.X = X;
  a.ldx = ldx;
  a.M = M;
  a.K = K;
  a.Y = Y;
  a.ldy = ldy;
  a.ksplit = pl.ksplit;
  a.ysplit = (size_t)M * ldy;
  return a;
}

}  // namespace

namespace {

// G = E W_ih^T + b_ih for every vocabulary row (fp32), so the GRU input half
// of a rollout step is a row gather.  Built with the same matrix-core GEMM as the
// projections, over the embedding in row chunks.
hipError_t build_gtab(domino_model *m, const void *w_ih, const void *b_ih) {
  const Dims &D = m->D;
  const int KSTEP = kstep(m);
  const int N = 3 * D.ds, K = D.d;
  Packed pk;
  pk.NT = (N + 15) / 16;
  pk.KS = (K + KSTEP - 1) / KSTEP;
  pk.off = 0;
  const int CH = 8192;
  void *P = nullptr, *XF = nullptr;
  float *X = nullptr;
  hipError_t e = hipMalloc(&P, (size_t)pk.NT * pk.KS * 1024);
  if (e != hipSuccess) return e;
  e = hipMalloc(&X, (size_t)CH * K * 4);
  if (e == hipSuccess && m->bf16) e = hipMalloc(&XF, gemm_wide_scratch_bytes(CH, K));
  if (e != hipSuccess) {
    (void)hipFree(P);
    if (X) (void)hipFree(X);
    return e;
  }
  launch_pack(m->bf16, w_ih, N, K, K, P, pk.NT, pk.KS, 1, 0, nullptr);
  float *G = (float *)((char *)m->mem + m->gtab_off);
  for (int r0 = 0; r0 < D.V; r0 += CH) {
    const int rows = std::min(CH, D.V - r0);
    launch_to_f32((const char *)m->embed + (size_t)r0 * K * m->esz, m->bf16, X, (size_t)rows * K, nullptr);
    const GemmPlan pl = plan_proj(m, pk, rows, EPI_STORE, 1);
    GemmArgs a = gemm_args(P, pk, 0, pk.NT, N, X, K, rows, K, G + (size_t)r0 * N, N, pl);
    a.xf = XF;
    if (!launch_proj(m, EPI_STORE, a, pl, nullptr)) {
      e = hipErrorInvalidValue;
      break;
    }
    launch_add_row_bias(G + (size_t)r0 * N, rows, N, b_ih, m->bf16, nullptr);
  }
  // finish what was launched before anything is freed, whatever stopped the loop
  const hipError_t le = hipGetLastError(), se = hipDeviceSynchronize();
  if (e == hipSuccess) e = le;
  if (e == hipSuccess) e = se;
  (void)hipFree(P);
  (void)hipFree(X);
  if (XF) (void)hipFree(XF);
  return e;
}

}  // namespace

extern "C" {

const char *domino_last_error(void) { return g_err.c_str(); }

namespace {
domino_status create_impl(const domino_config *cfg, const domino_weights *w, domino_model_t *out, bool with_head) {
  if (!out) return fail(DOMINO_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  domino_status s = check_config(cfg, with_head);
  if (s != DOMINO_OK) return s;
  if (!w) return fail(DOMINO_ERR_INVALID_ARG, "weights is NULL");
  const int L = cfg->n_layers;
  if (!w->embed || !w->lm_head || !w->final_norm)
    return fail(DOMINO_ERR_INVALID_ARG, "a weight pointer is NULL");
  if (with_head && (!w->gru_w_ih || !w->gru_w_hh || !w->gru_b_ih || !w->gru_b_hh || !w->w1 || !w->w2))
    return fail(DOMINO_ERR_INVALID_ARG, "a weight pointer is NULL");
  if (with_head && cfg->ctx_fuse_layers > 0 && !w->ctx_fc)
    return fail(DOMINO_ERR_INVALID_ARG, "ctx_fc is NULL (ctx_fuse_layers > 0)");
  const void *const *arrs[] = {w->attn_norm, w->wq, w->wk, w->wv, w->q_norm, w->k_norm,
                               w->wo, w->ffn_norm, w->w_gate, w->w_up, w->w_down};
  for (auto a : arrs) {
    if (!a) return fail(DOMINO_ERR_INVALID_ARG, "a per-layer weight array is NULL");
    for (int l = 0; l < L; ++l)
      if (!a[l]) return fail(DOMINO_ERR_INVALID_ARG, "a per-layer weight pointer is NULL (layer %d)", l);
  }

  domino_model *m = new domino_model();
  m->cfg = *cfg;
  m->has_head = with_head;
  {
    const char *ro = std::getenv("DOMINO_ROLLOUT");
    m->persistent = !(ro && std::strcmp(ro, "loop") == 0);
  }
  m->bf16 = cfg->dtype == DOMINO_BF16;
  m->esz = m->bf16 ? 2 : 4;
  Dims &D = m->D;
  D.bs = 0;
  D.B = cfg->block;
  D.d = cfg->hidden;
  D.nq = cfg->n_q_heads;
  D.nkv = cfg->n_kv_heads;
  D.dh = cfg->head_dim;
  D.ffn = cfg->ffn;
  D.V = cfg->vocab;
  D.ds = cfg->gru_hidden;
  D.r = cfg->rank;
  D.mask_id = cfg->mask_token_id;
  D.eps = cfg->rms_eps;
  D.theta = cfg->rope_theta;
  D.bf16 = m->bf16;
  D.inv_freq = nullptr;  // set once the model memory exists
  m->embed = w->embed;
  m->final_norm = w->final_norm;
  for (int l = 0; l < L; ++l) {
    m->attn_norm.push_back(w->attn_norm[l]);
    m->q_norm.push_back(w->q_norm[l]);
    m->k_norm.push_back(w->k_norm[l]);
    m->ffn_norm.push_back(w->ffn_norm[l]);
  }

  int dev = 0;
  hipError_t he = hipGetDevice(&dev);
  if (he == hipSuccess) he = hipDeviceGetAttribute(&m->n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (he != hipSuccess) {
    delete m;
    return fail(DOMINO_ERR_HIP, "querying the device: %s", hipGetErrorString(he));
  }

  // ---- plan packed storage
  const int KSTEP = kstep(m);
  auto ks_of = [&](int K) { return (K + KSTEP - 1) / KSTEP; };
  size_t off = 0;
  auto add = [&](int N, int K) {
    Packed p;
    p.NT = (N + 15) / 16;
    p.KS = ks_of(K);
    p.off = off;
    off = align_up(off + (size_t)p.NT * p.KS * 1024);
    return p;
  };
  const int qd = D.nq * D.dh, kvd = D.nkv * D.dh;
  for (int l = 0; l < L; ++l) {
    m->qkv.push_back(add(qd + 2 * kvd, D.d));
    m->wo.push_back(add(D.d, qd));
    Packed gu = add(2 * ((D.ffn + 15) / 16) * 16, D.d);
    m->gateup.push_back(gu);
    m->down.push_back(add(D.d, D.ffn));
  }
  // LM head and W1's H half share the input H: one packed matrix, W1 tiles after the vocabulary tiles
  m->lm = add(((D.V + 15) / 16) * 16 + (with_head ? D.r : 0), D.d);
  if (with_head) {
    m->w2 = add(D.V, D.r);
    m->w1s = add(D.r, D.ds);  // W1's S half on its own (training forward; state GEMMs of large batches)
    m->whh = add(3 * D.ds, D.ds);
    m->fuse_k = cfg->ctx_fuse_layers;
    if (m->fuse_k > 0) m->fc = add(D.d, m->fuse_k * D.d);
    m->gtab_off = off;
    off = align_up(off + (size_t)D.V * 3 * D.ds * 4);
    m->w_hh_off = off;
    off = align_up(off + (size_t)3 * D.ds * D.ds * m->esz);
    m->w1_off = off;
    off = align_up(off + (size_t)D.r * (D.d + D.ds) * m->esz);
    m->bhh_off = off;
    off = align_up(off + (size_t)3 * D.ds * 4);
  }
  m->freq_off = off;
  off = align_up(off + (size_t)(D.dh / 2) * sizeof(double));
  m->mem_bytes = off;

  he = hipMalloc(&m->mem, m->mem_bytes);
  if (he != hipSuccess) {
    delete m;
    return fail(DOMINO_ERR_HIP, "hipMalloc(%zu): %s", off, hipGetErrorString(he));
  }
  hipStream_t st = nullptr;
  char *base = (char *)m->mem;
  D.inv_freq = (const double *)(base + m->freq_off);
  const bool bf = m->bf16;
  for (int l = 0; l < L; ++l) {
    const Packed &p = m->qkv[l];
    // rows: [wq | wk | wv]; each block starts on a tile boundary (qd, kvd multiples of 16)
    launch_pack(bf, w->wq[l], qd, D.d, D.d, base + p.off, qd / 16, p.KS, 1, 0, st);
    launch_pack(bf, w->wk[l], kvd, D.d, D.d, base + p.off + (size_t)(qd / 16) * p.KS * 1024, kvd / 16, p.KS, 1, 0,
                st);
    launch_pack(bf, w->wv[l], kvd, D.d, D.d, base + p.off + (size_t)((qd + kvd) / 16) * p.KS * 1024, kvd / 16,
                p.KS, 1, 0, st);
    const Packed &o = m->wo[l];
    launch_pack(bf, w->wo[l], D.d, qd, qd, base + o.off, o.NT, o.KS, 1, 0, st);
    const Packed &g = m->gateup[l];
    const int ft = (D.ffn + 15) / 16;
    launch_pack(bf, w->w_gate[l], D.ffn, D.d, D.d, base + g.off, ft, g.KS, 2, 0, st);
    launch_pack(bf, w->w_up[l], D.ffn, D.d, D.d, base + g.off, ft, g.KS, 2, 1, st);
    const Packed &dn = m->down[l];
    launch_pack(bf, w->w_down[l], D.d, D.ffn, D.ffn, base + dn.off, dn.NT, dn.KS, 1, 0, st);
  }
  const int vt = (D.V + 15) / 16;
  launch_pack(bf, w->lm_head, D.V, D.d, D.d, base + m->lm.off, vt, m->lm.KS, 1, 0, st);
  if (with_head) {
    launch_pack(bf, w->w1, D.r, D.d, D.d + D.ds, base + m->lm.off + (size_t)vt * m->lm.KS * 1024, D.r / 16,
                m->lm.KS, 1, 0, st);
    launch_pack(bf, w->w2, D.V, D.r, D.r, base + m->w2.off, m->w2.NT, m->w2.KS, 1, 0, st);
    launch_pack(bf, (const char *)w->w1 + (size_t)D.d * m->esz, D.r, D.ds, D.d + D.ds, base + m->w1s.off,
                m->w1s.NT, m->w1s.KS, 1, 0, st);
    launch_pack(bf, w->gru_w_hh, 3 * D.ds, D.ds, D.ds, base + m->whh.off, m->whh.NT, m->whh.KS, 1, 0, st);
    if (m->fuse_k > 0) {
      const int kf = m->fuse_k * D.d;
      launch_pack(bf, w->ctx_fc, D.d, kf, kf, base + m->fc.off, m->fc.NT, m->fc.KS, 1, 0, st);
    }
  }
  he = hipGetLastError();
  if (he == hipSuccess && with_head) he = build_gtab(m, w->gru_w_ih, w->gru_b_ih);
  if (he == hipSuccess && with_head) {
    launch_to_f32(w->gru_b_hh, m->bf16, (float *)(base + m->bhh_off), (size_t)3 * D.ds, nullptr);
    he = hipGetLastError();
  }
  if (he == hipSuccess) {
    // RoPE inverse frequencies theta^(-2i/dh), exact in fp64 on the host
    std::vector<double> f(D.dh / 2);
    for (int i = 0; i < D.dh / 2; ++i) f[i] = std::pow((double)cfg->rope_theta, -2.0 * i / (double)D.dh);
    he = hipMemcpy(base + m->freq_off, f.data(), f.size() * sizeof(double), hipMemcpyHostToDevice);
  }
  if (he == hipSuccess && with_head)
    he = hipMemcpy(base + m->w_hh_off, w->gru_w_hh, (size_t)3 * D.ds * D.ds * m->esz, hipMemcpyDeviceToDevice);
  if (he == hipSuccess && with_head)
    he = hipMemcpy(base + m->w1_off, w->w1, (size_t)D.r * (D.d + D.ds) * m->esz, hipMemcpyDeviceToDevice);
  if (he == hipSuccess) he = hipDeviceSynchronize();
  if (he != hipSuccess) {
    (void)hipFree(m->mem);
    delete m;
    return fail(DOMINO_ERR_HIP, "packing weights: %s", hipGetErrorString(he));
  }
  *out = m;
  return DOMINO_OK;
}
}  // namespace

domino_status domino_model_create(const domino_config *cfg, const domino_weights *w, domino_model_t *out) {
  return create_impl(cfg, w, out, true);
}

domino_status domino_target_create(const domino_config *cfg, const domino_weights *w, domino_model_t *out) {
  return create_impl(cfg, w, out, false);
}

void domino_model_destroy(domino_model_t m) {
  if (!m) return;
  for (auto &e : m->ev) {
    for (auto x : e.a) (void)hipEventDestroy(x);
    for (auto x : e.b) (void)hipEventDestroy(x);
  }
  if (m->fork) (void)hipEventDestroy(m->fork);
  if (m->join) (void)hipEventDestroy(m->join);
  if (m->side) (void)hipStreamDestroy(m->side);
  if (m->mem) (void)hipFree(m->mem);
  delete m;
}

size_t domino_workspace_bytes(domino_model_t m, int32_t batch, int32_t max_ctx, int32_t max_new, int32_t branch) {
  if (!m || !m->has_head || batch < 1 || batch > 64 || max_ctx < 0 || max_new < 0 || max_new > max_ctx || branch < 1 ||
      branch > 8)
    return 0;
  WsLayout w;
  layout(m, batch, max_ctx, max_new, branch, w);
  return w.total;
}

namespace {
struct SampleOpt {
  float temperature;
  uint64_t seed;
};

domino_status check_step_args(domino_model_t m, int32_t batch, const int32_t *anchor_ids, const int32_t *ctx_lens,
                              void *ctx_k, void *ctx_v, int32_t max_ctx, const void *ctx_hidden_new, int32_t n_new) {
  if (!m) return fail(DOMINO_ERR_INVALID_ARG, "model is NULL");
  if (!m->has_head) return fail(DOMINO_ERR_INVALID_ARG, "model has no Domino head (created as a target decoder)");
  if (batch < 1 || batch > 64) return fail(DOMINO_ERR_INVALID_ARG, "batch must be in [1, 64]");
  if (!anchor_ids || !ctx_lens) return fail(DOMINO_ERR_INVALID_ARG, "anchor_ids/ctx_lens is NULL");
  if (max_ctx < 0) return fail(DOMINO_ERR_INVALID_ARG, "max_ctx must be >= 0");
  if (max_ctx > 0 && (!ctx_k || !ctx_v)) return fail(DOMINO_ERR_INVALID_ARG, "ctx_k/ctx_v is NULL");
  if (n_new < 0 || n_new > max_ctx) return fail(DOMINO_ERR_INVALID_ARG, "n_new must be in [0, max_ctx]");
  if (n_new > 0 && !ctx_hidden_new) return fail(DOMINO_ERR_INVALID_ARG, "ctx_hidden_new is NULL");
  return DOMINO_OK;
}

// The masked block through the draft backbone, the final norm and the LM head
// (with W1's H half): leaves [L_base | pad | P] in the workspace's LP.
// How the B rows of each batch row enter the layers.  Default (the drafter):
// the masked block [anchor, MASK, ...] at positions n + j, bidirectional block
// attention, final norm and LM head over the B-1 draft rows.  A verify forward
// gives a token and a position per row, a tree mask, stores its first n_store
// rows' K/V into the cache at n + j, and takes every row through the LM head.
struct RowSpec {
  const int32_t *tokens = nullptr;
  const int32_t *pos = nullptr;
  const uint8_t *amask = nullptr;
  int n_store = 0;
  bool all_rows = false;
};

domino_status run_layers(domino_model_t m, const Dims &D, const Plans &p, const RowSpec &spec,
                         const int32_t *anchor_ids, const int32_t *ctx_lens, void *ctx_k, void *ctx_v,
                         int32_t max_ctx, const void *ctx_hidden_new, int32_t n_new, const domino_debug *debug,
                         char *ws, const WsLayout &w, hipStream_t st, bool clear_header) {
  const int batch = D.bs;
  auto F = [&](size_t off) { return (float *)(ws + off); };
  int32_t *err = (int32_t *)(ws + w.err);
  const char *base = (const char *)m->mem;
  const int M = batch * D.B, Mh = spec.all_rows ? M : batch * (D.B - 1);
  const int qd = D.nq * D.dh, kvd = D.nkv * D.dh, qkvw = qd + 2 * kvd;
  const size_t layer_elems = (size_t)batch * max_ctx * kvd;

  // the error word, the rollout's best keys and exchange slots are cleared by
  // layer 0's RMSNorm launch (clear_header)
  // appended context rows (target hidden states) ride along in the QKV
  // projection: they sit after the block rows of its input, and the RMSNorms
  // only ever rewrite the block rows.  With context fusion the rows are
  // k*d wide and enter as ctx_fc times the row (K-split GEMM, then the sum of
  // its partials written into place).
  const int Ma = M + batch * n_new;
  if (n_new > 0 && m->fuse_k > 0) {
    const int kf = m->fuse_k * D.d, rows = batch * n_new;
    prof_begin(m, DOMINO_KC_CTXPROJ, st);
    GemmArgs a = gemm_args(base + m->fc.off, m->fc, 0, m->fc.NT, D.d, (const float *)ctx_hidden_new, kf, rows, kf,
                           F(w.FC), D.d, p.fc);
    a.xf = ws + w.XF;
    if (!launch_proj(m, EPI_STORE, a, p.fc, st)) return fail(DOMINO_ERR_UNSUPPORTED, "context fusion projection refused");
    launch_sum_parts(F(w.FC), p.fc.ksplit, (size_t)rows * D.d, rows, D.d, F(w.A) + (size_t)M * D.d, D.d, st);
    prof_end(m, DOMINO_KC_CTXPROJ, st);
  } else if (n_new > 0) {
    hipError_t ce = hipMemcpyAsync(F(w.A) + (size_t)M * D.d, ctx_hidden_new, (size_t)batch * n_new * D.d * 4,
                                   hipMemcpyDeviceToDevice, st);
    if (ce != hipSuccess) return fail(DOMINO_ERR_HIP, "staging ctx_hidden_new: %s", hipGetErrorString(ce));
  }

  const size_t rstride = (size_t)M * D.d;  // partial-output stride of the residual projections
  // every projection of the step: wide plans split their activations into the workspace's fragment planes
  auto proj = [&](int epi, GemmArgs a, const GemmPlan &pl) {
    a.xf = ws + w.XF;
    return launch_proj(m, epi, a, pl, st);
  };
  // the residual stream ping-pongs between two buffers: every RMSNorm launch
  // reads one and writes the updated residual to the other
  float *xc = F(w.X), *xn = F(w.X2);
  // Fused norms (one batch row's block on the skinny kernel): the O and down
  // projections end with the residual update (EPI_RESID), which also leaves the
  // next RMSNorm's input times its gain in A and the row sums of squares in SSQ;
  // the gate/up and next QKV projections then scale their output rows by the
  // norm factor.  Only layer 0's RMSNorm (of the embedding rows) and the final
  // one remain launches of their own.  The tickets start at zero: layer 0's
  // RMSNorm clears the header (clear_header), or the caller cleared it before
  // (the training forward); a layout without tickets never fuses.
  auto fusable = [](const GemmPlan &pl) { return !pl.wide && pl.pgrid == 0 && pl.WPT == 1 && pl.mgroups == 1; };
  const bool fuse = w.tickets && w.SSQ && n_new == 0 && m->bf16 && fusable(p.qkv) && fusable(p.wo) &&
                    fusable(p.gateup) && fusable(p.down) && p.wo.groups <= kNormGroups &&
                    p.down.groups <= kNormGroups && D.d % 4 == 0;
  unsigned *tickets = fuse ? (unsigned *)(ws + w.tickets) : nullptr;
  float *SSQ = fuse ? F(w.SSQ) : nullptr;
  auto resid = [&](GemmArgs &a, const void *gain, int slot) {
    a.res_in = xc;
    a.res_out = xn;
    a.res_xg = F(w.A);
    a.res_ssq = SSQ;
    a.res_gain = gain;
    a.res_tickets = tickets + (size_t)slot * kNormGroups;
  };
  auto deferred = [&](GemmArgs &a, int ng) {
    a.rs_ssq = SSQ;
    a.rs_ng = ng;
    a.rs_d = D.d;
    a.rs_eps = m->cfg.rms_eps;
  };
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    const char *ck = (const char *)ctx_k + l * layer_elems * m->esz;
    const char *cv = (const char *)ctx_v + l * layer_elems * m->esz;
    // residual += previous layer's down projection, then the attention RMSNorm
    // (fused: done by that down projection, except at layer 0)
    if (l == 0 || !fuse) {
      prof_begin(m, DOMINO_KC_NORM, st);
      // (layer 0: the residual starts as the embedding of [anchor, MASK, ...])
      launch_add_norm(D, xc, xn, D.d, F(w.DNp), l > 0 ? p.down.ksplit : 0, rstride, m->attn_norm[l], F(w.A), D.d,
                      M, D.d, false, l == 0 ? m->embed : nullptr, anchor_ids, err, st, spec.tokens,
                      l == 0 && clear_header ? (uint32_t *)ws : nullptr, (int)w.hdr_words);
      std::swap(xc, xn);
      prof_end(m, DOMINO_KC_NORM, st);
    }

    prof_begin(m, DOMINO_KC_QKV, st);
    GemmArgs a = gemm_args(base + m->qkv[l].off, m->qkv[l], 0, m->qkv[l].NT, qkvw, F(w.A), D.d, Ma, D.d, F(w.QKV),
                           qkvw, p.qkv);
    if (fuse && l > 0) deferred(a, p.down.groups);
    if (!proj(EPI_STORE, a, p.qkv)) return fail(DOMINO_ERR_UNSUPPORTED, "qkv projection refused");
    prof_end(m, DOMINO_KC_QKV, st);

    prof_begin(m, DOMINO_KC_ROPE, st);
    launch_qk_norm_rope(D, F(w.QKV), p.qkv.ksplit, (size_t)Ma * qkvw, m->q_norm[l], m->k_norm[l], ctx_lens, max_ctx,
                        F(w.Q), F(w.Kb), F(w.Vb), n_new, (void *)ck, (void *)cv, err, st, spec.pos, spec.n_store);
    prof_end(m, DOMINO_KC_ROPE, st);

    prof_begin(m, DOMINO_KC_ATTN, st);
    launch_attention(D, F(w.Q), F(w.Kb), F(w.Vb), ck, cv, ctx_lens, max_ctx, F(w.attn), F(w.O), err, st, spec.amask);
    prof_end(m, DOMINO_KC_ATTN, st);

    prof_begin(m, DOMINO_KC_WO, st);
    a = gemm_args(base + m->wo[l].off, m->wo[l], 0, m->wo[l].NT, D.d, F(w.O), qd, M, qd, F(w.WOp), D.d, p.wo);
    if (fuse) {  // residual += attention output, and the FFN RMSNorm's statistics
      resid(a, m->ffn_norm[l], 2 * l);
      if (!proj(EPI_RESID, a, p.wo)) return fail(DOMINO_ERR_UNSUPPORTED, "wo projection refused");
      std::swap(xc, xn);
    } else if (!proj(EPI_STORE, a, p.wo)) {
      return fail(DOMINO_ERR_UNSUPPORTED, "wo projection refused");
    }
    prof_end(m, DOMINO_KC_WO, st);

    if (!fuse) {  // residual += attention output, then the FFN RMSNorm
      prof_begin(m, DOMINO_KC_NORM, st);
      launch_add_norm(D, xc, xn, D.d, F(w.WOp), p.wo.ksplit, rstride, m->ffn_norm[l], F(w.A), D.d, M, D.d, false,
                      nullptr, nullptr, err, st);
      std::swap(xc, xn);
      prof_end(m, DOMINO_KC_NORM, st);
    }

    prof_begin(m, DOMINO_KC_GATEUP, st);
    a = gemm_args(base + m->gateup[l].off, m->gateup[l], 0, m->gateup[l].NT, D.ffn, F(w.A), D.d, M, D.d, F(w.F),
                  D.ffn, p.gateup);
    if (fuse) deferred(a, p.wo.groups);
    if (!proj(EPI_SWIGLU, a, p.gateup)) return fail(DOMINO_ERR_UNSUPPORTED, "gateup projection refused");
    prof_end(m, DOMINO_KC_GATEUP, st);

    prof_begin(m, DOMINO_KC_DOWN, st);
    a = gemm_args(base + m->down[l].off, m->down[l], 0, m->down[l].NT, D.d, F(w.F), D.ffn, M, D.ffn, F(w.DNp), D.d,
                  p.down);
    if (fuse && l + 1 < m->cfg.n_layers) {  // residual += FFN output, and the next attention RMSNorm's statistics
      resid(a, m->attn_norm[l + 1], 2 * l + 1);
      if (!proj(EPI_RESID, a, p.down)) return fail(DOMINO_ERR_UNSUPPORTED, "down projection refused");
      std::swap(xc, xn);
    } else if (!proj(EPI_STORE, a, p.down)) {
      return fail(DOMINO_ERR_UNSUPPORTED, "down projection refused");
    }
    prof_end(m, DOMINO_KC_DOWN, st);
  }

  // residual += last down projection; final RMSNorm of the draft rows -> H
  float *H = (debug && debug->hidden) ? debug->hidden : F(w.H);
  prof_begin(m, DOMINO_KC_NORM, st);
  launch_add_norm(D, xc, nullptr, D.d, F(w.DNp), p.down.ksplit, rstride, m->final_norm, H, D.d, Mh, D.d, !spec.all_rows,
                  nullptr, nullptr, err, st);
  prof_end(m, DOMINO_KC_NORM, st);

  // LM head and W1's H half in one pass over H: columns [0, V) are L_base, [ldl - r, ldl) are P
  float *LP = F(w.LP);
  prof_begin(m, DOMINO_KC_LMHEAD, st);
  GemmArgs a = gemm_args(base + m->lm.off, m->lm, 0, m->lm.NT, w.ldl, H, D.d, Mh, D.d, LP, w.ldl, p.lm);
  if (!proj(EPI_STORE, a, p.lm)) return fail(DOMINO_ERR_UNSUPPORTED, "lm projection refused");
  prof_end(m, DOMINO_KC_LMHEAD, st);
  if (!spec.all_rows && debug && debug->base_logits) {
    hipError_t ce = hipMemcpy2DAsync(debug->base_logits, (size_t)D.V * 4, LP, (size_t)w.ldl * 4, (size_t)D.V * 4, Mh,
                                     hipMemcpyDeviceToDevice, st);
    if (ce != hipSuccess) return fail(DOMINO_ERR_HIP, "copying base logits: %s", hipGetErrorString(ce));
  }

  return DOMINO_OK;
}

domino_status run_backbone(domino_model_t m, int32_t batch, const int32_t *anchor_ids, const int32_t *ctx_lens,
                           void *ctx_k, void *ctx_v, int32_t max_ctx, const void *ctx_hidden_new, int32_t n_new,
                           const domino_debug *debug, char *ws, const WsLayout &w, hipStream_t st,
                           bool clear_header = true) {
  return run_layers(m, make_dims(m, batch), make_plans(m, batch, n_new), RowSpec(), anchor_ids, ctx_lens, ctx_k, ctx_v,
                    max_ctx, ctx_hidden_new, n_new, debug, ws, w, st, clear_header);
}

HeadArgs head_args(domino_model_t m, int32_t batch, int32_t branch, char *ws, const WsLayout &w,
                   const int32_t *anchor_ids, const int32_t *forced_tokens, const domino_debug *debug) {
  const Dims D = make_dims(m, batch);
  const char *base = (const char *)m->mem;
  auto F = [&](size_t off) { return (float *)(ws + off); };
  float *LP = F(w.LP);
  HeadArgs h;
  h.D = D;
  h.beta = branch;
  h.gtab = (const float *)(base + m->gtab_off);
  h.w_hh = base + m->w_hh_off;
  h.bhh = (const float *)(base + m->bhh_off);
  h.w1 = base + m->w1_off;
  h.w2p = base + m->w2.off;
  h.P = LP + (w.ldl - D.r);
  h.ldp = w.ldl;
  h.Lbase = LP;
  h.ldl = w.ldl;
  h.best = (unsigned long long *)(ws + w.best);
  h.anchor = anchor_ids;
  h.forced = forced_tokens;
  h.topk_ids = nullptr;
  h.topk_vals = nullptr;
  h.final_logits = debug ? debug->final_logits : nullptr;
  h.states = debug ? debug->states : nullptr;
  h.hbuf = F(w.hbuf);
  h.ghbuf = F(w.ghbuf);
  h.ubuf = F(w.ubuf);
  h.u_ld = D.r;
  h.u_pos = 0;
  h.skip_u = 0;
  h.pval = F(w.pval);
  h.pid = (int32_t *)(ws + w.pid);
  h.err = (int32_t *)(ws + w.err);
  h.GC = w.GC;
  h.sample = 0;
  h.inv_temp = 1.0f;
  h.seed_lo = 0u;
  h.seed_hi = 0u;
  h.praw = F(w.praw);
  h.uslot = (unsigned long long *)(ws + w.slots);
  h.kslot = h.uslot + (size_t)batch * D.r * kSlotStride;
  h.abort_flag = (unsigned *)(ws + w.err + 128);
  h.poll_limit = m->poll_limit;
  h.whh_p = base + m->whh.off;
  h.w1s_p = base + m->w1s.off;
  h.whh_NT = m->whh.NT;
  h.whh_KS = m->whh.KS;
  h.w1s_NT = m->w1s.NT;
  h.w1s_KS = m->w1s.KS;
  h.hpart = head_part_floats(D) ? F(w.HP) : nullptr;
  h.n_cu = m->n_cu;
  return h;
}

domino_status draft_step_impl(domino_model_t m, int32_t batch, const int32_t *anchor_ids, const int32_t *ctx_lens,
                              void *ctx_k, void *ctx_v, int32_t max_ctx, const void *ctx_hidden_new, int32_t n_new,
                              int32_t branch, const int32_t *forced_tokens, int32_t *topk_ids, float *topk_vals,
                              const domino_debug *debug, void *workspace, size_t workspace_bytes, void *stream,
                              const SampleOpt *smp) {
  domino_status s = check_step_args(m, batch, anchor_ids, ctx_lens, ctx_k, ctx_v, max_ctx, ctx_hidden_new, n_new);
  if (s != DOMINO_OK) return s;
  if (branch < 1 || branch > 8 || branch > m->D.V) return fail(DOMINO_ERR_INVALID_ARG, "branch must be in [1, 8]");
  if (!topk_ids || !topk_vals) return fail(DOMINO_ERR_INVALID_ARG, "topk_ids/topk_vals is NULL");
  if (!workspace) return fail(DOMINO_ERR_WORKSPACE, "workspace is NULL");
  WsLayout w;
  layout(m, batch, max_ctx, n_new, branch, w);
  if (workspace_bytes < w.total)
    return fail(DOMINO_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, w.total);

  hipStream_t st = (hipStream_t)stream;
  char *ws = (char *)workspace;
  m->last_paths = 0;
  s = run_backbone(m, batch, anchor_ids, ctx_lens, ctx_k, ctx_v, max_ctx, ctx_hidden_new, n_new, debug, ws, w, st);
  if (s != DOMINO_OK) return s;

  HeadArgs h = head_args(m, batch, branch, ws, w, anchor_ids, forced_tokens, debug);
  h.topk_ids = topk_ids;
  h.topk_vals = topk_vals;
  h.sample = smp ? 1 : 0;
  h.inv_temp = smp ? 1.0f / smp->temperature : 1.0f;
  h.seed_lo = smp ? (uint32_t)smp->seed : 0u;
  h.seed_hi = smp ? (uint32_t)(smp->seed >> 32) : 0u;
  prof_begin(m, DOMINO_KC_HEADLOOP, st);
  hipError_t he = hipSuccess;
  // one persistent launch for the whole rollout where it applies, else a
  // launch pair per position
  if (m->persistent && launch_head_persistent(h, m->n_cu, st)) m->last_paths |= DOMINO_PATH_PERSISTENT_ROLLOUT;
  else he = launch_head(h, st);
  prof_end(m, DOMINO_KC_HEADLOOP, st);
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "head loop launch: %s", hipGetErrorString(he));
  he = hipGetLastError();
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "draft step launch: %s", hipGetErrorString(he));
  return DOMINO_OK;
}

}  // namespace

domino_status domino_draft_step(domino_model_t m, int32_t batch, const int32_t *anchor_ids, const int32_t *ctx_lens,
                                void *ctx_k, void *ctx_v, int32_t max_ctx, const void *ctx_hidden_new, int32_t n_new,
                                int32_t branch, const int32_t *forced_tokens, int32_t *topk_ids, float *topk_vals,
                                const domino_debug *debug, void *workspace, size_t workspace_bytes, void *stream) {
  return draft_step_impl(m, batch, anchor_ids, ctx_lens, ctx_k, ctx_v, max_ctx, ctx_hidden_new, n_new, branch,
                         forced_tokens, topk_ids, topk_vals, debug, workspace, workspace_bytes, stream, nullptr);
}

domino_status domino_draft_step_sampled(domino_model_t m, int32_t batch, const int32_t *anchor_ids,
                                        const int32_t *ctx_lens, void *ctx_k, void *ctx_v, int32_t max_ctx,
                                        const void *ctx_hidden_new, int32_t n_new, float temperature, uint64_t seed,
                                        const int32_t *forced_tokens, int32_t *topk_ids, float *topk_vals,
                                        float *final_logits, const domino_debug *debug, void *workspace,
                                        size_t workspace_bytes, void *stream) {
  if (!(temperature > 0.f) || !std::isfinite(temperature) || 1.0f / temperature > 1e30f)
    return fail(DOMINO_ERR_INVALID_ARG, "temperature must be positive and finite");
  if (!final_logits) return fail(DOMINO_ERR_INVALID_ARG, "final_logits is NULL (the verifier needs them)");
  domino_debug dbg = {};
  if (debug) dbg = *debug;
  dbg.final_logits = final_logits;
  const SampleOpt smp = {temperature, seed};
  return draft_step_impl(m, batch, anchor_ids, ctx_lens, ctx_k, ctx_v, max_ctx, ctx_hidden_new, n_new, 1,
                         forced_tokens, topk_ids, topk_vals, &dbg, workspace, workspace_bytes, stream, &smp);
}

namespace {
// training forward: the draft-step layout (branch 1) plus every position's u,
// the per-workgroup log-sum-exp pairs, the label logits and the per-row CEs
struct TrainLayout {
  WsLayout w;
  size_t S, Y, part, lab, ce, total;
  int GCt;
};
void train_layout(const domino_model *m, int bs, int max_ctx, int max_new, TrainLayout &t) {
  layout(m, bs, max_ctx, max_new, 1, t.w);
  const Dims &D = m->D;
  const size_t Mr = (size_t)bs * (D.B - 1);
  t.GCt = train_ce_grid(D.V, D.r, m->bf16);
  size_t o = t.w.total;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  t.S = take(Mr * D.ds * 4);
  t.Y = take(Mr * D.r * 4);
  t.part = take(Mr * t.GCt * 16);
  t.lab = take(2 * Mr * 4);
  t.ce = take(2 * Mr * 4);
  t.total = o;
}
}  // namespace

size_t domino_train_workspace_bytes(domino_model_t m, int32_t batch, int32_t max_ctx, int32_t max_new) {
  if (!m || !m->has_head || batch < 1 || batch > 64 || max_ctx < 0 || max_new < 0 || max_new > max_ctx) return 0;
  TrainLayout t;
  train_layout(m, batch, max_ctx, max_new, t);
  return t.total;
}

domino_status domino_train_forward(domino_model_t m, int32_t batch, const int32_t *anchor_ids,
                                   const int32_t *ctx_lens, void *ctx_k, void *ctx_v, int32_t max_ctx,
                                   const void *ctx_hidden_new, int32_t n_new, const int32_t *labels, float lambda,
                                   float gamma, float *loss, float *ce, const domino_debug *debug, void *workspace,
                                   size_t workspace_bytes, void *stream) {
  domino_status s = check_step_args(m, batch, anchor_ids, ctx_lens, ctx_k, ctx_v, max_ctx, ctx_hidden_new, n_new);
  if (s != DOMINO_OK) return s;
  if (!labels) return fail(DOMINO_ERR_INVALID_ARG, "labels is NULL");
  if (!loss) return fail(DOMINO_ERR_INVALID_ARG, "loss is NULL");
  if (!(lambda >= 0.f && lambda <= 1.f)) return fail(DOMINO_ERR_INVALID_ARG, "lambda must be in [0, 1]");
  if (!(gamma > 0.f) || !std::isfinite(gamma)) return fail(DOMINO_ERR_INVALID_ARG, "gamma must be positive and finite");
  if (!workspace) return fail(DOMINO_ERR_WORKSPACE, "workspace is NULL");
  TrainLayout tl;
  train_layout(m, batch, max_ctx, n_new, tl);
  if (workspace_bytes < tl.total)
    return fail(DOMINO_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, tl.total);

  hipStream_t st = (hipStream_t)stream;
  char *ws = (char *)workspace;
  const WsLayout &w = tl.w;
  const Dims D = make_dims(m, batch);
  const int depth = D.B - 1, Mr = batch * depth;
  m->last_paths = 0;
  if (!m->side) {
    HIP_TRY(hipStreamCreateWithFlags(&m->side, hipStreamNonBlocking));
    HIP_TRY(hipEventCreateWithFlags(&m->fork, hipEventDisableTiming));
    HIP_TRY(hipEventCreateWithFlags(&m->join, hipEventDisableTiming));
  }

  // the state recurrence depends on the labels only, not on the backbone: it
  // runs on the side stream (after the error word is cleared) while the
  // backbone streams its weights on the caller's stream
  launch_fill_u32((uint32_t *)ws, w.hdr_words, 0u, st);
  HIP_TRY(hipEventRecord(m->fork, st));
  HIP_TRY(hipStreamWaitEvent(m->side, m->fork, 0));
  HeadArgs h = head_args(m, batch, 1, ws, w, anchor_ids, labels, debug);
  h.final_logits = nullptr;
  h.states = (debug && debug->states) ? debug->states : (float *)(ws + tl.S);
  h.skip_u = 1;
  prof_begin(m, DOMINO_KC_HEADLOOP, m->side);
  hipError_t he = launch_head_states(h, m->side);
  prof_end(m, DOMINO_KC_HEADLOOP, m->side);
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "state recurrence launch: %s", hipGetErrorString(he));
  HIP_TRY(hipEventRecord(m->join, m->side));

  s = run_backbone(m, batch, anchor_ids, ctx_lens, ctx_k, ctx_v, max_ctx, ctx_hidden_new, n_new, debug, ws, w, st,
                   false);
  if (s != DOMINO_OK) {
    (void)hipStreamWaitEvent(st, m->join, 0);
    return s;
  }
  HIP_TRY(hipStreamWaitEvent(st, m->join, 0));

  // Y = W1[:, d:] S for every (row, position) at once
  prof_begin(m, DOMINO_KC_TRAINLOSS, st);
  const GemmPlan py = plan_proj(m, m->w1s, Mr, EPI_STORE, 1);
  const GemmArgs ga = gemm_args((const char *)m->mem + m->w1s.off, m->w1s, 0, m->w1s.NT, D.r, h.states, D.ds, Mr,
                                D.ds, (float *)(ws + tl.Y), D.r, py);
  GemmArgs gx = ga;
  gx.xf = ws + w.XF;
  if (!launch_proj(m, EPI_STORE, gx, py, st)) return fail(DOMINO_ERR_UNSUPPORTED, "W1 state projection refused");

  TrainArgs t;
  t.V = D.V;
  t.r = D.r;
  t.Mr = batch * depth;
  t.depth = depth;
  t.w2p = (const char *)m->mem + m->w2.off;
  t.P = (const float *)(ws + w.LP) + (w.ldl - D.r);
  t.ldp = w.ldl;
  t.Y = (const float *)(ws + tl.Y);
  t.Lbase = (const float *)(ws + w.LP);
  t.ldl = w.ldl;
  t.labels = labels;
  t.part = (float *)(ws + tl.part);
  t.lab = (float *)(ws + tl.lab);
  t.ce = ce ? ce : (float *)(ws + tl.ce);
  t.loss = loss;
  t.final_logits = debug ? debug->final_logits : nullptr;
  t.lambda = lambda;
  t.gamma = gamma;
  t.err = (int32_t *)(ws + w.err);
  he = launch_train_loss(t, m->bf16, st);
  prof_end(m, DOMINO_KC_TRAINLOSS, st);
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "training loss launch: %s", hipGetErrorString(he));
  return DOMINO_OK;
}

size_t domino_target_workspace_bytes(domino_model_t m, int32_t batch, int32_t n_nodes, int32_t max_ctx) {
  if (!m || m->has_head || batch < 1 || batch > 64 || n_nodes < 1 || n_nodes > 64 || max_ctx < n_nodes) return 0;
  TargetLayout t;
  if (!target_layout(m, batch, n_nodes, max_ctx, t)) return 0;
  return t.total;
}

domino_status domino_target_verify(domino_model_t m, int32_t batch, int32_t n_nodes, const int32_t *node_token,
                                   const int32_t *node_pos, const uint8_t *ancestor_mask, const int32_t *ctx_lens,
                                   void *ctx_k, void *ctx_v, int32_t max_ctx, void *logits, domino_dtype logits_dtype,
                                   void *workspace, size_t workspace_bytes, void *stream) {
  if (!m) return fail(DOMINO_ERR_INVALID_ARG, "model is NULL");
  if (m->has_head) return fail(DOMINO_ERR_INVALID_ARG, "model is a drafter (create the target with domino_target_create)");
  if (batch < 1 || batch > 64) return fail(DOMINO_ERR_INVALID_ARG, "batch must be in [1, 64]");
  if (n_nodes < 1 || n_nodes > 64) return fail(DOMINO_ERR_INVALID_ARG, "n_nodes must be in [1, 64]");
  if (!node_token || !node_pos || !ancestor_mask || !ctx_lens || !logits)
    return fail(DOMINO_ERR_INVALID_ARG, "a node array, ctx_lens or logits is NULL");
  if (max_ctx < n_nodes) return fail(DOMINO_ERR_INVALID_ARG, "max_ctx must leave room for the %d nodes", n_nodes);
  if (!ctx_k || !ctx_v) return fail(DOMINO_ERR_INVALID_ARG, "ctx_k/ctx_v is NULL");
  if (logits_dtype != DOMINO_F32 && logits_dtype != DOMINO_BF16) return fail(DOMINO_ERR_INVALID_ARG, "bad logits dtype");
  if (!workspace) return fail(DOMINO_ERR_WORKSPACE, "workspace is NULL");
  TargetLayout tl;
  if (!target_layout(m, batch, n_nodes, max_ctx, tl))
    return fail(DOMINO_ERR_UNSUPPORTED, "%d nodes exceed the largest block the attention supports for %d/%d heads",
                n_nodes, m->D.nq, m->D.nkv);
  if (workspace_bytes < tl.total)
    return fail(DOMINO_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, tl.total);

  hipStream_t st = (hipStream_t)stream;
  char *ws = (char *)workspace;
  const WsLayout &w = tl.w;
  Dims D = make_dims(m, batch);
  D.B = tl.Bp;
  const int M = batch * tl.Bp;
  const Plans p = make_plans_rows(m, M, M, M);
  int32_t *err = (int32_t *)(ws + w.err);
  int32_t *tok_p = (int32_t *)(ws + tl.tok), *pos_p = (int32_t *)(ws + tl.pos);
  uint8_t *mask_p = (uint8_t *)(ws + tl.mask);
  launch_fill_u32((uint32_t *)ws, w.hdr_words, 0u, st);
  launch_target_prep(batch, n_nodes, tl.Bp, D.V, node_token, node_pos, ancestor_mask, tok_p, pos_p, mask_p, err, st);
  RowSpec spec;
  spec.tokens = tok_p;
  spec.pos = pos_p;
  spec.amask = mask_p;
  spec.n_store = n_nodes;
  spec.all_rows = true;
  domino_status s = run_layers(m, D, p, spec, nullptr, ctx_lens, ctx_k, ctx_v, max_ctx, nullptr, 0, nullptr, ws, w, st,
                               false);
  if (s != DOMINO_OK) return s;
  launch_target_out(batch, n_nodes, tl.Bp, D.V, (const float *)(ws + w.LP), w.ldl, logits,
                    logits_dtype == DOMINO_BF16, st);
  hipError_t he = hipGetLastError();
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "verify forward launch: %s", hipGetErrorString(he));
  return DOMINO_OK;
}

domino_status domino_target_commit(domino_model_t m, int32_t batch, int32_t n_nodes, int32_t max_depth,
                                   const int32_t *ctx_lens, const int32_t *accept_len, const int32_t *accepted_nodes,
                                   void *ctx_k, void *ctx_v, int32_t max_ctx, int32_t *new_ctx_lens, void *workspace,
                                   void *stream) {
  if (!m) return fail(DOMINO_ERR_INVALID_ARG, "model is NULL");
  if (m->has_head) return fail(DOMINO_ERR_INVALID_ARG, "model is a drafter (create the target with domino_target_create)");
  if (batch < 1 || batch > 64) return fail(DOMINO_ERR_INVALID_ARG, "batch must be in [1, 64]");
  if (n_nodes < 1 || n_nodes > 64 || max_depth < 1 || max_depth > 63)
    return fail(DOMINO_ERR_INVALID_ARG, "n_nodes must be in [1, 64] and max_depth in [1, 63]");
  if (!ctx_lens || !accept_len || !accepted_nodes || !ctx_k || !ctx_v || !new_ctx_lens)
    return fail(DOMINO_ERR_INVALID_ARG, "an argument array is NULL");
  if ((const void *)new_ctx_lens == (const void *)ctx_lens)
    return fail(DOMINO_ERR_INVALID_ARG, "new_ctx_lens must not alias ctx_lens");
  if (max_ctx < n_nodes) return fail(DOMINO_ERR_INVALID_ARG, "max_ctx must be at least n_nodes");
  if (!workspace) return fail(DOMINO_ERR_WORKSPACE, "workspace is NULL");
  const Dims &D = m->D;
  launch_target_commit(m->bf16, m->cfg.n_layers, batch, n_nodes, max_depth, ctx_lens, accept_len, accepted_nodes,
                       ctx_k, ctx_v, max_ctx, D.nkv * D.dh, new_ctx_lens, (int32_t *)workspace, (hipStream_t)stream);
  hipError_t he = hipGetLastError();
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "commit launch: %s", hipGetErrorString(he));
  return DOMINO_OK;
}

domino_status domino_build_tree(int32_t batch, int32_t depth, int32_t branch, const int32_t *topk_ids,
                                const int32_t *anchor_ids, const int32_t *ctx_lens, int32_t *node_token,
                                int32_t *node_parent, int32_t *node_depth, int32_t *node_pos, uint8_t *ancestor_mask,
                                void *stream) {
  if (batch < 1) return fail(DOMINO_ERR_INVALID_ARG, "batch must be >= 1");
  if (depth < 1 || depth > 63) return fail(DOMINO_ERR_INVALID_ARG, "depth must be in [1, 63]");
  if (branch < 1 || branch > 8) return fail(DOMINO_ERR_INVALID_ARG, "branch must be in [1, 8]");
  if (!topk_ids || !anchor_ids || !ctx_lens || !node_token || !node_parent || !node_depth || !node_pos)
    return fail(DOMINO_ERR_INVALID_ARG, "a required pointer is NULL");
  launch_build_tree(batch, depth, branch, topk_ids, anchor_ids, ctx_lens, node_token, node_parent, node_depth,
                    node_pos, ancestor_mask, (hipStream_t)stream);
  hipError_t he = hipGetLastError();
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "build_tree launch: %s", hipGetErrorString(he));
  return DOMINO_OK;
}

size_t domino_verify_workspace_bytes(int32_t batch, int32_t n_nodes, int32_t vocab) {
  if (batch < 1 || n_nodes < 1 || n_nodes > 1024 || vocab < 1) return 0;
  return accept_ws_bytes(batch, n_nodes, vocab);
}

domino_status domino_verify_accept(int32_t batch, int32_t n_nodes, int32_t vocab, int32_t block,
                                   const int32_t *node_token, const int32_t *node_parent, const void *target_logits,
                                   domino_dtype logits_dtype, int32_t *accept_len, int32_t *accepted_nodes,
                                   int32_t *out_tokens, void *workspace, size_t workspace_bytes, void *stream) {
  if (batch < 1) return fail(DOMINO_ERR_INVALID_ARG, "batch must be >= 1");
  if (n_nodes < 1 || n_nodes > 1024) return fail(DOMINO_ERR_INVALID_ARG, "n_nodes must be in [1, 1024]");
  if (vocab < 1) return fail(DOMINO_ERR_INVALID_ARG, "vocab must be >= 1");
  if (block < 2 || block > 64) return fail(DOMINO_ERR_INVALID_ARG, "block must be in [2, 64]");
  if (logits_dtype != DOMINO_F32 && logits_dtype != DOMINO_BF16) return fail(DOMINO_ERR_INVALID_ARG, "bad logits dtype");
  if (!node_token || !node_parent || !target_logits || !accept_len || !accepted_nodes || !out_tokens)
    return fail(DOMINO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (!workspace) return fail(DOMINO_ERR_WORKSPACE, "workspace is NULL");
  const size_t need = accept_ws_bytes(batch, n_nodes, vocab);
  if (workspace_bytes < need) return fail(DOMINO_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  hipStream_t st = (hipStream_t)stream;
  launch_accept(batch, n_nodes, vocab, block, node_token, node_parent, target_logits, logits_dtype == DOMINO_BF16,
                accept_len, accepted_nodes, out_tokens, workspace, st);
  hipError_t he = hipGetLastError();
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "verify_accept launch: %s", hipGetErrorString(he));
  return DOMINO_OK;
}

// ---- acceptance without a workspace: the argmax partials live in a fixed
// device array, one copy per GPU, held until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is only a stand-in for the
// symbol); it uses the address hipGetSymbolAddress returns for the current
// device, looked up once per device.
namespace {
constexpr size_t kNoAllocScratchBytes = (size_t)DOMINO_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

domino_status scratch_for_current_device(void **out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(DOMINO_ERR_UNSUPPORTED, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(DOMINO_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DOMINO_OK;
}
}  // namespace

domino_status domino_verify_accept_noalloc(int32_t batch, int32_t n_nodes, int32_t vocab, int32_t block,
                                           const int32_t *node_token, const int32_t *node_parent,
                                           const void *target_logits, domino_dtype logits_dtype,
                                           int32_t *accept_len, int32_t *accepted_nodes, int32_t *out_tokens,
                                           int32_t *error_word, void *stream) {
  if (batch < 1) return fail(DOMINO_ERR_INVALID_ARG, "batch must be >= 1");
  if (n_nodes < 1 || n_nodes > 1024) return fail(DOMINO_ERR_INVALID_ARG, "n_nodes must be in [1, 1024]");
  if (vocab < 1) return fail(DOMINO_ERR_INVALID_ARG, "vocab must be >= 1");
  if (block < 2 || block > 64) return fail(DOMINO_ERR_INVALID_ARG, "block must be in [2, 64]");
  if (logits_dtype != DOMINO_F32 && logits_dtype != DOMINO_BF16) return fail(DOMINO_ERR_INVALID_ARG, "bad logits dtype");
  if (!node_token || !node_parent || !target_logits || !accept_len || !accepted_nodes || !out_tokens || !error_word)
    return fail(DOMINO_ERR_INVALID_ARG, "a required pointer is NULL");
  const size_t ent = accept_part_entries(batch, n_nodes, vocab);
  if (ent * 8 > kNoAllocScratchBytes)
    return fail(DOMINO_ERR_UNSUPPORTED,
                "batch %d x %d nodes x vocab %d needs %zu bytes of argmax partials; the fixed scratch holds %zu "
                "(use domino_verify_accept with a workspace)",
                batch, n_nodes, vocab, ent * 8, kNoAllocScratchBytes);
  void *sp = nullptr;
  domino_status s = scratch_for_current_device(&sp);
  if (s != DOMINO_OK) return s;
  float *pv = (float *)sp;
  launch_accept_parts(batch, n_nodes, vocab, block, node_token, node_parent, target_logits,
                      logits_dtype == DOMINO_BF16, accept_len, accepted_nodes, out_tokens, pv,
                      (int32_t *)(pv + ent), error_word, (hipStream_t)stream);
  hipError_t he = hipGetLastError();
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "verify_accept_noalloc launch: %s", hipGetErrorString(he));
  return DOMINO_OK;
}

size_t domino_verify_sample_workspace_bytes(int32_t batch, int32_t block, int32_t vocab) {
  if (batch < 1 || block < 2 || block > 64 || vocab < 1) return 0;
  return vs_ws_bytes(batch, block, vocab);
}

domino_status domino_verify_sample(int32_t batch, int32_t block, int32_t vocab, const int32_t *node_token,
                                   const void *target_logits, domino_dtype logits_dtype, const float *draft_logits,
                                   float temperature, uint64_t seed, int32_t *accept_len, int32_t *accepted_nodes,
                                   int32_t *out_tokens, void *workspace, size_t workspace_bytes, void *stream) {
  if (batch < 1) return fail(DOMINO_ERR_INVALID_ARG, "batch must be >= 1");
  if (block < 2 || block > 64) return fail(DOMINO_ERR_INVALID_ARG, "block must be in [2, 64]");
  if (vocab < 1) return fail(DOMINO_ERR_INVALID_ARG, "vocab must be >= 1");
  if (logits_dtype != DOMINO_F32 && logits_dtype != DOMINO_BF16) return fail(DOMINO_ERR_INVALID_ARG, "bad logits dtype");
  if (!(temperature > 0.f) || !std::isfinite(temperature) || 1.0f / temperature > 1e30f)
    return fail(DOMINO_ERR_INVALID_ARG, "temperature must be positive and finite");
  if (!node_token || !target_logits || !draft_logits || !accept_len || !accepted_nodes || !out_tokens)
    return fail(DOMINO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (!workspace) return fail(DOMINO_ERR_WORKSPACE, "workspace is NULL");
  const size_t need = vs_ws_bytes(batch, block, vocab);
  if (workspace_bytes < need) return fail(DOMINO_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  hipStream_t st = (hipStream_t)stream;
  launch_fill_u32((uint32_t *)workspace, 1, 0u, st);
  launch_verify_sample(batch, block, vocab, node_token, target_logits, logits_dtype == DOMINO_BF16, draft_logits,
                       temperature, seed, accept_len, accepted_nodes, out_tokens, workspace, st);
  hipError_t he = hipGetLastError();
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "verify_sample launch: %s", hipGetErrorString(he));
  return DOMINO_OK;
}

domino_status domino_philox4x32_10(const uint32_t *counters, uint64_t key, uint32_t *out, int32_t n, void *stream) {
  if (n < 0) return fail(DOMINO_ERR_INVALID_ARG, "n must be >= 0");
  if (n > 0 && (!counters || !out)) return fail(DOMINO_ERR_INVALID_ARG, "counters/out is NULL");
  launch_philox_words(counters, key, out, n, (hipStream_t)stream);
  hipError_t he = hipGetLastError();
  if (he != hipSuccess) return fail(DOMINO_ERR_HIP, "philox launch: %s", hipGetErrorString(he));
  return DOMINO_OK;
}

domino_status domino_workspace_error(const void *workspace, void *stream, int32_t *out) {
  if (!workspace || !out) return fail(DOMINO_ERR_INVALID_ARG, "workspace/out is NULL");
  int32_t v = 0;
  HIP_TRY(hipMemcpyAsync(&v, workspace, 4, hipMemcpyDeviceToHost, (hipStream_t)stream));
  HIP_TRY(hipStreamSynchronize((hipStream_t)stream));
  *out = v;
  if (v) return fail(DOMINO_ERR_DEVICE, "device error word 0x%x", v);
  return DOMINO_OK;
}

domino_status domino_workspace_clear_error(void *workspace, void *stream) {
  if (!workspace) return fail(DOMINO_ERR_INVALID_ARG, "workspace is NULL");
  launch_fill_u32((uint32_t *)workspace, 1, 0u, (hipStream_t)stream);
  HIP_TRY(hipGetLastError());
  return DOMINO_OK;
}

domino_status domino_profile_enable(domino_model_t m, uint32_t class_mask) {
  if (!m) return fail(DOMINO_ERR_INVALID_ARG, "model is NULL");
  for (int c = 0; c < DOMINO_KC_COUNT; ++c) {
    if (!(class_mask & (1u << c))) continue;
    auto &e = m->ev[c];
    while (e.a.size() < 4096) {
      hipEvent_t x, y;
      HIP_TRY(hipEventCreate(&x));
      HIP_TRY(hipEventCreate(&y));
      e.a.push_back(x);
      e.b.push_back(y);
    }
  }
  m->prof_mask = class_mask;
  return DOMINO_OK;
}

domino_status domino_profile_reset(domino_model_t m) {
  if (!m) return fail(DOMINO_ERR_INVALID_ARG, "model is NULL");
  for (auto &e : m->ev) e.used = 0;
  return DOMINO_OK;
}

domino_status domino_debug_last_paths(domino_model_t m, uint32_t *paths) {
  if (!m || !paths) return fail(DOMINO_ERR_INVALID_ARG, "NULL argument");
  *paths = m->last_paths;
  return DOMINO_OK;
}

domino_status domino_debug_set_poll_limit(domino_model_t m, int32_t polls) {
  if (!m) return fail(DOMINO_ERR_INVALID_ARG, "model is NULL");
  m->poll_limit = polls < 0 ? kDefaultPollLimit : (uint32_t)polls;
  return DOMINO_OK;
}

domino_status domino_profile_read(domino_model_t m, int32_t kernel_class, double *total_ms, int32_t *launches) {
  if (!m || !total_ms || !launches) return fail(DOMINO_ERR_INVALID_ARG, "NULL argument");
  if (kernel_class < 0 || kernel_class >= DOMINO_KC_COUNT) return fail(DOMINO_ERR_INVALID_ARG, "bad kernel class");
  auto &e = m->ev[kernel_class];
  double tot = 0;
  for (int i = 0; i < e.used; ++i) {
    HIP_TRY(hipEventSynchronize(e.b[i]));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, e.a[i], e.b[i]));
    tot += ms;
  }
  *total_ms = tot;
  *launches = e.used;
  return DOMINO_OK;
}

}  // extern "C"
