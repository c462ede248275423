// Domino-head rollout (Sec. 4.1.2 causal encoder and low-rank correction,
// Fig. 3 sequential rollout), as three short kernels per draft position j:
//
//   gru    y_{j-1} = top-1 of position j-1 (merged from the logits kernel's
//          per-workgroup lists; the anchor for j = 1; a forced token when
//          teacher forcing), then S_{j-1} = GRU(E[y_{j-1}], S_{j-2}) for a
//          slice of the d_s state indices per workgroup.  The input half of
//          the gates, E[y] W_ih^T, is a row of the table G = E W_ih^T built at
//          model creation, so a step gathers 3*d_s values instead of streaming
//          W_ih.
//   u      u = SiLU(W1[:, :d] H_j + W1[:, d:] S_{j-1}) (the H half comes from
//          the LM-head GEMM).
//   logits L_j = L_base_j + W2 u over a vocabulary slice per workgroup, the
//          slice's top-beta under (value desc, id asc), and an atomic max of
//          its top-1 into the position's key.
// A kernel boundary is the cheapest grid-wide handshake on this device (about
// 1.6 us against about 4 us for a 256-workgroup spin barrier), so the
// rollout is 3(B-1)+1 launches rather than one persistent kernel; the top-1
// of each position is a 64-bit atomic max, so no launch merges lists inside
// the loop (the full top-beta lists are merged once at the end).
#include "common.h"
#include "kernels.h"
#include "mfma.h"
#include "philox.h"

namespace dk {

// Insert (v, id) into a sorted 8-entry list (best first) by bubbling.
DEVI void list_insert(float (&lv)[8], int (&li)[8], float v, int id) {
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    if (better(v, id, lv[q], li[q])) {
      const float tv = lv[q];
      const int ti = li[q];
      lv[q] = v;
      li[q] = id;
      v = tv;
      id = ti;
    }
  }
}

// Extract the wave's top-beta from per-lane sorted lists: lane k (< beta)
// receives the k-th best in (mv, mi); other lanes get (-inf, INT_MAX).
DEVI void wave_extract(float (&lv)[8], int (&li)[8], int beta, float &mv, int &mi) {
  const int lane = threadIdx.x & 63;
  mv = -INFINITY;
  mi = INT_MAX;
  for (int k = 0; k < beta; ++k) {
    float bv = lv[0];
    int bi = li[0];
    wave_best(bv, bi);
    if (lane == k) {
      mv = bv;
      mi = bi;
    }
    if (li[0] == bi && bi != INT_MAX) {  // ids are unique: exactly one owner advances
#pragma unroll
      for (int q = 0; q < 7; ++q) {
        lv[q] = lv[q + 1];
        li[q] = li[q + 1];
      }
      lv[7] = -INFINITY;
      li[7] = INT_MAX;
    }
  }
}

// Wave-level top-beta of the candidates c in [c0, c1) produced by get(c);
// lane k (< beta) ends with the k-th best in (mv, mi).
template <typename Get>
DEVI void wave_select(Get get, int c0, int c1, int beta, float &mv, int &mi) {
  const int lane = threadIdx.x & 63;
  if (beta == 1) {  // a running best is enough
    float bv = -INFINITY;
    int bi = INT_MAX;
    for (int c = c0 + lane; c < c1; c += 64) {
      float v;
      int id;
      get(c, v, id);
      v = order_val(v);
      if (id != INT_MAX && better(v, id, bv, bi)) {
        bv = v;
        bi = id;
      }
    }
    wave_best(bv, bi);
    mv = lane == 0 ? bv : -INFINITY;
    mi = lane == 0 ? bi : INT_MAX;
    return;
  }
  float lv[8];
  int li[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    lv[q] = -INFINITY;
    li[q] = INT_MAX;
  }
  for (int c = c0 + lane; c < c1; c += 64) {
    float v;
    int id;
    get(c, v, id);
    if (id == INT_MAX) continue;
    list_insert(lv, li, order_val(v), id);
  }
  wave_extract(lv, li, beta, mv, mi);
}

// wave_select over candidates in global memory: each lane loads its
// candidates 8 at a time, all loads of a batch in flight together.
DEVI void wave_select_mem(const float *__restrict__ pv, const int32_t *__restrict__ pi, int cnt, int beta,
                          float &mv, int &mi) {
  const int lane = threadIdx.x & 63;
  float lv[8];
  int li[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    lv[q] = -INFINITY;
    li[q] = INT_MAX;
  }
  for (int c0 = 0; c0 < cnt; c0 += 8 * 64) {
    float v[8];
    int id[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int c = c0 + u * 64 + lane;
      const int cc = c < cnt ? c : cnt - 1;
      v[u] = pv[cc];
      id[u] = c < cnt ? pi[cc] : INT_MAX;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (id[u] != INT_MAX) list_insert(lv, li, order_val(v[u]), id[u]);
  }
  wave_extract(lv, li, beta, mv, mi);
}

DEVI float sigm(float x) { return 1.f / (1.f + expf(-x)); }
// The GRU's new state (1 - z) n + z h, written as n + z (h - n) with one
// explicit fused multiply-add: left to the compiler, the two products of the
// plain form get contracted differently from one kernel instantiation to the
// next, and the instantiations would disagree in the last bit.
DEVI float gru_mix(float z, float n, float h) { return fmaf(z, h - n, n); }

constexpr int kBestSlots = 8;  // atomic targets per (position, row), spread to cut contention

template <typename WT>
DEVI void unpack16(const u32x4 &w, float *f);
template <>
DEVI void unpack16<bf16_t>(const u32x4 &w, float *f) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    f[2 * q] = __uint_as_float(w[q] << 16);
    f[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
  }
}
template <>
DEVI void unpack16<float>(const u32x4 &w, float *f) {
#pragma unroll
  for (int q = 0; q < 4; ++q) f[q] = __uint_as_float(w[q]);
}

// ---------------------------------------------------------------------------
// state (batches up to kFusedBatch; replaces gru + u): every workgroup forms
// the whole S_{j-1} itself from the gathered input gates G[y_{j-1}], the
// hidden gates W_hh S_{j-2} that the previous position left in ghbuf, and
// S_{j-2}; its waves then take rows of the stacked matrix [W1[:, d:]; W_hh]
// against S_{j-1}.  The first r rows give u_j = SiLU(P_j + W1[:, d:] S_{j-1}),
// the other 3 d_s rows the hidden gates of position j+1, so the elementwise
// update is the only step repeated per workgroup and no launch sits between
// the state and u.  Weight rows are loaded before the state is formed.
// ---------------------------------------------------------------------------
constexpr int kFusedBatch = kHeadFusedBatch;
constexpr int kStateWaves = 8;
constexpr int kStateMaxGrid = 256;

template <typename WT>
__global__ __launch_bounds__(kStateWaves * 64) void head_state_kernel(HeadArgs h, int j) {
  constexpr int EPL = 16 / sizeof(WT);
  const Dims &D = h.D;
  const int bs = D.bs, ds = D.ds, r = D.r, d = D.d, depth = D.B - 1, V = D.V;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  extern __shared__ __align__(16) float sl[];  // S_{j-1} [bs][ds]
  __shared__ int ys[kFusedBatch];
  const int nchunk = ds / EPL;  // <= 256
  const int nrows = r + (j < depth ? 3 * ds : 0);
  const int rbeg = h.skip_u ? r : 0;  // skip_u: only the W_hh rows (u is formed later, batched)
  const int nw = gridDim.x * kStateWaves;
  const int w0 = blockIdx.x * kStateWaves + wave;
  const WT *w1 = (const WT *)h.w1, *whh = (const WT *)h.w_hh;

  // ---- the sources of y_{j-1} first (every thread, clamped batch row, so no
  // branch holds the later loads back), then this wave's weight rows
  const int bq = min(tid, bs - 1);
  const int anc = h.anchor[bq];
  unsigned long long keys[kBestSlots];
  {
    const unsigned long long *bk = h.best + ((size_t)(j > 1 ? j - 2 : 0) * bs + bq) * kBestSlots;
#pragma unroll
    for (int q = 0; q < kBestSlots; ++q) keys[q] = bk[q];
  }
  // two rows per wave per round (rows w0 + k*nw); the first round's loads go out now
  u32x4 w[2][4];
  auto load_rows = [&](int base) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int row = min(base + q * nw, nrows - 1);
      const WT *p = row < r ? w1 + (size_t)row * (d + ds) + d : whh + (size_t)(row - r) * ds;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int ch = min(lane + 64 * c, nchunk - 1);
        w[q][c] = *(const u32x4 *)(p + (size_t)ch * EPL);
      }
    }
  };
  load_rows(rbeg + w0);

  // ---- y_{j-1}: the anchor, a forced token, or the decoded best key of position j-1
  if (tid < bs) {
    int y;
    if (j == 1) y = clamp_token(anc, V, h.err);
    else if (h.forced) y = clamp_token(h.forced[(size_t)tid * depth + (j - 2)], V, h.err);  // teacher forcing
    else {
      unsigned long long key = keys[0];
#pragma unroll
      for (int q = 1; q < kBestSlots; ++q) key = keys[q] > key ? keys[q] : key;
      y = decode_best_id(key, V);
    }
    ys[tid] = y;
  }
  __syncthreads();

  // ---- S_{j-1} = GRU(x = E[y_{j-1}], S_{j-2}), four state indices per item.
  // G holds E W_ih^T + b_ih; the stored gates hold W_hh S_{j-2} + b_hh (at j = 1,
  // S = 0: the gates are b_hh).  Every load is unconditional (the position-1
  // values are selected after), so none waits behind a branch.
  const float *ghp = h.ghbuf + (size_t)((j - 1) & 1) * bs * 3 * ds;  // W_hh S_{j-2} + b_hh
  const float *sprev = h.hbuf + (size_t)(j & 1) * bs * ds;            // S_{j-2}
  float *scur = h.hbuf + (size_t)((j - 1) & 1) * bs * ds;             // S_{j-1}
  for (int it = tid; it < bs * ds / 4; it += kStateWaves * 64) {
    const int b = it / (ds / 4), i = (it % (ds / 4)) * 4;
    const float *gy = h.gtab + (size_t)ys[b] * 3 * ds;
    float gi[3][4], gh[3][4], hold[4];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      const float4 a = *(const float4 *)(gy + q * ds + i);
      const float4 c = *(const float4 *)(ghp + (size_t)b * 3 * ds + q * ds + i);
      const float4 c0 = *(const float4 *)(h.bhh + q * ds + i);
      gi[q][0] = a.x; gi[q][1] = a.y; gi[q][2] = a.z; gi[q][3] = a.w;
      gh[q][0] = j > 1 ? c.x : c0.x; gh[q][1] = j > 1 ? c.y : c0.y;
      gh[q][2] = j > 1 ? c.z : c0.z; gh[q][3] = j > 1 ? c.w : c0.w;
    }
    {
      const float4 c = *(const float4 *)(sprev + (size_t)b * ds + i);
      hold[0] = j > 1 ? c.x : 0.f; hold[1] = j > 1 ? c.y : 0.f;
      hold[2] = j > 1 ? c.z : 0.f; hold[3] = j > 1 ? c.w : 0.f;
    }
    float out[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float rg = sigm(gi[0][e] + gh[0][e]);
      const float zg = sigm(gi[1][e] + gh[1][e]);
      const float ng = tanhf(fmaf(rg, gh[2][e], gi[2][e]));
      out[e] = gru_mix(zg, ng, hold[e]);
    }
    const float4 o = make_float4(out[0], out[1], out[2], out[3]);
    *(float4 *)(sl + (size_t)b * ds + i) = o;
    if (blockIdx.x == 0) {
      *(float4 *)(scur + (size_t)b * ds + i) = o;
      if (h.states) *(float4 *)(h.states + ((size_t)b * depth + (j - 1)) * ds + i) = o;
    }
  }
  __syncthreads();

  // ---- rows of [W1[:, d:]; W_hh] against S_{j-1}
  float *ghn = h.ghbuf + (size_t)(j & 1) * bs * 3 * ds;  // W_hh S_{j-1}
  for (int base = rbeg + w0; base < nrows; base += 2 * nw) {
    if (base != rbeg + w0) load_rows(base);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int row = base + q * nw;
      if (row >= nrows) continue;  // wave-uniform
      float wf[4][EPL];
#pragma unroll
      for (int c = 0; c < 4; ++c) unpack16<WT>(w[q][c], wf[c]);
      for (int b = 0; b < bs; ++b) {
        const float *sb = sl + (size_t)b * ds;
        float acc = 0.f;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int ch = lane + 64 * c;
          if (ch < nchunk) {
#pragma unroll
            for (int e = 0; e < EPL; e += 4) {
              const float4 t = *(const float4 *)(sb + (size_t)ch * EPL + e);
              acc = fmaf(wf[c][e], t.x, acc);
              acc = fmaf(wf[c][e + 1], t.y, acc);
              acc = fmaf(wf[c][e + 2], t.z, acc);
              acc = fmaf(wf[c][e + 3], t.w, acc);
            }
          }
        }
        acc = wave_sum(acc);
        if (lane == 0) {
          if (row < r) {
            const float x = h.P[((size_t)b * depth + (j - 1)) * h.ldp + row] + acc;
            h.ubuf[(size_t)b * h.u_ld + (size_t)(j - 1) * h.u_pos + row] = x / (1.f + expf(-x));
          } else {
            ghn[(size_t)b * 3 * ds + (row - r)] = acc + h.bhh[row - r];
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Batches above kFusedBatch: W_hh S_{j-1} and W1[:, d:] S_j run as K-split
// GEMMs (the projections' weight-streaming kernel over packed copies of the
// two matrices), which stage the states once per workgroup; these kernels add
// the partials in split order and finish each step elementwise.
// ---------------------------------------------------------------------------
// S_j = GRU(G[y_{j-1}], S_{j-1}), one workgroup row per batch row
__global__ __launch_bounds__(256) void head_gru_elem_kernel(HeadArgs h, int j, const float *__restrict__ gp, int np,
                                                            size_t pstride) {
  const Dims &D = h.D;
  const int bs = D.bs, ds = D.ds, depth = D.B - 1, V = D.V;
  const int b = blockIdx.y;
  __shared__ int ysh;
  if (threadIdx.x == 0) {  // y_{j-1}: the anchor, a forced token, or the decoded best key of position j-1
    int y;
    if (j == 1) y = clamp_token(h.anchor[b], V, h.err);
    else if (h.forced) y = clamp_token(h.forced[(size_t)b * depth + (j - 2)], V, h.err);
    else {
      const unsigned long long *bk = h.best + ((size_t)(j - 2) * bs + b) * kBestSlots;
      unsigned long long key = bk[0];
#pragma unroll
      for (int q = 1; q < kBestSlots; ++q) key = bk[q] > key ? bk[q] : key;
      y = decode_best_id(key, V);
    }
    ysh = y;
  }
  __syncthreads();
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= ds) return;
  const float *hprev = h.hbuf + (size_t)((j - 1) & 1) * bs * ds;
  float *hnext = h.hbuf + (size_t)(j & 1) * bs * ds;
  float gh[3];
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    float acc = 0.f;  // W_hh S_{j-1} (S_0 = 0: no product at j = 1)
    for (int p = 0; p < np; ++p) acc += gp[(size_t)p * pstride + (size_t)b * 3 * ds + q * ds + i];
    gh[q] = acc + h.bhh[q * ds + i];
  }
  const float *gy = h.gtab + (size_t)ysh * 3 * ds;  // b_ih is in G
  const float rg = sigm(gy[i] + gh[0]), zg = sigm(gy[ds + i] + gh[1]);
  const float ng = tanhf(fmaf(rg, gh[2], gy[2 * ds + i]));
  const float hold = j > 1 ? hprev[(size_t)b * ds + i] : 0.f;
  const float hn = gru_mix(zg, ng, hold);
  hnext[(size_t)b * ds + i] = hn;
  if (h.states) h.states[((size_t)b * depth + (j - 1)) * ds + i] = hn;
}

// u_j = SiLU(W1[:, :d] H_j + W1[:, d:] S_j) from the summed partials
__global__ __launch_bounds__(256) void head_u_elem_kernel(HeadArgs h, int j, const float *__restrict__ up, int np,
                                                          size_t pstride) {
  const Dims &D = h.D;
  const int r = D.r, depth = D.B - 1;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= D.bs * r) return;
  const int b = e / r, k = e % r;
  float acc = 0.f;
  for (int p = 0; p < np; ++p) acc += up[(size_t)p * pstride + e];
  const float x = h.P[((size_t)b * depth + (j - 1)) * h.ldp + k] + acc;
  h.ubuf[(size_t)b * h.u_ld + (size_t)(j - 1) * h.u_pos + k] = x / (1.f + expf(-x));
}

// ---------------------------------------------------------------------------
// logits: matrix-core W2 tiles times the staged u (batch rows as the 16
// columns of the B operand, hi/lo split for bf16), plus L_base, then each
// workgroup's top-beta per batch row.  A workgroup covers ROWS vocabulary
// rows (8 waves x kTPW tiles of 16).
// ---------------------------------------------------------------------------
constexpr int kLogitWaves = 8;
// W2 tiles per wave: as many as fit the registers (all of a wave's loads are
// issued at once, and the grid then fits the GPU in one round)
constexpr int kTpwSmall = 5;
constexpr int logit_tpw(int KS, int MT) { return KS * MT <= 8 ? kTpwSmall : (KS * MT <= 16 ? 3 : 1); }

// Compare-exchange under the selection order: (a, b) -> (better, worse).
DEVI void sel_ce(float &va, int &ia, float &vb, int &ib) {
  const bool t = better(vb, ib, va, ia);
  const float v0 = t ? vb : va, v1 = t ? va : vb;
  const int i0 = t ? ib : ia, i1 = t ? ia : ib;
  va = v0;
  ia = i0;
  vb = v1;
  ib = i1;
}
// a (sorted best first) <- the best L of a and b (both sorted): the pairwise
// better of a[i] and b[L-1-i] is a bitonic sequence holding exactly those L,
// which a bitonic merge network sorts.
template <int L>
DEVI void sel_merge(float (&av)[L], int (&ai)[L], const float (&bv)[L], const int (&bi)[L]) {
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const bool t = better(bv[L - 1 - i], bi[L - 1 - i], av[i], ai[i]);
    av[i] = t ? bv[L - 1 - i] : av[i];
    ai[i] = t ? bi[L - 1 - i] : ai[i];
  }
#pragma unroll
  for (int st = L / 2; st >= 1; st >>= 1)
#pragma unroll
    for (int i = 0; i < L; ++i)
      if ((i & st) == 0) sel_ce(av[i], ai[i], av[i + st], ai[i + st]);
}

// Top-beta (beta <= L) of a logits workgroup's rows for every batch row, in
// registers: each lane sorts its own candidates of a batch row into an
// L-entry list; within a wave the four lanes of a row (g) hand their lists to
// lane g = 0 through LDS, which merges them; the waves' lists meet in LDS,
// where one thread per batch row merges them and emits the first beta
// entries (and the top-1 into the position's key).  (Merging by cross-lane
// shuffles instead made the compiler take minutes per instantiation.)
// LDS the lists need (after the u fragments): a wave's lane lists of one
// m-tile, and each wave's list per batch row
constexpr size_t topl_lds_bytes(int L, int MT) {
  return (size_t)kLogitWaves * (4 * 16 + MT * 16) * L * (sizeof(float) + sizeof(int));
}
template <int L, int kTPW, int MT>
DEVI void logits_topl(const HeadArgs &h, int j, const int (&tiles)[kTPW], const float4 (&lb)[kTPW][MT],
                      const floatx4 (&acc)[kTPW][MT], unsigned char *sbuf) {
  const Dims &D = h.D;
  const int bs = D.bs, V = D.V, beta = h.beta;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, cc = lane & 15;
  auto xg_v = (float(*)[4][16][L])sbuf;  // [kLogitWaves][4][16][L]
  auto xg_i = (int(*)[4][16][L])(sbuf + sizeof(float) * kLogitWaves * 4 * 16 * L);
  auto cand_v = (float(*)[MT * 16][L])(sbuf + (sizeof(float) + sizeof(int)) * kLogitWaves * 4 * 16 * L);
  auto cand_i = (int(*)[MT * 16][L])(sbuf + (sizeof(float) + sizeof(int)) * kLogitWaves * 4 * 16 * L +
                                     sizeof(float) * kLogitWaves * MT * 16 * L);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    float lv[L];
    int li[L];
#pragma unroll
    for (int k = 0; k < L; ++k) {
      lv[k] = -INFINITY;
      li[k] = INT_MAX;
    }
#pragma unroll
    for (int q = 0; q < kTPW; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int n = tiles[q] * 16 + 4 * g + e;
        const float lbe = e == 0 ? lb[q][mt].x : (e == 1 ? lb[q][mt].y : (e == 2 ? lb[q][mt].z : lb[q][mt].w));
        float v = n < V ? order_val(lbe + acc[q][mt][e]) : -INFINITY;
        int id = n < V ? n : INT_MAX;
#pragma unroll
        for (int k = 0; k < L; ++k) sel_ce(lv[k], li[k], v, id);  // bubble (v, id) into place
      }
    // a wave's LDS accesses complete in order, so lane g = 0 reads the lists
    // the other lanes of its wave wrote just before (and the next m-tile's
    // writes follow its reads)
    if (g > 0) {
#pragma unroll
      for (int k = 0; k < L; ++k) {
        xg_v[wave][g][cc][k] = lv[k];
        xg_i[wave][g][cc][k] = li[k];
      }
    }
    __builtin_amdgcn_wave_barrier();
    if (g == 0) {
#pragma unroll
      for (int o = 1; o < 4; ++o) {
        float ov[L];
        int oi[L];
#pragma unroll
        for (int k = 0; k < L; ++k) {
          ov[k] = xg_v[wave][o][cc][k];
          oi[k] = xg_i[wave][o][cc][k];
        }
        sel_merge<L>(lv, li, ov, oi);
      }
#pragma unroll
      for (int k = 0; k < L; ++k) {
        cand_v[wave][mt * 16 + cc][k] = lv[k];
        cand_i[wave][mt * 16 + cc][k] = li[k];
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  __syncthreads();
  for (int bb = tid; bb < bs; bb += kLogitWaves * 64) {
    float lv[L];
    int li[L];
#pragma unroll
    for (int k = 0; k < L; ++k) {
      lv[k] = cand_v[0][bb][k];
      li[k] = cand_i[0][bb][k];
    }
    for (int w = 1; w < kLogitWaves; ++w) {
      float ov[L];
      int oi[L];
#pragma unroll
      for (int k = 0; k < L; ++k) {
        ov[k] = cand_v[w][bb][k];
        oi[k] = cand_i[w][bb][k];
      }
      sel_merge<L>(lv, li, ov, oi);
    }
    const size_t o = (((size_t)(j - 1) * bs + bb) * h.GC + blockIdx.x) * beta;
#pragma unroll
    for (int k = 0; k < L; ++k)
      if (k < beta) {
        h.pval[o + k] = lv[k];
        h.pid[o + k] = li[k];
      }
    // top-1 of this workgroup into the position's best key (order-independent max)
    if (li[0] != INT_MAX)
      atomicMax(&h.best[((size_t)(j - 1) * bs + bb) * kBestSlots + (blockIdx.x % kBestSlots)], encode_best(lv[0], li[0]));
  }
}

template <typename WT, int KS, int MT>
__global__ __launch_bounds__(kLogitWaves * 64) void head_logits_kernel(HeadArgs h, int j) {
  constexpr int EPL = Frag<WT>::EPL, KSTEP = Frag<WT>::KSTEP, XF = XStage<WT>::XF;
  constexpr int kTPW = logit_tpw(KS, MT);
  const Dims &D = h.D;
  const int bs = D.bs, r = D.r, V = D.V, depth = D.B - 1, beta = h.beta;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, cc = lane & 15;
  const int NT = (V + 15) / 16;
  extern __shared__ __align__(16) unsigned char smem[];
  u32x4 *us = (u32x4 *)smem;                                      // [KS][MT][64][XF]

  // u_j first (a few L2-resident values), so the matrix-core work can follow
  // the W2 stream as its fragments arrive
  constexpr int kUIt = (KS * MT * 64 + kLogitWaves * 64 - 1) / (kLogitWaves * 64);
  float4 uv[kUIt][EPL / 4];
#pragma unroll
  for (int q = 0; q < kUIt; ++q) {
    const int it = min(tid + q * kLogitWaves * 64, KS * MT * 64 - 1);
    const int l = it & 63, mt = (it >> 6) % MT, s = (it >> 6) / MT;
    const int bb = mt * 16 + (l & 15);
    const int k0 = s * KSTEP + (l >> 4) * EPL;
    // unconditional loads at a clamped row: a guarded load becomes a branch
    // whose join drains every outstanding load, holding back the W2 stream
    // issued below.  Columns of padding rows (bb >= bs) only reach output
    // columns that are never read, so their values do not matter.
    const float *src = h.ubuf + (size_t)min(bb, bs - 1) * h.u_ld + (size_t)(j - 1) * h.u_pos + k0;
#pragma unroll
    for (int e = 0; e < EPL / 4; ++e) uv[q][e] = *(const float4 *)(src + 4 * e);
  }
  // then the L_base values this wave will add (rows are padded to whole tiles,
  // ldl >= 16 * NT, so a tile's four values load as one float4; entries past V
  // are masked below), then the W2 fragments of its tiles
  int tiles[kTPW];
#pragma unroll
  for (int q = 0; q < kTPW; ++q) tiles[q] = (blockIdx.x * kLogitWaves + wave) * kTPW + q;
  float4 lb[kTPW][MT];
#pragma unroll
  for (int q = 0; q < kTPW; ++q)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int bb = mt * 16 + cc;
      const int t = tiles[q] < NT ? tiles[q] : NT - 1;
      // clamped row, unconditional (lanes of padding rows are never read)
      lb[q][mt] = *(const float4 *)(h.Lbase + ((size_t)min(bb, bs - 1) * depth + (j - 1)) * h.ldl + t * 16 + 4 * g);
    }
  const u32x4 *w2p = (const u32x4 *)h.w2p;
  u32x4 wf[kTPW][KS];
#pragma unroll
  for (int q = 0; q < kTPW; ++q) {
    const int t = tiles[q] < NT ? tiles[q] : NT - 1;
#pragma unroll
    for (int s = 0; s < KS; ++s) wf[q][s] = w2p[((size_t)t * KS + s) * 64 + lane];
  }
  // u staged as matrix-core B fragments
#pragma unroll
  for (int q = 0; q < kUIt; ++q) {
    const int it = tid + q * kLogitWaves * 64;
    if (it < KS * MT * 64) XStage<WT>::put(us + (size_t)it * XF, uv[q]);
  }
  __syncthreads();

  floatx4 acc[kTPW][MT];
#pragma unroll
  for (int q = 0; q < kTPW; ++q)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[q][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
  // tile-major, in the order the fragments were requested: tile q's products
  // start as soon as its fragments arrive, overlapping the rest of the stream
#pragma unroll
  for (int q = 0; q < kTPW; ++q)
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      u32x4 xf[MT * XF];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int f = 0; f < XF; ++f) xf[mt * XF + f] = us[((size_t)(s * MT + mt) * 64 + lane) * XF + f];
      Mac2<WT, MT>::step(wf[q][s], xf, acc[q]);
    }

  // corrected logits of this workgroup's rows: lane (g, cc) holds rows
  // 16 t + 4 g + e of batch row mt * 16 + cc
  if (beta == 1) {
    // top-1 without staging: a running best per batch row in registers, the
    // four lanes of a row combined by shuffles, then one entry per (wave, row)
    // With sampling the key is L / T + Gumbel noise of (row, position, id): the
    // maximum is a draw from softmax(L / T); raw carries the chosen L.
    __shared__ float best_v[kLogitWaves][64], best_r[kLogitWaves][64];
    __shared__ int best_i[kLogitWaves][64];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int bb = mt * 16 + cc;
      float bv = -INFINITY, br = 0.f;
      int bi = INT_MAX;
#pragma unroll
      for (int q = 0; q < kTPW; ++q) {
        Philox4 noise = {{0u, 0u, 0u, 0u}};
        if (h.sample && bb < bs) noise = rng_block(h.seed_lo, h.seed_hi, RNG_DRAFT, bb, j, tiles[q] * 4 + g);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int n = tiles[q] * 16 + 4 * g + e;
          const float lbe = e == 0 ? lb[q][mt].x : (e == 1 ? lb[q][mt].y : (e == 2 ? lb[q][mt].z : lb[q][mt].w));
          const float val = lbe + acc[q][mt][e];
          if (bb < bs && n < V) {
            if (h.final_logits) h.final_logits[((size_t)bb * depth + (j - 1)) * V + n] = val;
            const float key = h.sample ? val * h.inv_temp + rng_gumbel(noise.x[e]) : val;
            const float ov = order_val(key);
            if (better(ov, n, bv, bi)) {
              bv = ov;
              bi = n;
              br = val;
            }
          }
        }
      }
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float ov = __shfl_xor(bv, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        const float orw = __shfl_xor(br, o, 64);
        if (better(ov, oi, bv, bi)) {
          bv = ov;
          bi = oi;
          br = orw;
        }
      }
      if (g == 0) {
        best_v[wave][bb] = bv;
        best_i[wave][bb] = bi;
        best_r[wave][bb] = br;
      }
    }
    __syncthreads();
    for (int bb = tid; bb < bs; bb += kLogitWaves * 64) {
      float v = best_v[0][bb], raw = best_r[0][bb];
      int id = best_i[0][bb];
#pragma unroll
      for (int w = 1; w < kLogitWaves; ++w)
        if (better(best_v[w][bb], best_i[w][bb], v, id)) {
          v = best_v[w][bb];
          id = best_i[w][bb];
          raw = best_r[w][bb];
        }
      const size_t o = ((size_t)(j - 1) * bs + bb) * h.GC + blockIdx.x;
      h.pval[o] = v;
      h.pid[o] = id;
      if (h.sample) h.praw[o] = raw;
      if (id != INT_MAX)
        atomicMax(&h.best[((size_t)(j - 1) * bs + bb) * kBestSlots + (blockIdx.x % kBestSlots)], encode_best(v, id));
    }
    return;
  }
  if (h.final_logits) {
#pragma unroll
    for (int q = 0; q < kTPW; ++q)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int bb = mt * 16 + cc;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int n = tiles[q] * 16 + 4 * g + e;
          const float lbe = e == 0 ? lb[q][mt].x : (e == 1 ? lb[q][mt].y : (e == 2 ? lb[q][mt].z : lb[q][mt].w));
          if (bb < bs && n < V) h.final_logits[((size_t)bb * depth + (j - 1)) * V + n] = lbe + acc[q][mt][e];
        }
      }
  }
  unsigned char *sbuf = smem + sizeof(u32x4) * KS * MT * 64 * XF;
  if (beta <= 4) logits_topl<4, kTPW, MT>(h, j, tiles, lb, acc, sbuf);
  else logits_topl<8, kTPW, MT>(h, j, tiles, lb, acc, sbuf);
}

// Merge every workgroup's top-beta list of one (position, batch row) after the
// rollout; one wave per (j, b).
__global__ __launch_bounds__(64) void head_merge_kernel(HeadArgs h) {
  const int j = blockIdx.x, b = blockIdx.y;
  const int bs = h.D.bs, depth = h.D.B - 1, beta = h.beta;
  const int lane = threadIdx.x;
  const size_t base = ((size_t)j * bs + b) * h.GC * beta;
  if (h.sample) {  // branch 1: the largest key wins; its raw logit is the reported value
    float bv = -INFINITY, br = 0.f;
    int bi = INT_MAX;
    for (int c = lane; c < h.GC; c += 64) {
      const float v = order_val(h.pval[base + c]);
      const int id = h.pid[base + c];
      const float raw = h.praw[base + c];
      if (id != INT_MAX && better(v, id, bv, bi)) {
        bv = v;
        bi = id;
        br = raw;
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      const float orw = __shfl_xor(br, o, 64);
      if (better(ov, oi, bv, bi)) {
        bv = ov;
        bi = oi;
        br = orw;
      }
    }
    if (lane == 0) {
      h.topk_ids[(size_t)b * depth + j] = bi;
      h.topk_vals[(size_t)b * depth + j] = br;
    }
    return;
  }
  float mv;
  int mi;
  wave_select_mem(h.pval + base, h.pid + base, h.GC * beta, beta, mv, mi);
  if (lane < beta) {
    h.topk_ids[((size_t)b * depth + j) * beta + lane] = mi;
    h.topk_vals[((size_t)b * depth + j) * beta + lane] = mv;
  }
}

// ---------------------------------------------------------------------------
// Persistent rollout (bf16 weights, r = 256, one or two batch rows, greedy or
// sampled; three or four rows as one launch per pair): one
// launch of at most one workgroup per CU runs all B-1 positions.  Each workgroup keeps its slice
// of W2 resident for the whole rollout (kPersTiles tiles per wave, the last
// one in LDS, the rest in registers: 77.8 MB over 238 workgroups at the Qwen3
// vocabulary) and its rows of [W1[:, d:]; W_hh] in LDS, so W2 leaves HBM once
// per step instead of once per position.
//
// Workgroups exchange data through tagged 64-bit slots in the workspace
// header (zeroed at every step), written with device-scope atomic stores and
// polled with device-scope atomic loads by one wave; a slot is ready when its
// top bits carry the position's tag, so a poll both waits and delivers:
//   u slot [b][k]   (j << 32) | bits of u_j[k], written by the owner of row k
//   key slot [b][g] (j << 50) | value(32) << 18 | (2^18 - 1 - id): workgroup
//                   g's top-1 for position j; the maximum over g is the argmax
//                   under (value desc, id asc)
// The hidden gates W_hh S for the next position go out as plain device-scope
// stores while one wave waits for u; each thread waits for its own stores
// before its workgroup publishes its key, so "all key slots ready" also means
// "all gates stored".
// Waits are bounded: a timeout sets DEV_BARRIER_TIMEOUT and the abort flag,
// and every workgroup leaves; the kernel always ends.  Workgroup 0 writes the
// drafted token and its value of every position (no merge kernel).
// ---------------------------------------------------------------------------
constexpr int kPersWaves = 8, kPersTiles = 5, kPersKS = 8, kPersRegTiles = kPersTiles - 1;
constexpr int kPersMaxBatch = 4;  // batch rows the persistent rollout takes (in launches of two)
constexpr int kKeyIdBits = 18;

DEVI unsigned long long ld_slot(const unsigned long long *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
DEVI void st_slot(unsigned long long *p, unsigned long long v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
DEVI unsigned long long pack_key50(float v, int id) {
  uint32_t u = __float_as_uint(order_val(v));
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((unsigned long long)u << kKeyIdBits) | (unsigned long long)((1 << kKeyIdBits) - 1 - id);
}
DEVI int key50_id(unsigned long long k) { return (1 << kKeyIdBits) - 1 - (int)(k & ((1ull << kKeyIdBits) - 1)); }

// Wave 0 polls `n` slots (kSlotStride words apart) until each carries `tag`
// (top bits from `shift`); lane l holds slots l, l+64, ... in w[].  Returns
// false on timeout (`limit` polls made, none complete) or when another
// workgroup has aborted.
template <int MAXQ>
DEVI bool poll_tagged(const unsigned long long *slots, int n, unsigned long long tag, int shift,
                      unsigned *abort_flag, int32_t *err, unsigned limit, unsigned long long (&w)[MAXQ]) {
  const int lane = threadIdx.x & 63;
  unsigned polls = 0;
  while (true) {
    if (polls++ >= limit) {  // this wait gives up: every workgroup is told to leave
      if (lane == 0) {
        __hip_atomic_store(abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        raise_error(err, DEV_BARRIER_TIMEOUT);
      }
      return false;
    }
#pragma unroll
    for (int q = 0; q < MAXQ; ++q) w[q] = ld_slot(slots + (size_t)min(lane + 64 * q, n - 1) * kSlotStride);
    bool ready = true;
#pragma unroll
    for (int q = 0; q < MAXQ; ++q) ready = ready && (w[q] >> shift) == tag;
    if (__all(ready)) return true;
    if ((polls & 63) == 0 && __hip_atomic_load(abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return false;
  }
}

// BS: the largest batch the instantiation serves (1 or 2; arrays sized by it);
// DBG: the final logits are also written out (h.final_logits);
// SAMPLE: temperature sampling, the selection key is L / T + Gumbel noise
// (Philox stream RNG_DRAFT, as in the launch-pair rollout) and the reported
// value is the chosen token's raw logit
template <int BS, bool DBG, bool SAMPLE>
__global__ __launch_bounds__(kPersWaves * 64) void head_persist_kernel(HeadArgs h, int nr) {
  using WT = bf16_t;
  constexpr int EPL = 8, KSTEP = 32;
  const Dims &D = h.D;
  const int bs = D.bs, ds = D.ds, r = D.r, d = D.d, depth = D.B - 1, V = D.V;
  // the wave index is uniform in a wave: held in a scalar register, so the
  // per-wave offsets below cost no vector registers (the resident W2 tiles
  // take 128 of the 256)
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, cc = lane & 15;
  const int G = gridDim.x, NT = (V + 15) / 16;
  const int nchunk = ds / EPL;  // 16-byte chunks of a row (<= 256 by the config check)
  const int nrows_all = r + 3 * ds;
  extern __shared__ __align__(16) unsigned char smem[];
  u32x4 *rows = (u32x4 *)smem;                          // [nr][nchunk] rows of [W1s; W_hh]
  float *S = (float *)(rows + (size_t)nr * nchunk);     // [bs][ds] the state
  u32x4 *us = (u32x4 *)(S + (size_t)bs * ds);           // [KS][64] u as B fragments
  u32x4 *w2s = us + kPersKS * 64;                       // [waves][KS][64] each wave's last W2 tile
  float4 *lbs = (float4 *)(w2s + kPersWaves * kPersKS * 64);  // [waves][tiles][64] this lane's L_base values
  const int nu = (r + G - 1) / G;                              // u rows per workgroup: k < nu (R < r)
  float *P_s = (float *)(lbs + kPersWaves * kPersTiles * 64);  // [depth][bs][nu] W1[:, :d] H at the u rows
  // each lane's best of its tiles: [wave][row group g][column]
  __shared__ float best_v[kPersWaves][4][16], best_r[SAMPLE ? kPersWaves : 1][4][16];
  __shared__ int best_i[kPersWaves][4][16];
  __shared__ int win_id[SAMPLE ? 64 : 1][BS];  // workgroup 0: each position's drafted token
  __shared__ int ys[kFusedBatch];
  __shared__ int s_ok;
  const WT *w1 = (const WT *)h.w1, *whh = (const WT *)h.w_hh;
  const int tile0 = (blockIdx.x * kPersWaves + wave) * kPersTiles;  // this wave's tiles tile0 + q

  // ---- resident operands, loaded once: W2 tiles, rows, b_ih
  u32x4 wf[kPersRegTiles][kPersKS];
  {
    const u32x4 *w2p = (const u32x4 *)h.w2p;
#pragma unroll
    for (int q = 0; q < kPersTiles; ++q) {
      const int t = min(tile0 + q, NT - 1);
#pragma unroll
      for (int s = 0; s < kPersKS; ++s) {
        const u32x4 v = w2p[((size_t)t * kPersKS + s) * 64 + lane];
        if (q < kPersRegTiles) wf[q < kPersRegTiles ? q : 0][s] = v;
        else w2s[((size_t)wave * kPersKS + s) * 64 + lane] = v;
      }
    }
  }
  for (int e = tid; e < nr * nchunk; e += kPersWaves * 64) {
    const int k = e / nchunk, ch = e % nchunk;
    const int R = min(blockIdx.x + k * G, nrows_all - 1);
    const WT *src = R < r ? w1 + (size_t)R * (d + ds) + d : whh + (size_t)(R - r) * ds;
    rows[e] = *(const u32x4 *)(src + (size_t)ch * EPL);
  }
  for (int e = tid; e < bs * ds; e += kPersWaves * 64) S[e] = 0.f;
  // the u fragments' unused columns (2 bs and up) stay zero for the whole launch
  for (int e = tid; e < kPersKS * 64; e += kPersWaves * 64) us[e] = u32x4{0u, 0u, 0u, 0u};
  for (int e = tid; e < depth * bs * nu; e += kPersWaves * 64) {
    const int k = e % nu, b = (e / nu) % bs, jj = e / (nu * bs);
    const int R = min(blockIdx.x + k * G, r - 1);
    P_s[e] = h.P[((size_t)b * depth + jj) * h.ldp + R];
  }
  __syncthreads();

  // state items: two indices of one batch row each, so that all eight waves
  // share the GRU's transcendental arithmetic (one item per thread at one
  // batch row and d_s = 1024)
  constexpr int GE = 2;
  const int nit = bs * ds / GE;
  for (int j = 1; j <= depth; ++j) {
    // the thread index, opaque to the compiler once per position: addresses
    // derived from it are recomputed here (a few instructions) instead of being
    // hoisted out of the loop, where they would not fit the registers the
    // resident W2 tiles leave and would be reloaded from scratch every position
    int tj = threadIdx.x;
    __asm__ volatile("" : "+v"(tj));
    const int lane_j = tj & 63, cc_j = lane_j & 15;
    // ---- y_{j-1}: anchor, forced token, or the argmax the previous wait delivered
    if (tj < bs) {
      int y;
      if (j == 1) y = clamp_token(h.anchor[tj], V, h.err);
      else if (h.forced) y = clamp_token(h.forced[(size_t)tj * depth + (j - 2)], V, h.err);
      else y = ys[tj];
      ys[tj] = y;
    }
    __syncthreads();
    // L_base of this lane's row and tiles, straight from memory into LDS (no
    // registers held).  Issued after the barrier above, whose wait would
    // otherwise take in its whole latency, and alongside the GRU's loads: the
    // barrier after the GRU finds both complete.
    {
      const int bb = min(cc, bs - 1);
#pragma unroll
      for (int q = 0; q < kPersTiles; ++q) {
        const int t = min(tile0 + q, NT - 1);
        __builtin_amdgcn_global_load_lds(
            (const void *)(h.Lbase + ((size_t)bb * depth + (j - 1)) * h.ldl + t * 16 + 4 * g),
            (void __attribute__((address_space(3))) *)(lbs + ((size_t)wave * kPersTiles + q) * 64), 16, 0, 0);
      }
    }
    // ---- S_{j-1} = GRU(E[y_{j-1}], S_{j-2}) in place
    for (int it = tid; it < nit; it += kPersWaves * 64) {
      const int b = it / (ds / GE), i = (it % (ds / GE)) * GE;
      // W_hh S_{j-2} + b_hh (stored by the previous position's row owners) and the G row, loaded together
      float ghv[3][GE];
      {
        const float *gb = h.ghbuf + (size_t)((j - 1) & 1) * bs * 3 * ds + (size_t)b * 3 * ds + i;
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          const float2 c0 = *(const float2 *)(h.bhh + q * ds + i);  // the gates at j = 1 (S = 0)
          const float v0 = ld_coherent(gb + q * ds), v1 = ld_coherent(gb + q * ds + 1);
          ghv[q][0] = j > 1 ? v0 : c0.x;
          ghv[q][1] = j > 1 ? v1 : c0.y;
        }
      }
      const float *gy = h.gtab + (size_t)ys[b] * 3 * ds + i;
      const float2 g0 = *(const float2 *)gy, g1 = *(const float2 *)(gy + ds), g2 = *(const float2 *)(gy + 2 * ds);
      const float gi[3][GE] = {{g0.x, g0.y}, {g1.x, g1.y}, {g2.x, g2.y}};
      float2 s2 = *(const float2 *)(S + (size_t)b * ds + i);
      const float hold[GE] = {s2.x, s2.y};
      float out[GE];
#pragma unroll
      for (int e = 0; e < GE; ++e) {
        const float rg = sigm(gi[0][e] + ghv[0][e]), zg = sigm(gi[1][e] + ghv[1][e]);
        const float ng = tanhf(fmaf(rg, ghv[2][e], gi[2][e]));
        out[e] = gru_mix(zg, ng, hold[e]);
      }
      s2 = make_float2(out[0], out[1]);
      *(float2 *)(S + (size_t)b * ds + i) = s2;
      if (blockIdx.x == 0 && h.states) *(float2 *)(h.states + ((size_t)b * depth + (j - 1)) * ds + i) = s2;
    }
    __syncthreads();
    // ---- this workgroup's u rows against S_{j-1} into the tagged u slots
    for (int it = wave; it < nu * bs; it += kPersWaves) {
      const int k = it / bs, b = it % bs;
      const int R = blockIdx.x + k * G;
      if (R >= r) continue;  // wave-uniform
      float acc = 0.f;
      for (int c = 0; c < 4; ++c) {
        const int ch = lane + 64 * c;
        if (ch >= nchunk) break;
        float wfl[EPL];
        unpack16<WT>(rows[(size_t)k * nchunk + ch], wfl);
        const float *sb = S + (size_t)b * ds + (size_t)ch * EPL;
        const float4 s0 = *(const float4 *)sb, s1 = *(const float4 *)(sb + 4);
        acc = fmaf(wfl[0], s0.x, acc);
        acc = fmaf(wfl[1], s0.y, acc);
        acc = fmaf(wfl[2], s0.z, acc);
        acc = fmaf(wfl[3], s0.w, acc);
        acc = fmaf(wfl[4], s1.x, acc);
        acc = fmaf(wfl[5], s1.y, acc);
        acc = fmaf(wfl[6], s1.z, acc);
        acc = fmaf(wfl[7], s1.w, acc);
      }
      acc = wave_sum_dpp(acc);
      if (lane == 0) {
        const float x = P_s[((size_t)(j - 1) * bs + b) * nu + k] + acc;
        const float u = x / (1.f + expf(-x));
        st_slot(h.uslot + ((size_t)b * r + R) * kSlotStride, ((unsigned long long)j << 32) | __float_as_uint(u));
      }
    }
    // ---- gates of the next position, W_hh S_{j-1} + b_hh (plain device-scope
    // stores), by waves 1.. while wave 0 waits for u; the stores are waited for
    // before this workgroup publishes its top-1, so "every key slot of position
    // j ready" also means "every gate of position j + 1 stored"
    if (wave > 0 && j < depth) {
      float *gh_out = h.ghbuf + (size_t)(j & 1) * bs * 3 * ds;
      for (int k = wave - 1; k < nr; k += kPersWaves - 1) {
        const int R = blockIdx.x + k * G;
        if (R < r || R >= nrows_all) continue;  // wave-uniform
        float accb[BS];
#pragma unroll
        for (int b = 0; b < BS; ++b) accb[b] = 0.f;
        for (int c = 0; c < 4; ++c) {
          const int ch = lane + 64 * c;
          if (ch >= nchunk) break;
          float wfl[EPL];
          unpack16<WT>(rows[(size_t)k * nchunk + ch], wfl);
#pragma unroll
          for (int b = 0; b < BS; ++b) {
            if (b >= bs) break;
            const float *sb = S + (size_t)b * ds + (size_t)ch * EPL;
            const float4 s0 = *(const float4 *)sb, s1 = *(const float4 *)(sb + 4);
            accb[b] = fmaf(wfl[0], s0.x, accb[b]);
            accb[b] = fmaf(wfl[1], s0.y, accb[b]);
            accb[b] = fmaf(wfl[2], s0.z, accb[b]);
            accb[b] = fmaf(wfl[3], s0.w, accb[b]);
            accb[b] = fmaf(wfl[4], s1.x, accb[b]);
            accb[b] = fmaf(wfl[5], s1.y, accb[b]);
            accb[b] = fmaf(wfl[6], s1.z, accb[b]);
            accb[b] = fmaf(wfl[7], s1.w, accb[b]);
          }
        }
        const float bias = h.bhh[R - r];
#pragma unroll
        for (int b = 0; b < BS; ++b) {
          if (b >= bs) break;
          const float acc = wave_sum_dpp(accb[b]);
          if (lane == 0) st_coherent(gh_out + (size_t)b * 3 * ds + (R - r), acc + bias);
        }
      }
    }
    // ---- wait for u (wave 0 polls all u slots; the slots deliver the values)
    if (wave == 0) {
      unsigned long long w[4 * BS];
      const bool ok = poll_tagged<4 * BS>(h.uslot, bs * r, (unsigned long long)j, 32, h.abort_flag, h.err, h.poll_limit, w);
      // u goes straight into the B fragments of the logits product: element
      // (b, k) sits at k-step k / 32, lane 16 ((k / 8) mod 4) + column, slot k mod 8,
      // where column b holds the bf16 high part of batch row b's u and column
      // bs + b its low part (u - hi).  One product per tile and k-step then
      // carries both; the two columns are summed after the k loop.
      unsigned short *us16 = (unsigned short *)us;
#pragma unroll
      for (int q = 0; q < 4 * BS; ++q) {
        const int e = lane_j + 64 * q;  // slot b * r + k (r = 256)
        if (BS == 1 || e < bs * r) {
          const float u = __uint_as_float((uint32_t)(w[q] & 0xffffffffu));
          const __bf16 hi = (__bf16)u, lo = (__bf16)(u - (float)hi);
          const int b = e >> 8, k = e & 255;
          const int at = ((k >> 5) * 64 + ((k >> 3) & 3) * 16 + b) * 8 + (k & 7);
          us16[at] = __builtin_bit_cast(unsigned short, hi);
          us16[at + bs * 8] = __builtin_bit_cast(unsigned short, lo);
        }
      }
      if (lane == 0) s_ok = ok;
    }
    __syncthreads();
    if (!s_ok) return;
    // ---- logits: u as B fragments against the resident W2
    floatx4 acc[kPersTiles];
#pragma unroll
    for (int q = 0; q < kPersTiles; ++q) acc[q] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < kPersKS; ++s) {
      const bf16x8 xb = __builtin_bit_cast(bf16x8, us[(size_t)s * 64 + lane]);
#pragma unroll
      for (int q = 0; q < kPersRegTiles; ++q)
        acc[q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf[q][s]), xb, acc[q], 0, 0, 0);
      acc[kPersRegTiles] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          __builtin_bit_cast(bf16x8, w2s[((size_t)wave * kPersKS + s) * 64 + lane]), xb, acc[kPersRegTiles], 0, 0, 0);
    }
    // lane (g, cc) holds vocabulary ids 16 (tile0 + q) + 4 g + e: column cc < bs
    // adds the low-part column of lane cc + bs (a row shift within 16 lanes).
    // Each tile's four corrected logits are formed, written (DBG) and folded
    // into the running best before the next tile's, so only one tile's values
    // are live at a time.
    const bool rowok = cc < bs;
    {
      // ids grow along (q, e) within a lane, so a strict comparison keeps the
      // smallest id of equal keys; ids past V occur only in the last workgroup
      float bv = -INFINITY, br = 0.f;
      int bi = (tile0 * 16 + 4 * g) < V ? tile0 * 16 + 4 * g : INT_MAX;
      const bool full = (tile0 + kPersTiles) * 16 <= V;
      float *fl = DBG ? h.final_logits + ((size_t)min(cc, bs - 1) * depth + (j - 1)) * V : nullptr;
#pragma unroll
      for (int q = 0; q < kPersTiles; ++q) {
        const float4 l4 = lbs[((size_t)wave * kPersTiles + q) * 64 + lane];
        const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
        float val[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int a = __float_as_int(acc[q][e]);
          const int lo1 = __builtin_amdgcn_update_dpp(0, a, 0x101, 0xf, 0xf, false);  // lane + 1
          const int lo2 = __builtin_amdgcn_update_dpp(0, a, 0x102, 0xf, 0xf, false);  // lane + 2
          val[e] = lv[e] + (acc[q][e] + __int_as_float(BS == 1 || bs == 1 ? lo1 : lo2));
        }
        if (DBG && rowok) {  // the final logits (output of sampled drafting, debug output otherwise)
          const int n = (tile0 + q) * 16 + 4 * g;
          if ((V & 3) == 0 && n + 4 <= V) {  // rows start 16-byte aligned: four ids per store
            *(float4 *)(fl + n) = make_float4(val[0], val[1], val[2], val[3]);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (n + e < V) fl[n + e] = val[e];
          }
        }
        Philox4 noise = {{0u, 0u, 0u, 0u}};
        if (SAMPLE) noise = rng_block(h.seed_lo, h.seed_hi, RNG_DRAFT, h.row0 + cc, j, (tile0 + q) * 4 + g);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int n = (tile0 + q) * 16 + 4 * g + e;
          const float key = SAMPLE ? val[e] * h.inv_temp + rng_gumbel(noise.x[e]) : val[e];
          const float ov = (full || n < V) ? order_val(key) : -INFINITY;
          const bool take = ov > bv;
          bv = take ? ov : bv;
          bi = take ? n : bi;
          if (SAMPLE) br = take ? val[e] : br;
        }
      }
      // every lane's best goes to LDS as it is (no cross-row exchange here):
      // the merge below takes 32 candidates per batch row
      // (lanes of columns past the batch are written too and never read)
      (&best_v[wave][0][0])[lane_j] = bv;
      (&best_i[wave][0][0])[lane_j] = bi;
      if (SAMPLE) (&best_r[SAMPLE ? wave : 0][0][0])[lane_j] = br;
    }
    __builtin_amdgcn_s_waitcnt(0);  // this thread's gate stores are done
    __syncthreads();                // ... and every thread's
    if (wave == 0) {
      // wave 0 merges the 32 candidates (8 waves x 4 row groups) of batch row b
      // in lanes 32 b ..: rotations within each 16-lane row, then across the
      // two rows of a batch row
      const int bb = lane_j >> 5, c = lane_j & 31;
      const bool have = bb < bs;
      float v = have ? best_v[c >> 2][c & 3][bb] : -INFINITY;
      float raw = (SAMPLE && have) ? best_r[SAMPLE ? c >> 2 : 0][c & 3][bb] : 0.f;
      int id = have ? best_i[c >> 2][c & 3][bb] : INT_MAX;
      auto step = [&](float ov, int oi, float orw) {
        const bool take = better(ov, oi, v, id);
        v = take ? ov : v;
        id = take ? oi : id;
        if (SAMPLE) raw = take ? orw : raw;
      };
      step(row_ror<8>(v), row_ror<8>(id), SAMPLE ? row_ror<8>(raw) : 0.f);
      step(row_ror<4>(v), row_ror<4>(id), SAMPLE ? row_ror<4>(raw) : 0.f);
      step(row_ror<2>(v), row_ror<2>(id), SAMPLE ? row_ror<2>(raw) : 0.f);
      step(row_ror<1>(v), row_ror<1>(id), SAMPLE ? row_ror<1>(raw) : 0.f);
      // the odd rows take the best of the row before them (DPP row_bcast:15:
      // lane 15 of rows 0 and 2 to every lane of rows 1 and 3), so lanes 16 and
      // 48 hold the workgroup's best of batch rows 0 and 1
      step(__int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x142, 0xa, 0xf, false)),
           __builtin_amdgcn_update_dpp(id, id, 0x142, 0xa, 0xf, false),
           SAMPLE ? __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(raw), __float_as_int(raw), 0x142, 0xa, 0xf, false))
                  : 0.f);
      if (c == 16 && have) {
        if (SAMPLE) {  // the raw logit goes out before the key that announces it
          st_coherent(h.praw + ((size_t)(j - 1) * bs + bb) * h.GC + blockIdx.x, raw);
          __builtin_amdgcn_s_waitcnt(0);
        }
        // an empty slice (no valid id) publishes the smallest key
        const unsigned long long key = id == INT_MAX ? 0ull : pack_key50(v, id);
        st_slot(h.kslot + ((size_t)bb * G + blockIdx.x) * kSlotStride, ((unsigned long long)j << 50) | key);
      }
    }
    // ---- wait for every workgroup's top-1: the maximum key is y_j.  Also the
    // guard that no workgroup writes the next position's slots while another
    // still polls this position's, so it runs with forced tokens as well.
    // Workgroup 0 reports (y_j, its value) for every position, the last included.
    if (j < depth || blockIdx.x == 0) {
      if (wave == 0) {
        unsigned long long w[4 * BS];
        const bool ok = poll_tagged<4 * BS>(h.kslot, bs * G, (unsigned long long)j, 50, h.abort_flag, h.err, h.poll_limit, w);
        // lane holds slots lane + 64 q: slot e = b * G + g
        for (int b = 0; b < bs; ++b) {
          unsigned long long best = 0;
#pragma unroll
          for (int q = 0; q < 4 * BS; ++q) {
            const int e = lane + 64 * q;
            const unsigned long long k = w[q] & ((1ull << 50) - 1);
            if (e >= b * G && e < (b + 1) * G && e < bs * G) best = k > best ? k : best;
          }
          best = wave_max_u64(best);
          if (lane == 0) {
            const int id = key50_id(best);
            ys[b] = min(max(id, 0), V - 1);
            if (blockIdx.x == 0) {
              const uint32_t u = (uint32_t)(best >> kKeyIdBits);
              h.topk_ids[(size_t)b * depth + (j - 1)] = id;
              if (SAMPLE) win_id[SAMPLE ? j - 1 : 0][b] = id;
              else h.topk_vals[(size_t)b * depth + (j - 1)] = __uint_as_float((u & 0x80000000u) ? (u ^ 0x80000000u) : ~u);
            }
          }
        }
        if (lane == 0) s_ok = ok;
      }
      __syncthreads();
      if (!s_ok) return;
    }
  }
  if (SAMPLE && blockIdx.x == 0) {  // reported values: the drafted tokens' raw logits, from their owners
    __syncthreads();
    for (int e = tid; e < depth * bs; e += kPersWaves * 64) {
      const int jj = e / bs, b = e % bs;
      const int id = win_id[SAMPLE ? jj : 0][b];
      const int owner = min(max(id, 0), V - 1) / (16 * kPersWaves * kPersTiles);
      h.topk_vals[(size_t)b * depth + jj] = ld_coherent(h.praw + ((size_t)jj * bs + b) * h.GC + owner);
    }
  }
}

// The persistent kernel for one or two batch rows of `h` (D.bs <= 2): checks
// the shapes and the device, and picks the instantiation and its LDS size.
static bool persist_plan(const HeadArgs &h, int n_cu, const void **fn, size_t *lds_out, int *nr_out) {
  const Dims &D = h.D;
  if (!D.bf16 || D.r != kPersKS * 32 || D.bs < 1 || D.bs > 2 || h.beta != 1 || D.ds % 32 || D.ds > 256 * 8 ||
      D.V >= (1 << kKeyIdBits) || D.B > 64 || !h.uslot || !h.kslot || !h.abort_flag || (h.sample && !h.praw))
    return false;
  const int NT = (D.V + 15) / 16;
  const int G = (NT + kPersWaves * kPersTiles - 1) / (kPersWaves * kPersTiles);
  // every workgroup must own a u row (its u slot doubles as its "gates stored" signal),
  // and the polls cover at most 4 * kFusedBatch slots per lane
  if (G != h.GC || G > n_cu || G > D.r || G > 256) return false;  // polls: 4 slots per lane per batch row
  const int nr = (D.r + 3 * D.ds + G - 1) / G;
  const size_t lds = (size_t)nr * (D.ds / 8) * 16 + sizeof(float) * (size_t)D.bs * D.ds +
                     sizeof(u32x4) * kPersKS * 64 + sizeof(u32x4) * kPersWaves * kPersKS * 64 +
                     sizeof(float4) * kPersWaves * kPersTiles * 64 +
                     sizeof(float) * (size_t)(D.B - 1) * D.bs * ((D.r + G - 1) / G);
  if (lds > 160 * 1024) return false;
  const bool dbg = h.final_logits != nullptr, smp = h.sample != 0;
  switch ((D.bs == 1 ? 0 : 4) + (dbg ? 2 : 0) + (smp ? 1 : 0)) {
    case 0: *fn = (const void *)head_persist_kernel<1, false, false>; break;
    case 1: *fn = (const void *)head_persist_kernel<1, false, true>; break;
    case 2: *fn = (const void *)head_persist_kernel<1, true, false>; break;
    case 3: *fn = (const void *)head_persist_kernel<1, true, true>; break;
    case 4: *fn = (const void *)head_persist_kernel<2, false, false>; break;
    case 5: *fn = (const void *)head_persist_kernel<2, false, true>; break;
    case 6: *fn = (const void *)head_persist_kernel<2, true, false>; break;
    default: *fn = (const void *)head_persist_kernel<2, true, true>; break;
  }
  if (hipFuncSetAttribute(*fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  // Every workgroup waits for all others, so the grid must be resident at once:
  // one workgroup per CU at most (its LDS share allows no second), G <= CUs.  An
  // ordinary launch is used (a cooperative one cost ~60 us per step in
  // queue synchronisation); it gets the whole device once the previous kernel
  // on the stream has drained.  Should other work hold CUs, the waits are
  // bounded and end in DEV_BARRIER_TIMEOUT rather than a hang.
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, *fn, kPersWaves * 64, lds) != hipSuccess || per_cu < 1) {
    (void)hipGetLastError();
    return false;
  }
  *lds_out = lds;
  *nr_out = nr;
  return true;
}

// The rollout of `h` with the batch rows [b0, b0 + nb) only: every per-row
// pointer moves to row b0 (the exchange slots too, so each launch has slots
// of its own, zeroed with the step's header), the batch becomes nb.
static HeadArgs rows_of(const HeadArgs &h, int b0, int nb) {
  HeadArgs a = h;
  const int depth = h.D.B - 1;
  a.D.bs = nb;
  a.row0 = h.row0 + b0;
  a.anchor = h.anchor + b0;
  if (h.forced) a.forced = h.forced + (size_t)b0 * depth;
  a.topk_ids = h.topk_ids + (size_t)b0 * depth * h.beta;
  a.topk_vals = h.topk_vals + (size_t)b0 * depth * h.beta;
  if (h.final_logits) a.final_logits = h.final_logits + (size_t)b0 * depth * h.D.V;
  if (h.states) a.states = h.states + (size_t)b0 * depth * h.D.ds;
  a.P = h.P + (size_t)b0 * depth * h.ldp;
  a.Lbase = h.Lbase + (size_t)b0 * depth * h.ldl;
  a.uslot = h.uslot + (size_t)b0 * h.D.r * kSlotStride;
  a.kslot = h.kslot + (size_t)b0 * h.GC * kSlotStride;
  return a;
}

bool launch_head_persistent(const HeadArgs &h, int n_cu, hipStream_t st) {
  const Dims &D = h.D;
  // one or two batch rows per launch (more would spill the per-lane state);
  // three or four rows run as one launch per pair of rows, one after the
  // other (each re-reads W2: 2 x ~140 us against ~480 us for the launch-pair
  // rollout of four rows, measured at the Qwen3-4B shape); larger batches
  // run the launch-pair rollout
  if (D.bs < 1 || D.bs > kPersMaxBatch) return false;
  const int npair = (D.bs + 1) / 2;
  const void *fn[2];
  size_t lds[2];
  int nr[2];
  for (int p = 0; p < npair; ++p) {  // every launch's plan first: all or nothing
    const int nb = std::min(2, D.bs - 2 * p);
    if (!persist_plan(rows_of(h, 2 * p, nb), n_cu, &fn[nb - 1], &lds[nb - 1], &nr[nb - 1])) return false;
  }
  for (int p = 0; p < npair; ++p) {
    const int nb = std::min(2, D.bs - 2 * p);
    HeadArgs a = rows_of(h, 2 * p, nb);
    int nrv = nr[nb - 1];
    void *args[] = {&a, &nrv};
    if (hipLaunchKernel(fn[nb - 1], dim3(a.GC), dim3(kPersWaves * 64), args, lds[nb - 1], st) != hipSuccess) {
      // (a failure after the first pair leaves nothing wrong behind: the
      // launch-pair rollout that follows rewrites every row's outputs)
      (void)hipGetLastError();
      return false;
    }
  }
  return true;
}

static int logit_rows(const Dims &D) {
  const int KS = D.r / (D.bf16 ? 32 : 16);
  const int MT = D.bs <= 16 ? 1 : (D.bs <= 32 ? 2 : 4);
  return kLogitWaves * logit_tpw(KS, MT) * 16;
}
int head_logits_grid(const Dims &D) { return (D.V + logit_rows(D) - 1) / logit_rows(D); }



// One position's state (and u) for batches above kFusedBatch: the two GEMMs
// and their elementwise finishes
static void states_gemm_step(const HeadArgs &h, int j, bool with_u, hipStream_t st) {
  const Dims &D = h.D;
  const int bs = D.bs, ds = D.ds, r = D.r;
  float *gp = h.hpart, *up = h.hpart + (size_t)kHeadMaxSplit * bs * 3 * ds;
  int npg = 0;
  if (j > 1) {
    const GemmPlan pg = plan_gemm(h.whh_NT, h.whh_KS, bs, EPI_STORE, h.n_cu, kHeadMaxSplit);
    GemmArgs a;
    a.P = h.whh_p;
    a.KS = h.whh_KS;
    a.tile0 = 0;
    a.ntiles = h.whh_NT;
    a.N = 3 * ds;
    a.X = h.hbuf + (size_t)((j - 1) & 1) * bs * ds;
    a.ldx = ds;
    a.M = bs;
    a.K = ds;
    a.Y = gp;
    a.ldy = 3 * ds;
    a.ysplit = (size_t)bs * 3 * ds;
    a.ksplit = pg.ksplit;
    launch_gemm(D.bf16, EPI_STORE, a, pg, st);
    npg = pg.ksplit;
  }
  hipLaunchKernelGGL(head_gru_elem_kernel, dim3((ds + 255) / 256, bs), dim3(256), 0, st, h, j, gp, npg,
                     (size_t)bs * 3 * ds);
  if (!with_u) return;
  const GemmPlan pu = plan_gemm(h.w1s_NT, h.w1s_KS, bs, EPI_STORE, h.n_cu, kHeadMaxSplit);
  GemmArgs a;
  a.P = h.w1s_p;
  a.KS = h.w1s_KS;
  a.tile0 = 0;
  a.ntiles = h.w1s_NT;
  a.N = r;
  a.X = h.hbuf + (size_t)(j & 1) * bs * ds;
  a.ldx = ds;
  a.M = bs;
  a.K = ds;
  a.Y = up;
  a.ldy = r;
  a.ysplit = (size_t)bs * r;
  a.ksplit = pu.ksplit;
  launch_gemm(D.bf16, EPI_STORE, a, pu, st);
  hipLaunchKernelGGL(head_u_elem_kernel, dim3((bs * r + 255) / 256), dim3(256), 0, st, h, j, up, pu.ksplit,
                     (size_t)bs * r);
}
static bool states_by_gemm(const HeadArgs &h) {
  return h.D.bs > kFusedBatch && h.whh_p && h.w1s_p && h.hpart && h.n_cu > 0;
}

template <typename WT, int KS, int MT>
static void launch_loop(const HeadArgs &h, hipStream_t st) {
  const Dims &D = h.D;
  const int depth = D.B - 1;
  constexpr int XF = XStage<WT>::XF;
  // the largest request (beta 8) plus the kernel's 6 KB of static LDS fits a CU's 160 KB
  static_assert(sizeof(u32x4) * KS * MT * 64 * XF + topl_lds_bytes(8, MT) + 8192 <= 160 * 1024, "logits LDS");
  const size_t lds = sizeof(u32x4) * KS * MT * 64 * XF + (h.beta == 1 ? 0 : topl_lds_bytes(h.beta <= 4 ? 4 : 8, MT));
  (void)hipFuncSetAttribute((const void *)head_logits_kernel<WT, KS, MT>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  const bool fused = D.bs <= kFusedBatch;
  const size_t slds = sizeof(float) * (size_t)D.bs * D.ds;
  const int gs = min((D.r + 3 * D.ds + 2 * kStateWaves - 1) / (2 * kStateWaves), kStateMaxGrid);
  if (fused)
    (void)hipFuncSetAttribute((const void *)head_state_kernel<WT>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)slds);
  for (int j = 1; j <= depth; ++j) {
    if (fused) hipLaunchKernelGGL(head_state_kernel<WT>, dim3(gs), dim3(kStateWaves * 64), slds, st, h, j);
    else states_gemm_step(h, j, true, st);
    hipLaunchKernelGGL((head_logits_kernel<WT, KS, MT>), dim3(h.GC), dim3(kLogitWaves * 64), lds, st, h, j);
  }
  hipLaunchKernelGGL(head_merge_kernel, dim3(depth, D.bs), dim3(64), 0, st, h);
}

template <typename WT>
static void launch_states_t(const HeadArgs &h, hipStream_t st) {
  const Dims &D = h.D;
  const bool fused = D.bs <= kFusedBatch;
  const size_t slds = sizeof(float) * (size_t)D.bs * D.ds;
  const int rows = (h.skip_u ? 0 : D.r) + 3 * D.ds;
  const int gs = min((rows + 2 * kStateWaves - 1) / (2 * kStateWaves), kStateMaxGrid);
  if (fused)
    (void)hipFuncSetAttribute((const void *)head_state_kernel<WT>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)slds);
  for (int j = 1; j <= D.B - 1; ++j) {
    if (fused) hipLaunchKernelGGL(head_state_kernel<WT>, dim3(gs), dim3(kStateWaves * 64), slds, st, h, j);
    else states_gemm_step(h, j, !h.skip_u, st);
  }
}

hipError_t launch_head_states(const HeadArgs &h, hipStream_t st) {
  if (!h.forced) return hipErrorInvalidValue;
  if (h.D.bs > kFusedBatch && !states_by_gemm(h)) return hipErrorInvalidValue;
  if (h.D.bf16) launch_states_t<bf16_t>(h, st);
  else launch_states_t<float>(h, st);
  return hipGetLastError();
}

template <typename WT, int KS>
static void launch_mt(const HeadArgs &h, hipStream_t st) {
  if (h.D.bs <= 16) launch_loop<WT, KS, 1>(h, st);
  else if (h.D.bs <= 32) launch_loop<WT, KS, 2>(h, st);
  else launch_loop<WT, KS, 4>(h, st);
}

hipError_t launch_head(const HeadArgs &h, hipStream_t st) {
  if (h.D.bs > kFusedBatch && !states_by_gemm(h)) return hipErrorInvalidValue;
  const bool bf = h.D.bf16;
  const int KS = h.D.r / (bf ? 32 : 16);
  if (bf) {
    if (KS == 8) launch_mt<bf16_t, 8>(h, st);
    else return hipErrorInvalidValue;
  } else {
    if (KS == 16) launch_mt<float, 16>(h, st);
    else if (KS == 8) launch_mt<float, 8>(h, st);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dk

namespace dk {
int head_best_slots() { return kBestSlots; }
}  // namespace dk
