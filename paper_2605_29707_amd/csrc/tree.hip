// Draft-tree construction and greedy acceptance (Sec. 3.1: the longest valid
// prefix plus the target's bonus token).  Integer / compare work only; every
// argmax uses the total order (value desc, id asc) with NaN as -inf, so the
// results are exact and independent of reduction order.
#include "common.h"
#include "kernels.h"

namespace dk {

// One workgroup per batch row.
__global__ __launch_bounds__(256) void build_tree_kernel(int depth, int beta,
                                                         const int32_t *__restrict__ topk,
                                                         const int32_t *__restrict__ anchor,
                                                         const int32_t *__restrict__ ctx_lens,
                                                         int32_t *tok, int32_t *par, int32_t *dep,
                                                         int32_t *pos, uint8_t *mask) {
  const int b = blockIdx.x;
  const int nn = 1 + depth * beta;
  const int n = ctx_lens[b];
  for (int i = threadIdx.x; i < nn; i += blockDim.x) {
    int t, p, d;
    if (i == 0) {
      t = anchor[b];
      p = -1;
      d = 0;
    } else {
      d = (i - 1) / beta + 1;
      const int rho = (i - 1) % beta;
      t = topk[((size_t)b * depth + (d - 1)) * beta + rho];
      p = d == 1 ? 0 : 1 + (d - 2) * beta;
    }
    tok[(size_t)b * nn + i] = t;
    par[(size_t)b * nn + i] = p;
    dep[(size_t)b * nn + i] = d;
    pos[(size_t)b * nn + i] = n + d;
  }
  if (!mask) return;
  for (int e = threadIdx.x; e < nn * nn; e += blockDim.x) {
    const int i = e / nn, k = e % nn;
    // ancestors of i: i itself, then the spine nodes of depths dep(i)-1 .. 1, then the root
    uint8_t m = 0;
    if (k == i || k == 0) {
      m = 1;
    } else if (i > 0) {
      const int di = (i - 1) / beta + 1;
      const int dk = (k - 1) / beta + 1;
      const bool spine = ((k - 1) % beta) == 0;
      m = (spine && dk < di) ? 1 : 0;
    }
    mask[((size_t)b * nn + i) * nn + k] = m;
  }
}

void launch_build_tree(int bs, int depth, int beta, const int32_t *topk, const int32_t *anchor,
                       const int32_t *ctx_lens, int32_t *tok, int32_t *par, int32_t *dep,
                       int32_t *pos, uint8_t *mask, hipStream_t st) {
  hipLaunchKernelGGL(build_tree_kernel, dim3(bs), dim3(256), 0, st, depth, beta, topk, anchor, ctx_lens,
                     tok, par, dep, pos, mask);
}

// ---------------------------------------------------------------------------
// acceptance: two launches.  (1) the argmax of the rows of nodes that have
// children (the walk can only continue from those), split into vocabulary
// chunks; (2) one workgroup per batch row checks the tree and walks it from
// the root.  When the walk stops on a node without children (a leaf of a
// tree, or the end of a fully accepted chain) the bonus token is that row's
// argmax, which the walk's workgroup scans itself: one row, and only then.
// workspace: [err:int32][pad to 256 B][partials: (float,int) bs*nn*nchunk]
// ---------------------------------------------------------------------------
constexpr int ACH = 4096;  // vocabulary elements per argmax chunk

static size_t acc_part_off() { return 256; }
size_t accept_ws_bytes(int bs, int nn, int V) {
  const int nch = (V + ACH - 1) / ACH;
  return acc_part_off() + (size_t)bs * nn * nch * 8;
}

template <typename LT>
DEVI float ld_logit(const LT *p);
template <>
DEVI float ld_logit<float>(const float *p) {
  return *p;
}
template <>
DEVI float ld_logit<bf16_t>(const bf16_t *p) {
  return to_f32(*p);
}

// 16 bytes of logits as values: 8 bf16 or 4 fp32
template <typename LT>
struct LVec;
template <>
struct LVec<bf16_t> {
  static constexpr int N = 8;
  DEVI static float get(const u32x4 &x, int e) {
    const uint32_t w = x[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
  }
};
template <>
struct LVec<float> {
  static constexpr int N = 4;
  DEVI static float get(const u32x4 &x, int e) { return __uint_as_float(x[e]); }
};

// Fold the values of one 16-byte load (ids id0 .. id0 + N - 1, those below v1)
// into a running best; ids grow within a thread, so a strict comparison keeps
// the smallest id of equal values.
template <typename LT>
DEVI void fold_vec(const u32x4 &x, int id0, int v1, float &bv, int &bi) {
#pragma unroll
  for (int e = 0; e < LVec<LT>::N; ++e) {
    const int v = id0 + e;
    const float o = order_val(LVec<LT>::get(x, e));
    if (v < v1 && (o > bv || bi == INT_MAX)) {
      bv = o;
      bi = v;
    }
  }
}

// (bv, bi) of the 256-thread workgroup: every thread gets the best
DEVI void block_best(float &bv, int &bi, float (&sv)[4], int (&si)[4]) {
  wave_best(bv, bi);
  __syncthreads();  // the arrays may hold the previous reduction
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = bv;
    si[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  bv = sv[0];
  bi = si[0];
  for (int w = 1; w < 4; ++w)
    if (better(sv[w], si[w], bv, bi)) {
      bv = sv[w];
      bi = si[w];
    }
}

// Partial argmax of rows m0 .. m0 + kArgRows - 1 of batch row b over one
// vocabulary chunk (one row per workgroup for small grids, several when there
// are many node rows), for the rows of nodes that have children (the walk scans
// another row itself if it ends there).  Rows are 16-byte aligned when V is a
// multiple of 8 (bf16) or 4 (fp32); then every value comes from 16-byte loads,
// all of the workgroup's rows in flight together; otherwise one value per
// load.  The first workgroup also clears the error word (only the walk, a
// later launch, raises errors).
template <typename LT, int kArgRows>
__global__ __launch_bounds__(256) void argmax_partial_kernel(int nn, int V, const LT *__restrict__ logits,
                                                             const int32_t *__restrict__ par, float *part_v,
                                                             int32_t *part_i, int32_t *err) {
  constexpr int EV = LVec<LT>::N, VPT = ACH / EV / 256;  // 16-byte loads per thread and row
  const int ch = blockIdx.x, m0 = blockIdx.y * kArgRows, b = blockIdx.z;
  const int nch = gridDim.x, tid = threadIdx.x;
  if ((ch | blockIdx.y | b) == 0 && tid == 0) *err = 0;
  __shared__ int s_has[kArgRows];
  __shared__ float sv[4];
  __shared__ int si[4];
  if (tid < kArgRows) s_has[tid] = 0;
  __syncthreads();
  // children come after their parent
  for (int c = m0 + 1 + tid; c < nn; c += blockDim.x) {
    const int p = par[(size_t)b * nn + c];
    if (p >= m0 && p < m0 + kArgRows && p < c) s_has[p - m0] = 1;
  }
  __syncthreads();
  const int v0 = ch * ACH, v1 = min(V, v0 + ACH);
  if (V % EV == 0) {
    u32x4 x[kArgRows][VPT];
#pragma unroll
    for (int r = 0; r < kArgRows; ++r) {
      if (!s_has[r] || m0 + r >= nn) continue;  // uniform: a leaf's row is not read
      const LT *row = logits + ((size_t)b * nn + m0 + r) * V;
#pragma unroll
      for (int q = 0; q < VPT; ++q) {  // clamped within the row: every lane's load valid
        const int id0 = min(v0 + (q * 256 + tid) * EV, V - EV);
        x[r][q] = *(const u32x4 *)(row + id0);
      }
    }
#pragma unroll
    for (int r = 0; r < kArgRows; ++r) {
      if (!s_has[r] || m0 + r >= nn) continue;  // uniform over the workgroup
      float bv = -INFINITY;
      int bi = INT_MAX;
#pragma unroll
      for (int q = 0; q < VPT; ++q) fold_vec<LT>(x[r][q], v0 + (q * 256 + tid) * EV, v1, bv, bi);
      block_best(bv, bi, sv, si);
      if (tid == 0) {
        const size_t o = ((size_t)b * nn + m0 + r) * nch + ch;
        part_v[o] = bv;
        part_i[o] = bi;
      }
    }
    return;
  }
  for (int r = 0; r < kArgRows; ++r) {
    if (!s_has[r] || m0 + r >= nn) continue;  // uniform over the workgroup
    const LT *row = logits + ((size_t)b * nn + m0 + r) * V;
    constexpr int PER = ACH / 256;
    float x[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) x[q] = ld_logit<LT>(row + min(v0 + tid + q * 256, v1 - 1));
    float bv = -INFINITY;
    int bi = INT_MAX;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int v = v0 + tid + q * 256;  // increasing in q: a strict > keeps the smallest id
      const float o = v < v1 ? order_val(x[q]) : -INFINITY;
      if (v < v1 && (o > bv || bi == INT_MAX)) {
        bv = o;
        bi = v;
      }
    }
    block_best(bv, bi, sv, si);
    if (tid == 0) {
      const size_t o = ((size_t)b * nn + m0 + r) * nch + ch;
      part_v[o] = bv;
      part_i[o] = bi;
    }
  }
}

// The walk of one batch row.  Every table the walk needs is formed in
// parallel first, with all of its memory reads in flight together: which nodes
// have children (the rows argmax_partial_kernel took), each such node's argmax
// R from its chunk partials (a wave per node, four nodes per pass), and the
// first child of each node whose token is that R.  The walk from the root is
// then a chase through LDS.  Only if it stops on a node without children (a
// leaf of a tree, or the end of a fully accepted chain) is that row's argmax
// needed, which the workgroup scans itself.
constexpr int kWalkMaxNodes = 1024;

template <typename LT>
__global__ __launch_bounds__(256) void accept_walk_kernel(int nn, int V, int B, const int32_t *__restrict__ tok,
                                                          const int32_t *__restrict__ par,
                                                          const float *__restrict__ part_v,
                                                          const int32_t *__restrict__ part_i,
                                                          const LT *__restrict__ logits,
                                                          int32_t *acc_len, int32_t *acc_nodes,
                                                          int32_t *out_tok, int32_t *err) {
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nch = (V + ACH - 1) / ACH;
  __shared__ float sv[4];
  __shared__ int si[4];
  __shared__ int s_R[kWalkMaxNodes], s_next[kWalkMaxNodes];
  __shared__ unsigned char s_kid[kWalkMaxNodes];
  const int32_t *pr = par + (size_t)b * nn, *tk = tok + (size_t)b * nn;
  for (int c = tid; c < nn; c += blockDim.x) {
    s_kid[c] = 0;
    s_next[c] = INT_MAX;
  }
  __syncthreads();
  // the tree: node 0 is the root, every other node's parent comes before it
  for (int c = tid; c < nn; c += blockDim.x) {
    const int p = pr[c];
    if (!((c == 0) ? (p == -1) : (p >= 0 && p < c))) raise_error(err, DEV_BAD_TREE);
    if (c > 0 && p >= 0 && p < c) s_kid[p] = 1;
  }
  __syncthreads();
  // R of every node with children: wave w takes nodes w + 4 q (+ 16 per pass),
  // lanes over the vocabulary chunks
  for (int c0 = wave; c0 < nn; c0 += 16) {
    float bv[4];
    int bi[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      bv[q] = -INFINITY;
      bi[q] = INT_MAX;
    }
    for (int k0 = 0; k0 < nch; k0 += 64) {
      float lv[4];
      int li[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {  // clamped: every load valid, all in flight together
        const int c = min(c0 + 4 * q, nn - 1), k = min(k0 + lane, nch - 1);
        const size_t o = ((size_t)b * nn + c) * nch + k;
        lv[q] = part_v[o];
        li[q] = part_i[o];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = c0 + 4 * q;
        if (c < nn && s_kid[c] && k0 + lane < nch && better(lv[q], li[q], bv[q], bi[q])) {
          bv[q] = lv[q];
          bi[q] = li[q];
        }
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      wave_best(bv[q], bi[q]);
      const int c = c0 + 4 * q;
      if (lane == 0 && c < nn) s_R[c] = bi[q];
    }
  }
  __syncthreads();
  // each node's child carrying R (children have distinct tokens; the first one)
  for (int c = 1 + tid; c < nn; c += blockDim.x) {
    const int p = pr[c];
    if (p >= 0 && p < c && tk[c] == s_R[p]) atomicMin(&s_next[p], c);
  }
  __syncthreads();
  // the walk (every thread follows it)
  int cur = 0, a = 0, R = 0;
  bool leaf = false;
  while (true) {
    if (!s_kid[cur]) {
      leaf = true;
      break;
    }
    R = s_R[cur];
    if (a >= B - 1) break;  // walk bound
    const int nx = s_next[cur];
    if (nx == INT_MAX || nx <= cur) break;
    if (tid == 0) {
      acc_nodes[(size_t)b * (B - 1) + a] = nx;
      out_tok[(size_t)b * B + a] = R;
    }
    ++a;
    cur = nx;
  }
  if (leaf) {  // the bonus token: the argmax of this row, scanned here
    float bv = -INFINITY;
    int bi = INT_MAX;
    // ids visited in increasing order per thread: a strict > keeps the smallest id
    const LT *row = logits + ((size_t)b * nn + cur) * V;
    constexpr int EV = LVec<LT>::N, U = 16;
    if (V % EV == 0) {  // 16-byte rows: U loads of EV values per thread in flight
      const int nv = V / EV;
      for (int g0 = 0; g0 < nv; g0 += 256 * U) {
        u32x4 x[U];
#pragma unroll
        for (int q = 0; q < U; ++q) x[q] = *(const u32x4 *)(row + (size_t)min(g0 + q * 256 + tid, nv - 1) * EV);
#pragma unroll
        for (int q = 0; q < U; ++q) {
          const int gi = g0 + q * 256 + tid;
          fold_vec<LT>(x[q], gi * EV, gi < nv ? V : 0, bv, bi);
        }
      }
    } else {
      for (int v0 = tid; v0 < V; v0 += 256 * U) {
        float x[U];
#pragma unroll
        for (int q = 0; q < U; ++q) x[q] = ld_logit<LT>(row + min(v0 + q * 256, V - 1));
#pragma unroll
        for (int q = 0; q < U; ++q) {
          const int v = v0 + q * 256;
          const float ov = order_val(x[q]);
          if (v < V && (ov > bv || bi == INT_MAX)) {
            bv = ov;
            bi = v;
          }
        }
      }
    }
    block_best(bv, bi, sv, si);
    R = bi;
  }
  if (tid == 0) {
    acc_len[b] = a;
    out_tok[(size_t)b * B + a] = R;
  }
  for (int q = a + 1 + tid; q < B; q += blockDim.x) out_tok[(size_t)b * B + q] = -1;
  for (int q = a + tid; q < B - 1; q += blockDim.x) acc_nodes[(size_t)b * (B - 1) + q] = -1;
}

size_t accept_part_entries(int bs, int nn, int V) { return (size_t)bs * nn * ((V + ACH - 1) / ACH); }

void launch_accept(int bs, int nn, int V, int B, const int32_t *tok, const int32_t *par,
                   const void *logits, bool bf16, int32_t *acc_len, int32_t *acc_nodes,
                   int32_t *out_tok, void *ws, hipStream_t st) {
  unsigned char *w = (unsigned char *)ws;
  float *pv = (float *)(w + acc_part_off());
  launch_accept_parts(bs, nn, V, B, tok, par, logits, bf16, acc_len, acc_nodes, out_tok, pv,
                      (int32_t *)(pv + accept_part_entries(bs, nn, V)), (int32_t *)w, st);
}

void launch_accept_parts(int bs, int nn, int V, int B, const int32_t *tok, const int32_t *par,
                         const void *logits, bool bf16, int32_t *acc_len, int32_t *acc_nodes,
                         int32_t *out_tok, float *pv, int32_t *pi, int32_t *err, hipStream_t st) {
  const int nch = (V + ACH - 1) / ACH;
  // a workgroup per row while the grid is small; eight rows per workgroup for
  // many rows (most of them leaves of a tree), which keeps the grid of
  // workgroups that only find no children from dominating
  const bool many = (long)nch * nn * bs > 4096;
  const int rpw = many ? 8 : 1;
  dim3 grid(nch, (nn + rpw - 1) / rpw, bs);
  if (bf16) {
    if (many)
      hipLaunchKernelGGL((argmax_partial_kernel<bf16_t, 8>), grid, dim3(256), 0, st, nn, V, (const bf16_t *)logits,
                         par, pv, pi, err);
    else
      hipLaunchKernelGGL((argmax_partial_kernel<bf16_t, 1>), grid, dim3(256), 0, st, nn, V, (const bf16_t *)logits,
                         par, pv, pi, err);
    hipLaunchKernelGGL(accept_walk_kernel<bf16_t>, dim3(bs), dim3(256), 0, st, nn, V, B, tok, par, pv, pi,
                       (const bf16_t *)logits, acc_len, acc_nodes, out_tok, err);
  } else {
    if (many)
      hipLaunchKernelGGL((argmax_partial_kernel<float, 8>), grid, dim3(256), 0, st, nn, V, (const float *)logits, par,
                         pv, pi, err);
    else
      hipLaunchKernelGGL((argmax_partial_kernel<float, 1>), grid, dim3(256), 0, st, nn, V, (const float *)logits, par,
                         pv, pi, err);
    hipLaunchKernelGGL(accept_walk_kernel<float>, dim3(bs), dim3(256), 0, st, nn, V, B, tok, par, pv, pi,
                       (const float *)logits, acc_len, acc_nodes, out_tok, err);
  }
}

}  // namespace dk
