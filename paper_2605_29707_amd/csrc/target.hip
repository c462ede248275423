// Target-side pieces of a speculative cycle (Sec. 3.1): the tree-verify
// forward's input preparation and output copy, and the cache commit after
// acceptance.  The forward itself runs the backbone kernels with per-row
// tokens and positions, a tree mask in the attention, and every node's K/V
// stored into the cache at n + i (node i) by the RoPE kernel.
//
//   prep    the caller's [bs][N+1] node tokens / positions and [bs][N+1][N+1]
//           tree mask, padded to Bp rows per batch row (the attention's
//           supported block sizes): a padding row holds token 0 at node 0's
//           position and sees only itself; real rows never see padding.  The
//           diagonal is always visible (a node attends to itself).
//   out     the LM-head rows of the real nodes into the caller's logits, fp32
//           or bf16 (round to nearest even).
//   commit  per (layer, batch row): the accepted path's rows n + node(d) move
//           to n + d, d = 1..a (a round's sources are all read before its
//           writes); ctx_len becomes n + 1 + a.
#include "common.h"
#include "kernels.h"

namespace dk {

__global__ __launch_bounds__(256) void target_prep_kernel(const int32_t *__restrict__ tok,
                                                          const int32_t *__restrict__ pos,
                                                          const uint8_t *__restrict__ mask, int nn, int Bp,
                                                          int V, int32_t *__restrict__ tok_p,
                                                          int32_t *__restrict__ pos_p, uint8_t *__restrict__ mask_p,
                                                          int32_t *err) {
  const int b = blockIdx.x;
  for (int i = threadIdx.x; i < Bp; i += blockDim.x) {
    int t = 0, p = pos[(size_t)b * nn];
    if (i < nn) {
      t = tok[(size_t)b * nn + i];
      p = pos[(size_t)b * nn + i];
      if (t < 0 || t >= V) {
        raise_error(err, DEV_BAD_TOKEN);
        t = t < 0 ? 0 : V - 1;
      }
    }
    tok_p[(size_t)b * Bp + i] = t;
    pos_p[(size_t)b * Bp + i] = p;
  }
  for (int e = threadIdx.x; e < Bp * Bp; e += blockDim.x) {
    const int i = e / Bp, k = e % Bp;
    uint8_t v = 0;
    if (i == k) v = 1;
    else if (i < nn && k < nn) v = mask[((size_t)b * nn + i) * nn + k] ? 1 : 0;
    mask_p[(size_t)b * Bp * Bp + e] = v;
  }
}

template <typename OT>
__global__ __launch_bounds__(256) void target_out_kernel(const float *__restrict__ lg, int ldl, int nn, int Bp, int V,
                                                         OT *__restrict__ out) {
  const int r = blockIdx.y;  // output row b * nn + i
  const int b = r / nn, i = r % nn;
  const float *src = lg + ((size_t)b * Bp + i) * ldl;
  OT *dst = out + (size_t)r * V;
  const int v0 = (blockIdx.x * blockDim.x + threadIdx.x) * 4;  // four values per thread, loads issued together
  float x[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] = src[min(v0 + e, V - 1)];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (v0 + e < V) store_as(dst + v0 + e, x[e]);
}

constexpr int kCommitThreads = 256, kCommitPer = 16;  // 16-byte items per thread per round

// Rows move in rounds of as many rows as fit kCommitPer items per thread: all
// of a round's sources are read (unconditionally, clamped) before any
// destination is written.  Moves of later rounds are safe after earlier ones:
// the node at depth d has id >= d (breadth-first order), so every source
// n + node(d') of a later depth lies above every earlier destination n + d.
__global__ __launch_bounds__(kCommitThreads) void target_commit_kernel(
    const int32_t *__restrict__ ctx_lens, const int32_t *__restrict__ accept_len,
    const int32_t *__restrict__ accepted_nodes, int max_depth, int nn, uint4 *__restrict__ ck, uint4 *__restrict__ cv,
    int max_ctx, int bs, int row16, int32_t *__restrict__ new_lens, int32_t *err) {
  const int l = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int n = ctx_lens[b];
  const int a = accept_len[b];
  __shared__ int node[64];
  __shared__ int bad;
  if (tid == 0) bad = (n < 0 || a < 0 || a > max_depth || n + nn > max_ctx) ? 1 : 0;
  __syncthreads();
  if (bad) {
    if (tid == 0 && l == 0) {
      raise_error(err, DEV_BAD_CTX_LEN);
      new_lens[b] = n;
    }
    return;
  }
  for (int d = tid; d <= a; d += kCommitThreads) {
    const int x = d == 0 ? 0 : accepted_nodes[(size_t)b * max_depth + d - 1];
    if (x < d || x >= nn) bad = 2;  // breadth-first ids: the node at depth d is at least d
    node[d] = x < 0 ? 0 : (x >= nn ? nn - 1 : x);
  }
  __syncthreads();
  if (bad) {
    if (tid == 0 && l == 0) {
      raise_error(err, DEV_BAD_TREE);
      new_lens[b] = n;
    }
    return;
  }
  if (tid == 0 && l == 0) new_lens[b] = n + 1 + a;
  const size_t base = ((size_t)l * bs + b) * max_ctx * row16;
  const int rows_per_round = max(1, kCommitThreads * kCommitPer / (2 * row16));
  for (int d0 = 1; d0 <= a; d0 += rows_per_round) {
    const int nr = min(rows_per_round, a + 1 - d0);
    const int items = nr * row16 * 2;  // K rows, then V rows
    uint4 v[kCommitPer];
#pragma unroll
    for (int q = 0; q < kCommitPer; ++q) {
      const int it = min(tid + q * kCommitThreads, items - 1);
      const int isv = it / (nr * row16), rem = it % (nr * row16);
      const int d = d0 + rem / row16, c = rem % row16;
      const uint4 *src = (isv ? cv : ck) + base + (size_t)(n + node[d]) * row16 + c;
      v[q] = *src;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kCommitPer; ++q) {
      const int it = tid + q * kCommitThreads;
      if (it >= items) continue;
      const int isv = it / (nr * row16), rem = it % (nr * row16);
      const int d = d0 + rem / row16, c = rem % row16;
      if (node[d] != d) *((isv ? cv : ck) + base + (size_t)(n + d) * row16 + c) = v[q];
    }
    __syncthreads();
  }
}

void launch_target_prep(int bs, int nn, int Bp, int V, const int32_t *tok, const int32_t *pos, const uint8_t *mask,
                        int32_t *tok_p, int32_t *pos_p, uint8_t *mask_p, int32_t *err, hipStream_t st) {
  hipLaunchKernelGGL(target_prep_kernel, dim3(bs), dim3(256), 0, st, tok, pos, mask, nn, Bp, V, tok_p, pos_p, mask_p,
                     err);
}

void launch_target_out(int bs, int nn, int Bp, int V, const float *lg, int ldl, void *out, bool out_bf16,
                       hipStream_t st) {
  const dim3 grid((V + 1023) / 1024, bs * nn);
  if (out_bf16)
    hipLaunchKernelGGL(target_out_kernel<bf16_t>, grid, dim3(256), 0, st, lg, ldl, nn, Bp, V, (bf16_t *)out);
  else
    hipLaunchKernelGGL(target_out_kernel<float>, grid, dim3(256), 0, st, lg, ldl, nn, Bp, V, (float *)out);
}

void launch_target_commit(bool bf16, int L, int bs, int nn, int max_depth, const int32_t *ctx_lens,
                          const int32_t *accept_len, const int32_t *accepted_nodes, void *ck, void *cv, int max_ctx,
                          int width, int32_t *new_lens, int32_t *err, hipStream_t st) {
  const int row16 = width * (bf16 ? 2 : 4) / 16;  // a cache row (n_kv * d_h values) in 16-byte items
  hipLaunchKernelGGL(target_commit_kernel, dim3(L, bs), dim3(kCommitThreads), 0, st, ctx_lens, accept_len,
                     accepted_nodes, max_depth, nn, (uint4 *)ck, (uint4 *)cv, max_ctx, bs, row16, new_lens, err);
}

}  // namespace dk
