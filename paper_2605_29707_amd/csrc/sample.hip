// Speculative-sampling verification of a drafted chain at temperature T
// (Sec. 3.1: the standard speculative verification rule; Fig. 3: draft tokens
// sampled from the final logits).  For batch row b and depth j = 1..B-1 the
// draft token x_j was drawn from q_j = softmax(draft_j / T); the target's
// distribution there is p_j = softmax(target_{j-1} / T) (target row m follows
// node m).  x_j is accepted iff u_j q_j(x_j) < p_j(x_j), i.e. with probability
// min(1, p_j / q_j), u_j the acceptance uniform of (b, j).  At the first
// rejection j the bonus token is a draw from max(0, p_j - q_j); if all B-1 are
// accepted it is a draw from p_B.  Draws use the Philox streams of philox.h
// and the Gumbel-max form.
//
// Three launches: per (row, vocabulary chunk) log-sum-exp partials of every
// target and draft row; per (row, stop depth, chunk) the chunk's best bonus
// candidate for every possible stop depth (so the walk never waits for a
// vocabulary pass); one wave per batch row for the walk.
#include "common.h"
#include "kernels.h"
#include "philox.h"

namespace dk {

constexpr int kVsChunk = 4096;  // vocabulary ids per workgroup
constexpr int kVsThreads = 256;
constexpr int kVsPer = kVsChunk / kVsThreads;  // 16 ids per thread, 4 groups of 4

template <typename LT>
DEVI float ld_logit(const LT *p, size_t i);
template <>
DEVI float ld_logit<float>(const float *p, size_t i) { return p[i]; }
template <>
DEVI float ld_logit<bf16_t>(const bf16_t *p, size_t i) { return to_f32(p[i]); }

// block-wide max / sum over kVsThreads threads
DEVI float block_max(float v, float *red) {
  v = wave_max(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < kVsThreads / 64; ++w) r = fmaxf(r, red[w]);
  __syncthreads();
  return r;
}
DEVI float block_sum(float v, float *red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float r = 0.f;
#pragma unroll
  for (int w = 0; w < kVsThreads / 64; ++w) r += red[w];
  __syncthreads();
  return r;
}

// Row r of the 2B-1 softmax rows of batch row b: r < B the target row r,
// r >= B the draft row of depth r - B + 1.
template <typename LT>
DEVI float row_logit(const LT *target, const float *draft, int b, int r, int B, int V, int v) {
  return r < B ? ld_logit<LT>(target, ((size_t)b * B + r) * V + v)
               : draft[((size_t)b * (B - 1) + (r - B)) * V + v];
}

// (1) max and sum of exp over one vocabulary chunk of one row (NaN as -inf)
template <typename LT>
__global__ __launch_bounds__(kVsThreads) void vs_lse_partial_kernel(const LT *__restrict__ target,
                                                                    const float *__restrict__ draft, int B, int V,
                                                                    float inv_t, int nch, float2 *__restrict__ part) {
  const int c = blockIdx.x, r = blockIdx.y, b = blockIdx.z;
  __shared__ float red[kVsThreads / 64];
  float z[kVsPer];
  float m = -INFINITY;
#pragma unroll
  for (int q = 0; q < kVsPer; ++q) {  // unconditional loads at clamped ids, masked afterwards
    const int v = c * kVsChunk + q * kVsThreads + threadIdx.x;
    const float raw = row_logit<LT>(target, draft, b, r, B, V, min(v, V - 1));
    const float x = v < V ? order_val(raw * inv_t) : -INFINITY;
    z[q] = x;
    m = fmaxf(m, x);
  }
  m = block_max(m, red);
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < kVsPer; ++q) s += z[q] == -INFINITY ? 0.f : expf(z[q] - m);
  s = block_sum(s, red);
  if (threadIdx.x == 0) part[((size_t)b * (2 * B - 1) + r) * nch + c] = make_float2(m, s);
}

// log-sum-exp of one row from its chunk partials (one wave; lanes over chunks)
DEVI float row_lse(const float2 *__restrict__ part, int nch) {
  const int lane = threadIdx.x & 63;
  float m = -INFINITY;
  for (int c = lane; c < nch; c += 64) m = fmaxf(m, part[c].x);
  m = wave_max(m);
  float s = 0.f;
  for (int c = lane; c < nch; c += 64) {
    const float2 t = part[c];
    s += t.x == -INFINITY ? 0.f : t.y * expf(t.x - m);
  }
  s = wave_sum(s);
  return m + logf(s);
}

// (2) best bonus candidate of one chunk for stop depth j = blockIdx.y + 1
template <typename LT>
__global__ __launch_bounds__(kVsThreads) void vs_bonus_partial_kernel(
    const LT *__restrict__ target, const float *__restrict__ draft, int B, int V, float inv_t, int nch,
    const float2 *__restrict__ part, uint32_t seed_lo, uint32_t seed_hi, unsigned long long *__restrict__ bkey) {
  const int c = blockIdx.x, j = blockIdx.y + 1, b = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __shared__ float lse[2];
  __shared__ unsigned long long red[kVsThreads / 64];
  const float2 *prow = part + (size_t)b * (2 * B - 1) * nch;
  if (wave == 0) {
    const float lt = row_lse(prow + (size_t)(j - 1) * nch, nch);
    const float ld = j < B ? row_lse(prow + (size_t)(B + j - 1) * nch, nch) : 0.f;
    if (lane == 0) {
      lse[0] = lt;
      lse[1] = ld;
    }
  }
  __syncthreads();
  const float lt = lse[0], ld = lse[1];
  float bv = -INFINITY;
  int bi = INT_MAX;
  // all loads first, at clamped ids (masked afterwards), so none waits on another
  float tl[kVsPer], dl[kVsPer];
  const int jd = j < B ? j - 1 : B - 2;  // the last depth has no draft row (its q is 0)
#pragma unroll
  for (int q = 0; q < kVsPer; ++q) {
    const int v = min(c * kVsChunk + ((q / 4) * kVsThreads + threadIdx.x) * 4 + (q % 4), V - 1);
    tl[q] = row_logit<LT>(target, draft, b, j - 1, B, V, v);
    dl[q] = draft[((size_t)b * (B - 1) + jd) * V + v];
  }
#pragma unroll
  for (int grp = 0; grp < kVsPer / 4; ++grp) {
    const int v0 = c * kVsChunk + (grp * kVsThreads + threadIdx.x) * 4;  // four consecutive ids
    const Philox4 noise = rng_block(seed_lo, seed_hi, RNG_BONUS, b, j, v0 / 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int v = v0 + e;
      const float p = expf(order_val(tl[grp * 4 + e] * inv_t) - lt);
      const float q = j < B ? expf(order_val(dl[grp * 4 + e] * inv_t) - ld) : 0.f;
      const float w = v < V ? fmaxf(p - q, 0.f) : 0.f;
      if (w > 0.f) {
        const float key = logf(w) + rng_gumbel(noise.x[e]);
        if (better(key, v, bv, bi)) {
          bv = key;
          bi = v;
        }
      }
    }
  }
  wave_best(bv, bi);
  if (lane == 0) red[wave] = bi == INT_MAX ? 0ull : encode_best(bv, bi);
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long k = red[0];
#pragma unroll
    for (int w = 1; w < kVsThreads / 64; ++w) k = red[w] > k ? red[w] : k;
    bkey[((size_t)b * B + (j - 1)) * nch + c] = k;
  }
}

// (3) the acceptance walk, one wave per batch row
template <typename LT>
__global__ __launch_bounds__(64) void vs_walk_kernel(const int32_t *__restrict__ node_token,
                                                    const LT *__restrict__ target, const float *__restrict__ draft,
                                                    int B, int V, float inv_t, int nch, const float2 *__restrict__ part,
                                                    const unsigned long long *__restrict__ bkey, uint32_t seed_lo,
                                                    uint32_t seed_hi, int32_t *__restrict__ accept_len,
                                                    int32_t *__restrict__ accepted_nodes,
                                                    int32_t *__restrict__ out_tokens, int32_t *err) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const float2 *prow = part + (size_t)b * (2 * B - 1) * nch;
  int a = 0, stop = B;
  for (int j = 1; j < B; ++j) {
    const float lt = row_lse(prow + (size_t)(j - 1) * nch, nch);
    const float ld = row_lse(prow + (size_t)(B + j - 1) * nch, nch);
    int x = node_token[(size_t)b * B + j];
    if (x < 0 || x >= V) {
      if (lane == 0) raise_error(err, DEV_BAD_TOKEN);
      stop = j;
      break;
    }
    const float p = expf(order_val(ld_logit<LT>(target, ((size_t)b * B + (j - 1)) * V + x) * inv_t) - lt);
    const float q = expf(order_val(draft[((size_t)b * (B - 1) + (j - 1)) * V + x] * inv_t) - ld);
    const float u = rng_uniform(rng_block(seed_lo, seed_hi, RNG_ACCEPT, b, j, 0).x[0]);
    if (!(u * q < p)) {
      stop = j;
      break;
    }
    if (lane == 0) {
      accepted_nodes[(size_t)b * (B - 1) + a] = j;
      out_tokens[(size_t)b * B + a] = x;
    }
    ++a;
  }
  // bonus: best candidate over the chunks of the stop depth
  unsigned long long k = 0ull;
  for (int c = lane; c < nch; c += 64) {
    const unsigned long long t = bkey[((size_t)b * B + (stop - 1)) * nch + c];
    k = t > k ? t : k;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const unsigned long long t = __shfl_xor(k, o, 64);
    k = t > k ? t : k;
  }
  if (lane == 0) {
    accept_len[b] = a;
    out_tokens[(size_t)b * B + a] = k ? decode_best_id(k, V) : 0;
    for (int i = a; i < B - 1; ++i) accepted_nodes[(size_t)b * (B - 1) + i] = -1;
    for (int i = a + 1; i < B; ++i) out_tokens[(size_t)b * B + i] = -1;
  }
}

int vs_nchunks(int V) { return (V + kVsChunk - 1) / kVsChunk; }

size_t vs_ws_bytes(int bs, int B, int V) {
  const size_t nch = vs_nchunks(V);
  return 256 + (size_t)bs * (2 * B - 1) * nch * sizeof(float2) + (size_t)bs * B * nch * 8 + 256;
}

void launch_verify_sample(int bs, int B, int V, const int32_t *node_token, const void *target, bool bf16,
                          const float *draft, float temperature, uint64_t seed, int32_t *accept_len,
                          int32_t *accepted_nodes, int32_t *out_tokens, void *ws, hipStream_t st) {
  const int nch = vs_nchunks(V);
  int32_t *err = (int32_t *)ws;
  float2 *part = (float2 *)((char *)ws + 256);
  unsigned long long *bkey =
      (unsigned long long *)((char *)part + (((size_t)bs * (2 * B - 1) * nch * sizeof(float2) + 255) & ~(size_t)255));
  const float inv_t = 1.0f / temperature;
  const uint32_t slo = (uint32_t)seed, shi = (uint32_t)(seed >> 32);
  if (bf16) {
    const bf16_t *t = (const bf16_t *)target;
    hipLaunchKernelGGL(vs_lse_partial_kernel<bf16_t>, dim3(nch, 2 * B - 1, bs), dim3(kVsThreads), 0, st, t, draft, B,
                       V, inv_t, nch, part);
    hipLaunchKernelGGL(vs_bonus_partial_kernel<bf16_t>, dim3(nch, B, bs), dim3(kVsThreads), 0, st, t, draft, B, V,
                       inv_t, nch, part, slo, shi, bkey);
    hipLaunchKernelGGL(vs_walk_kernel<bf16_t>, dim3(bs), dim3(64), 0, st, node_token, t, draft, B, V, inv_t, nch,
                       part, bkey, slo, shi, accept_len, accepted_nodes, out_tokens, err);
  } else {
    const float *t = (const float *)target;
    hipLaunchKernelGGL(vs_lse_partial_kernel<float>, dim3(nch, 2 * B - 1, bs), dim3(kVsThreads), 0, st, t, draft, B,
                       V, inv_t, nch, part);
    hipLaunchKernelGGL(vs_bonus_partial_kernel<float>, dim3(nch, B, bs), dim3(kVsThreads), 0, st, t, draft, B, V,
                       inv_t, nch, part, slo, shi, bkey);
    hipLaunchKernelGGL(vs_walk_kernel<float>, dim3(bs), dim3(64), 0, st, node_token, t, draft, B, V, inv_t, nch, part,
                       bkey, slo, shi, accept_len, accepted_nodes, out_tokens, err);
  }
}

// Philox words for explicit counters (tests and callers that need the same draws)
__global__ void philox_words_kernel(const uint32_t *__restrict__ ctr, uint32_t k0, uint32_t k1, uint32_t *__restrict__ out,
                                    int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const Philox4 r = philox4x32_10(ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3], k0, k1);
#pragma unroll
  for (int e = 0; e < 4; ++e) out[4 * i + e] = r.x[e];
}

void launch_philox_words(const uint32_t *ctr, uint64_t key, uint32_t *out, int n, hipStream_t st) {
  if (n <= 0) return;
  hipLaunchKernelGGL(philox_words_kernel, dim3((n + 255) / 256), dim3(256), 0, st, ctr, (uint32_t)key,
                     (uint32_t)(key >> 32), out, n);
}

}  // namespace dk
