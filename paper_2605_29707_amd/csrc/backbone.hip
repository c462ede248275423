// Draft-backbone kernels other than the projections (Sec. 4.1.1): block
// embedding, RMSNorm, per-head q/k RMSNorm + rotate-half RoPE, projection of
// context hidden states into the KV cache, and split-KV block attention.
// All arithmetic is fp32; RoPE angles are formed in fp64 so that positions in
// the thousands keep full fp32 accuracy in the rotated values.
#include "common.h"
#include "kernels.h"

namespace dk {

template <typename WT>
__global__ __launch_bounds__(256) void embed_block_kernel(const WT *__restrict__ embed,
                                                          const int32_t *__restrict__ anchor,
                                                          float *__restrict__ X, int B, int d, int V,
                                                          int mask_id, int32_t *err) {
  const int row = blockIdx.x;
  const int b = row / B, j = row % B;
  int tok = mask_id;
  if (j == 0) {
    tok = anchor[b];
    if (tok < 0 || tok >= V) {
      if (threadIdx.x == 0) raise_error(err, DEV_BAD_TOKEN);
      tok = tok < 0 ? 0 : V - 1;
    }
  }
  const WT *src = embed + (size_t)tok * d;
  float *dst = X + (size_t)row * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) dst[c] = to_f32(src[c]);
}

template <typename WT>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float *__restrict__ x, int ldx,
                                                      const WT *__restrict__ gain, float *__restrict__ y,
                                                      int ldy, int width, float eps, int skip_anchor,
                                                      int depth) {
  const int i = blockIdx.x;
  const int in_row = skip_anchor ? i + i / depth + 1 : i;
  const float *xr = x + (size_t)in_row * ldx;
  float ss = 0.f;
  for (int c = threadIdx.x; c < width; c += blockDim.x) ss = fmaf(xr[c], xr[c], ss);
  ss = wave_sum(ss);
  __shared__ float red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)width + eps);
  float *yr = y + (size_t)i * ldy;
  for (int c = threadIdx.x; c < width; c += blockDim.x) yr[c] = xr[c] * inv * to_f32(gain[c]);
}

// One wave per (row, head).  Lane l holds elements l and l+64 (dh = 128) or
// l (dh = 64); RoPE pairs element i with i + dh/2.
template <typename WT>
DEVI void norm_rope_head(float (&v)[2], int dh, const WT *__restrict__ gain, float eps, int pos,
                         float theta, bool rotate, int lane) {
  const int per = dh / 64;
  float ss = 0.f;
  for (int q = 0; q < per; ++q) ss = fmaf(v[q], v[q], ss);
  ss = wave_sum(ss);
  const float inv = 1.0f / sqrtf(ss / (float)dh + eps);
  for (int q = 0; q < per; ++q) v[q] = v[q] * inv * to_f32(gain[lane + 64 * q]);
  if (!rotate) return;
  if (dh == 128) {
    const double w = pow((double)theta, -2.0 * (double)lane / 128.0);
    double sd, cd;
    sincos((double)pos * w, &sd, &cd);
    const float c = (float)cd, s = (float)sd;
    const float x1 = v[0], x2 = v[1];
    v[0] = x1 * c - x2 * s;
    v[1] = x2 * c + x1 * s;
  } else {  // dh == 64: partner lives 32 lanes away
    const int i = lane & 31;
    const double w = pow((double)theta, -2.0 * (double)i / 64.0);
    double sd, cd;
    sincos((double)pos * w, &sd, &cd);
    const float c = (float)cd, s = (float)sd;
    const float p = __shfl_xor(v[0], 32, 64);
    v[0] = (lane < 32) ? (v[0] * c - p * s) : (v[0] * c + p * s);
  }
}

template <typename WT>
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(const float *__restrict__ qkv,
                                                           const WT *__restrict__ qn,
                                                           const WT *__restrict__ kn,
                                                           const int32_t *__restrict__ ctx_lens,
                                                           int max_ctx, float *__restrict__ Q,
                                                           float *__restrict__ Kb,
                                                           float *__restrict__ Vb, int M, int B, int nq,
                                                           int nkv, int dh, float eps, float theta) {
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nh = nq + 2 * nkv;
  if (item >= M * nh) return;
  const int m = item / nh, hh = item % nh;
  const int b = m / B, j = m % B;
  int n = ctx_lens[b];
  n = n < 0 ? 0 : (n > max_ctx ? max_ctx : n);
  const int pos = n + j;
  const float *src = qkv + (size_t)m * nh * dh + (size_t)hh * dh;
  float v[2] = {0.f, 0.f};
  const int per = dh / 64;
  for (int q = 0; q < per; ++q) v[q] = src[lane + 64 * q];
  float *dst;
  if (hh < nq) {
    norm_rope_head<WT>(v, dh, qn, eps, pos, theta, true, lane);
    dst = Q + ((size_t)m * nq + hh) * dh;
  } else if (hh < nq + nkv) {
    norm_rope_head<WT>(v, dh, kn, eps, pos, theta, true, lane);
    dst = Kb + ((size_t)m * nkv + (hh - nq)) * dh;
  } else {
    dst = Vb + ((size_t)m * nkv + (hh - nq - nkv)) * dh;
  }
  for (int q = 0; q < per; ++q) dst[lane + 64 * q] = v[q];
}

// kv: [bs*n_new][2*nkv*dh] = [K heads | V heads] of the projected hidden rows.
template <typename WT>
__global__ __launch_bounds__(256) void ctx_store_kernel(const float *__restrict__ kv, int n_new,
                                                        const WT *__restrict__ kn,
                                                        const int32_t *__restrict__ ctx_lens,
                                                        int max_ctx, WT *__restrict__ ck,
                                                        WT *__restrict__ cv, int bs, int nkv, int dh,
                                                        float eps, float theta, int32_t *err) {
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= bs * n_new * 2 * nkv) return;
  const int row = item / (2 * nkv), hh = item % (2 * nkv);
  const int b = row / n_new, i = row % n_new;
  int n = ctx_lens[b];
  if (n < n_new || n > max_ctx) {
    if (lane == 0 && i == 0 && hh == 0) raise_error(err, DEV_BAD_CTX_LEN);
    n = n < n_new ? n_new : max_ctx;
  }
  const int pos = n - n_new + i;
  if (pos < 0 || pos >= max_ctx) return;
  const float *src = kv + (size_t)row * 2 * nkv * dh + (size_t)hh * dh;
  float v[2] = {0.f, 0.f};
  const int per = dh / 64;
  for (int q = 0; q < per; ++q) v[q] = src[lane + 64 * q];
  WT *dst;
  const size_t off = (((size_t)b * max_ctx + pos) * nkv) * dh;
  if (hh < nkv) {
    norm_rope_head<WT>(v, dh, kn, eps, pos, theta, true, lane);
    dst = ck + off + (size_t)hh * dh;
  } else {
    dst = cv + off + (size_t)(hh - nkv) * dh;
  }
  for (int q = 0; q < per; ++q) store_as(dst + lane + 64 * q, v[q]);
}

// ---------------------------------------------------------------------------
// block attention: queries = the B block rows of the G query heads sharing one
// kv head; keys = context[0, n) followed by the B block keys; no mask.
// Split over key chunks of CH; each chunk writes (max, sum, unnormalised
// output) per query row and a second kernel merges chunks with log-sum-exp.
// ---------------------------------------------------------------------------
constexpr int CH = 32;
int attn_chunk_len() { return CH; }
int attn_nchunks(int max_ctx, int B) { return (max_ctx + B + CH - 1) / CH; }
size_t attn_part_floats(const Dims &D, int max_ctx) {
  return (size_t)D.bs * D.nq * D.B * attn_nchunks(max_ctx, D.B) * (D.dh + 2);
}

template <typename WT>
__global__ __launch_bounds__(256) void attn_partial_kernel(
    const float *__restrict__ Q, const float *__restrict__ Kb, const float *__restrict__ Vb,
    const WT *__restrict__ ck, const WT *__restrict__ cv, const int32_t *__restrict__ ctx_lens,
    int max_ctx, float *__restrict__ part, int B, int nq, int nkv, int dh, int nch, float scale) {
  extern __shared__ float smem[];
  const int c = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int G = nq / nkv, R = G * B;
  int n = ctx_lens[b];
  n = n < 0 ? 0 : (n > max_ctx ? max_ctx : n);
  const int total = n + B;
  const int c0 = c * CH;
  if (c0 >= total) return;
  const int nk = min(CH, total - c0);
  const int dp = dh + 1;
  float *Qs = smem;               // [R][dh]
  float *Ks = Qs + R * dh;        // [CH][dh+1]
  float *Vs = Ks + CH * dp;       // [CH][dh]
  float *S = Vs + CH * dh;        // [R][CH]
  const int tid = threadIdx.x;

  for (int e = tid; e < R * dh; e += 256) {
    const int qi = e / dh, dd = e % dh;
    const int qh = kvh * G + qi / B, j = qi % B;
    Qs[e] = Q[(((size_t)b * B + j) * nq + qh) * dh + dd];
  }
  for (int e = tid; e < CH * dh; e += 256) {
    const int t = e / dh, dd = e % dh;
    float kvk = 0.f, kvv = 0.f;
    if (t < nk) {
      const int kk = c0 + t;
      if (kk < n) {
        const size_t off = ((((size_t)b * max_ctx + kk) * nkv) + kvh) * dh + dd;
        kvk = to_f32(ck[off]);
        kvv = to_f32(cv[off]);
      } else {
        const size_t off = ((((size_t)b * B + (kk - n)) * nkv) + kvh) * dh + dd;
        kvk = Kb[off];
        kvv = Vb[off];
      }
    }
    Ks[t * dp + dd] = kvk;
    Vs[t * dh + dd] = kvv;
  }
  __syncthreads();

  for (int e = tid; e < R * CH; e += 256) {
    const int qi = e / CH, t = e % CH;
    float s = -INFINITY;
    if (t < nk) {
      const float *qr = Qs + qi * dh;
      const float *kr = Ks + t * dp;
      float a0 = 0.f, a1 = 0.f;
      for (int dd = 0; dd < dh; dd += 2) {
        a0 = fmaf(qr[dd], kr[dd], a0);
        a1 = fmaf(qr[dd + 1], kr[dd + 1], a1);
      }
      s = (a0 + a1) * scale;
    }
    S[e] = s;
  }
  __syncthreads();

  // per-row max and exp; one wave per row at a time
  const int wave = tid >> 6, lane = tid & 63;
  float *rowstat = part;  // written below per row
  for (int qi = wave; qi < R; qi += 4) {
    float s = lane < CH ? S[qi * CH + lane] : -INFINITY;
    const float m = wave_max(s);
    const float p = (lane < nk) ? expf(s - m) : 0.f;
    const float l = wave_sum(p);
    if (lane < CH) S[qi * CH + lane] = p;
    if (lane == 0) {
      const int qh = kvh * G + qi / B, j = qi % B;
      float *dst = rowstat + ((((size_t)b * nq + qh) * B + j) * nch + c) * (dh + 2);
      dst[dh] = m;
      dst[dh + 1] = l;
    }
  }
  __syncthreads();
  for (int e = tid; e < R * dh; e += 256) {
    const int qi = e / dh, dd = e % dh;
    const float *pr = S + qi * CH;
    float acc = 0.f;
    for (int t = 0; t < nk; ++t) acc = fmaf(pr[t], Vs[t * dh + dd], acc);
    const int qh = kvh * G + qi / B, j = qi % B;
    part[((((size_t)b * nq + qh) * B + j) * nch + c) * (dh + 2) + dd] = acc;
  }
}

__global__ __launch_bounds__(256) void attn_combine_kernel(const float *__restrict__ part,
                                                           const int32_t *__restrict__ ctx_lens,
                                                           int max_ctx, float *__restrict__ O, int bs,
                                                           int B, int nq, int dh, int nch) {
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);  // (b, qh, j)
  if (item >= bs * nq * B) return;
  const int j = item % B, qh = (item / B) % nq, b = item / (B * nq);
  int n = ctx_lens[b];
  n = n < 0 ? 0 : (n > max_ctx ? max_ctx : n);
  const int nc = (n + B + CH - 1) / CH;
  const float *base = part + (((size_t)b * nq + qh) * B + j) * nch * (dh + 2);
  float M = -INFINITY;
  for (int c = 0; c < nc; ++c) M = fmaxf(M, base[c * (dh + 2) + dh]);
  float den = 0.f, o0 = 0.f, o1 = 0.f;
  for (int c = 0; c < nc; ++c) {
    const float *pc = base + c * (dh + 2);
    const float w = expf(pc[dh] - M);
    den = fmaf(w, pc[dh + 1], den);
    o0 = fmaf(w, pc[lane], o0);
    if (dh == 128) o1 = fmaf(w, pc[lane + 64], o1);
  }
  const float inv = 1.0f / den;
  float *dst = O + ((size_t)(b * B + j) * nq + qh) * dh;
  dst[lane] = o0 * inv;
  if (dh == 128) dst[lane + 64] = o1 * inv;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
void launch_embed_block(const Dims &D, const void *embed, const int32_t *anchor, float *X,
                        int32_t *err, hipStream_t st) {
  dim3 grid(D.bs * D.B);
  if (D.bf16)
    hipLaunchKernelGGL(embed_block_kernel<bf16_t>, grid, dim3(256), 0, st, (const bf16_t *)embed, anchor,
                       X, D.B, D.d, D.V, D.mask_id, err);
  else
    hipLaunchKernelGGL(embed_block_kernel<float>, grid, dim3(256), 0, st, (const float *)embed, anchor, X,
                       D.B, D.d, D.V, D.mask_id, err);
}

void launch_rmsnorm(const Dims &D, const float *x, int ldx, const void *gain, float *y, int ldy,
                    int rows, int width, bool skip_anchor, hipStream_t st) {
  if (rows <= 0) return;
  if (D.bf16)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(rows), dim3(256), 0, st, x, ldx, (const bf16_t *)gain, y,
                       ldy, width, D.eps, (int)skip_anchor, D.B - 1);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(rows), dim3(256), 0, st, x, ldx, (const float *)gain, y,
                       ldy, width, D.eps, (int)skip_anchor, D.B - 1);
}

void launch_qk_norm_rope(const Dims &D, const float *qkv, const void *q_norm, const void *k_norm,
                         const int32_t *ctx_lens, int max_ctx, float *Q, float *Kb, float *Vb,
                         hipStream_t st) {
  const int M = D.bs * D.B;
  const int items = M * (D.nq + 2 * D.nkv);
  dim3 grid((items + 3) / 4);
  if (D.bf16)
    hipLaunchKernelGGL(qk_norm_rope_kernel<bf16_t>, grid, dim3(256), 0, st, qkv, (const bf16_t *)q_norm,
                       (const bf16_t *)k_norm, ctx_lens, max_ctx, Q, Kb, Vb, M, D.B, D.nq, D.nkv, D.dh,
                       D.eps, D.theta);
  else
    hipLaunchKernelGGL(qk_norm_rope_kernel<float>, grid, dim3(256), 0, st, qkv, (const float *)q_norm,
                       (const float *)k_norm, ctx_lens, max_ctx, Q, Kb, Vb, M, D.B, D.nq, D.nkv, D.dh,
                       D.eps, D.theta);
}

void launch_ctx_store(const Dims &D, const float *kv, int n_new, const void *k_norm,
                      const int32_t *ctx_lens, int max_ctx, void *ck, void *cv, int32_t *err,
                      hipStream_t st) {
  const int items = D.bs * n_new * 2 * D.nkv;
  if (items <= 0) return;
  dim3 grid((items + 3) / 4);
  if (D.bf16)
    hipLaunchKernelGGL(ctx_store_kernel<bf16_t>, grid, dim3(256), 0, st, kv, n_new, (const bf16_t *)k_norm,
                       ctx_lens, max_ctx, (bf16_t *)ck, (bf16_t *)cv, D.bs, D.nkv, D.dh, D.eps, D.theta,
                       err);
  else
    hipLaunchKernelGGL(ctx_store_kernel<float>, grid, dim3(256), 0, st, kv, n_new, (const float *)k_norm,
                       ctx_lens, max_ctx, (float *)ck, (float *)cv, D.bs, D.nkv, D.dh, D.eps, D.theta, err);
}

static size_t attn_lds_bytes(const Dims &D) {
  const int R = (D.nq / D.nkv) * D.B;
  return sizeof(float) * ((size_t)R * D.dh + CH * (D.dh + 1) + CH * D.dh + (size_t)R * CH);
}

void launch_attention(const Dims &D, const float *Q, const float *Kb, const float *Vb,
                      const void *ck, const void *cv, const int32_t *ctx_lens, int max_ctx,
                      float *part, float *O, int32_t *err, hipStream_t st) {
  (void)err;
  const int nch = attn_nchunks(max_ctx, D.B);
  const size_t lds = attn_lds_bytes(D);
  const float scale = 1.0f / sqrtf((float)D.dh);
  dim3 grid(nch, D.nkv, D.bs);
  if (D.bf16) {
    (void)hipFuncSetAttribute((const void *)attn_partial_kernel<bf16_t>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(attn_partial_kernel<bf16_t>, grid, dim3(256), lds, st, Q, Kb, Vb,
                       (const bf16_t *)ck, (const bf16_t *)cv, ctx_lens, max_ctx, part, D.B, D.nq, D.nkv,
                       D.dh, nch, scale);
  } else {
    (void)hipFuncSetAttribute((const void *)attn_partial_kernel<float>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(attn_partial_kernel<float>, grid, dim3(256), lds, st, Q, Kb, Vb, (const float *)ck,
                       (const float *)cv, ctx_lens, max_ctx, part, D.B, D.nq, D.nkv, D.dh, nch, scale);
  }
  const int items = D.bs * D.nq * D.B;
  hipLaunchKernelGGL(attn_combine_kernel, dim3((items + 3) / 4), dim3(256), 0, st, part, ctx_lens, max_ctx,
                     O, D.bs, D.B, D.nq, D.dh, nch);
}

__global__ void fill_u32_kernel(uint32_t *p, size_t n, uint32_t v) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}
void launch_fill_u32(uint32_t *p, size_t n, uint32_t v, hipStream_t st) {
  if (n == 0) return;
  hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n, v);
}

}  // namespace dk
