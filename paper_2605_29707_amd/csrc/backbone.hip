// Draft-backbone kernels other than the projections (Sec. 4.1.1): block
// embedding, RMSNorm, per-head q/k RMSNorm + rotate-half RoPE, projection of
// context hidden states into the KV cache, and split-KV block attention.
// All arithmetic is fp32; RoPE angles are formed and range-reduced in fp64 so
// that positions in the thousands keep full fp32 accuracy in the rotated values.
#include <algorithm>

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

// x_out[in_row] = x[in_row] + the `np` (<= 16) partial outputs (split order),
// y[i] = RMSNorm(x_out[in_row]) * gain.  With skip_anchor, output row i reads
// input row i + i/(B-1) + 1 (the draft rows of each block); a null x_out skips
// the residual write.  x and x_out are distinct buffers (ping-pong): the
// workgroups of one row each write a slice while the others still read x.  With `embed` given, the row is first replaced by the embedding
// row of its token: tokens[row] when `tokens` is given, else the anchor for
// block position 0 and MASK otherwise.  One
// workgroup per output row; a thread keeps its 16 columns in registers and
// issues all of its loads together.
template <typename WT, int MAXP>
__global__ __launch_bounds__(512) void add_norm_kernel(const float *__restrict__ x, float *__restrict__ x_out,
                                                       int ldx,
                                                       const float *__restrict__ parts, int np,
                                                       size_t pstride, const WT *__restrict__ gain,
                                                       float *__restrict__ y, int ldy, int width, float eps,
                                                       int skip_anchor, int depth, const WT *__restrict__ embed,
                                                       const int32_t *__restrict__ anchor, int mask_id, int V,
                                                       int32_t *err, const int32_t *__restrict__ tokens,
                                                       int nsplit, uint32_t *hdr, int hdr_words) {
  // nsplit workgroups per row: each forms the whole row's sum of squares but
  // writes only its slice of the columns
  const int i = blockIdx.x / nsplit, part = blockIdx.x % nsplit;
  // hdr: the step's workspace header (word 0 the error word) is cleared here
  // instead of by a launch of its own; then only thread 0 of workgroup 0 checks
  // the tokens, after clearing the error word, so no error raised in this launch
  // is lost to the clear
  if (hdr) {
    for (int e = blockIdx.x * blockDim.x + threadIdx.x + 1; e < hdr_words; e += gridDim.x * blockDim.x) hdr[e] = 0u;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      hdr[0] = 0u;
      const int B = depth + 1;
      for (int row = 0; row < (int)gridDim.x / nsplit; ++row) {
        const int tk = tokens ? tokens[row] : (row % B == 0 ? anchor[row / B] : 0);
        if (tk < 0 || tk >= V) raise_error(err, DEV_BAD_TOKEN);
      }
    }
  }
  const bool raise = hdr == nullptr;
  const int cs = width / nsplit;  // columns per slice (a multiple of 8)
  const int in_row = skip_anchor ? i + i / depth + 1 : i;
  const float *xr = x + (size_t)in_row * ldx;
  const float *pr = parts + (size_t)in_row * ldx;
  constexpr int PER = 8, IT = 2;
  const WT *er = nullptr;
  if (embed) {
    const int B = depth + 1;
    int tok = mask_id;
    if (tokens) {  // one token per row (a tree's nodes)
      tok = tokens[in_row];
      if (tok < 0 || tok >= V) {
        if (threadIdx.x == 0 && raise) raise_error(err, DEV_BAD_TOKEN);
        tok = tok < 0 ? 0 : V - 1;
      }
    } else if (in_row % B == 0) {
      tok = anchor[in_row / B];
      if (tok < 0 || tok >= V) {
        if (threadIdx.x == 0 && raise) raise_error(err, DEV_BAD_TOKEN);
        tok = tok < 0 ? 0 : V - 1;
      }
    }
    er = embed + (size_t)tok * width;
  }
  // the gains of this thread's columns, loaded with the inputs (not after the reduction)
  float gv[IT][PER];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int c0 = min((int)(threadIdx.x + it * blockDim.x) * PER, width - PER);
#pragma unroll
    for (int e = 0; e < PER; ++e) gv[it][e] = to_f32(gain[c0 + e]);
  }
  float v[IT][PER];
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int c0 = (threadIdx.x + it * blockDim.x) * PER;
    if (c0 >= width) continue;
    if (er) {
#pragma unroll
      for (int e = 0; e < PER; ++e) v[it][e] = to_f32(er[c0 + e]);
    } else {
      const float4 a = *(const float4 *)(xr + c0), c = *(const float4 *)(xr + c0 + 4);
      v[it][0] = a.x; v[it][1] = a.y; v[it][2] = a.z; v[it][3] = a.w;
      v[it][4] = c.x; v[it][5] = c.y; v[it][6] = c.z; v[it][7] = c.w;
    }
    // MAXP slots loaded unconditionally (slot index clamped to a valid
    // partial) and added only below np: a guarded load would end in a branch
    // join that drains every outstanding load, serialising the partials
    float4 pa[MAXP], pc[MAXP];
#pragma unroll
    for (int p = 0; p < MAXP; ++p) {
      const int pp = min(p, max(np, 1) - 1);
      pa[p] = *(const float4 *)(pr + pp * pstride + c0);
      pc[p] = *(const float4 *)(pr + pp * pstride + c0 + 4);
    }
#pragma unroll
    for (int p = 0; p < MAXP; ++p)
      if (p < np) {
        v[it][0] += pa[p].x; v[it][1] += pa[p].y; v[it][2] += pa[p].z; v[it][3] += pa[p].w;
        v[it][4] += pc[p].x; v[it][5] += pc[p].y; v[it][6] += pc[p].z; v[it][7] += pc[p].w;
      }
    if (x_out && c0 / cs == part) {  // the updated residual goes to the other buffer (other slices still read x)
      float *xo = x_out + (size_t)in_row * ldx;
      *(float4 *)(xo + c0) = make_float4(v[it][0], v[it][1], v[it][2], v[it][3]);
      *(float4 *)(xo + c0 + 4) = make_float4(v[it][4], v[it][5], v[it][6], v[it][7]);
    }
#pragma unroll
    for (int e = 0; e < PER; ++e) ss = fmaf(v[it][e], v[it][e], ss);
  }
  ss = wave_sum_dpp(ss);
  __shared__ float red[8];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)width + eps);
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int c0 = (threadIdx.x + it * blockDim.x) * PER;
    if (c0 >= width || c0 / cs != part) continue;
    float o[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) o[e] = v[it][e] * inv * gv[it][e];
    float *yr = y + (size_t)i * ldy + c0;
    *(float4 *)(yr) = make_float4(o[0], o[1], o[2], o[3]);
    *(float4 *)(yr + 4) = make_float4(o[4], o[5], o[6], o[7]);
  }
}

// One wave per (row, head).  Lane l holds elements l and l+64 (dh = 128) or
// l (dh = 64); RoPE pairs element i with i + dh/2.
DEVI void norm_rope_head(float (&v)[2], int dh, const float (&gain)[2], float eps, int pos, double freq,
                         bool rotate, int lane) {
  const int per = dh / 64;
  float ss = 0.f;
  for (int q = 0; q < per; ++q) ss = fmaf(v[q], v[q], ss);
  ss = wave_sum_dpp(ss);
  const float inv = 1.0f / sqrtf(ss / (float)dh + eps);
  for (int q = 0; q < per; ++q) v[q] = v[q] * inv * gain[q];
  if (!rotate) return;
  // angle pos * theta^(-2i/dh) (freq = theta^(-2i/dh) of this lane's pair):
  // formed and reduced modulo 2*pi in fp64, then an fp32 sine/cosine of the
  // reduced angle (|error| ~ 1e-7 at positions of 10^4)
  const double ang = (double)pos * freq;
  const double k = rint(ang * 0.15915494309189535);
  const double red = fma(-k, 6.283185307179586, ang) - k * 2.4492935982947064e-16;
  float s, c;
  sincosf((float)red, &s, &c);
  if (dh == 128) {
    const float x1 = v[0], x2 = v[1];
    v[0] = x1 * c - x2 * s;
    v[1] = x2 * c + x1 * s;
  } else {  // dh == 64: partner lives 32 lanes away
    const float p = __shfl_xor(v[0], 32, 64);
    v[0] = (lane < 32) ? (v[0] * c - p * s) : (v[0] * c + p * s);
  }
}

// Block rows m < M: Q and K heads get their RMSNorm and RoPE (position n_b + j),
// V heads are copied; Q, Kb, Vb are [M][heads][dh].  Rows M + b*n_new + i are
// context rows appended from target hidden states (the same GEMM projected
// them): their K heads get the k-norm and RoPE at position n_b - n_new + i and
// are stored, with their V heads, into the cache in the storage type.
template <typename WT, int MAXP>
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(const float *__restrict__ qkv, int np,
                                                           size_t pstride, const WT *__restrict__ qn,
                                                           const WT *__restrict__ kn,
                                                           const int32_t *__restrict__ ctx_lens,
                                                           int max_ctx, float *__restrict__ Q,
                                                           float *__restrict__ Kb,
                                                           float *__restrict__ Vb, int M, int B, int nq,
                                                           int nkv, int dh, float eps,
                                                           const double *__restrict__ inv_freq, int n_new,
                                                           WT *__restrict__ ck, WT *__restrict__ cv,
                                                           int32_t *err, const int32_t *__restrict__ pos_rows,
                                                           int n_store) {
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nh = nq + 2 * nkv;
  int m, hh;
  if (item < M * nh) {
    m = item / nh;
    hh = item % nh;
  } else {  // appended context rows: K and V heads only
    const int a = item - M * nh;
    const int bs = M / B;
    if (a >= bs * n_new * 2 * nkv) return;
    m = M + a / (2 * nkv);
    hh = nq + a % (2 * nkv);
  }
  const float *src = qkv + (size_t)m * nh * dh + (size_t)hh * dh;
  float v[2] = {0.f, 0.f};
  const int per = dh / 64;
  // everything the head needs besides the projection, loaded with it: the
  // context length, the row's position, the norm gains, the RoPE frequency
  const bool appended = m >= M;
  const int b = appended ? (m - M) / n_new : m / B;
  const int n_raw = ctx_lens[b];
  const int prow = (!appended && pos_rows) ? pos_rows[m] : 0;
  float gv[2];
  {
    const WT *gp = hh < nq ? qn : kn;
#pragma unroll
    for (int q = 0; q < 2; ++q) gv[q] = to_f32(gp[lane + 64 * min(q, per - 1)]);
  }
  const double freq = inv_freq[dh == 128 ? lane : (lane & 31)];
  {
    // K-split partial outputs, added in split order; all loads issued together
    // (MAXP slots, clamped to a valid partial, added only below np)
    float t[MAXP][2];
#pragma unroll
    for (int p = 0; p < MAXP; ++p) {
      const int pp = min(p, max(np, 1) - 1);
#pragma unroll
      for (int q = 0; q < 2; ++q) t[p][q] = src[pp * pstride + lane + 64 * min(q, per - 1)];
    }
#pragma unroll
    for (int p = 0; p < MAXP; ++p)
      if (p < np)
#pragma unroll
        for (int q = 0; q < 2; ++q) v[q] += q < per ? t[p][q] : 0.f;
  }
  if (appended) {
    const int i = (m - M) % n_new;
    int n = n_raw;
    if (n < n_new || n > max_ctx) {
      if (lane == 0 && i == 0 && hh == nq) raise_error(err, DEV_BAD_CTX_LEN);
      n = n < n_new ? n_new : max_ctx;
    }
    const int pos = n - n_new + i;
    const size_t off = (((size_t)b * max_ctx + pos) * nkv) * dh;
    WT *dst;
    if (hh < nq + nkv) {
      norm_rope_head(v, dh, gv, eps, pos, freq, true, lane);
      dst = ck + off + (size_t)(hh - nq) * dh;
    } else {
      dst = cv + off + (size_t)(hh - nq - nkv) * dh;
    }
    for (int q = 0; q < per; ++q) store_as(dst + lane + 64 * q, v[q]);
    return;
  }
  const int j = m % B;
  int n = n_raw;
  n = n < 0 ? 0 : (n > max_ctx ? max_ctx : n);
  const int pos = pos_rows ? prow : n + j;
  float *dst;
  if (hh < nq) {
    norm_rope_head(v, dh, gv, eps, pos, freq, true, lane);
    dst = Q + ((size_t)m * nq + hh) * dh;
  } else if (hh < nq + nkv) {
    norm_rope_head(v, dh, gv, eps, pos, freq, true, lane);
    dst = Kb + ((size_t)m * nkv + (hh - nq)) * dh;
  } else {
    dst = Vb + ((size_t)m * nkv + (hh - nq - nkv)) * dh;
  }
  for (int q = 0; q < per; ++q) dst[lane + 64 * q] = v[q];
  // the first n_store rows of each block also go to the cache at n + j (a
  // verify forward leaves every node's K/V there for the commit)
  if (j < n_store && hh >= nq) {
    if (n + j < max_ctx) {
      const bool isk = hh < nq + nkv;
      WT *cd = (isk ? ck : cv) + (((size_t)b * max_ctx + n + j) * nkv + (hh - nq - (isk ? 0 : nkv))) * dh;
      for (int q = 0; q < per; ++q) store_as(cd + lane + 64 * q, v[q]);
    } else if (lane == 0) {
      raise_error(err, DEV_BAD_CTX_LEN);
    }
  }
}

// ---------------------------------------------------------------------------
// block attention: queries = the B block rows of the G query heads sharing one
// kv head (R = G*B rows); keys = context[0, n) followed by the B block keys;
// no mask.  One workgroup per (key chunk of CH, kv head, batch row) writes the
// chunk's row max, row sum of exp and unnormalised output; a second kernel
// merges the chunks with log-sum-exp weights.  Both products run on the
// matrix cores (see attn_partial_kernel).
// ---------------------------------------------------------------------------
constexpr int kAttnThreads = 256;

DEVI float4 ld4_f32(const float *p) { return *(const float4 *)p; }
// component-wise select (a whole-vector select can be lowered through scratch memory)
DEVI float4 keep4(bool ok, const float4 &v) {
  return make_float4(ok ? v.x : 0.f, ok ? v.y : 0.f, ok ? v.z : 0.f, ok ? v.w : 0.f);
}
DEVI float4 ld4_f32(const bf16_t *p) {
  const uint2 u = *(const uint2 *)p;
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                     __uint_as_float(u.y & 0xffff0000u));
}

// keys per chunk, by the query rows R = (n_q / n_kv) * B of a workgroup (the
// partial kernel's dispatch and the merge must agree)
static int attn_ch(int R) { return R >= 64 ? 32 : 64; }
int attn_nchunks(int max_ctx, int B) { return (max_ctx + B + 31) / 32; }  // upper bound for any G
size_t attn_part_floats(const Dims &D, int max_ctx) {
  return (size_t)D.bs * D.nq * D.B * attn_nchunks(max_ctx, D.B) * (D.dh + 2);
}

// Four fp32 values as hi and lo bf16 quads (8 bytes each), the split of split8.
DEVI void split4(const float4 &v, uint2 &hi, uint2 &lo) {
  const float f[8] = {v.x, v.y, v.z, v.w, 0.f, 0.f, 0.f, 0.f};
  bf16x8 h, l;
  split8(f, h, l);
  const u32x4 hu = __builtin_bit_cast(u32x4, h), lu = __builtin_bit_cast(u32x4, l);
  hi = make_uint2(hu[0], hu[1]);
  lo = make_uint2(lu[0], lu[1]);
}
DEVI bf16x8 ld_frag(const uint16_t *p) { return __builtin_bit_cast(bf16x8, *(const u32x4 *)p); }
// the product with an exact bf16 first operand (its lo part is zero)
DEVI floatx4 mfma2(const bf16x8 &ah, const bf16x8 &bh, const bf16x8 &bl, floatx4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, acc, 0, 0, 0);
  return acc;
}
// the product with an exact bf16 second operand, in mfma3's order without its zero term
DEVI floatx4 mfma2b(const bf16x8 &ah, const bf16x8 &al, const bf16x8 &bh, floatx4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, acc, 0, 0, 0);
  return acc;
}
DEVI floatx4 mfma3(const bf16x8 &ah, const bf16x8 &al, const bf16x8 &bh, const bf16x8 &bl, floatx4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, acc, 0, 0, 0);
  return acc;
}

// Matrix-core attention partial for one (key chunk, kv head, batch row):
//   S^T = K Q^T  (16-key x 16-query tiles), softmax statistics per query row,
//   O   = P V    (16-query x 16-dim tiles), with every fp32 operand split into
//   hi + lo bf16 parts (three passes, the lo*lo term dropped: ~2^-16 relative).
// Q, K, P live in LDS row-major as bf16 hi and lo parts (split once, when
// staged or produced; P takes K's place once the scores are formed); V is staged transposed so a B fragment (8 consecutive
// keys of one dim) is one contiguous read.  A chunk of bf16 cache keys has
// exact K and V (zero lo parts): the products with them are skipped.
// MASKED: block key k is visible to block query j only where amask[b][j][k] is
// set (a verify forward's tree mask, [bs][B][B] bytes, B a multiple of 4);
// context keys are always visible.  Rows whose keys in a chunk are all hidden
// leave (max -inf, sum 0), which the merge weighs as zero.
template <typename WT, int QT, int CH, int DH, bool MASKED, bool MULTI>
__global__ __launch_bounds__(kAttnThreads) void attn_partial_kernel(
    const float *__restrict__ Q, const float *__restrict__ Kb, const float *__restrict__ Vb,
    const WT *__restrict__ ck, const WT *__restrict__ cv, const int32_t *__restrict__ ctx_lens,
    int max_ctx, float *__restrict__ part, int B, int nq, int nkv, int nch, float scale,
    const uint8_t *__restrict__ amask, int cpw) {
  constexpr int R = QT * 16;      // query rows of the group
  constexpr int KT = CH / 16;     // key tiles
  constexpr int DT = DH / 16;     // output dim tiles
  constexpr int QTW = QT * KT / 4;  // query tiles per wave in the score phase
  constexpr int DTW = DT / 4;     // dim tiles per wave in the output phase
  // operands are held as bf16 hi and lo parts, split once while staging
  constexpr int DP = DH + 8, CP = CH + 8;  // row strides in bf16 values (16-byte rows, staggered banks)
  extern __shared__ __align__(16) float smem[];
  uint16_t *Qh = (uint16_t *)smem, *Ql = Qh + R * DP;  // [R][DP]
  uint16_t *Kh = Ql + R * DP, *Kl = Kh + CH * DP;        // [CH][DP]
  uint16_t *Vh = Kl + CH * DP, *Vl = Vh + DH * CP;       // [DH][CP]  (transposed)
  // [R][CP], over K where it fits: P is written after the barrier that
  // follows the last read of K
  constexpr bool kPinK = R * CP <= CH * DP;
  uint16_t *Ph = kPinK ? Kh : Vl + DH * CP, *Pl = Ph + R * CP;
  float *Rm = (float *)(kPinK ? Vl + DH * CP : Pl + R * CP);  // [KT][R] partial row max
  float *Rl = Rm + KT * R;             // [KT][R] partial row sum
  // MULTI: running row max and sum over the chunks folded so far, and each
  // row's rescale factor for the current chunk
  float *Mrun = Rl + KT * R, *Lrun = Mrun + R, *Alpha = Lrun + R;
  uint32_t *Ms = (uint32_t *)(Rl + KT * R + (MULTI ? 3 * R : 0));  // MASKED: [B][B] bytes of this batch row's tree mask
  constexpr int kMaskIt = 64 * 64 / 4 / kAttnThreads;  // words per thread for B <= 64

  const int c = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int G = nq / nkv;
  int n = ctx_lens[b];
  n = n < 0 ? 0 : (n > max_ctx ? max_ctx : n);
  const int total = n + B;
  // MULTI: this workgroup folds chunks c*cpw .. c*cpw + cpw - 1 into one
  // partial with a running (online) softmax; otherwise it takes chunk c alone
  const int nsub = MULTI ? cpw : 1;
  if (c * nsub * CH >= total) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, cc = lane & 15;
  if constexpr (MULTI)
    for (int q = tid; q < R; q += kAttnThreads) {
      Mrun[q] = -INFINITY;
      Lrun[q] = 0.f;
    }
  floatx4 oacc[QT][DTW];
#pragma unroll
  for (int i = 0; i < QT; ++i)
#pragma unroll
    for (int x = 0; x < DTW; ++x) oacc[i][x] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int cs = 0; cs < nsub; ++cs) {
  const int c0 = (c * nsub + cs) * CH;
  if (c0 >= total) break;  // uniform over the workgroup
  const int nk = min(CH, total - c0);

  // ---- stage Q rows (first chunk only), the K chunk (row-major) and the V chunk (transposed)
  {
    constexpr int NQ = R * DH / 4 / kAttnThreads;
    float4 qv[NQ];
    if (cs == 0) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int e = tid + q * kAttnThreads;
        const int qi = e / (DH / 4), d4 = e % (DH / 4);
        const int qh = kvh * G + qi / B, j = qi % B;
        qv[q] = *(const float4 *)(Q + (((size_t)b * B + j) * nq + qh) * DH + 4 * d4);
      }
    }
    // Each key comes from the cache (index < n) or the block (index >= n).
    // Both candidates are loaded unconditionally at clamped, valid addresses
    // and selected per lane: a per-lane guarded load would become a branch
    // whose join drains every outstanding load, serialising the staging into
    // one memory round trip per load.  Without a context the cache candidate
    // reads the block buffer instead (discarded: no index is < 0).
    constexpr int NE = CH * DH / 4 / kAttnThreads;
    const WT *ckb = n > 0 ? ck : (const WT *)Kb, *cvb = n > 0 ? cv : (const WT *)Vb;
    const int nl = n > 0 ? n - 1 : 0;
    float4 kc[NE], kbk[NE], vc[NE], vbk[NE];
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      const int e = tid + q * kAttnThreads;
      const int t = e / (DH / 4), d4 = e % (DH / 4);
      const int kk = min(c0 + t, total - 1);
      const size_t crow = n > 0 ? (((size_t)b * max_ctx + min(kk, nl)) * nkv + kvh) * DH : (size_t)kvh * DH;
      kc[q] = ld4_f32(ckb + crow + 4 * d4);
      kbk[q] = *(const float4 *)(Kb + ((((size_t)b * B + min(max(kk - n, 0), B - 1)) * nkv) + kvh) * DH + 4 * d4);
      const int tv = e % CH, dv = e / CH;                   // V: consecutive lanes, consecutive keys
      const int kv2 = min(c0 + tv, total - 1);
      const size_t vrow = n > 0 ? (((size_t)b * max_ctx + min(kv2, nl)) * nkv + kvh) * DH : (size_t)kvh * DH;
      vc[q] = ld4_f32(cvb + vrow + 4 * dv);
      vbk[q] = *(const float4 *)(Vb + ((((size_t)b * B + min(max(kv2 - n, 0), B - 1)) * nkv) + kvh) * DH + 4 * dv);
    }
    uint32_t mw[MASKED ? kMaskIt : 1];
    if constexpr (MASKED) {  // unconditional loads at clamped word indices
      const int words = B * B / 4;
      const uint32_t *src = (const uint32_t *)amask + (size_t)b * words;
#pragma unroll
      for (int q = 0; q < kMaskIt; ++q) mw[q] = src[min(tid + q * kAttnThreads, words - 1)];
    }
    float4 kv[NE], vv[NE];
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      const int e = tid + q * kAttnThreads;
      const int kk = min(c0 + e / (DH / 4), total - 1);
      const int kv2 = min(c0 + e % CH, total - 1);
      kv[q] = kk < n ? kc[q] : kbk[q];
      vv[q] = kv2 < n ? vc[q] : vbk[q];
    }
    if (cs == 0) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int e = tid + q * kAttnThreads;
        const int qi = e / (DH / 4), d4 = e % (DH / 4);
        uint2 hi, lo;
        split4(qv[q], hi, lo);
        *(uint2 *)(Qh + qi * DP + 4 * d4) = hi;
        *(uint2 *)(Ql + qi * DP + 4 * d4) = lo;
      }
    }
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      const int e = tid + q * kAttnThreads;
      const int t = e / (DH / 4), d4 = e % (DH / 4);
      uint2 hi, lo;
      split4(keep4(t < nk, kv[q]), hi, lo);
      *(uint2 *)(Kh + t * DP + 4 * d4) = hi;
      *(uint2 *)(Kl + t * DP + 4 * d4) = lo;
      const int tv = e % CH, dv = e / CH;
      split4(keep4(tv < nk, vv[q]), hi, lo);
      Vh[(4 * dv + 0) * CP + tv] = (uint16_t)hi.x;
      Vh[(4 * dv + 1) * CP + tv] = (uint16_t)(hi.x >> 16);
      Vh[(4 * dv + 2) * CP + tv] = (uint16_t)hi.y;
      Vh[(4 * dv + 3) * CP + tv] = (uint16_t)(hi.y >> 16);
      Vl[(4 * dv + 0) * CP + tv] = (uint16_t)lo.x;
      Vl[(4 * dv + 1) * CP + tv] = (uint16_t)(lo.x >> 16);
      Vl[(4 * dv + 2) * CP + tv] = (uint16_t)lo.y;
      Vl[(4 * dv + 3) * CP + tv] = (uint16_t)(lo.y >> 16);
    }
    if constexpr (MASKED) {
#pragma unroll
      for (int q = 0; q < kMaskIt; ++q)
        if (tid + q * kAttnThreads < B * B / 4) Ms[tid + q * kAttnThreads] = mw[q];
    }
  }
  __syncthreads();

  // ---- scores: wave w owns key tile kt = w % KT and QTW query tiles.  A
  // chunk of bf16 cache keys only has exact keys: their lo parts are zero,
  // so those products are skipped (the sums are the same bits).
  const bool exact = sizeof(WT) == 2 && c0 + CH <= n;
  const int kt = wave % KT, qt0 = (wave / KT) * QTW;
  floatx4 sacc[QTW];
#pragma unroll
  for (int i = 0; i < QTW; ++i) sacc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < DH / 32; ++s) {
    const bf16x8 kh = ld_frag(Kh + (16 * kt + cc) * DP + 32 * s + 8 * g);
    const bf16x8 kl = ld_frag(Kl + (16 * kt + cc) * DP + 32 * s + 8 * g);
#pragma unroll
    for (int i = 0; i < QTW; ++i) {
      const bf16x8 qh = ld_frag(Qh + (16 * (qt0 + i) + cc) * DP + 32 * s + 8 * g);
      const bf16x8 ql = ld_frag(Ql + (16 * (qt0 + i) + cc) * DP + 32 * s + 8 * g);
      sacc[i] = exact ? mfma2(kh, qh, ql, sacc[i]) : mfma3(kh, kl, qh, ql, sacc[i]);
    }
  }
  // lane (g, cc) holds S[q = 16*qt + cc][key = 16*kt + 4g + e]
#pragma unroll
  for (int i = 0; i < QTW; ++i) {
    float m = -INFINITY;
    const int jq = (16 * (qt0 + i) + cc) % B;  // the query's block row
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int key = 16 * kt + 4 * g + e;
      bool ok = key < nk;
      if constexpr (MASKED) {
        const int kb = c0 + key - n;  // block key index (< 0: a context key; < B wherever key < nk)
        ok = ok && (kb < 0 || ((const uint8_t *)Ms)[jq * B + min(kb, B - 1)] != 0);
      }
      sacc[i][e] = ok ? sacc[i][e] * scale : -INFINITY;
      m = fmaxf(m, sacc[i][e]);
    }
    m = fmaxf(m, __shfl_xor(m, 16, 64));
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    if (g == 0) Rm[kt * R + 16 * (qt0 + i) + cc] = m;
  }
  __syncthreads();
  if constexpr (MULTI) {  // running max and the rescale of what was folded before
    for (int q = tid; q < R; q += kAttnThreads) {
      float mc = Rm[q];
      for (int k2 = 1; k2 < KT; ++k2) mc = fmaxf(mc, Rm[k2 * R + q]);
      const float mo = Mrun[q], mn = fmaxf(mo, mc);
      Alpha[q] = mo == -INFINITY ? 0.f : expf(mo - mn);
      Mrun[q] = mn;
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < QTW; ++i) {
    const int q = 16 * (qt0 + i) + cc;
    float m;
    if constexpr (MULTI) {
      m = Mrun[q];
    } else {
      m = Rm[q];
#pragma unroll
      for (int k2 = 1; k2 < KT; ++k2) m = fmaxf(m, Rm[k2 * R + q]);
    }
    float p[4], l = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int key = 16 * kt + 4 * g + e;
      if constexpr (MASKED)  // hidden keys hold -inf (and m too if all of them are hidden)
        p[e] = sacc[i][e] != -INFINITY ? expf(sacc[i][e] - m) : 0.f;
      else
        p[e] = key < nk ? expf(sacc[i][e] - m) : 0.f;
      l += p[e];
    }
    uint2 hi, lo;
    split4(make_float4(p[0], p[1], p[2], p[3]), hi, lo);
    *(uint2 *)(Ph + q * CP + 16 * kt + 4 * g) = hi;
    *(uint2 *)(Pl + q * CP + 16 * kt + 4 * g) = lo;
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (g == 0) Rl[kt * R + q] = l;
  }
  __syncthreads();
  // softmax statistics of the chunk per query row
  if constexpr (MULTI) {
    for (int q = tid; q < R; q += kAttnThreads) {
      float l = 0.f;
      for (int k2 = 0; k2 < KT; ++k2) l += Rl[k2 * R + q];
      Lrun[q] = Alpha[q] * Lrun[q] + l;
    }
  } else {
    for (int q = tid; q < R; q += kAttnThreads) {
      float m = Rm[q], l = 0.f;
      for (int k2 = 1; k2 < KT; ++k2) m = fmaxf(m, Rm[k2 * R + q]);
      for (int k2 = 0; k2 < KT; ++k2) l += Rl[k2 * R + q];
      const int qh = kvh * G + q / B, j = q % B;
      float *dst = part + ((((size_t)b * nq + qh) * B + j) * nch + c) * (DH + 2);
      dst[DH] = m;
      dst[DH + 1] = l;
    }
  }

  // ---- output: wave w owns DTW dim tiles, all query tiles
  if constexpr (MULTI) {  // what was folded before is rescaled to the new running max
#pragma unroll
    for (int i = 0; i < QT; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float al = Alpha[16 * i + 4 * g + e];
#pragma unroll
        for (int x = 0; x < DTW; ++x) oacc[i][x][e] *= al;
      }
  }
#pragma unroll
  for (int s = 0; s < CH / 32; ++s) {
    bf16x8 vh[DTW], vl[DTW];
#pragma unroll
    for (int x = 0; x < DTW; ++x) {
      vh[x] = ld_frag(Vh + (16 * (wave * DTW + x) + cc) * CP + 32 * s + 8 * g);
      vl[x] = ld_frag(Vl + (16 * (wave * DTW + x) + cc) * CP + 32 * s + 8 * g);
    }
#pragma unroll
    for (int i = 0; i < QT; ++i) {
      const bf16x8 ph = ld_frag(Ph + (16 * i + cc) * CP + 32 * s + 8 * g);
      const bf16x8 pl = ld_frag(Pl + (16 * i + cc) * CP + 32 * s + 8 * g);
#pragma unroll
      for (int x = 0; x < DTW; ++x)  // exact V (zero lo part): the zero product is left out
        oacc[i][x] = exact ? mfma2b(ph, pl, vh[x], oacc[i][x]) : mfma3(ph, pl, vh[x], vl[x], oacc[i][x]);
    }
  }
  if constexpr (MULTI) __syncthreads();  // K/P, V and the row statistics are reused by the next chunk
  }  // chunks

  // lane (g, cc) holds O[q = 16*i + 4g + e][dim = 16*dt + cc]
#pragma unroll
  for (int i = 0; i < QT; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int q = 16 * i + 4 * g + e;
      const int qh = kvh * G + q / B, j = q % B;
      float *dst = part + ((((size_t)b * nq + qh) * B + j) * nch + c) * (DH + 2);
#pragma unroll
      for (int x = 0; x < DTW; ++x) dst[16 * (wave * DTW + x) + cc] = oacc[i][x][e];
    }
  if constexpr (MULTI)
    for (int q = tid; q < R; q += kAttnThreads) {
      const int qh = kvh * G + q / B, j = q % B;
      float *dst = part + ((((size_t)b * nq + qh) * B + j) * nch + c) * (DH + 2);
      dst[DH] = Mrun[q];
      dst[DH + 1] = Lrun[q];
    }
}

// ---------------------------------------------------------------------------
// Context attention over a bf16 cache, one online-softmax pass per workgroup
// (batched steps): workgroup (c, kv head, batch row) takes keys
// [c * kpw, (c + 1) * kpw) of the sequence context[0, n) + block[0, B) and
// writes the same partial (unnormalised output, row max, row sum) as
// attn_partial_kernel, for the same merge.
//
// Wave w owns query rows 16 w .. 16 w + 15 of the group (R = G * B = 16 NW
// rows) and keeps their Q fragments (hi and lo) in registers.  Context keys
// go in blocks of 64 through two LDS buffers (K row-major, V transposed),
// staged from registers loaded one block ahead.  Per block a wave forms
// S^T = K Q^T (exact bf16 keys: two products per tile), updates its rows'
// running max and sum, and adds P V.  S^T leaves lane (g, cc) holding row
// cc's scores of keys 16 t + 4 g + e, which is already the A fragment of P V
// when the 32 keys of a product step are ordered (4 g .. 4 g + 3,
// 16 + 4 g .. 16 + 4 g + 3); V's B fragment is read in that order from the
// transposed copy.  The block's own keys (fp32) come last, in one more block
// with hi and lo parts in the two buffers and three products per tile.
// ---------------------------------------------------------------------------
constexpr int kFlashKB = 64;                 // keys per block
constexpr int kFlashKP = 128 + 8;            // K row stride (bf16): conflict-free 16-byte fragment reads
constexpr int kFlashVP = kFlashKB + 4;       // transposed V row stride (bf16): conflict-free 8-byte reads
constexpr size_t kFlashK = (size_t)kFlashKB * kFlashKP, kFlashV = (size_t)128 * kFlashVP;  // bf16 per buffer part
constexpr size_t kFlashLds = 2 * (kFlashK + kFlashV) * sizeof(uint16_t);

DEVI uint32_t pack_lo16(uint32_t a, uint32_t b) { return (a & 0xffffu) | (b << 16); }
DEVI uint32_t pack_hi16(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }

template <int NW, int PD>
__global__ __launch_bounds__(NW * 64) void attn_flash_kernel(const float *__restrict__ Q, const float *__restrict__ Kb,
                                                             const float *__restrict__ Vb, const bf16_t *__restrict__ ck,
                                                             const bf16_t *__restrict__ cv,
                                                             const int32_t *__restrict__ ctx_lens, int max_ctx,
                                                             float *__restrict__ part, int B, int nq, int nkv, int nch,
                                                             float scale, int kpw) {
  constexpr int DH = 128, T = NW * 64, KCH = kFlashKB * DH / 8 / T;  // 16-byte K chunks per thread per block
  extern __shared__ __align__(16) uint16_t fsm[];
  auto Kbuf = [&](int bb) { return fsm + bb * (kFlashK + kFlashV); };  // buffer bb: K, then transposed V
  auto Vbuf = [&](int bb) { return fsm + bb * (kFlashK + kFlashV) + kFlashK; };

  const int c = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int G = nq / nkv;
  int n = ctx_lens[b];
  n = n < 0 ? 0 : (n > max_ctx ? max_ctx : n);
  const int total = n + B;
  const int k0 = c * kpw, k1 = min(total, k0 + kpw);
  if (k0 >= total) return;  // workgroup-uniform
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, cc = lane & 15;

  bf16x8 qhf[DH / 32], qlf[DH / 32];  // this wave's query rows as Q^T fragments (loaded below)
  floatx4 oacc[DH / 16];
#pragma unroll
  for (int x = 0; x < DH / 16; ++x) oacc[x] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;  // of query row cc (the same in every g)

  // scores of one block against this wave's rows -> online softmax -> P V.
  // HILO: the block's keys are fp32 (hi parts in buffer 0, lo parts in buffer 1).
  // Only the 16-key tiles holding valid keys are multiplied (and only the
  // 32-key steps of P V that cover them): a short run, such as the block's own
  // 16 keys, skips three quarters of the products.
  auto fold = [&](int nvalid, bool hilo, int bb) {
    const uint16_t *Kh = Kbuf(bb), *Vh = Vbuf(bb), *Kl = Kbuf(1), *Vl = Vbuf(1);
    const int nkt = (nvalid + 15) / 16;  // workgroup-uniform
    floatx4 sacc[kFlashKB / 16];
#pragma unroll
    for (int t = 0; t < kFlashKB / 16; ++t) {
      sacc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
      if (t >= nkt) continue;
#pragma unroll
      for (int s = 0; s < DH / 32; ++s) {
        const bf16x8 kh = ld_frag(Kh + (16 * t + cc) * kFlashKP + 32 * s + 8 * g);
        if (hilo) {
          const bf16x8 kl = ld_frag(Kl + (16 * t + cc) * kFlashKP + 32 * s + 8 * g);
          sacc[t] = mfma3(kh, kl, qhf[s], qlf[s], sacc[t]);
        } else {
          sacc[t] = mfma2(kh, qhf[s], qlf[s], sacc[t]);
        }
      }
    }
    float mb = -INFINITY;
#pragma unroll
    for (int t = 0; t < kFlashKB / 16; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float v = 16 * t + 4 * g + e < nvalid ? sacc[t][e] * scale : -INFINITY;
        sacc[t][e] = v;
        mb = fmaxf(mb, v);
      }
    mb = fmaxf(mb, __shfl_xor(mb, 16, 64));
    mb = fmaxf(mb, __shfl_xor(mb, 32, 64));
    const float mn = fmaxf(m_run, mb);  // finite: every block has a valid key
    const float alpha = m_run == -INFINITY ? 0.f : expf(m_run - mn);
    m_run = mn;
    float p[kFlashKB / 16][4], lb = 0.f;
#pragma unroll
    for (int t = 0; t < kFlashKB / 16; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        p[t][e] = sacc[t][e] == -INFINITY ? 0.f : expf(sacc[t][e] - mn);
        lb += p[t][e];
      }
    lb += __shfl_xor(lb, 16, 64);
    lb += __shfl_xor(lb, 32, 64);
    l_run = alpha * l_run + lb;
    // output rows are 4 g + e: their factors come from lanes 4 g + e
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float ae = __shfl(alpha, 4 * g + e, 64);
#pragma unroll
      for (int x = 0; x < DH / 16; ++x) oacc[x][e] *= ae;
    }
#pragma unroll
    for (int u = 0; u < kFlashKB / 32; ++u) {
      if (2 * u >= nkt) break;  // (keys past the valid tiles have p = 0)
      const float f[8] = {p[2 * u][0], p[2 * u][1], p[2 * u][2], p[2 * u][3],
                          p[2 * u + 1][0], p[2 * u + 1][1], p[2 * u + 1][2], p[2 * u + 1][3]};
      bf16x8 ph, pl;
      split8(f, ph, pl);
#pragma unroll
      for (int x = 0; x < DH / 16; ++x) {
        const uint16_t *vr = Vh + (16 * x + cc) * kFlashVP + 32 * u + 4 * g;
        const uint2 v0 = *(const uint2 *)vr, v1 = *(const uint2 *)(vr + 16);
        const bf16x8 vh = __builtin_bit_cast(bf16x8, u32x4{v0.x, v0.y, v1.x, v1.y});
        if (hilo) {
          const uint16_t *vq = Vl + (16 * x + cc) * kFlashVP + 32 * u + 4 * g;
          const uint2 w0 = *(const uint2 *)vq, w1 = *(const uint2 *)(vq + 16);
          const bf16x8 vl = __builtin_bit_cast(bf16x8, u32x4{w0.x, w0.y, w1.x, w1.y});
          oacc[x] = mfma3(ph, pl, vh, vl, oacc[x]);
        } else {
          oacc[x] = mfma2b(ph, pl, vh, oacc[x]);
        }
      }
    }
  };

  // ---- context keys [k0, c1) from the cache, 64 per block
  const int c1 = min(k1, n);
  const int nblk = c1 > k0 ? (c1 - k0 + kFlashKB - 1) / kFlashKB : 0;
  // PD register stages: block i's loads land in stage i % PD
  u32x4 kr[PD][KCH], vr[PD][4];
  auto load_blk = [&](int i, int sg) {  // rows clamped into [k0, c1): every load valid and unconditional
    const int base = k0 + i * kFlashKB;
#pragma unroll
    for (int q = 0; q < KCH; ++q) {
      const int e = tid + q * T, key = min(base + e / (DH / 8), c1 - 1);
      kr[sg][q] = *(const u32x4 *)(ck + (((size_t)b * max_ctx + key) * nkv + kvh) * DH + 8 * (e % (DH / 8)));
    }
    const int u = min(tid, 255), dof = u % 16, kq = u / 16;  // V: 4 keys x 8 dims per thread (threads < 256)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int key = min(base + 4 * kq + r, c1 - 1);
      vr[sg][r] = *(const u32x4 *)(cv + (((size_t)b * max_ctx + key) * nkv + kvh) * DH + 8 * dof);
    }
  };
  auto store_blk = [&](int i, int bb, int sg) {  // keys past c1 get zero values (their scores are masked)
    const int base = k0 + i * kFlashKB;
#pragma unroll
    for (int q = 0; q < KCH; ++q) {
      const int e = tid + q * T;
      *(u32x4 *)(Kbuf(bb) + (e / (DH / 8)) * kFlashKP + 8 * (e % (DH / 8))) = kr[sg][q];
    }
    if (tid < 256) {
      const int dof = tid % 16, kq = tid / 16;
      u32x4 v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = base + 4 * kq + r < c1 ? vr[sg][r] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int w = 0; w < 4; ++w) {  // dims 8 dof + 2 w (low halves) and + 1 (high halves)
        uint16_t *row = Vbuf(bb) + (8 * dof + 2 * w) * kFlashVP + 4 * kq;
        *(uint2 *)row = make_uint2(pack_lo16(v[0][w], v[1][w]), pack_lo16(v[2][w], v[3][w]));
        *(uint2 *)(row + kFlashVP) = make_uint2(pack_hi16(v[0][w], v[1][w]), pack_hi16(v[2][w], v[3][w]));
      }
    }
  };
  if constexpr (PD == 1) {
    if (nblk > 0) load_blk(0, 0);
  } else if (nblk > 0) {  // (no context keys here: c1 - 1 may be no row at all)
#pragma unroll
    for (int sg = 0; sg < PD; ++sg) load_blk(sg, sg);  // clamped: issued even past the last block
  }
  // the block's own keys [max(k0, n), k1): this thread's first PB items (rows
  // kk = e / 32 of e = tid + T q, 4 dims each; every row of a 16-row block at
  // 256 threads) are loaded now, in flight with the context keys and Q, not
  // after the context blocks
  const int b0 = max(k0, n) - n, nb = k1 - n - b0;
  constexpr int PB = 2;
  float4 pk[PB], pv[PB];
  if (nb > 0) {
#pragma unroll
    for (int q = 0; q < PB; ++q) {
      const int e = tid + T * q, kk = e / (DH / 4), d4 = e % (DH / 4);
      const size_t row = (((size_t)b * B + b0 + min(kk, nb - 1)) * nkv + kvh) * DH;
      pk[q] = *(const float4 *)(Kb + row + 4 * d4);
      pv[q] = *(const float4 *)(Vb + row + 4 * d4);
    }
  }
  // this wave's query rows: Q^T fragments (dims 32 s + 8 g .. of row 16 wave + cc),
  // loaded after the first block's keys so the two memory round trips overlap
  {
    const int qi = 16 * wave + cc, qh = kvh * G + qi / B, j = qi % B;
    const float *qrow = Q + (((size_t)b * B + j) * nq + qh) * DH;
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) {
      const float4 a = *(const float4 *)(qrow + 32 * s + 8 * g), d = *(const float4 *)(qrow + 32 * s + 8 * g + 4);
      const float f[8] = {a.x, a.y, a.z, a.w, d.x, d.y, d.z, d.w};
      split8(f, qhf[s], qlf[s]);
    }
  }
  if constexpr (PD == 1) {
    for (int i = 0; i < nblk; ++i) {
      // buffer i & 1 was last read by block i - 2, which every wave finished
      // before the barrier of block i - 1
      store_blk(i, i & 1, 0);
      if (i + 1 < nblk) load_blk(i + 1, 0);
      __syncthreads();
      fold(min(kFlashKB, c1 - (k0 + i * kFlashKB)), false, i & 1);
    }
  } else {
    // PD blocks in flight while one is multiplied.  The loads are
    // unconditional (clamped rows past the last block), so every path through
    // the loop leaves the same loads outstanding and the compiler's waits for
    // a stage cover only that stage's loads, not the younger ones.
    for (int i = 0; i < nblk; i += PD) {
#pragma unroll
      for (int sg = 0; sg < PD; ++sg) {
        const int ii = i + sg;
        store_blk(ii, ii & 1, sg);
        load_blk(ii + PD, sg);
        __syncthreads();
        if (ii < nblk) fold(min(kFlashKB, c1 - (k0 + ii * kFlashKB)), false, ii & 1);  // workgroup-uniform
      }
    }
  }

  // ---- block keys [max(k0, n), k1): fp32, hi parts in buffer 0, lo in buffer 1
  if (nb > 0) {
    __syncthreads();  // both buffers free
    // rows the fold reads: the 32-key steps covering the nb keys (the rest stay unwritten)
    const int nrow = (nb + 31) / 32 * 32;
#pragma unroll
    for (int qi = 0; qi < kFlashKB * DH / 4 / T; ++qi) {
      const int e = tid + T * qi, kk = e / (DH / 4), d4 = e % (DH / 4);
      if (T * qi >= nrow * (DH / 4)) break;  // workgroup-uniform
      const size_t row = (((size_t)b * B + b0 + min(kk, nb - 1)) * nkv + kvh) * DH;
      const float4 kv = kk >= nb ? make_float4(0.f, 0.f, 0.f, 0.f) : qi < PB ? pk[qi < PB ? qi : 0]
                                                                             : *(const float4 *)(Kb + row + 4 * d4);
      const float4 vv = kk >= nb ? make_float4(0.f, 0.f, 0.f, 0.f) : qi < PB ? pv[qi < PB ? qi : 0]
                                                                             : *(const float4 *)(Vb + row + 4 * d4);
      uint2 hi, lo;
      split4(kv, hi, lo);
      *(uint2 *)(Kbuf(0) + kk * kFlashKP + 4 * d4) = hi;
      *(uint2 *)(Kbuf(1) + kk * kFlashKP + 4 * d4) = lo;
      split4(vv, hi, lo);
      const uint32_t hv[4] = {hi.x & 0xffffu, hi.x >> 16, hi.y & 0xffffu, hi.y >> 16};
      const uint32_t lv[4] = {lo.x & 0xffffu, lo.x >> 16, lo.y & 0xffffu, lo.y >> 16};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        Vbuf(0)[(4 * d4 + q) * kFlashVP + kk] = (uint16_t)hv[q];
        Vbuf(1)[(4 * d4 + q) * kFlashVP + kk] = (uint16_t)lv[q];
      }
    }
    __syncthreads();
    fold(nb, true, 0);
  }

  // ---- partial: unnormalised rows 4 g + e of this wave, and row cc's statistics
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int qi = 16 * wave + 4 * g + e, qh = kvh * G + qi / B, j = qi % B;
    float *dst = part + ((((size_t)b * nq + qh) * B + j) * nch + c) * (DH + 2);
#pragma unroll
    for (int x = 0; x < DH / 16; ++x) dst[16 * x + cc] = oacc[x][e];
  }
  if (g == 0) {
    const int qi = 16 * wave + cc, qh = kvh * G + qi / B, j = qi % B;
    float *dst = part + ((((size_t)b * nq + qh) * B + j) * nch + c) * (DH + 2);
    dst[DH] = m_run;
    dst[DH + 1] = l_run;
  }
}

// Merge the chunks of one (batch, query head, block row) with log-sum-exp
// weights; one wave per row.  The first CB chunks' output rows and maxima are
// loaded together with the statistics pass (at clamped chunk indices, so
// CB sized to the usual chunk count: 40 for the chunked kernel at one batch
// row, 8 or 24 after the one-pass kernel), so a context of up to CB chunks costs
// one memory round trip: lane c folds chunks c, c + 64, ... into a
// running (max, sum) pair, the wave combines the pairs, then the rows are
// weighted and summed in chunk order.
template <int DH, int CB = 40>
__global__ __launch_bounds__(256) void attn_combine_kernel(const float *__restrict__ part,
                                                           const int32_t *__restrict__ ctx_lens,
                                                           int max_ctx, float *__restrict__ O, int bs,
                                                           int B, int nq, int nch, int CH) {
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);  // (b, qh, j)
  if (item >= bs * nq * B) return;
  const int j = item % B, qh = (item / B) % nq, b = item / (B * nq);
  int n = ctx_lens[b];
  n = n < 0 ? 0 : (n > max_ctx ? max_ctx : n);
  const int nc = (n + B + CH - 1) / CH;
  const float *base = part + (((size_t)b * nq + qh) * B + j) * nch * (DH + 2);
  constexpr int PER = DH / 64;
  float w[CB], v[CB][PER];
#pragma unroll
  for (int u = 0; u < CB; ++u) {  // chunk u's max and this lane's output values (clamped, in flight together)
    const int cu = min(u, nc - 1);
    w[u] = base[cu * (DH + 2) + DH];
#pragma unroll
    for (int q = 0; q < PER; ++q) v[u][q] = base[cu * (DH + 2) + lane + 64 * q];
  }
  float M = -INFINITY, den = 0.f;
  for (int c = lane; c < nc; c += 64) {
    const float m = base[c * (DH + 2) + DH], l = base[c * (DH + 2) + DH + 1];
    const float Mn = fmaxf(M, m);
    den = (M == -INFINITY ? 0.f : den * expf(M - Mn)) + (m == -INFINITY ? 0.f : l * expf(m - Mn));
    M = Mn;
  }
  const float Mw = wave_max(M);
  den = wave_sum(M == -INFINITY ? 0.f : den * expf(M - Mw));
  M = Mw;
  float acc[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) acc[q] = 0.f;
#pragma unroll
  for (int u = 0; u < CB; ++u) {
    const float wu = u < nc ? expf(w[u] - M) : 0.f;
#pragma unroll
    for (int q = 0; q < PER; ++q) acc[q] = fmaf(wu, v[u][q], acc[q]);
  }
  for (int c0 = CB; c0 < nc; c0 += CB) {  // longer contexts: further batches
#pragma unroll
    for (int u = 0; u < CB; ++u) {
      const int cu = min(c0 + u, nc - 1);
      w[u] = base[cu * (DH + 2) + DH];
#pragma unroll
      for (int q = 0; q < PER; ++q) v[u][q] = base[cu * (DH + 2) + lane + 64 * q];
    }
#pragma unroll
    for (int u = 0; u < CB; ++u) {
      const float wu = c0 + u < nc ? expf(w[u] - M) : 0.f;
#pragma unroll
      for (int q = 0; q < PER; ++q) acc[q] = fmaf(wu, v[u][q], acc[q]);
    }
  }
  const float inv = 1.0f / den;
  float *dst = O + ((size_t)(b * B + j) * nq + qh) * DH;
#pragma unroll
  for (int q = 0; q < PER; ++q) dst[lane + 64 * q] = acc[q] * inv;
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

template <typename WT, int MAXP>
static void add_norm_t(const Dims &D, const float *x, float *x_out, int ldx, const float *parts, int np, size_t pstride,
                       const void *gain, float *y, int ldy, int rows, int width, bool skip_anchor,
                       const void *embed, const int32_t *anchor, int32_t *err, hipStream_t st,
                       const int32_t *tokens, uint32_t *hdr, int hdr_words) {
  // a few workgroups per row when there are few rows: a GEMM that reads rows
  // written by one workgroup each was measured ~5 us slower (QKV after the
  // attention RMSNorm at 16 rows), with two or more per row it is not
  int split = 1;
  while (split < 4 && rows * split < 64 && width % (2 * split * 8) == 0) split *= 2;
  hipLaunchKernelGGL((add_norm_kernel<WT, MAXP>), dim3(rows * split), dim3(512), 0, st, x, x_out, ldx, parts, np, pstride,
                     (const WT *)gain, y, ldy, width, D.eps, (int)skip_anchor, D.B - 1, (const WT *)embed, anchor,
                     D.mask_id, D.V, err, tokens, split, hdr, hdr_words);
}

void launch_add_norm(const Dims &D, const float *x, float *x_out, int ldx, const float *parts, int np, size_t pstride,
                     const void *gain, float *y, int ldy, int rows, int width, bool skip_anchor,
                     const void *embed, const int32_t *anchor, int32_t *err, hipStream_t st,
                     const int32_t *tokens, uint32_t *hdr, int hdr_words) {
  if (rows <= 0) return;
  if (np < 0 || np > 16) return;  // partial counts come from the GEMM planner (<= 16)
  if (D.bf16) {
    if (np <= 8) add_norm_t<bf16_t, 8>(D, x, x_out, ldx, parts, np, pstride, gain, y, ldy, rows, width, skip_anchor, embed, anchor, err, st, tokens, hdr, hdr_words);
    else add_norm_t<bf16_t, 16>(D, x, x_out, ldx, parts, np, pstride, gain, y, ldy, rows, width, skip_anchor, embed, anchor, err, st, tokens, hdr, hdr_words);
  } else {
    if (np <= 8) add_norm_t<float, 8>(D, x, x_out, ldx, parts, np, pstride, gain, y, ldy, rows, width, skip_anchor, embed, anchor, err, st, tokens, hdr, hdr_words);
    else add_norm_t<float, 16>(D, x, x_out, ldx, parts, np, pstride, gain, y, ldy, rows, width, skip_anchor, embed, anchor, err, st, tokens, hdr, hdr_words);
  }
}

template <typename WT, int MAXP>
static void qk_norm_rope_t(const Dims &D, const float *qkv, int np, size_t pstride, const void *q_norm,
                           const void *k_norm, const int32_t *ctx_lens, int max_ctx, float *Q, float *Kb, float *Vb,
                           int n_new, void *ck, void *cv, int32_t *err, hipStream_t st, const int32_t *pos_rows,
                           int n_store) {
  const int M = D.bs * D.B;
  const int items = M * (D.nq + 2 * D.nkv) + D.bs * n_new * 2 * D.nkv;
  hipLaunchKernelGGL((qk_norm_rope_kernel<WT, MAXP>), dim3((items + 3) / 4), dim3(256), 0, st, qkv, np, pstride,
                     (const WT *)q_norm, (const WT *)k_norm, ctx_lens, max_ctx, Q, Kb, Vb, M, D.B, D.nq, D.nkv, D.dh,
                     D.eps, D.inv_freq, n_new, (WT *)ck, (WT *)cv, err, pos_rows, n_store);
}

void launch_qk_norm_rope(const Dims &D, const float *qkv, int np, size_t pstride, const void *q_norm,
                         const void *k_norm, const int32_t *ctx_lens, int max_ctx, float *Q, float *Kb,
                         float *Vb, int n_new, void *ck, void *cv, int32_t *err, hipStream_t st,
                         const int32_t *pos_rows, int n_store) {
  if (np < 1 || np > 16) return;  // partial counts come from the GEMM planner (1..16)
  if (D.bf16) {
    if (np <= 8) qk_norm_rope_t<bf16_t, 8>(D, qkv, np, pstride, q_norm, k_norm, ctx_lens, max_ctx, Q, Kb, Vb, n_new, ck, cv, err, st, pos_rows, n_store);
    else qk_norm_rope_t<bf16_t, 16>(D, qkv, np, pstride, q_norm, k_norm, ctx_lens, max_ctx, Q, Kb, Vb, n_new, ck, cv, err, st, pos_rows, n_store);
  } else {
    if (np <= 8) qk_norm_rope_t<float, 8>(D, qkv, np, pstride, q_norm, k_norm, ctx_lens, max_ctx, Q, Kb, Vb, n_new, ck, cv, err, st, pos_rows, n_store);
    else qk_norm_rope_t<float, 16>(D, qkv, np, pstride, q_norm, k_norm, ctx_lens, max_ctx, Q, Kb, Vb, n_new, ck, cv, err, st, pos_rows, n_store);
  }
}

template <typename WT, int RPT, int CH, int DH, bool MASKED, bool MULTI>
static void attn_launch_mt(const Dims &D, const float *Q, const float *Kb, const float *Vb, const void *ck,
                           const void *cv, const int32_t *ctx_lens, int max_ctx, float *part, int nch,
                           const uint8_t *amask, int cpw, hipStream_t st) {
  constexpr int R = RPT * 16, DP = DH + 8, CP = CH + 8, KT = CH / 16;
  const size_t ps = R * CP <= CH * DP ? 0 : (size_t)R * CP;  // P over K where it fits
  const size_t lds = 2 * sizeof(uint16_t) * ((size_t)R * DP + (size_t)CH * DP + (size_t)DH * CP + ps) +
                     sizeof(float) * (2 * KT * R + (MULTI ? 3 * R : 0)) + (MASKED ? (size_t)64 * 64 : 0);
  const float scale = 1.0f / sqrtf((float)DH);
  const int nc = (max_ctx + D.B + CH - 1) / CH;
  const int ngrp = (nc + cpw - 1) / cpw;
  (void)hipFuncSetAttribute((const void *)attn_partial_kernel<WT, RPT, CH, DH, MASKED, MULTI>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hipLaunchKernelGGL((attn_partial_kernel<WT, RPT, CH, DH, MASKED, MULTI>), dim3(ngrp, D.nkv, D.bs),
                     dim3(kAttnThreads), lds, st, Q, Kb, Vb, (const WT *)ck, (const WT *)cv, ctx_lens, max_ctx, part,
                     D.B, D.nq, D.nkv, nch, scale, amask, cpw);
}

template <typename WT, int RPT, int CH, int DH, bool MASKED>
static void attn_launch_t(const Dims &D, const float *Q, const float *Kb, const float *Vb, const void *ck,
                          const void *cv, const int32_t *ctx_lens, int max_ctx, float *part, int nch,
                          const uint8_t *amask, int cpw, hipStream_t st) {
  if (cpw > 1)
    attn_launch_mt<WT, RPT, CH, DH, MASKED, true>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, cpw, st);
  else
    attn_launch_mt<WT, RPT, CH, DH, MASKED, false>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, 1, st);
}

template <typename WT, int DH, bool MASKED>
static bool attn_dispatch(const Dims &D, const float *Q, const float *Kb, const float *Vb, const void *ck,
                          const void *cv, const int32_t *ctx_lens, int max_ctx, float *part, int nch,
                          const uint8_t *amask, int cpw, hipStream_t st) {
  const int R = (D.nq / D.nkv) * D.B;
  switch (R) {
    case 32: attn_launch_t<WT, 2, 64, DH, MASKED>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, cpw, st); return true;
    case 64: attn_launch_t<WT, 4, 32, DH, MASKED>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, cpw, st); return true;
    case 128: attn_launch_t<WT, 8, 32, DH, MASKED>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, cpw, st); return true;
    default: return false;
  }
}

template <typename WT, int DH>
static bool attn_dispatch_m(const Dims &D, const float *Q, const float *Kb, const float *Vb, const void *ck,
                            const void *cv, const int32_t *ctx_lens, int max_ctx, float *part, int nch,
                            const uint8_t *amask, int cpw, hipStream_t st) {
  if (amask) return attn_dispatch<WT, DH, true>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, cpw, st);
  return attn_dispatch<WT, DH, false>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, nullptr, cpw, st);
}

// Chunks folded per workgroup: 1 (a workgroup per chunk, the lowest latency)
// unless the grid has enough (batch row, kv head) pairs that, doubling the
// chunks per workgroup, it still holds at least four workgroups per CU; then
// the partial outputs and the merge shrink by that factor.
static int attn_cu_count() {
  static int n_cu = 0;
  if (n_cu == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      n_cu = v;
    else
      n_cu = 256;
  }
  return n_cu;
}
static int attn_chunks_per_wg(const Dims &D, int nc) {
  const int n_cu = attn_cu_count();
  const long pairs = (long)D.bs * D.nkv;
  int cpw = 1;
  while (cpw < 64 && pairs * ((nc + 2 * cpw - 1) / (2 * cpw)) >= 4L * n_cu) cpw *= 2;
  return cpw;
}

bool attn_supported(int nq, int nkv, int B) {
  const int R = (nq / nkv) * B;
  return R == 32 || R == 64 || R == 128;
}

void launch_attention(const Dims &D, const float *Q, const float *Kb, const float *Vb,
                      const void *ck, const void *cv, const int32_t *ctx_lens, int max_ctx,
                      float *part, float *O, int32_t *err, hipStream_t st, const uint8_t *amask) {
  (void)err;
  // batched steps over a bf16 cache: the one-pass kernel, about two
  // workgroups per CU, each over a contiguous run of keys
  {
    const int G = D.nq / D.nkv, R = G * D.B;
    const long pairs = (long)D.bs * D.nkv;
    if (D.bf16 && D.dh == 128 && !amask && (R == 64 || R == 128) && pairs >= 8) {
      const int n_cu = attn_cu_count();
      const int nkeys = max_ctx + D.B;
      // workgroups resident per CU: two of 4 waves (LDS), one of 8 (registers)
      const long target = std::max(1L, (R == 64 ? 2L : 1L) * n_cu / pairs);
      const int kpw = (int)(((nkeys + target - 1) / target + kFlashKB - 1) / kFlashKB * kFlashKB);
      const int ngrp = (nkeys + kpw - 1) / kpw;
      const int nch = attn_nchunks(max_ctx, D.B);
      const float scale = 1.0f / sqrtf(128.f);
      const dim3 grid(ngrp, D.nkv, D.bs);
      if (R == 64) {
        (void)hipFuncSetAttribute((const void *)attn_flash_kernel<4, 1>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)kFlashLds);
        hipLaunchKernelGGL((attn_flash_kernel<4, 1>), grid, dim3(256), kFlashLds, st, Q, Kb, Vb, (const bf16_t *)ck,
                           (const bf16_t *)cv, ctx_lens, max_ctx, part, D.B, D.nq, D.nkv, nch, scale, kpw);
      } else {
        (void)hipFuncSetAttribute((const void *)attn_flash_kernel<8, 2>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)kFlashLds);
        hipLaunchKernelGGL((attn_flash_kernel<8, 2>), grid, dim3(512), kFlashLds, st, Q, Kb, Vb, (const bf16_t *)ck,
                           (const bf16_t *)cv, ctx_lens, max_ctx, part, D.B, D.nq, D.nkv, nch, scale, kpw);
      }
      const int items = D.bs * D.nq * D.B;
      if (ngrp <= 8)
        hipLaunchKernelGGL((attn_combine_kernel<128, 8>), dim3((items + 3) / 4), dim3(256), 0, st, part, ctx_lens,
                           max_ctx, O, D.bs, D.B, D.nq, nch, kpw);
      else if (ngrp <= 24)  // one batch row at a 1024-key context: 17 runs
        hipLaunchKernelGGL((attn_combine_kernel<128, 24>), dim3((items + 3) / 4), dim3(256), 0, st, part, ctx_lens,
                           max_ctx, O, D.bs, D.B, D.nq, nch, kpw);
      else
        hipLaunchKernelGGL((attn_combine_kernel<128, 40>), dim3((items + 3) / 4), dim3(256), 0, st, part, ctx_lens,
                           max_ctx, O, D.bs, D.B, D.nq, nch, kpw);
      return;
    }
  }
  const int nch = attn_nchunks(max_ctx, D.B);
  const int CH0 = attn_ch((D.nq / D.nkv) * D.B);
  const int cpw = attn_chunks_per_wg(D, (max_ctx + D.B + CH0 - 1) / CH0);
  const int CH = CH0 * cpw;  // keys per partial, as the merge sees them
  if (D.dh == 128) {
    if (D.bf16) attn_dispatch_m<bf16_t, 128>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, cpw, st);
    else attn_dispatch_m<float, 128>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, cpw, st);
  } else {
    if (D.bf16) attn_dispatch_m<bf16_t, 64>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, cpw, st);
    else attn_dispatch_m<float, 64>(D, Q, Kb, Vb, ck, cv, ctx_lens, max_ctx, part, nch, amask, cpw, st);
  }
  const int items = D.bs * D.nq * D.B;
  if (D.dh == 128)
    hipLaunchKernelGGL(attn_combine_kernel<128>, dim3((items + 3) / 4), dim3(256), 0, st, part, ctx_lens, max_ctx,
                       O, D.bs, D.B, D.nq, nch, CH);
  else
    hipLaunchKernelGGL(attn_combine_kernel<64>, dim3((items + 3) / 4), dim3(256), 0, st, part, ctx_lens, max_ctx,
                       O, D.bs, D.B, D.nq, nch, CH);
}

template <typename WT>
__global__ void to_f32_kernel(const WT *__restrict__ src, float *__restrict__ dst, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = to_f32(src[i]);
}
void launch_to_f32(const void *src, bool bf16, float *dst, size_t n, hipStream_t st) {
  if (n == 0) return;
  const unsigned blocks = (unsigned)((n + 255) / 256);
  if (bf16) hipLaunchKernelGGL(to_f32_kernel<bf16_t>, dim3(blocks), dim3(256), 0, st, (const bf16_t *)src, dst, n);
  else hipLaunchKernelGGL(to_f32_kernel<float>, dim3(blocks), dim3(256), 0, st, (const float *)src, dst, n);
}

template <typename WT>
__global__ void add_row_bias_kernel(float *__restrict__ Y, size_t n, int N, const WT *__restrict__ bias) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    Y[i] += to_f32(bias[i % N]);
}
void launch_add_row_bias(float *Y, size_t rows, int N, const void *bias, bool bf16, hipStream_t st) {
  const size_t n = rows * (size_t)N;
  const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 65536);
  if (bf16) hipLaunchKernelGGL(add_row_bias_kernel<bf16_t>, dim3(blocks), dim3(256), 0, st, Y, n, N, (const bf16_t *)bias);
  else hipLaunchKernelGGL(add_row_bias_kernel<float>, dim3(blocks), dim3(256), 0, st, Y, n, N, (const float *)bias);
}

// y[r][c] = sum over p < np of parts[p * pstride + r * width + c], four
// columns per thread (width % 4 == 0, pstride % 4 == 0, ldy % 4 == 0)
__global__ void sum_parts_kernel(const float *__restrict__ parts, int np, size_t pstride, int rows, int width,
                                 float *__restrict__ y, int ldy) {
  const int w4 = width / 4;
  const size_t n = (size_t)rows * w4;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const size_t r = i / w4, c = (i % w4) * 4;
    const float *src = parts + r * width + c;
    float4 acc = *(const float4 *)src;
    for (int p = 1; p < np; ++p) {
      const float4 v = *(const float4 *)(src + (size_t)p * pstride);
      acc.x += v.x;
      acc.y += v.y;
      acc.z += v.z;
      acc.w += v.w;
    }
    *(float4 *)(y + r * ldy + c) = acc;
  }
}
void launch_sum_parts(const float *parts, int np, size_t pstride, int rows, int width, float *y, int ldy,
                      hipStream_t st) {
  const size_t n = (size_t)rows * (width / 4);
  if (n == 0) return;
  const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(sum_parts_kernel, dim3(blocks), dim3(256), 0, st, parts, np, pstride, rows, width, y, ldy);
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
