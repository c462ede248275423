// Domino-head rollout (Sec. 4.1.2 causal encoder and low-rank correction,
// Fig. 3 sequential rollout) as one persistent, cooperatively launched kernel.
//
// For draft position j = 1 .. B-1 (all batch rows together):
//   A  S_{j-1} = GRU(E[y_{j-1}], S_{j-2})      each workgroup owns a slice of
//      the d_s state indices (its W_ih / W_hh rows stay in LDS for the whole
//      rollout when they fit)
//   B  u = SiLU(W1[:, :d] H_j + W1[:, d:] S_{j-1})  (the H half is precomputed
//      for all j by a GEMM before the loop); each workgroup owns a slice of r
//   C  L_j = L_base_j + W2 u over the workgroup's vocabulary slice, then the
//      slice's top-beta under (value desc, id asc)
//   D  every workgroup merges all slices' top-beta lists (redundantly, so no
//      further barrier is needed) and takes y_j = top-1 (or the forced token)
// Grid barriers separate A|B, B|C and C|D.  Each barrier's spin is bounded; on
// timeout the kernel records DEV_BARRIER_TIMEOUT and every workgroup exits.
#include "common.h"
#include "kernels.h"

namespace dk {

constexpr unsigned kSpinLimit = 1u << 22;

struct Lds {
  int ipw, upw, tpw_max, rows_max;
  bool gru_lds;
  size_t gru_off, lv_off, u_off, ys_off, abort_off, total;
};

static Lds plan_lds(const Dims &D, int G, bool bf16) {
  Lds L;
  const int esz = bf16 ? 2 : 4;
  const int NT = (D.V + 15) / 16;
  L.ipw = (D.ds + G - 1) / G;
  L.upw = (D.r + G - 1) / G;
  L.tpw_max = (NT + G - 1) / G;
  L.rows_max = L.tpw_max * 16;
  size_t off = 0;
  L.lv_off = off;
  off += (size_t)D.bs * L.rows_max * 4;
  L.u_off = off;
  off += (size_t)D.bs * D.r * 4;
  L.ys_off = off;
  off += (size_t)D.bs * 4;
  L.abort_off = off;
  off += 16;
  off = (off + 15) & ~(size_t)15;
  const size_t gru = (size_t)L.ipw * 3 * (D.d + D.ds) * esz;
  const size_t budget = 150 * 1024;
  L.gru_lds = off + gru <= budget;
  L.gru_off = off;
  if (L.gru_lds) off += gru;
  L.total = off;
  return L;
}

template <typename WT>
struct HeadKernelArgs {
  HeadArgs h;
  Lds L;
};

// Bounded grid barrier.  Returns false if this or another workgroup gave up.
DEVI bool grid_sync(unsigned *bar, unsigned *abort_flag, unsigned target, int32_t *err,
                    volatile int *s_ok) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0) {
    int ok = 1;
    atomicAdd(bar, 1u);
    unsigned spins = 0;
    while (true) {
      const unsigned v = __hip_atomic_load(bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (v >= target) break;
      if (__hip_atomic_load(abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        ok = 0;
        break;
      }
      if (++spins > kSpinLimit) {
        raise_error(err, DEV_BARRIER_TIMEOUT);
        atomicExch(abort_flag, 1u);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    *s_ok = ok;
  }
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  return *s_ok != 0;
}

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

// Wave-level top-beta of `cnt` candidates; candidate c is produced by get(c).
// Lane 0 ends with the result in ov/oi (first beta entries valid).
template <typename Get>
DEVI void wave_select(Get get, int cnt, int beta, float (&ov)[8], int (&oi)[8]) {
  const int lane = threadIdx.x & 63;
  float lv[8];
  int li[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    lv[q] = -INFINITY;
    li[q] = INT_MAX;
  }
  for (int c = lane; c < cnt; c += 64) {
    float v;
    int id;
    get(c, v, id);
    if (id == INT_MAX) continue;
    list_insert(lv, li, order_val(v), id);
  }
  for (int k = 0; k < beta; ++k) {
    float bv = lv[0];
    int bi = li[0];
    wave_best(bv, bi);
    ov[k] = bv;
    oi[k] = bi;
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

template <typename WT>
DEVI float2 ld2(const WT *p);
template <>
DEVI float2 ld2<float>(const float *p) {
  return *(const float2 *)p;
}
template <>
DEVI float2 ld2<bf16_t>(const bf16_t *p) {
  const uint32_t u = *(const uint32_t *)p;
  return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
}

DEVI float sigm(float x) { return 1.f / (1.f + expf(-x)); }

template <typename WT>
__global__ __launch_bounds__(256) void head_kernel(HeadKernelArgs<WT> ka) {
  const HeadArgs &h = ka.h;
  const Lds &L = ka.L;
  const Dims &D = h.D;
  extern __shared__ __align__(16) unsigned char smem[];
  float *lv = (float *)(smem + L.lv_off);
  float *us = (float *)(smem + L.u_off);
  int *ys = (int *)(smem + L.ys_off);
  volatile int *s_ok = (volatile int *)(smem + L.abort_off);
  WT *gw = (WT *)(smem + L.gru_off);

  const int G = h.G, g = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bs = D.bs, d = D.d, ds = D.ds, r = D.r, V = D.V, depth = D.B - 1;
  const int beta = h.beta;
  const int kw = d + ds;
  const int i0 = min(ds, g * L.ipw), i1 = min(ds, i0 + L.ipw);
  const int k0 = min(r, g * L.upw), k1 = min(r, k0 + L.upw);
  const int NT = (V + 15) / 16;
  const int t0 = (int)((long long)g * NT / G), t1 = (int)((long long)(g + 1) * NT / G);
  const int row0 = t0 * 16, nrows = min(V, t1 * 16) - row0;
  unsigned *bar = h.barrier, *abort_flag = h.barrier + 1;
  unsigned nbar = 0;

  // GRU rows of this workgroup into LDS: local row (li*3 + q) = [W_ih | W_hh] of gate q, index i0+li
  const WT *w_ih = (const WT *)h.w_ih, *w_hh = (const WT *)h.w_hh;
  if (L.gru_lds) {
    const int nr = (i1 - i0) * 3;
    for (int e = tid; e < nr * kw; e += 256) {
      const int lr = e / kw, c = e % kw;
      const int i = i0 + lr / 3, q = lr % 3;
      gw[e] = c < d ? w_ih[(size_t)(q * ds + i) * d + c] : w_hh[(size_t)(q * ds + i) * ds + (c - d)];
    }
  }
  for (int b = tid; b < bs; b += 256) ys[b] = clamp_token(h.anchor[b], V, h.err);
  __syncthreads();

  const WT *embed = (const WT *)h.embed;
  const WT *b_ih = (const WT *)h.b_ih, *b_hh = (const WT *)h.b_hh;
  const WT *w1 = (const WT *)h.w1s_rows;
  constexpr int EPL = sizeof(WT) == 2 ? 8 : 4, KSTEP = 4 * EPL;
  const int KS = r / KSTEP;
  const u32x4 *w2p = (const u32x4 *)h.w2p;

  for (int j = 1; j <= depth; ++j) {
    const float *hprev = h.hbuf + (size_t)((j - 1) & 1) * bs * ds;
    float *hnext = h.hbuf + (size_t)(j & 1) * bs * ds;
    const bool first = (j == 1);

    // ---------------- A: GRU state slice
    for (int item = wave; item < (i1 - i0) * bs; item += 4) {
      const int li = item % (i1 - i0), b = item / (i1 - i0);
      const int i = i0 + li;
      const WT *e = embed + (size_t)ys[b] * d;
      const float *hp = hprev + (size_t)b * ds;
      float acc[6] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int c = 2 * lane; c < d; c += 128) {
        const float2 ev = ld2<WT>(e + c);
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          const float2 wv = L.gru_lds ? ld2<WT>(gw + (size_t)(li * 3 + q) * kw + c)
                                      : ld2<WT>(w_ih + (size_t)(q * ds + i) * d + c);
          acc[q] = fmaf(wv.x, ev.x, fmaf(wv.y, ev.y, acc[q]));
        }
      }
      if (!first) {
        for (int c = 2 * lane; c < ds; c += 128) {
          const float2 hv = *(const float2 *)(hp + c);
#pragma unroll
          for (int q = 0; q < 3; ++q) {
            const float2 wv = L.gru_lds ? ld2<WT>(gw + (size_t)(li * 3 + q) * kw + d + c)
                                        : ld2<WT>(w_hh + (size_t)(q * ds + i) * ds + c);
            acc[3 + q] = fmaf(wv.x, hv.x, fmaf(wv.y, hv.y, acc[3 + q]));
          }
        }
      }
#pragma unroll
      for (int q = 0; q < 6; ++q) acc[q] = wave_sum(acc[q]);
      if (lane == 0) {
        const float gir = acc[0] + to_f32(b_ih[i]), giz = acc[1] + to_f32(b_ih[ds + i]),
                    gin = acc[2] + to_f32(b_ih[2 * ds + i]);
        const float ghr = acc[3] + to_f32(b_hh[i]), ghz = acc[4] + to_f32(b_hh[ds + i]),
                    ghn = acc[5] + to_f32(b_hh[2 * ds + i]);
        const float rg = sigm(gir + ghr), zg = sigm(giz + ghz);
        const float ng = tanhf(gin + rg * ghn);
        const float hold = first ? 0.f : hp[i];
        const float hn = (1.f - zg) * ng + zg * hold;
        hnext[(size_t)b * ds + i] = hn;
        if (h.states) h.states[((size_t)b * depth + (j - 1)) * ds + i] = hn;
      }
    }
    if (!grid_sync(bar, abort_flag, (++nbar) * G, h.err, s_ok)) return;

    // ---------------- B: u slice
    for (int item = wave; item < (k1 - k0) * bs; item += 4) {
      const int lk = item % (k1 - k0), b = item / (k1 - k0);
      const int k = k0 + lk;
      const float *hn = hnext + (size_t)b * ds;
      const WT *wr = w1 + (size_t)k * (d + ds) + d;
      float acc = 0.f;
      for (int c = 2 * lane; c < ds; c += 128) {
        const float2 wv = ld2<WT>(wr + c);
        const float2 hv = *(const float2 *)(hn + c);
        acc = fmaf(wv.x, hv.x, fmaf(wv.y, hv.y, acc));
      }
      acc = wave_sum(acc);
      if (lane == 0) {
        const float x = h.P[((size_t)b * depth + (j - 1)) * r + k] + acc;
        h.ubuf[(size_t)b * r + k] = x / (1.f + expf(-x));
      }
    }
    if (!grid_sync(bar, abort_flag, (++nbar) * G, h.err, s_ok)) return;

    // ---------------- C: corrected logits of this slice
    for (int e = tid; e < bs * r; e += 256) us[e] = h.ubuf[e];
    __syncthreads();
    {
      const int gq = lane >> 4, rr = lane & 15;
      for (int t = t0 + wave; t < t1; t += 4) {
        u32x4 wf[16];
#pragma unroll
        for (int s = 0; s < 16; ++s)
          if (s < KS) wf[s] = w2p[((size_t)t * KS + s) * 64 + lane];
        const int n = t * 16 + rr;
        for (int b = 0; b < bs; ++b) {
          const float *ub = us + (size_t)b * r;
          float acc = 0.f;
#pragma unroll
          for (int s = 0; s < 16; ++s) {
            if (s < KS) {
              const float *uu = ub + s * KSTEP + gq * EPL;
              if (EPL == 8) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                  const uint32_t wv = wf[s][q];
                  acc = fmaf(__uint_as_float(wv << 16), uu[2 * q], acc);
                  acc = fmaf(__uint_as_float(wv & 0xffff0000u), uu[2 * q + 1], acc);
                }
              } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) acc = fmaf(__uint_as_float(wf[s][q]), uu[q], acc);
              }
            }
          }
          acc += __shfl_xor(acc, 16, 64);
          acc += __shfl_xor(acc, 32, 64);
          if (gq == 0 && n < V) {
            const float val = h.Lbase[((size_t)b * depth + (j - 1)) * V + n] + acc;
            lv[(size_t)b * L.rows_max + (n - row0)] = val;
            if (h.final_logits) h.final_logits[((size_t)b * depth + (j - 1)) * V + n] = val;
          }
        }
      }
    }
    __syncthreads();
    for (int b = wave; b < bs; b += 4) {
      float ov[8];
      int oi[8];
      const float *lb = lv + (size_t)b * L.rows_max;
      wave_select([&](int c, float &v, int &id) { v = lb[c]; id = row0 + c; }, nrows, beta, ov, oi);
      if (lane < beta) {
        float v = ov[0];
        int id = oi[0];
#pragma unroll
        for (int q = 1; q < 8; ++q)
          if (lane == q) {
            v = ov[q];
            id = oi[q];
          }
        h.pval[((size_t)b * G + g) * beta + lane] = v;
        h.pid[((size_t)b * G + g) * beta + lane] = id;
      }
    }
    if (!grid_sync(bar, abort_flag, (++nbar) * G, h.err, s_ok)) return;

    // ---------------- D: merge all slices, choose y_j
    for (int b = wave; b < bs; b += 4) {
      float ov[8];
      int oi[8];
      const float *pv = h.pval + (size_t)b * G * beta;
      const int32_t *pi = h.pid + (size_t)b * G * beta;
      wave_select([&](int c, float &v, int &id) { v = pv[c]; id = pi[c]; }, G * beta, beta, ov, oi);
      if (lane == 0) {
        int y = oi[0];
        if (h.forced) y = clamp_token(h.forced[(size_t)b * depth + (j - 1)], V, h.err);
        ys[b] = y;
        if (g == 0) {
          for (int q = 0; q < beta; ++q) {
            h.topk_ids[((size_t)b * depth + (j - 1)) * beta + q] = oi[q];
            h.topk_vals[((size_t)b * depth + (j - 1)) * beta + q] = ov[q];
          }
        }
      }
    }
    __syncthreads();
  }
}

int head_grid(const Dims &D, int n_cu, size_t *lds_bytes) {
  const int G = n_cu;
  Lds L = plan_lds(D, G, D.bf16);
  *lds_bytes = L.total;
  return G;
}

size_t head_exchange_floats(const Dims &D, int G, int beta) {
  // hbuf [2][bs][ds] + ubuf [bs][r] + pval/pid [bs][G][beta]
  return (size_t)2 * D.bs * D.ds + (size_t)D.bs * D.r + (size_t)2 * D.bs * G * beta;
}

template <typename WT>
static hipError_t launch_t(const HeadArgs &h, size_t lds_bytes, hipStream_t st) {
  HeadKernelArgs<WT> ka;
  ka.h = h;
  ka.L = plan_lds(h.D, h.G, h.D.bf16);
  if (ka.L.total != lds_bytes) return hipErrorInvalidValue;
  hipError_t e = hipFuncSetAttribute((const void *)head_kernel<WT>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds_bytes);
  if (e != hipSuccess) return e;
  void *args[] = {&ka};
  return hipLaunchCooperativeKernel((const void *)head_kernel<WT>, dim3(h.G), dim3(256), args,
                                    (unsigned)lds_bytes, st);
}

hipError_t launch_head(const HeadArgs &h, size_t lds_bytes, hipStream_t st) {
  if (h.D.bf16) return launch_t<bf16_t>(h, lds_bytes, st);
  return launch_t<float>(h, lds_bytes, st);
}

}  // namespace dk
