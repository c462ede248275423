// Weight-streaming matrix-core GEMM for skinny activations:
//   Y[m][n] = sum_k X[m][k] * W[n][k]      (X fp32 [M][K], W [N][K] bf16 or fp32)
// as used by every projection of the draft step (QKV, O, gate/up, down, LM
// head, W1's H half, context K/V).  M is small (16 rows per batch row of the
// block), so the kernel is bound by streaming W from HBM once.
//
// Packed weight layout (built once at model creation): W is cut into tiles of
// 16 rows; tile t is stored as KS consecutive 1 KB blocks, block s holding,
// for lane l = 16*g + r of a wave, the 16 bytes W[16t + r][s*KSTEP + g*EPL ..
// + EPL-1] (EPL = 8 bf16 or 4 fp32; KSTEP = 4*EPL).  A wave's fragment load is
// therefore one contiguous, fully coalesced 1 KB read, and it is directly the
// A operand of v_mfma_f32_16x16x32_bf16 (or four v_mfma_f32_16x16x4_f32).
//
// bf16 weights meet fp32 activations split into hi + lo bf16 parts (two MFMAs
// per fragment; products are exact in fp32), so the GEMM keeps fp32 accuracy.
//
// Work split: a workgroup of 4 waves owns T consecutive tiles and one of
// `ksplit` K-ranges; its 4 waves split that range again.  Partial tiles are
// summed in LDS in wave order, and across workgroups through a workspace in
// K-range order by whichever workgroup finishes last — the sum order never
// depends on timing, so results are bitwise reproducible.
#include "common.h"
#include "kernels.h"

namespace dk {

template <typename WT> struct Frag;
template <> struct Frag<bf16_t> {
  static constexpr int EPL = 8, KSTEP = 32;
};
template <> struct Frag<float> {
  static constexpr int EPL = 4, KSTEP = 16;
};

template <typename WT>
__global__ void pack_kernel(const WT *__restrict__ W, int N, int K, int ldw, WT *__restrict__ P,
                            int NT, int KS, int tile_mul, int tile_off) {
  constexpr int EPL = Frag<WT>::EPL, KSTEP = Frag<WT>::KSTEP;
  size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t total = (size_t)NT * KS * 64;
  if (idx >= total) return;
  int lane = (int)(idx & 63);
  size_t ts = idx >> 6;
  int s = (int)(ts % KS);
  int t = (int)(ts / KS);
  int r = lane & 15, g = lane >> 4;
  int n = 16 * t + r;
  int k0 = s * KSTEP + g * EPL;
  WT vals[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    int k = k0 + e;
    if (n < N && k < K) vals[e] = W[(size_t)n * ldw + k];
    else {
      WT z;
      __builtin_memset(&z, 0, sizeof(z));
      vals[e] = z;
    }
  }
  size_t dst_tile = (size_t)t * tile_mul + tile_off;
  WT *dst = P + ((dst_tile * KS + s) * 64 + lane) * EPL;
  *(u32x4 *)dst = *(u32x4 *)vals;
}

// Load this lane's activation fragment (EPL consecutive k of row m), zero
// outside [0, M) x [0, K).
template <int EPL>
DEVI void load_x(const float *__restrict__ X, int ldx, int M, int K, int m, int k0, float *out) {
  if (m < M && k0 + EPL <= K) {
    const float4 *p = (const float4 *)(X + (size_t)m * ldx + k0);
#pragma unroll
    for (int q = 0; q < EPL / 4; ++q) {
      float4 v = p[q];
      out[4 * q + 0] = v.x;
      out[4 * q + 1] = v.y;
      out[4 * q + 2] = v.z;
      out[4 * q + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < EPL; ++e) out[e] = (m < M && k0 + e < K) ? X[(size_t)m * ldx + k0 + e] : 0.f;
  }
}

template <typename WT, int T, int MT>
struct Mac;

template <int T, int MT>
struct Mac<bf16_t, T, MT> {
  DEVI static void step(const u32x4 (&w)[T], const float (&x)[MT][8], floatx4 (&acc)[T][MT]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      bf16x8 hi, lo;
      split8(x[mt], hi, lo);
#pragma unroll
      for (int i = 0; i < T; ++i) {
        bf16x8 a = __builtin_bit_cast(bf16x8, w[i]);
        acc[i][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, hi, acc[i][mt], 0, 0, 0);
        acc[i][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, lo, acc[i][mt], 0, 0, 0);
      }
    }
  }
};

template <int T, int MT>
struct Mac<float, T, MT> {
  DEVI static void step(const u32x4 (&w)[T], const float (&x)[MT][4], floatx4 (&acc)[T][MT]) {
#pragma unroll
    for (int i = 0; i < T; ++i) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float a = __uint_as_float(w[i][e]);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          acc[i][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, x[mt][e], acc[i][mt], 0, 0, 0);
      }
    }
  }
};

DEVI float silu_f(float x) { return x / (1.f + expf(-x)); }

template <typename WT, int T, int MT, int EPI, int U>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a) {
  constexpr int EPL = Frag<WT>::EPL, KSTEP = Frag<WT>::KSTEP;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, r = lane & 15;
  const int grp = blockIdx.x, ky = blockIdx.y, mz = blockIdx.z;
  const int KS = a.KS;

  const int nw = a.ksplit * 4;
  const int per = (KS + nw - 1) / nw;
  const int s0 = (ky * 4 + wave) * per;
  const int s1 = min(KS, s0 + per);

  floatx4 acc[T][MT];
#pragma unroll
  for (int i = 0; i < T; ++i)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[i][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  const u32x4 *__restrict__ Pv = (const u32x4 *)a.P;
  size_t tbase[T];
  bool tval[T];
#pragma unroll
  for (int i = 0; i < T; ++i) {
    int t = grp * T + i;
    tval[i] = t < a.ntiles;
    tbase[i] = ((size_t)(a.tile0 + (tval[i] ? t : 0)) * KS) * 64 + lane;
  }
  int mrow[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) mrow[mt] = (mz * MT + mt) * 16 + r;

  int s = s0;
  for (; s + U <= s1; s += U) {
    u32x4 w[U][T];
    float x[U][MT][EPL];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < T; ++i)
        w[u][i] = tval[i] ? __builtin_nontemporal_load(&Pv[tbase[i] + (size_t)(s + u) * 64])
                          : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        load_x<EPL>(a.X, a.ldx, a.M, a.K, mrow[mt], (s + u) * KSTEP + g * EPL, x[u][mt]);
#pragma unroll
    for (int u = 0; u < U; ++u) Mac<WT, T, MT>::step(w[u], x[u], acc);
  }
  for (; s < s1; ++s) {
    u32x4 w[T];
    float x[MT][EPL];
#pragma unroll
    for (int i = 0; i < T; ++i)
      w[i] = tval[i] ? __builtin_nontemporal_load(&Pv[tbase[i] + (size_t)s * 64]) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) load_x<EPL>(a.X, a.ldx, a.M, a.K, mrow[mt], s * KSTEP + g * EPL, x[mt]);
    Mac<WT, T, MT>::step(w, x, acc);
  }

  // ---- reduce the 4 waves' partial tiles in LDS (fixed wave order)
  __shared__ floatx4 red[4][T][MT][64];
  __shared__ int s_last;
#pragma unroll
  for (int i = 0; i < T; ++i)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) red[wave][i][mt][lane] = acc[i][mt];
  __syncthreads();

  constexpr int ITEMS = T * MT * 64;
  const int Mpad = gridDim.z * MT * 16;
  const int ncols = a.ntiles * 16;  // columns covered by the launch (partials)
  for (int it = threadIdx.x; it < ITEMS; it += 256) {
    const int l = it & 63, mt = (it >> 6) % MT, i = (it >> 6) / MT;
    floatx4 v = red[0][i][mt][l];
#pragma unroll
    for (int wv = 1; wv < 4; ++wv) v += red[wv][i][mt][l];
    red[0][i][mt][l] = v;
    if (a.ksplit > 1) {
      const int m = (mz * MT + mt) * 16 + (l & 15);
      const int n = (grp * T + i) * 16 + 4 * (l >> 4);
      if (grp * T + i < a.ntiles)
        *(floatx4 *)(a.part + ((size_t)ky * Mpad + m) * ncols + n) = v;
    }
  }
  if (a.ksplit > 1) {
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
      int *tk = a.tickets + (size_t)blockIdx.z * gridDim.x + grp;
      int prev = atomicAdd(tk, 1);
      s_last = (prev == a.ksplit - 1);
      if (s_last) atomicExch(tk, 0);  // ready for the next launch
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
  } else {
    __syncthreads();
  }

  // ---- epilogue
  if (EPI == EPI_SWIGLU) {
    // tiles come in (gate, up) pairs; output column = 16*pair + 4g + e
    constexpr int PAIRS = T / 2;
    for (int it = threadIdx.x; it < PAIRS * MT * 64; it += 256) {
      const int l = it & 63, mt = (it >> 6) % MT, q = (it >> 6) / MT;
      const int m = (mz * MT + mt) * 16 + (l & 15);
      const int tg = grp * T + 2 * q;
      if (m >= a.M || tg + 1 >= a.ntiles) continue;
      floatx4 gv, uv;
      if (a.ksplit > 1) {
        gv = floatx4{0.f, 0.f, 0.f, 0.f};
        uv = gv;
        const int n = tg * 16 + 4 * (l >> 4);
        for (int kz = 0; kz < a.ksplit; ++kz) {
          const float *row = a.part + ((size_t)kz * Mpad + m) * ncols;
          gv += *(const floatx4 *)(row + n);
          uv += *(const floatx4 *)(row + n + 16);
        }
      } else {
        gv = red[0][2 * q][mt][l];
        uv = red[0][2 * q + 1][mt][l];
      }
      const int col = (tg / 2) * 16 + 4 * (l >> 4);
      float *y = a.Y + (size_t)m * a.ldy + col;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (col + e < a.N) y[e] = silu_f(gv[e]) * uv[e];
    }
    return;
  }
  for (int it = threadIdx.x; it < ITEMS; it += 256) {
    const int l = it & 63, mt = (it >> 6) % MT, i = (it >> 6) / MT;
    const int m = (mz * MT + mt) * 16 + (l & 15);
    const int t = grp * T + i;
    if (m >= a.M || t >= a.ntiles) continue;
    const int n = t * 16 + 4 * (l >> 4);
    floatx4 v;
    if (a.ksplit > 1) {
      v = floatx4{0.f, 0.f, 0.f, 0.f};
      for (int kz = 0; kz < a.ksplit; ++kz) v += *(const floatx4 *)(a.part + ((size_t)kz * Mpad + m) * ncols + n);
    } else {
      v = red[0][i][mt][l];
    }
    float *y = a.Y + (size_t)m * a.ldy + n;
    if (n + 4 <= a.N && ((a.ldy & 3) == 0)) {
      if (EPI == EPI_ADD) {
        floatx4 o = *(floatx4 *)y;
        *(floatx4 *)y = o + v;
      } else {
        *(floatx4 *)y = v;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < a.N) {
          if (EPI == EPI_ADD) y[e] += v[e];
          else y[e] = v[e];
        }
    }
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
GemmPlan plan_gemm(int ntiles, int KS, int M, int epi, int n_cu) {
  GemmPlan p;
  p.MT = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  p.T = (epi == EPI_SWIGLU) ? 2 : (ntiles >= 2 ? 2 : 1);
  p.groups = (ntiles + p.T - 1) / p.T;
  p.mgroups = (M + 16 * p.MT - 1) / (16 * p.MT);
  const int target = 2 * n_cu;  // workgroups wanted in flight
  int ks = 1;
  const int base = p.groups * p.mgroups;
  while (base * ks < target && KS / ((ks + 1) * 4) >= 8) ++ks;
  p.ksplit = ks;
  p.part_floats = ks > 1 ? (size_t)ks * p.mgroups * p.MT * 16 * ntiles * 16 : 0;
  p.tickets = ks > 1 ? (size_t)p.groups * p.mgroups : 0;
  return p;
}

template <typename WT, int T, int MT, int EPI>
static void launch_t(const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  dim3 grid(p.groups, p.ksplit, p.mgroups);
  hipLaunchKernelGGL((gemm_kernel<WT, T, MT, EPI, 4>), grid, dim3(256), 0, st, a);
}

template <typename WT, int T, int MT>
static void launch_epi(int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  if (epi == EPI_STORE) launch_t<WT, T, MT, EPI_STORE>(a, p, st);
  else if (epi == EPI_ADD) launch_t<WT, T, MT, EPI_ADD>(a, p, st);
  else launch_t<WT, 2, MT, EPI_SWIGLU>(a, p, st);
}

template <typename WT>
static void launch_w(int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  if (p.T == 1) {
    if (p.MT == 1) launch_epi<WT, 1, 1>(epi, a, p, st);
    else if (p.MT == 2) launch_epi<WT, 1, 2>(epi, a, p, st);
    else launch_epi<WT, 1, 4>(epi, a, p, st);
  } else {
    if (p.MT == 1) launch_epi<WT, 2, 1>(epi, a, p, st);
    else if (p.MT == 2) launch_epi<WT, 2, 2>(epi, a, p, st);
    else launch_epi<WT, 2, 4>(epi, a, p, st);
  }
}

void launch_gemm(bool bf16, int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  if (bf16) launch_w<bf16_t>(epi, a, p, st);
  else launch_w<float>(epi, a, p, st);
}

void launch_pack(bool bf16, const void *W, int N, int K, int ldw, void *P, int NT, int KS,
                 int tile_mul, int tile_off, hipStream_t st) {
  size_t total = (size_t)NT * KS * 64;
  unsigned blocks = (unsigned)((total + 255) / 256);
  if (bf16)
    hipLaunchKernelGGL(pack_kernel<bf16_t>, dim3(blocks), dim3(256), 0, st, (const bf16_t *)W, N, K, ldw,
                       (bf16_t *)P, NT, KS, tile_mul, tile_off);
  else
    hipLaunchKernelGGL(pack_kernel<float>, dim3(blocks), dim3(256), 0, st, (const float *)W, N, K, ldw,
                       (float *)P, NT, KS, tile_mul, tile_off);
}

}  // namespace dk
