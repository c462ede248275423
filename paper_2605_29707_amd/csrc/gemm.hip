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
// Work split: a workgroup of 8 (or 6) waves owns one tile per wave and a
// range of K chunks of KCM k-steps (16/MT, or 8/MT: half the registers, two
// workgroups per CU, finer K splits).  The activations of a chunk are staged
// once per workgroup into LDS, already split into hi/lo fragments, and shared
// by all its waves; weight fragments of the next chunk are in flight while the
// current chunk is multiplied.  Activations load before weights, at clamped
// addresses, so the in-order vector-memory counter never makes a wave wait for
// the weights it just prefetched.  When K is split across workgroups (ksplit > 1) each
// split writes its own partial output and the consuming kernel adds the
// partials in split order: no workgroup ever waits on another, and the sums
// are bitwise reproducible.  Grids larger than the device (the LM head: 1189
// groups of 8 tiles) run as one workgroup per CU that owns several groups and
// multiplies each staged activation chunk into all of them, with a single
// pipeline, which saves the pipeline fill of every further workgroup and all
// but one staging of each chunk.
#include "common.h"
#include "kernels.h"
#include "mfma.h"

#include <algorithm>
#include <type_traits>

namespace dk {

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


DEVI float silu_f(float x) { return x / (1.f + expf(-x)); }

// X fragment of (k-step s, m-tile mt, lane): EPL consecutive k of row m, zero
// outside [0, M) x [0, K).  The load itself is always issued at a clamped,
// valid address (K is a multiple of EPL), so the count of outstanding vector
// loads stays static.
template <int EPL>
DEVI void load_xfrag(const float *__restrict__ X, int ldx, int M, int K, int m, int k0, float4 (&v)[EPL / 4]) {
  const bool ok = m < M && k0 + EPL <= K;
  const int mc = m < M ? m : M - 1;
  const int kc = k0 + EPL <= K ? k0 : K - EPL;
  const float4 *p = (const float4 *)(X + (size_t)mc * ldx + kc);
  // `ok` enters as an opaque all-ones / zero mask ANDed into the loaded bits:
  // every lane then needs its load, so the compiler cannot sink the load into
  // a branch on `ok` (a branch whose join drains every load in flight), and
  // masked lanes get exact zeros whatever the clamped row holds
  uint32_t mask = ok ? 0xffffffffu : 0u;
  __asm__ volatile("" : "+v"(mask));
#pragma unroll
  for (int q = 0; q < EPL / 4; ++q) {
    const float4 t = p[q];
    v[q] = make_float4(__uint_as_float(__float_as_uint(t.x) & mask), __uint_as_float(__float_as_uint(t.y) & mask),
                       __uint_as_float(__float_as_uint(t.z) & mask), __uint_as_float(__float_as_uint(t.w) & mask));
  }
}

// load_xfrag in two parts: the load (clamped address) and the lane's mask,
// applied later by mask_xfrag (so that nothing needs the loaded values before
// the caller wants them)
template <int EPL>
DEVI uint32_t load_xfrag_raw(const float *__restrict__ X, int ldx, int M, int K, int m, int k0,
                             float4 (&v)[EPL / 4]) {
  const bool ok = m < M && k0 + EPL <= K;
  const int mc = m < M ? m : M - 1;
  const int kc = k0 + EPL <= K ? k0 : K - EPL;
  const float4 *p = (const float4 *)(X + (size_t)mc * ldx + kc);
#pragma unroll
  for (int q = 0; q < EPL / 4; ++q) v[q] = p[q];
  uint32_t mask = ok ? 0xffffffffu : 0u;
  __asm__ volatile("" : "+v"(mask));
  return mask;
}
template <int EPL>
DEVI void mask_xfrag(float4 (&v)[EPL / 4], uint32_t mask) {
#pragma unroll
  for (int q = 0; q < EPL / 4; ++q)
    v[q] = make_float4(__uint_as_float(__float_as_uint(v[q].x) & mask), __uint_as_float(__float_as_uint(v[q].y) & mask),
                       __uint_as_float(__float_as_uint(v[q].z) & mask), __uint_as_float(__float_as_uint(v[q].w) & mask));
}

// EPI_RESID, after this workgroup's partial went out (device-scope stores):
// wait for the stores, take a ticket of the column group, and if it is the
// group's last split, form res_in + partial_0 + ... + partial_{ksplit-1} (split
// order: the result does not depend on which split came last) over the group's
// TW * 16 columns and every row, write it and its gain-scaled copy, and the
// row sums of its squares.  `sq` is LDS scratch of `nsq` floats.
template <typename WT, int TW>
DEVI void resid_epilogue(const GemmArgs &a, int grp, float *sq, int nsq) {
  __shared__ int s_last;
  __builtin_amdgcn_s_waitcnt(0);  // this thread's partial stores are complete
  __syncthreads();                // ... and every thread's
  if (threadIdx.x == 0)
    s_last = __hip_atomic_fetch_add(a.res_tickets + grp, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
             (unsigned)(a.ksplit - 1);
  __syncthreads();
  if (!s_last) return;
  const int c0 = grp * TW * 16;
  constexpr int PR = TW * 4;  // float4 items per row of the group
  const WT *gain = (const WT *)a.res_gain;
  for (int it = threadIdx.x; it < a.M * PR; it += blockDim.x) {
    const int m = it / PR, n = c0 + 4 * (it % PR);
    float ss = 0.f;
    if (n < a.N) {  // N is a multiple of 4
      const size_t at = (size_t)m * a.ldy + n;
      float4 v = *(const float4 *)(a.res_in + at);
      for (int sp = 0; sp < a.ksplit; ++sp) {
        const unsigned long long *p = (const unsigned long long *)(a.Y + sp * a.ysplit + at);
        const unsigned long long p0 = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const unsigned long long p1 = __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        v.x += __uint_as_float((uint32_t)p0);
        v.y += __uint_as_float((uint32_t)(p0 >> 32));
        v.z += __uint_as_float((uint32_t)p1);
        v.w += __uint_as_float((uint32_t)(p1 >> 32));
      }
      *(float4 *)(a.res_out + at) = v;
      *(float4 *)(a.res_xg + at) = make_float4(v.x * to_f32(gain[n]), v.y * to_f32(gain[n + 1]),
                                               v.z * to_f32(gain[n + 2]), v.w * to_f32(gain[n + 3]));
      ss = fmaf(v.x, v.x, ss);
      ss = fmaf(v.y, v.y, ss);
      ss = fmaf(v.z, v.z, ss);
      ss = fmaf(v.w, v.w, ss);
    }
    if (it < nsq) sq[it] = ss;
  }
  __syncthreads();
  if ((int)threadIdx.x < a.M) {  // row sums in column order
    float t = 0.f;
    for (int i = 0; i < PR; ++i) t += sq[threadIdx.x * PR + i];
    a.res_ssq[(size_t)grp * a.M + threadIdx.x] = t;
  }
}

template <typename WT, int MT, int WPT, int EPI, int KCM, int kWaves>
__global__ __launch_bounds__(kWaves * 64) void gemm_kernel(GemmArgs a) {
  constexpr int EPL = Frag<WT>::EPL, KSTEP = Frag<WT>::KSTEP;
  constexpr int XF = XStage<WT>::XF;
  constexpr int KW = KCM / WPT;          // k-steps per wave per chunk
  constexpr int TW = kWaves / WPT;       // tiles per workgroup
  constexpr int ITEMS = KCM * MT * 64;   // staged fragments per chunk
  constexpr int IPT = (ITEMS + kWaves * 64 - 1) / (kWaves * 64);

  __shared__ u32x4 xs[2][KCM][MT][64][XF];
  __shared__ floatx4 xch[kWaves][MT][64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = blockIdx.x, ky = blockIdx.y, mz = blockIdx.z;
  const int KS = a.KS;
  const int nch = (KS + KCM - 1) / KCM;
  const int cpw = (nch + a.ksplit - 1) / a.ksplit;
  const int c0 = min(nch, ky * cpw), c1 = min(nch, c0 + cpw);
  const int tile = grp * TW + wave / WPT;
  const bool tvalid = tile < a.ntiles;
  const int ksub = (wave % WPT) * KW;    // this wave's first k-step within a chunk
  const u32x4 *__restrict__ Pv =
      (const u32x4 *)a.P + ((size_t)(a.tile0 + (tvalid ? tile : 0)) * KS) * 64 + lane;
  const int mbase = mz * MT * 16;

  floatx4 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // deferred RMSNorm: the producer's per-group sums of squares of this
  // workgroup's rows, one load per thread into LDS now (in flight with the
  // first chunks), summed by the epilogue (after the loop's barriers)
  __shared__ float rs_part[kNormGroups * MT * 16];
  const int rs_ng = min(a.rs_ng, kNormGroups);  // (the host keeps rs_ng within kNormGroups)
  const int rs_n = a.rs_ssq ? rs_ng * MT * 16 : 0;  // [group][row of the m-group]
  for (int e = tid; e < rs_n; e += kWaves * 64) {
    const int g = e / (MT * 16), m = min(mbase + e % (MT * 16), a.M - 1);
    rs_part[e] = a.rs_ssq[(size_t)g * a.M + m];
  }

  auto load_w = [&](u32x4 (&w)[KW], int c) {
#pragma unroll
    for (int u = 0; u < KW; ++u) {
      const int s = min(c * KCM + ksub + u, KS - 1);
      w[u] = __builtin_nontemporal_load(Pv + (size_t)s * 64);
    }
  };
  auto load_x = [&](float4 (&v)[IPT][EPL / 4], int c) {
#pragma unroll
    for (int q = 0; q < IPT; ++q) {
      const int it = min(tid + q * kWaves * 64, ITEMS - 1);  // clamped: loads stay unconditional
      const int l = it & 63, mt = (it >> 6) % MT, s = (it >> 6) / MT;
      const int m = mbase + mt * 16 + (l & 15);
      const int k0 = (c * KCM + s) * KSTEP + (l >> 4) * EPL;
      load_xfrag<EPL>(a.X, a.ldx, a.M, a.K, m, k0, v[q]);
    }
  };
  auto store_x = [&](const float4 (&v)[IPT][EPL / 4], int buf) {
#pragma unroll
    for (int q = 0; q < IPT; ++q) {
      const int it = tid + q * kWaves * 64;
      if (ITEMS % (kWaves * 64) != 0 && it >= ITEMS) continue;
      const int l = it & 63, mt = (it >> 6) % MT, s = (it >> 6) / MT;
      XStage<WT>::put(&xs[buf][s][mt][l][0], v[q]);
    }
  };
  auto mac = [&](const u32x4 &w, int buf, int u) {
    u32x4 xf[MT * XF];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int f = 0; f < XF; ++f) xf[mt * XF + f] = xs[buf][ksub + u][mt][lane][f];
    Mac2<WT, MT>::step(w, xf, acc);
  };
  auto compute = [&](const u32x4 (&w)[KW], int c, int buf) {
    if (c * KCM + ksub + KW <= KS) {  // every step of the chunk is in range: no per-step test
#pragma unroll
      for (int u = 0; u < KW; ++u) mac(w[u], buf, u);
    } else {
#pragma unroll
      for (int u = 0; u < KW; ++u)
        if (c * KCM + ksub + u < KS) mac(w[u], buf, u);
      consume(w);
    }
  };

  // Weights and activations one chunk ahead, in straight-line code over three
  // chunks at a time (a fresh pipeline fill per three chunks).  Measured
  // against loops that keep one or two chunks in flight throughout, on the
  // gate/up shape, this is the fastest: the compiler's waits in straight-line
  // code are exact, while a loop's are taken over every path it cannot rule
  // out (a path that leaves a load unconsumed makes it drain the prefetch).
  if (c0 < c1) {
    u32x4 wa[KW], wb[KW];
    float4 xr[IPT][EPL / 4];
    for (int cb = c0; cb < c1; cb += 3) {
      const int n = min(3, c1 - cb);
      if (cb > c0) __syncthreads();  // every wave is done reading the previous three's buffers
      load_x(xr, cb);
      load_w(wa, cb);
      store_x(xr, 0);
      __syncthreads();
      if (n == 1) {
        compute(wa, cb, 0);
      } else {
        load_x(xr, cb + 1);
        load_w(wb, cb + 1);
        compute(wa, cb, 0);
        store_x(xr, 1);
        __syncthreads();
        if (n == 2) {
          compute(wb, cb + 1, 1);
        } else {
          load_x(xr, cb + 2);
          load_w(wa, cb + 2);
          compute(wb, cb + 1, 1);
          store_x(xr, 0);
          __syncthreads();
          compute(wa, cb + 2, 0);
        }
      }
    }
  }

  if (a.rs_ssq) {  // (the loop's barriers have made rs_part visible)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      float t = 0.f;
      for (int g = 0; g < rs_ng; ++g) t += rs_part[g * MT * 16 + mt * 16 + (lane & 15)];
      const float rs = 1.0f / sqrtf(t / (float)a.rs_d + a.rs_eps);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[mt][e] *= rs;
    }
  }

  // waves sharing a tile: fold into the first one
  if (WPT > 1) {
    if (wave % WPT) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) xch[wave][mt][lane] = acc[mt];
    }
    __syncthreads();
    if (wave % WPT == 0) {
#pragma unroll
      for (int q = 1; q < WPT; ++q)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] += xch[wave + q][mt][lane];
    }
  }

  float *Y = a.Y + (size_t)ky * a.ysplit;
  if (EPI == EPI_SWIGLU) {
    // tiles come in (gate, up) pairs held by owner waves w and w + WPT
    __syncthreads();
    const bool owner = wave % WPT == 0;
    const bool up = ((wave / WPT) & 1) == 1;
    if (owner && up) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) xch[wave][mt][lane] = acc[mt];
    }
    __syncthreads();
    if (!owner || up || tile + 1 >= a.ntiles) return;
    const int col = (tile / 2) * 16 + 4 * (lane >> 4);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = mbase + mt * 16 + (lane & 15);
      if (m >= a.M) continue;
      const floatx4 uv = xch[wave + WPT][mt][lane];
      float *y = Y + (size_t)m * a.ldy + col;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (col + e < a.N) y[e] = silu_f(acc[mt][e]) * uv[e];
    }
    return;
  }
  if (EPI == EPI_RESID) {
    // this split's partial, written through to the device coherence point
    if (wave % WPT == 0 && tvalid) {
      const int n = tile * 16 + 4 * (lane >> 4);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mbase + mt * 16 + (lane & 15);
        if (m >= a.M) continue;
        unsigned long long *y = (unsigned long long *)(Y + (size_t)m * a.ldy + n);  // n + 4 <= N, ldy % 4 == 0
        __hip_atomic_store(y, ((unsigned long long)__float_as_uint(acc[mt][1]) << 32) | __float_as_uint(acc[mt][0]),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(y + 1, ((unsigned long long)__float_as_uint(acc[mt][3]) << 32) | __float_as_uint(acc[mt][2]),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    resid_epilogue<WT, kWaves / WPT>(a, grp, (float *)&xch[0][0][0], sizeof(xch) / sizeof(float));
    return;
  }
  if (wave % WPT || !tvalid) return;
  const int n = tile * 16 + 4 * (lane >> 4);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mbase + mt * 16 + (lane & 15);
    if (m >= a.M) continue;
    float *y = Y + (size_t)m * a.ldy + n;
    if (n + 4 <= a.N && ((a.ldy & 3) == 0)) {
      *(floatx4 *)y = acc[mt];
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < a.N) y[e] = acc[mt][e];
    }
  }
}

// Most column groups one workgroup of the persistent variant below owns.
constexpr int kStreamMaxGroups = 8;

// Stored-output variant for grids larger than the device (the LM head: 1189
// groups of 8 tiles): pgrid workgroups, workgroup b owning groups b, b + pgrid,
// ... (at most GR of them).  The loop runs chunk-outer: a chunk of activations
// is staged once and multiplied into the tiles of every owned group (GR sets of
// sums), so the staging and its barrier come once per chunk instead of once per
// group and chunk.  One pipeline covers every item (chunk, group), weights one
// item ahead, so a workgroup never refills it.  Each tile still sums its
// k-steps in ascending order: its results equal the other kernels'.
// The host launches it for whole chunks only, an even number of them and no K
// split, so the loop body has no branch at all: a workgroup owning fewer than
// GR groups multiplies its last group's weights again (loaded from L2) into
// sums it never stores.
template <typename WT, int MT, int KCM, int kWaves, int GR>
__global__ __launch_bounds__(kWaves * 64) void gemm_stream_kernel(GemmArgs a, int ngroups) {
  constexpr int EPL = Frag<WT>::EPL, KSTEP = Frag<WT>::KSTEP;
  constexpr int XF = XStage<WT>::XF;
  constexpr int KW = KCM;
  constexpr int ITEMS = KCM * MT * 64;
  constexpr int IPT = (ITEMS + kWaves * 64 - 1) / (kWaves * 64);
  __shared__ u32x4 xs[2][KCM][MT][64][XF];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int mz = blockIdx.z;
  const int KS = a.KS;
  const int nch = KS / KCM;  // whole chunks, an even number of them
  // owned groups (the host keeps every workgroup's count within GR)
  const int mine = (int)blockIdx.x < ngroups ? min(GR, (ngroups - 1 - (int)blockIdx.x) / (int)gridDim.x + 1) : 0;
  if (mine <= 0 || nch <= 0) return;
  const int mbase = mz * MT * 16;

  auto tile_of = [&](int j) { return ((int)blockIdx.x + j * (int)gridDim.x) * kWaves + wave; };
  // item (c, j): chunk c of owned group j.  A group past the owned ones loads
  // the first KW KB of the activations instead (in L2: every chunk's staging
  // reads them), never multiplied; a streamed weight chunk loaded again would
  // come from HBM, its lines being the first the cache gives up.
  auto load_w = [&](u32x4 (&w)[KW], int c, int j) {
    c = min(c, nch - 1);
    const int t = min(tile_of(min(j, mine - 1)), a.ntiles - 1);
    const u32x4 *Pv = j < mine ? (const u32x4 *)a.P + ((size_t)(a.tile0 + t) * KS + (size_t)c * KCM) * 64 + lane
                               : (const u32x4 *)a.X + lane;
#pragma unroll
    for (int u = 0; u < KW; ++u) w[u] = __builtin_nontemporal_load(Pv + u * 64);
  };
  uint32_t xm[IPT];  // the staged fragments' lane masks (zero outside [0, M) x [0, K))
  auto load_x = [&](float4 (&v)[IPT][EPL / 4], int c) {
    c = min(c, nch - 1);
#pragma unroll
    for (int q = 0; q < IPT; ++q) {
      const int i2 = min(tid + q * kWaves * 64, ITEMS - 1);
      const int l = i2 & 63, mt = (i2 >> 6) % MT, s = (i2 >> 6) / MT;
      const int m = mbase + mt * 16 + (l & 15);
      const int k0 = (c * KCM + s) * KSTEP + (l >> 4) * EPL;
      xm[q] = load_xfrag_raw<EPL>(a.X, a.ldx, a.M, a.K, m, k0, v[q]);
    }
  };
  auto store_x = [&](float4 (&v)[IPT][EPL / 4], int buf) {
#pragma unroll
    for (int q = 0; q < IPT; ++q) {
      const int i2 = tid + q * kWaves * 64;
      if (ITEMS % (kWaves * 64) != 0 && i2 >= ITEMS) continue;
      const int l = i2 & 63, mt = (i2 >> 6) % MT, s = (i2 >> 6) / MT;
      mask_xfrag<EPL>(v[q], xm[q]);
      XStage<WT>::put(&xs[buf][s][mt][l][0], v[q]);
    }
  };
  floatx4 acc[GR][MT];
#pragma unroll
  for (int j = 0; j < GR; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](floatx4 (&ac)[MT], const u32x4 (&w)[KW], int buf) {
#pragma unroll
    for (int u = 0; u < KW; ++u) {
      u32x4 xf[MT * XF];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int f = 0; f < XF; ++f) xf[mt * XF + f] = xs[buf][u][mt][lane][f];
      Mac2<WT, MT>::step(w[u], xf, ac);
    }
  };

  u32x4 wa[KW], wb[KW];
  float4 xr[IPT][EPL / 4];
  load_x(xr, 0);
  load_w(wa, 0, 0);
  store_x(xr, 0);
  __syncthreads();
  // chunks in pairs, c in LDS buffer 0 and c + 1 in buffer 1; the 2 GR items
  // of a pair are unrolled, even ones holding their weights in wa and odd ones
  // in wb.  The next chunk's activations load with a chunk's first item and
  // are staged after its last.  The last pair is a copy that loads nothing past
  // the range (a load of the last item again would come from HBM).
  auto pair = [&](int c, auto last) {
    constexpr bool kLast = decltype(last)::value;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int cc = c + h;
      const bool final_chunk = kLast && h == 1;
#pragma unroll
      for (int j = 0; j < GR; ++j) {
        // each item issues the next item's loads, then multiplies: the
        // scheduler keeps that order (sunk into the products, the prefetch
        // would be waited for by the very next item)
        __builtin_amdgcn_sched_barrier(0);
        if (j == 0 && !final_chunk) load_x(xr, cc + 1);
        const int nc = j + 1 < GR ? cc : cc + 1, nj = j + 1 < GR ? j + 1 : 0;
        const bool even = ((h * GR + j) & 1) == 0;
        if (!(final_chunk && j == GR - 1)) {
          if (even) load_w(wb, nc, nj);
          else load_w(wa, nc, nj);
        }
        __builtin_amdgcn_sched_barrier(0);
        if (even) compute(acc[j], wa, h);
        else compute(acc[j], wb, h);
        if (j == GR - 1 && !final_chunk) {
          __builtin_amdgcn_sched_barrier(0);
          pin(xr);
          store_x(xr, h ^ 1);
          __syncthreads();
        }
      }
    }
  };
  for (int c = 0; c + 2 < nch; c += 2) pair(c, std::false_type{});
  pair(nch - 2, std::true_type{});

#pragma unroll
  for (int j = 0; j < GR; ++j) {
    const int tile = tile_of(j);
    if (j >= mine || tile >= a.ntiles) continue;
    const int n = tile * 16 + 4 * (lane >> 4);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = mbase + mt * 16 + (lane & 15);
      if (m >= a.M) continue;
      float *y = a.Y + (size_t)m * a.ldy + n;
      if (n + 4 <= a.N && ((a.ldy & 3) == 0)) {
        *(floatx4 *)y = acc[j][mt];
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n + e < a.N) y[e] = acc[j][mt][e];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
GemmPlan plan_gemm(int ntiles, int KS, int M, int epi, int n_cu, int max_split) {
  GemmPlan p;
  p.pgrid = 0;
  p.MT = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  p.mgroups = (M + 16 * p.MT - 1) / (16 * p.MT);
  p.WPT = 1;
  p.groups = (ntiles + 7) / 8;
  p.ksplit = 1;
  p.kcm = 16 / p.MT;
  (void)epi;
  // Cost model (bytes through the busiest CU): workgroups land evenly over the
  // CUs, so a CU streams ceil(W / n_cu) workgroups' weight slices; K-split
  // partial outputs are written and read back once (spread over all CUs).
  // Candidates: chunks of 16/MT or 8/MT k-steps, any split dividing the chunk count.
  // Workgroups of 8 or 6 waves (a wave per tile; 6 lets 1536 gate/up tiles
  // fill 256 CUs exactly).
  const int N = ntiles * 16;
  double best = 1e300;
  p.nw = 8;
  for (int nw : {8, 6}) {
    const int groups = (ntiles + nw - 1) / nw;
    for (int kcm : {16 / p.MT, 8 / p.MT}) {
      const int nch = (KS + kcm - 1) / kcm;
      for (int s = 1; s <= std::min(nch, max_split); ++s) {
        if (nch % s) continue;
        const long W = (long)groups * p.mgroups * s;
        const double wg_bytes = (double)nw * (nch / s) * kcm * 1024.0;
        const double cost = (double)((W + n_cu - 1) / n_cu) * wg_bytes +
                            (s > 1 ? 2.0 * s * (double)M * N * 4.0 / n_cu : 0.0);
        if (cost < best * 0.999) {
          best = cost;
          p.ksplit = s;
          p.kcm = kcm;
          p.nw = nw;
          p.groups = groups;
        }
      }
    }
  }
  // more workgroups than CUs (8 waves and 16-k-step chunks fill a CU): a
  // grid of at most n_cu workgroups loops over the groups instead, sized so
  // that every workgroup takes the same number of groups (or one fewer) and
  // rounded up to a multiple of 8 (the XCDs)
  p.pgrid = 0;
  const long wgs = (long)p.groups * p.ksplit * p.mgroups;
  if (epi == EPI_STORE && p.nw == 8 && p.kcm == 16 / p.MT && wgs > n_cu) {
    const int per = std::max(1, n_cu / (p.ksplit * p.mgroups));  // CUs per (split, m-group)
    const int rounds = (p.groups + per - 1) / per;
    const int pg = std::min(per, ((p.groups + rounds - 1) / rounds + 7) / 8 * 8);
    // (the persistent kernel takes whole chunks, an even number of them, and no K split)
    const bool shape_ok = p.ksplit == 1 && KS % p.kcm == 0 && (KS / p.kcm) % 2 == 0;
    if (shape_ok && pg < p.groups && (p.groups + pg - 1) / pg <= kStreamMaxGroups) p.pgrid = pg;
  }
  return p;
}

// the persistent kernel for a plan with pgrid > 0
template <typename WT, int MT, int KCM>
static void launch_stream(const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  // groups per workgroup: 2..6 or 8 (7 runs the 8 instance, its last group idle)
  const int gr = (p.groups + p.pgrid - 1) / p.pgrid;
  const dim3 grid(p.pgrid, p.ksplit, p.mgroups), block(8 * 64);
  if (gr <= 2) hipLaunchKernelGGL((gemm_stream_kernel<WT, MT, KCM, 8, 2>), grid, block, 0, st, a, p.groups);
  else if (gr == 3) hipLaunchKernelGGL((gemm_stream_kernel<WT, MT, KCM, 8, 3>), grid, block, 0, st, a, p.groups);
  else if (gr == 4) hipLaunchKernelGGL((gemm_stream_kernel<WT, MT, KCM, 8, 4>), grid, block, 0, st, a, p.groups);
  else if (gr == 5) hipLaunchKernelGGL((gemm_stream_kernel<WT, MT, KCM, 8, 5>), grid, block, 0, st, a, p.groups);
  else if (gr == 6) hipLaunchKernelGGL((gemm_stream_kernel<WT, MT, KCM, 8, 6>), grid, block, 0, st, a, p.groups);
  else hipLaunchKernelGGL((gemm_stream_kernel<WT, MT, KCM, 8, kStreamMaxGroups>), grid, block, 0, st, a, p.groups);
}

template <typename WT, int MT, int EPI, int KCM>
static void launch_t(const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  if constexpr (EPI == EPI_STORE && KCM == 16 / MT) {  // (the only shapes the planner makes persistent)
    // (the persistent kernel's idle groups read the first KCM KB of X)
    const bool x_covers = (size_t)(a.M - 1) * a.ldx + a.K >= (size_t)KCM * 256;
    if (p.pgrid > 0 && p.nw == 8 && x_covers) {
      launch_stream<WT, MT, KCM>(a, p, st);
      return;
    }
  }
  dim3 grid(p.groups, p.ksplit, p.mgroups);
  if (p.nw == 6) hipLaunchKernelGGL((gemm_kernel<WT, MT, 1, EPI, KCM, 6>), grid, dim3(6 * 64), 0, st, a);
  else hipLaunchKernelGGL((gemm_kernel<WT, MT, 1, EPI, KCM, 8>), grid, dim3(8 * 64), 0, st, a);
}

template <typename WT, int MT>
static void launch_m(int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  constexpr int K1 = 16 / MT, K2 = 8 / MT;
  if (p.kcm == K2) {
    if (epi == EPI_SWIGLU) launch_t<WT, MT, EPI_SWIGLU, K2>(a, p, st);
    else if (epi == EPI_RESID) launch_t<WT, MT, EPI_RESID, K2>(a, p, st);
    else launch_t<WT, MT, EPI_STORE, K2>(a, p, st);
  } else {
    if (epi == EPI_SWIGLU) launch_t<WT, MT, EPI_SWIGLU, K1>(a, p, st);
    else if (epi == EPI_RESID) launch_t<WT, MT, EPI_RESID, K1>(a, p, st);
    else launch_t<WT, MT, EPI_STORE, K1>(a, p, st);
  }
}

template <typename WT>
static void launch_w(int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  if (p.MT == 1) launch_m<WT, 1>(epi, a, p, st);
  else if (p.MT == 2) launch_m<WT, 2>(epi, a, p, st);
  else launch_m<WT, 4>(epi, a, p, st);
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
