// Matrix-core GEMM for wide activations (more than 64 rows: batched drafting,
// the training forward over many rows, the table build at model creation):
//   Y[m][n] = sum_k X[m][k] * W[n][k]      (X fp32 [M][K], W [N][K] bf16)
// with the packed weight tiles of the skinny kernel and the same hi + lo bf16
// split of the activations, so both kernels compute to the same precision.
//
// The activations are split once per projection (split_frag_kernel) into two
// bf16 planes, hi and lo, stored in MFMA fragment order: fragment (row block
// rb, k-step s) is 1 KB, lane l = 16 g + r holding the 8 k values
// 32 s + 8 g .. + 7 of row 16 rb + r.  A fragment is then one coalesced 1 KB
// wave load, exactly like a packed weight fragment, and no arithmetic is left
// between the loads and the products.
//
// A workgroup of 4 waves owns 8 weight tiles (128 output columns) and 16 row
// blocks (256 rows); wave w multiplies all 8 tiles by row blocks 4w .. 4w + 3,
// hi and lo: 64 products of 16x16x32 per k-step.  The weight fragments, used
// by all four waves, go through LDS (two 8 KB buffers, one barrier per
// k-step); the activation fragments, used by one wave only, are loaded
// straight into that wave's registers one k-step ahead.  Registers are capped
// at 256 per lane so that two workgroups share a CU: while one waits at its
// barrier, the other's products keep the matrix cores busy.  A K split
// (grid.y) writes partial outputs that the consumer adds in split order, as
// in the skinny kernel.
#include "common.h"
#include "kernels.h"
#include "mfma.h"

#include <algorithm>

namespace dk {

namespace {

constexpr int kWideTiles = 8;                    // weight tiles per workgroup (128 columns)
constexpr int kWideBlocks = 16;                  // row blocks per workgroup (256 rows)
constexpr int kWideRows = kWideBlocks * 16;
constexpr int kWideWaves = 4;                    // wave w: row blocks kWideTM * w ..
constexpr int kWideTM = kWideBlocks / kWideWaves;
constexpr int kWideThreads = kWideWaves * 64;
constexpr int kWideWPW = kWideTiles / kWideWaves;  // weight fragments each wave stages: 2
static_assert(kWideTiles % kWideWaves == 0, "weight fragments must divide over the waves");

DEVI float silu_w(float x) { return x / (1.f + expf(-x)); }

// One thread per (row block, k-step, lane): 8 values of one row, split.
__global__ __launch_bounds__(256) void split_frag_kernel(const float *__restrict__ X, int ldx, int M, int KS,
                                                         u32x4 *__restrict__ Xf, int nrb) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)nrb * KS * 64) return;
  const int lane = (int)(idx & 63);
  const size_t rs = idx >> 6;
  const int s = (int)(rs % KS), rb = (int)(rs / KS);
  const int m = rb * 16 + (lane & 15), k0 = s * 32 + (lane >> 4) * 8;
  float f[8];
  if (m < M) {
    const float4 *p = (const float4 *)(X + (size_t)m * ldx + k0);
    const float4 a = p[0], b = p[1];
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
    f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = 0.f;
  }
  bf16x8 hi, lo;
  split8(f, hi, lo);
  Xf[((size_t)rb * KS + s) * 64 + lane] = __builtin_bit_cast(u32x4, hi);
  Xf[(((size_t)nrb + rb) * KS + s) * 64 + lane] = __builtin_bit_cast(u32x4, lo);
}

// two workgroups per CU (80 KB of LDS and at most 256 registers each), so one
// workgroup's products run while the other waits at its barrier
// Workgroup order (a 1-D grid, workgroup L on XCD L % 8): the workgroups of
// one (column group, K split) pair u, one per row group, are L = (8 c + mz) *
// ... such that they share L % 8 and are dispatched 8 apart, so the second row
// group finds the weight tiles in its XCD's L2 instead of reading them again.
struct WideMap {
  int groups, ksplit, mgroups;
};
DEVI bool wide_coords(const WideMap &mp, int L, int &grp, int &ky, int &mz) {
  const int x = L & 7, r = L >> 3;
  const int c = r / mp.mgroups;
  mz = r % mp.mgroups;
  const int u = c * 8 + x;
  grp = u % mp.groups;
  ky = u / mp.groups;
  return ky < mp.ksplit;
}

template <int EPI>
__global__ __launch_bounds__(kWideThreads) __attribute__((amdgpu_waves_per_eu(2))) void gemm_wide_kernel(GemmArgs a,
                                                                                                       int nrb,
                                                                                                       WideMap mp) {
  __shared__ u32x4 lw[2][kWideTiles][64];  // [buffer][weight tile][lane]

  int grp, ky, mz;
  if (!wide_coords(mp, (int)blockIdx.x, grp, ky, mz)) return;  // past the last pair (workgroup-uniform)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int KS = a.KS;
  const int spw = (KS + a.ksplit - 1) / a.ksplit;
  const int s0 = min(KS, ky * spw), s1 = min(KS, s0 + spw);

  // weight tiles grp * 8 + 2 * wave + q staged by this wave; this wave's row
  // blocks in the two planes.  Tiles and blocks past the end are clamped: they
  // only feed outputs that are never stored.
  const u32x4 *wsrc[kWideWPW];
#pragma unroll
  for (int q = 0; q < kWideWPW; ++q) {
    const int t = min(grp * kWideTiles + kWideWPW * wave + q, a.ntiles - 1);
    wsrc[q] = (const u32x4 *)a.P + (size_t)(a.tile0 + t) * KS * 64;
  }
  const u32x4 *xsrc[2 * kWideTM];
#pragma unroll
  for (int f = 0; f < 2 * kWideTM; ++f) {
    const int rb = min(mz * kWideBlocks + kWideTM * wave + f % kWideTM, nrb - 1);
    xsrc[f] = (const u32x4 *)a.xf + ((size_t)(f / kWideTM) * nrb + rb) * KS * 64;
  }

  floatx4 acc[kWideTiles][kWideTM];
#pragma unroll
  for (int i = 0; i < kWideTiles; ++i)
#pragma unroll
    for (int j = 0; j < kWideTM; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // weight fragments on their way to LDS, two k-steps ahead (slot = k-step
  // parity); activation fragments of even / odd k-steps, one k-step ahead
  u32x4 wr[2][kWideWPW];
  u32x4 xa[2 * kWideTM], xb[2 * kWideTM];
  auto issue_w = [&](int d, int s) {
    const int sc = min(s, s1 - 1);  // clamped: every load stays valid and unconditional
#pragma unroll
    for (int q = 0; q < kWideWPW; ++q) wr[d][q] = __builtin_nontemporal_load(wsrc[q] + (size_t)sc * 64 + lane);
  };
  auto issue_x = [&](int s, u32x4 (&x)[2 * kWideTM]) {
    const int sc = min(s, s1 - 1);
#pragma unroll
    for (int f = 0; f < 2 * kWideTM; ++f) x[f] = xsrc[f][(size_t)sc * 64 + lane];
  };
  auto stage = [&](int d) {
#pragma unroll
    for (int q = 0; q < kWideWPW; ++q) lw[d][kWideWPW * wave + q][lane] = wr[d][q];
  };
  auto compute = [&](int buf, const u32x4 (&x)[2 * kWideTM]) {
    // tile i + 1's weight fragment is read from LDS before tile i's products
    // (scheduling barriers keep that order), so the read's latency hides
    // behind them; left to itself the compiler read each pair of tiles just
    // before their products (the registers allow two fragments)
    u32x4 wn = lw[buf][0][lane];
#pragma unroll
    for (int i = 0; i < kWideTiles; ++i) {
      const bf16x8 w = __builtin_bit_cast(bf16x8, wn);
      if (i + 1 < kWideTiles) wn = lw[buf][i + 1][lane];
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < kWideTM; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, __builtin_bit_cast(bf16x8, x[j]), acc[i][j], 0, 0, 0);
#pragma unroll
      for (int j = 0; j < kWideTM; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, __builtin_bit_cast(bf16x8, x[kWideTM + j]), acc[i][j],
                                                            0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  if (s0 < s1) {
    // k-step s0 + i: weights in slot and LDS buffer i & 1, activations in xa
    // (even i) or xb (odd i).  Each step stages its weights, issues the
    // weights of step i + 2 and the activations of step i + 1, passes the
    // barrier and multiplies.  A buffer is rewritten only after the barrier
    // that every wave passes once it has finished its products on it.  An odd
    // step past the end (odd count) stages a copy of the last step and skips
    // its products (a workgroup-uniform branch).  The prologue's loads go out
    // in order (no reordering across the scheduling barriers), so the waits
    // in the loop leave the later loads in flight.
    issue_w(0, s0);
    __builtin_amdgcn_sched_barrier(0);
    issue_x(s0, xa);
    __builtin_amdgcn_sched_barrier(0);
    issue_w(1, s0 + 1);
    __builtin_amdgcn_sched_barrier(0);
    const int nsteps = s1 - s0;
    for (int i0 = 0; i0 < nsteps; i0 += 2) {
      stage(0);
      issue_w(0, s0 + i0 + 2);
      issue_x(s0 + i0 + 1, xb);
      __syncthreads();
      compute(0, xa);
      stage(1);
      issue_w(1, s0 + i0 + 3);
      issue_x(s0 + i0 + 2, xa);
      __syncthreads();
      if (i0 + 1 < nsteps) compute(1, xb);
    }
  }

  float *Y = a.Y + (size_t)ky * a.ysplit;
  const int mbase = mz * kWideRows;
#pragma unroll
  for (int i = 0; i < kWideTiles; ++i) {
    const int tile = grp * kWideTiles + i;
    if (EPI == EPI_SWIGLU) {
      // packed tiles come in (gate, up) pairs; tile parity equals i's parity
      if ((i & 1) || tile + 1 >= a.ntiles) continue;
      const int col = (tile / 2) * 16 + 4 * (lane >> 4);
#pragma unroll
      for (int j = 0; j < kWideTM; ++j) {
        const int m = mbase + (wave * kWideTM + j) * 16 + (lane & 15);
        if (m >= a.M) continue;
        float *y = Y + (size_t)m * a.ldy + col;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (col + e < a.N) y[e] = silu_w(acc[i][j][e]) * acc[i + (i + 1 < kWideTiles ? 1 : 0)][j][e];
      }
    } else {
      if (tile >= a.ntiles) continue;
      const int n = tile * 16 + 4 * (lane >> 4);
#pragma unroll
      for (int j = 0; j < kWideTM; ++j) {
        const int m = mbase + (wave * kWideTM + j) * 16 + (lane & 15);
        if (m >= a.M) continue;
        float *y = Y + (size_t)m * a.ldy + n;
        if (n + 4 <= a.N && (a.ldy & 3) == 0) {
          *(floatx4 *)y = acc[i][j];
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (n + e < a.N) y[e] = acc[i][j][e];
        }
      }
    }
  }
}

}  // namespace

GemmPlan plan_gemm_wide(int ntiles, int KS, int M, int epi, int n_cu, int max_split) {
  GemmPlan p;
  p.wide = 1;
  p.MT = 0;
  p.WPT = 1;
  p.kcm = 1;
  p.nw = 8;
  p.pgrid = 0;
  p.groups = (ntiles + kWideTiles - 1) / kWideTiles;
  p.mgroups = (M + kWideRows - 1) / kWideRows;
  // K split (power of two, at least 8 k-steps per split) by a cost model in
  // k-step units of the busiest CU: rounds of workgroup pairs times (k-steps per
  // split + ~8 of pipeline fill and epilogue), plus the partial outputs
  // written and read back (a k-step moves ~40 KB per workgroup).  SwiGLU,
  // nonlinear in the sum, is never split.
  p.ksplit = 1;
  if (epi == EPI_STORE) {
    const long wgs = (long)p.groups * p.mgroups;
    double best = 1e300;
    for (int ks = 1; ks <= max_split && KS / ks >= 8; ks *= 2) {
      const double rounds = (double)((wgs * ks + 2 * n_cu - 1) / (2 * n_cu));  // two workgroups per CU
      const double part = ks > 1 ? 2.0 * ks * (double)M * ntiles * 16 * 4 / n_cu / 40960.0 : 0.0;
      const double cost = rounds * ((KS + ks - 1) / ks + 8) + part;
      if (cost < best * 0.999) {
        best = cost;
        p.ksplit = ks;
      }
    }
  }
  return p;
}

size_t gemm_wide_scratch_bytes(int M, int K) {
  const size_t nrb = (size_t)(M + 15) / 16, KS = (size_t)(K + 31) / 32;
  return 2 * nrb * KS * 1024;
}

bool launch_gemm_wide(int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  // the activation loads assume whole k-steps (K = 32 KS) and at least one row;
  // the model's config checks guarantee both for every projection
  if (a.K != a.KS * 32 || a.M <= 0 || a.ldx < a.K || !a.xf) return false;
  const int nrb = (a.M + 15) / 16;
  const size_t items = (size_t)nrb * a.KS * 64;
  hipLaunchKernelGGL(split_frag_kernel, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, st, a.X, a.ldx, a.M, a.KS,
                     (u32x4 *)a.xf, nrb);
  const WideMap mp{p.groups, p.ksplit, p.mgroups};
  const long pairs = (long)p.groups * p.ksplit;
  const dim3 grid((unsigned)((pairs + 7) / 8 * 8 * p.mgroups));
  if (epi == EPI_SWIGLU) hipLaunchKernelGGL(gemm_wide_kernel<EPI_SWIGLU>, grid, dim3(kWideThreads), 0, st, a, nrb, mp);
  else hipLaunchKernelGGL(gemm_wide_kernel<EPI_STORE>, grid, dim3(kWideThreads), 0, st, a, nrb, mp);
  return true;
}

}  // namespace dk
