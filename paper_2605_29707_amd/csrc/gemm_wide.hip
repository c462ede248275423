// Matrix-core GEMM for wide activations (more than 64 rows: batched drafting,
// the training forward over many rows, the table build at model creation):
//   Y[m][n] = sum_k X[m][k] * W[n][k]      (X fp32 [M][K], W [N][K] bf16)
// with the packed weight tiles of the skinny kernel and the same hi + lo bf16
// split of the activations, so both kernels compute to the same precision.
//
// The skinny kernel gives each wave one 16-column weight tile against all rows
// of its m-group (at most 64), so above 64 rows it re-reads every weight tile
// once per m-group and feeds each staged activation fragment to a single
// tile.  Here a workgroup of 8 waves owns 8 weight tiles (128 output columns)
// and 256 rows: waves form a 2 (columns) x 4 (rows) grid, each wave multiplies
// 4 weight tiles by 4 row blocks (16 accumulators), so a weight byte leaves
// HBM once per 256 rows and every fragment read from LDS feeds 4 products.
//
// Per k-step the workgroup stages 8 KB of weights and 32 KB of activations
// (256 rows x 32 k, split into hi/lo fragments) into one of two LDS buffers;
// each thread keeps kWideDepth k-steps of loads in flight in registers, so
// the loads of later k-steps overlap the products of the current one.  A K
// split (grid.y) writes partial outputs that the consumer adds in split
// order, as in the skinny kernel.
#include "common.h"
#include "kernels.h"
#include "mfma.h"

#include <algorithm>

namespace dk {

namespace {

constexpr int kWideTN = 4, kWideTM = 4;          // tiles and row blocks per wave
constexpr int kWideWN = 2, kWideWM = 4;          // wave grid
constexpr int kWideTiles = kWideTN * kWideWN;    // 8 weight tiles per workgroup
constexpr int kWideBlocks = kWideTM * kWideWM;   // 16 row blocks of 16
constexpr int kWideRows = kWideBlocks * 16;      // 256 rows per workgroup
constexpr int kWideDepth = 4;                    // k-steps of loads in flight per thread
constexpr int kWideThreads = 512;

DEVI float silu_w(float x) { return x / (1.f + expf(-x)); }

// 8 consecutive k of row m from k0 (K is a multiple of 32, so k0 + 8 <= K).
// Rows past M read row M - 1 instead: they only feed output rows that are
// never stored, and the load stays unconditional, so the compiler can count
// the loads in flight instead of waiting for all of them.
DEVI void load_row8(const float *__restrict__ X, int ldx, int M, int m, int k0, float4 (&v)[2]) {
  const int mc = m < M ? m : M - 1;
  const float4 *p = (const float4 *)(X + (size_t)mc * ldx + k0);
  v[0] = p[0];
  v[1] = p[1];
}

template <int EPI>
__global__ __launch_bounds__(kWideThreads) void gemm_wide_kernel(GemmArgs a) {
  __shared__ u32x4 wsm[2][kWideTiles][64];
  __shared__ u32x4 xsm[2][kWideBlocks][2][64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave % kWideWN, wm = wave / kWideWN;
  const int grp = blockIdx.x, ky = blockIdx.y, mz = blockIdx.z;
  const int KS = a.KS;
  const int spw = (KS + a.ksplit - 1) / a.ksplit;
  const int s0 = min(KS, ky * spw), s1 = min(KS, s0 + spw);
  const int mbase = mz * kWideRows;

  // this thread's loads of a k-step: 16 bytes of weight tile `wave`, and 8 k
  // (k-group g) of rows rr and rr + 128
  const int wt = grp * kWideTiles + wave;
  const u32x4 *__restrict__ Pw =
      (const u32x4 *)a.P + (size_t)(a.tile0 + min(wt, a.ntiles - 1)) * KS * 64 + lane;
  const int g = tid & 3, rr = tid >> 2;

  floatx4 acc[kWideTN][kWideTM];
#pragma unroll
  for (int i = 0; i < kWideTN; ++i)
#pragma unroll
    for (int j = 0; j < kWideTM; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  u32x4 wr[kWideDepth];
  float4 xr[kWideDepth][2][2];
  auto issue = [&](int d, int s) {
    const int sc = min(s, s1 - 1);  // clamped: every load stays valid and unconditional
    wr[d] = __builtin_nontemporal_load(Pw + (size_t)sc * 64);
#pragma unroll
    for (int h = 0; h < 2; ++h) load_row8(a.X, a.ldx, a.M, mbase + rr + 128 * h, sc * 32 + g * 8, xr[d][h]);
  };
  auto stage = [&](int d, int buf, bool live) {
    // a k-step past the split's end is staged as zeros (a select on loaded
    // data, not a skipped load), so it adds nothing to the products
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    wsm[buf][wave][lane] = live ? wr[d] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = rr + 128 * h;
      u32x4 hl[2];
      const float4 xv[2] = {live ? xr[d][h][0] : z, live ? xr[d][h][1] : z};
      XStage<bf16_t>::put(hl, xv);
      const int l = (r & 15) + 16 * g;
      xsm[buf][r >> 4][0][l] = hl[0];
      xsm[buf][r >> 4][1][l] = hl[1];
    }
  };
  auto compute = [&](int buf) {
    bf16x8 xb[kWideTM][2];
#pragma unroll
    for (int j = 0; j < kWideTM; ++j) {
      xb[j][0] = __builtin_bit_cast(bf16x8, xsm[buf][wm * kWideTM + j][0][lane]);
      xb[j][1] = __builtin_bit_cast(bf16x8, xsm[buf][wm * kWideTM + j][1][lane]);
    }
#pragma unroll
    for (int i = 0; i < kWideTN; ++i) {
      const bf16x8 w = __builtin_bit_cast(bf16x8, wsm[buf][wn * kWideTN + i][lane]);
#pragma unroll
      for (int j = 0; j < kWideTM; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, xb[j][0], acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, xb[j][1], acc[i][j], 0, 0, 0);
      }
    }
  };

  if (s0 < s1) {
#pragma unroll
    for (int d = 0; d < kWideDepth; ++d) issue(d, s0 + d);
    // k-step s0 + i sits in ring slot i % depth and LDS buffer i & 1 (the
    // depth is even); the ring index is a compile-time constant inside the
    // unrolled body.  The loop runs whole rounds of the ring with no branch
    // inside (k-steps past the end are staged as zeros), so the compiler can
    // keep the later rounds' loads in flight across the loop's back edge.
    const int nsteps = s1 - s0;
    for (int i0 = 0; i0 < nsteps; i0 += kWideDepth) {
#pragma unroll
      for (int d = 0; d < kWideDepth; ++d) {
        stage(d, d & 1, i0 + d < nsteps);
        issue(d, s0 + i0 + d + kWideDepth);
        __syncthreads();
        compute(d & 1);
      }
    }
  }

  float *Y = a.Y + (size_t)ky * a.ysplit;
#pragma unroll
  for (int i = 0; i < kWideTN; ++i) {
    const int tile = grp * kWideTiles + wn * kWideTN + i;
    if (EPI == EPI_SWIGLU) {
      // packed tiles come in (gate, up) pairs; tile parity equals i's parity
      if ((i & 1) || tile + 1 >= a.ntiles) continue;
      const int col = (tile / 2) * 16 + 4 * (lane >> 4);
#pragma unroll
      for (int j = 0; j < kWideTM; ++j) {
        const int m = mbase + (wm * kWideTM + j) * 16 + (lane & 15);
        if (m >= a.M) continue;
        float *y = Y + (size_t)m * a.ldy + col;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (col + e < a.N) y[e] = silu_w(acc[i][j][e]) * acc[i + (i + 1 < kWideTN ? 1 : 0)][j][e];
      }
    } else {
      if (tile >= a.ntiles) continue;
      const int n = tile * 16 + 4 * (lane >> 4);
#pragma unroll
      for (int j = 0; j < kWideTM; ++j) {
        const int m = mbase + (wm * kWideTM + j) * 16 + (lane & 15);
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
  // k-step units of the busiest CU: rounds of workgroups times (k-steps per
  // split + ~8 of pipeline fill and epilogue), plus the partial outputs
  // written and read back (a k-step moves ~40 KB per workgroup).  SwiGLU,
  // nonlinear in the sum, is never split.
  p.ksplit = 1;
  if (epi == EPI_STORE) {
    const long wgs = (long)p.groups * p.mgroups;
    double best = 1e300;
    for (int ks = 1; ks <= max_split && KS / ks >= 8; ks *= 2) {
      const double rounds = (double)((wgs * ks + n_cu - 1) / n_cu);
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

void launch_gemm_wide(int epi, const GemmArgs &a, const GemmPlan &p, hipStream_t st) {
  // the activation loads assume whole k-steps (K = 32 KS) and at least one row;
  // the model's config checks guarantee both for every projection
  if (a.K != a.KS * 32 || a.M <= 0 || a.ldx < a.K) return;
  const dim3 grid(p.groups, p.ksplit, p.mgroups);
  if (epi == EPI_SWIGLU) hipLaunchKernelGGL(gemm_wide_kernel<EPI_SWIGLU>, grid, dim3(kWideThreads), 0, st, a);
  else hipLaunchKernelGGL(gemm_wide_kernel<EPI_STORE>, grid, dim3(kWideThreads), 0, st, a);
}

}  // namespace dk
