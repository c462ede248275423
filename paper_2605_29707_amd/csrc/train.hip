// Teacher-forced training forward of the Domino head and its loss (Sec. 4.2).
//
// With ground-truth tokens fed to the causal encoder the rollout no longer
// waits on an argmax, so everything after the state recurrence is batched
// over positions:
//   ce     u = SiLU(P + Y) for every row (P = W1[:, :d] H from the LM-head
//          pass, Y = W1[:, d:] S from one small GEMM over all states), then
//          L_final = L_base + W2 u for all bs*(B-1) rows at once: W2 streams
//          from HBM once (tile-packed, matrix cores, hi/lo split of U as in the
//          rollout), L_base once, and the corrected logits never leave the
//          chip.  Each workgroup leaves, per row, the (max, sum exp) pair of
//          its vocabulary slice for the base and the final logits, and the
//          workgroup holding the label writes the label's two logits.
//   loss   one workgroup: a wave per row merges the pairs (CE = log-sum-exp
//          - label logit), then the position-weighted means (weights
//          exp(-k / gamma), k = 0 for the first draft position) and the
//          curriculum mix (1 - lambda) L_final + lambda L_base, in a fixed
//          order (deterministic).
#include "common.h"
#include "kernels.h"
#include "mfma.h"

namespace dk {

constexpr int kCeWaves = 8;
constexpr int ce_tpw(int KS) { return KS <= 8 ? 5 : 2; }  // W2 tiles per wave (fragments stay in registers)

// (m, s) <- merge of two (max, sum exp(x - max)) pairs
DEVI void lse_merge(float &m, float &s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) {
    m = mn;
    s = 0.f;
    return;
  }
  s = s * expf(m - mn) + s2 * expf(m2 - mn);
  m = mn;
}

template <typename WT, int KS>
__global__ __launch_bounds__(kCeWaves * 64) void train_ce_kernel(TrainArgs t) {
  constexpr int EPL = Frag<WT>::EPL, KSTEP = Frag<WT>::KSTEP, XF = XStage<WT>::XF;
  constexpr int kTPW = ce_tpw(KS);
  const int V = t.V, r = t.r, Mr = t.Mr;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, cc = lane & 15;
  const int NT = (V + 15) / 16;
  __shared__ u32x4 us[KS * 64 * XF];                 // U tile as B fragments
  __shared__ float4 red[kCeWaves][16];                // per-wave (mb, sb, mf, sf) of each row
  __shared__ float4 lbs[kCeWaves][kTPW][64];          // L_base values of each lane

  int tiles[kTPW];
#pragma unroll
  for (int q = 0; q < kTPW; ++q) tiles[q] = (blockIdx.x * kCeWaves + wave) * kTPW + q;
  // this wave's W2 fragments, loaded once and reused for every row tile
  const u32x4 *w2p = (const u32x4 *)t.w2p;
  u32x4 wf[kTPW][KS];
#pragma unroll
  for (int q = 0; q < kTPW; ++q) {
    const int tc = min(tiles[q], NT - 1);
#pragma unroll
    for (int s = 0; s < KS; ++s) wf[q][s] = w2p[((size_t)tc * KS + s) * 64 + lane];
  }

  constexpr int kUIt = (KS * 64 + kCeWaves * 64 - 1) / (kCeWaves * 64);
  for (int m0 = 0; m0 < Mr; m0 += 16) {
    // u = SiLU(P + Y) of this tile's rows (clamped rows: padding columns are never read)
    float4 uv[kUIt][EPL / 4];
#pragma unroll
    for (int q = 0; q < kUIt; ++q) {
      const int it = min(tid + q * kCeWaves * 64, KS * 64 - 1);
      const int l = it & 63, s = it >> 6;
      const int row = min(m0 + (l & 15), Mr - 1);
      const int k0 = s * KSTEP + (l >> 4) * EPL;
      const float *py = t.Y + (size_t)row * r + k0;
      const float *pp = t.P + (size_t)row * t.ldp + k0;
#pragma unroll
      for (int e = 0; e < EPL / 4; ++e) {
        const float4 a = *(const float4 *)(py + 4 * e), b = *(const float4 *)(pp + 4 * e);
        float4 x = make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
        x.x = x.x / (1.f + expf(-x.x));
        x.y = x.y / (1.f + expf(-x.y));
        x.z = x.z / (1.f + expf(-x.z));
        x.w = x.w / (1.f + expf(-x.w));
        uv[q][e] = x;
      }
    }
    // L_base of this lane's row and the four vocabulary ids of each tile (rows
    // are padded to whole tiles, so the float4 stays inside the row), parked
    // in LDS until the epilogue: the registers hold this wave's W2 fragments
    const int row = m0 + cc;
    const int rowc = min(row, Mr - 1);
    {
      float4 lb[kTPW];
#pragma unroll
      for (int q = 0; q < kTPW; ++q) {
        const int tc = min(tiles[q], NT - 1);
        lb[q] = *(const float4 *)(t.Lbase + (size_t)rowc * t.ldl + tc * 16 + 4 * g);
      }
#pragma unroll
      for (int q = 0; q < kTPW; ++q) lbs[wave][q][lane] = lb[q];
    }
    const int label = t.labels[rowc];
#pragma unroll
    for (int q = 0; q < kUIt; ++q) {
      const int it = tid + q * kCeWaves * 64;
      if (it < KS * 64) XStage<WT>::put(us + (size_t)it * XF, uv[q]);
    }
    __syncthreads();

    // k-step major: each staged U fragment is read from LDS once for all tiles
    floatx4 acc[kTPW][1];
#pragma unroll
    for (int q = 0; q < kTPW; ++q) acc[q][0] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      u32x4 xf[XF];
#pragma unroll
      for (int f = 0; f < XF; ++f) xf[f] = us[((size_t)s * 64 + lane) * XF + f];
#pragma unroll
      for (int q = 0; q < kTPW; ++q) Mac2<WT, 1>::step(wf[q][s], xf, acc[q]);
    }

    // lane (g, cc) holds vocabulary ids 16 tile + 4 g + e of row m0 + cc:
    // stores, the label's logits and the maximum first, then the sums
    // (values are re-formed from lb and acc rather than kept)
    float mb = -INFINITY, mf = -INFINITY;
#pragma unroll
    for (int q = 0; q < kTPW; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int n = tiles[q] * 16 + 4 * g + e;
        const bool ok = row < Mr && n < V;
        const float4 l4 = lbs[wave][q][lane];
        const float base = e == 0 ? l4.x : (e == 1 ? l4.y : (e == 2 ? l4.z : l4.w));
        const float fin = base + acc[q][0][e];
        if (ok && t.final_logits) t.final_logits[(size_t)row * V + n] = fin;
        if (ok && n == label) {
          t.lab[row] = base;
          t.lab[Mr + row] = fin;
        }
        mb = fmaxf(mb, ok ? order_val(base) : -INFINITY);
        mf = fmaxf(mf, ok ? order_val(fin) : -INFINITY);
      }
    float sb = 0.f, sf = 0.f;
#pragma unroll
    for (int q = 0; q < kTPW; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int n = tiles[q] * 16 + 4 * g + e;
        const bool ok = row < Mr && n < V;
        const float4 l4 = lbs[wave][q][lane];
        const float base = e == 0 ? l4.x : (e == 1 ? l4.y : (e == 2 ? l4.z : l4.w));
        const float fin = base + acc[q][0][e];
        // exp(-inf - m) is 0 for finite m; a slice with no finite value keeps its sum at 0
        if (ok && mb != -INFINITY) sb += expf(order_val(base) - mb);
        if (ok && mf != -INFINITY) sf += expf(order_val(fin) - mf);
      }
    // the four lanes of a row, then the waves
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float mb2 = __shfl_xor(mb, o, 64), sb2 = __shfl_xor(sb, o, 64);
      const float mf2 = __shfl_xor(mf, o, 64), sf2 = __shfl_xor(sf, o, 64);
      lse_merge(mb, sb, mb2, sb2);
      lse_merge(mf, sf, mf2, sf2);
    }
    if (g == 0) red[wave][cc] = make_float4(mb, sb, mf, sf);
    __syncthreads();
    if (tid < 16 && m0 + tid < Mr) {
      float4 p = red[0][tid];
#pragma unroll
      for (int w = 1; w < kCeWaves; ++w) {
        const float4 o = red[w][tid];
        lse_merge(p.x, p.y, o.x, o.y);
        lse_merge(p.z, p.w, o.z, o.w);
      }
      *(float4 *)(t.part + ((size_t)(m0 + tid) * gridDim.x + blockIdx.x) * 4) = p;
    }
  }
}

// One workgroup: each wave merges the workgroups' pairs of its rows
// (CE = log-sum-exp - label logit), then the position-weighted means and the
// curriculum mix, summed in a fixed order (deterministic).
constexpr int kLossThreads = 1024;
constexpr int kLoadsPerLane = 8;
__global__ __launch_bounds__(kLossThreads) void train_loss_kernel(TrainArgs t, int GC) {
  constexpr int kWaves = kLossThreads / 64;
  __shared__ double sb[kWaves], sf[kWaves], wk[64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < t.depth) wk[tid] = exp(-(double)tid / (double)t.gamma);  // position weights, depth <= 63
  __syncthreads();
  double ab = 0.0, af = 0.0;  // this wave's weighted sums, rows in a fixed order
  for (int row = wave; row < t.Mr; row += kWaves) {
    // the label and its two logits first, so their round trip overlaps the pairs'
    const int label = t.labels[row];
    const float lb = order_val(t.lab[row]), lf = order_val(t.lab[t.Mr + row]);
    float mb = -INFINITY, s_b = 0.f, mf = -INFINITY, s_f = 0.f;
    // kLoadsPerLane pairs per lane in flight together (clamped index, masked
    // after): a load per merge would pay one memory round trip each
    const float4 *pr = (const float4 *)t.part + (size_t)row * GC;
    for (int c0 = 0; c0 < GC; c0 += 64 * kLoadsPerLane) {
      float4 p[kLoadsPerLane];
#pragma unroll
      for (int q = 0; q < kLoadsPerLane; ++q) p[q] = pr[min(c0 + q * 64 + lane, GC - 1)];
#pragma unroll
      for (int q = 0; q < kLoadsPerLane; ++q)
        if (c0 + q * 64 + lane < GC) {
          lse_merge(mb, s_b, p[q].x, p[q].y);
          lse_merge(mf, s_f, p[q].z, p[q].w);
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float mb2 = __shfl_xor(mb, o, 64), sb2 = __shfl_xor(s_b, o, 64);
      const float mf2 = __shfl_xor(mf, o, 64), sf2 = __shfl_xor(s_f, o, 64);
      lse_merge(mb, s_b, mb2, sb2);
      lse_merge(mf, s_f, mf2, sf2);
    }
    if (lane == 0) {
      const bool ok = label >= 0 && label < t.V;
      if (!ok) raise_error(t.err, DEV_BAD_TOKEN);
      const float cb = ok ? mb + logf(s_b) - lb : NAN, cf = ok ? mf + logf(s_f) - lf : NAN;
      t.ce[row] = cb;
      t.ce[t.Mr + row] = cf;
      ab += wk[row % t.depth] * (double)cb;
      af += wk[row % t.depth] * (double)cf;
    }
  }
  if (lane == 0) {
    sb[wave] = ab;
    sf[wave] = af;
  }
  __syncthreads();
  if (tid == 0) {
    double tb = 0.0, tf = 0.0, wsum = 0.0;
    for (int w = 0; w < kWaves; ++w) {
      tb += sb[w];
      tf += sf[w];
    }
    for (int k = 0; k < t.depth; ++k) wsum += wk[k];
    const double n = wsum * (double)(t.Mr / t.depth);
    const double lb = tb / n, lf = tf / n;
    t.loss[0] = (float)((1.0 - (double)t.lambda) * lf + (double)t.lambda * lb);
    t.loss[1] = (float)lb;
    t.loss[2] = (float)lf;
  }
}

template <typename WT, int KS>
static void launch_ce_t(const TrainArgs &t, int GC, hipStream_t st) {
  hipLaunchKernelGGL((train_ce_kernel<WT, KS>), dim3(GC), dim3(kCeWaves * 64), 0, st, t);
}

int train_ce_grid(int V, int r, bool bf16) {
  const int KS = r / kstep_of(bf16);
  const int rows = kCeWaves * ce_tpw(KS) * 16;
  return (V + rows - 1) / rows;
}

hipError_t launch_train_loss(const TrainArgs &t, bool bf16, hipStream_t st) {
  const int KS = t.r / kstep_of(bf16);
  const int GC = train_ce_grid(t.V, t.r, bf16);
  if (bf16) {
    if (KS == 8) launch_ce_t<bf16_t, 8>(t, GC, st);
    else return hipErrorInvalidValue;
  } else {
    if (KS == 16) launch_ce_t<float, 16>(t, GC, st);
    else if (KS == 8) launch_ce_t<float, 8>(t, GC, st);
    else return hipErrorInvalidValue;
  }
  hipLaunchKernelGGL(train_loss_kernel, dim3(1), dim3(kLossThreads), 0, st, t, GC);
  return hipGetLastError();
}

}  // namespace dk
