// Matrix-core operand helpers shared by the GEMM and the rollout kernels.
//
// A 16x16 output tile is produced by v_mfma_f32_16x16x32_bf16 (bf16 storage)
// or four v_mfma_f32_16x16x4_f32 (fp32 storage).  For lane l = 16*g + r the
// A operand holds 16 bytes of row r (EPL consecutive k starting at g*EPL) and
// the B operand the same k range of column r; the accumulator holds rows
// 4g..4g+3 of column r.  fp32 activations are split into hi + lo bf16 parts
// for the bf16 path, so products with exact bf16 weights stay exact in fp32.
#pragma once
#include "common.h"

namespace dk {

template <typename WT> struct Frag;
template <> struct Frag<bf16_t> {
  static constexpr int EPL = 8, KSTEP = 32;
};
template <> struct Frag<float> {
  static constexpr int EPL = 4, KSTEP = 16;
};

template <typename WT> struct XStage;
template <> struct XStage<bf16_t> {
  static constexpr int XF = 2;  // u32x4 per fragment: hi, lo
  DEVI static void put(u32x4 *dst, const float4 (&v)[2]) {
    const float f[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
    bf16x8 hi, lo;
    split8(f, hi, lo);
    dst[0] = __builtin_bit_cast(u32x4, hi);
    dst[1] = __builtin_bit_cast(u32x4, lo);
  }
};
template <> struct XStage<float> {
  static constexpr int XF = 1;
  DEVI static void put(u32x4 *dst, const float4 (&v)[1]) { dst[0] = __builtin_bit_cast(u32x4, v[0]); }
};

// Marks loaded registers as used on a path that does not multiply them, so
// that the compiler waits for their loads there.  The compiler's wait
// insertion assumes the worst over all paths: a load left unconsumed on one
// path makes it drain every younger load (the next chunk's prefetch included)
// before the register is next written.
template <int N>
DEVI void consume(const u32x4 (&w)[N]) {
#pragma unroll
  for (int u = 0; u < N; ++u) __asm__ volatile("" ::"v"(w[u]));
}

// Passes loaded values through an empty asm that the compiler keeps in order
// with the scheduling barriers around it, so that work on them (and the wait
// for their loads) cannot move up to where they were loaded.
template <int N, int E>
DEVI void pin(float4 (&v)[N][E]) {
#pragma unroll
  for (int q = 0; q < N; ++q)
#pragma unroll
    for (int e = 0; e < E; ++e) __asm__ volatile("" : "+v"(v[q][e].x), "+v"(v[q][e].y), "+v"(v[q][e].z), "+v"(v[q][e].w));
}

template <typename WT, int MT>
struct Mac2 {
  // xf points at fragments [mt][XF] of one k-step
  DEVI static void step(const u32x4 &w, const u32x4 *xf, floatx4 (&acc)[MT]) {
    if constexpr (sizeof(WT) == 2) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, w);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, xf[mt * 2 + 0]), acc[mt], 0, 0, 0);
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, xf[mt * 2 + 1]), acc[mt], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float av = __uint_as_float(w[e]);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, __uint_as_float(xf[mt][e]), acc[mt], 0, 0, 0);
      }
    }
  }
};


}  // namespace dk
