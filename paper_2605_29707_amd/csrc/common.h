// Shared device helpers for the gfx950 kernels: storage types, bf16
// conversion, matrix-core operand types, wave reductions and the selection
// order used by every top-k / argmax.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define DEVI __device__ __forceinline__

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// bf16 values are stored as raw 16-bit patterns.
struct bf16_t {
  uint16_t v;
};

DEVI float to_f32(float x) { return x; }
DEVI float to_f32(bf16_t x) { return __uint_as_float(((uint32_t)x.v) << 16); }

DEVI bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return bf16_t{(uint16_t)((u >> 16) | 0x40)};  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return bf16_t{(uint16_t)(u >> 16)};
}
// Device-scope (all XCDs) loads and stores of single values, for data one
// workgroup hands to another within a launch: the store is complete at the
// device coherence point once the storing thread's vector-memory count drains,
// and the load does not hit a stale line in a CU or XCD cache.
DEVI float ld_coherent(const float *p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
DEVI void st_coherent(float *p, float v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }

DEVI void store_as(float *p, float v) { *p = v; }
DEVI void store_as(bf16_t *p, float v) { *p = f32_to_bf16(v); }

// Split 8 fp32 values into high and low bf16 parts: x = hi + lo + O(2^-17 |x|).
// Products of an exact bf16 weight with hi and lo are exact in fp32, so two
// matrix-core passes reproduce an fp32-accurate dot product.
DEVI void split8(const float *x, bf16x8 &hi, bf16x8 &lo) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    __bf16 h = (__bf16)x[e];
    hi[e] = h;
    lo[e] = (__bf16)(x[e] - (float)h);
  }
}

DEVI float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
// Whole-wave sum through DPP lane moves (no LDS round trips): pairs within
// quads, then the half-row and row mirrors give every lane its 16-lane row
// sum, and the four row sums are read out in order.  Every lane gets the total.
DEVI float wave_sum_dpp(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xf, 0xf, false));   // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xf, 0xf, false));   // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xf, 0xf, false));  // row_half_mirror
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xf, 0xf, false));  // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}
// Lane move within each 16-lane row: lane i reads lane (i + N) mod 16 of its row
// (DPP row_ror), an ALU-latency exchange.
template <int N>
DEVI int row_ror(int v) {
  static_assert(N >= 1 && N <= 15, "row_ror takes 1..15");
  return __builtin_amdgcn_update_dpp(0, v, 0x120 + N, 0xf, 0xf, false);
}
template <int N>
DEVI float row_ror(float v) { return __int_as_float(row_ror<N>(__float_as_int(v))); }
template <int N>
DEVI unsigned long long row_ror(unsigned long long v) {
  const int lo = row_ror<N>((int)(uint32_t)v), hi = row_ror<N>((int)(uint32_t)(v >> 32));
  return ((unsigned long long)(uint32_t)hi << 32) | (uint32_t)lo;
}
// Maximum of a 64-bit key over the whole wave: within rows by rotations, then
// the four row maxima read out.  Every lane gets the result.
DEVI unsigned long long wave_max_u64(unsigned long long k) {
  unsigned long long o;
  o = row_ror<8>(k); k = o > k ? o : k;
  o = row_ror<4>(k); k = o > k ? o : k;
  o = row_ror<2>(k); k = o > k ? o : k;
  o = row_ror<1>(k); k = o > k ? o : k;
  unsigned long long best = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)k, 16 * r);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(k >> 32), 16 * r);
    const unsigned long long v = ((unsigned long long)hi << 32) | lo;
    best = v > best ? v : best;
  }
  return best;
}
DEVI float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Selection order: larger value first, then smaller id; NaN counts as -inf.
DEVI float order_val(float v) { return (v != v) ? -INFINITY : v; }
DEVI bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// 64-bit key whose unsigned order is the selection order: the float mapped
// to an order-preserving unsigned value (NaN as -inf) in the high half, the
// complement of the id in the low half (smaller id wins a tie).
DEVI unsigned long long encode_best(float v, int id) {
  uint32_t u = __float_as_uint(order_val(v));
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((unsigned long long)u << 32) | (unsigned long long)(0xffffffffu - (uint32_t)id);
}
DEVI int decode_best_id(unsigned long long key, int V) {
  const int id = (int)(0xffffffffu - (uint32_t)(key & 0xffffffffu));
  return id < 0 ? 0 : (id >= V ? V - 1 : id);  // an unset key never reaches here
}

// Reduce a (value, id) pair to the wave's best under the selection order.
DEVI void wave_best(float &v, int &i) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    float ov = __shfl_xor(v, o, 64);
    int oi = __shfl_xor(i, o, 64);
    if (better(ov, oi, v, i)) {
      v = ov;
      i = oi;
    }
  }
}

// Device error word bits (mirrors include/domino.h).
enum : int32_t {
  DEV_BAD_TOKEN = 1,
  DEV_BAD_CTX_LEN = 2,
  DEV_BAD_TREE = 4,
  DEV_BARRIER_TIMEOUT = 8
};

DEVI void raise_error(int32_t *err, int32_t bit) { atomicOr(err, bit); }

DEVI int clamp_token(int t, int vocab, int32_t *err) {
  if (t < 0 || t >= vocab) {
    raise_error(err, DEV_BAD_TOKEN);
    return t < 0 ? 0 : vocab - 1;
  }
  return t;
}
