// Device helpers shared by the SmallKV HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smallkv.h"

namespace smallkv {

constexpr int kWave = 64;

// bf16 is carried as its 16-bit pattern; widening to fp32 is exact.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T> struct elem;
template <> struct elem<float> {
  static constexpr int per16 = 4;  // elements per 16-byte vector
  // Unpack one 16-byte vector into per16 floats.
  __device__ __forceinline__ static void unpack(const uint4 &v, float *o) {
    o[0] = __uint_as_float(v.x);
    o[1] = __uint_as_float(v.y);
    o[2] = __uint_as_float(v.z);
    o[3] = __uint_as_float(v.w);
  }
  __device__ __forceinline__ static float load1(const void *p, int64_t i) {
    return reinterpret_cast<const float *>(p)[i];
  }
  __device__ __forceinline__ static void store1(void *p, int64_t i, float x) {
    reinterpret_cast<float *>(p)[i] = x;
  }
};
template <> struct elem<bf16_t> {
  static constexpr int per16 = 8;
  __device__ __forceinline__ static void unpack(const uint4 &v, float *o) {
    o[0] = bf16_lo(v.x);
    o[1] = bf16_hi(v.x);
    o[2] = bf16_lo(v.y);
    o[3] = bf16_hi(v.y);
    o[4] = bf16_lo(v.z);
    o[5] = bf16_hi(v.z);
    o[6] = bf16_lo(v.w);
    o[7] = bf16_hi(v.w);
  }
  __device__ __forceinline__ static float load1(const void *p, int64_t i) {
    return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t *>(p)[i] << 16);
  }
  __device__ __forceinline__ static void store1(void *p, int64_t i, float x) {
    reinterpret_cast<uint16_t *>(p)[i] = f32_to_bf16(x);
  }
};

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

// Per-sequence set sizes, exactly as documented in smallkv.h: the last nr
// tokens are recent (kept, not ranked); of the older n - nr tokens the top
// ntop are critical and the next nm marginal; |C| = nc = nr + ntop.
struct Sizes {
  int n, nc, nm, nr, ntop;
};
__device__ __forceinline__ Sizes set_sizes(const int32_t *seq_len, const int32_t *k_crit,
                                           const int32_t *k_marg, const int32_t *k_recent, int b,
                                           int n_cap, int kc_cap, int km_cap) {
  Sizes s;
  s.n = clampi(seq_len[b], 1, n_cap);
  s.nr = k_recent ? clampi(k_recent[b], 0, min(s.n, kc_cap)) : 0;
  s.ntop = min(max(k_crit[b], 1), min(s.n - s.nr, kc_cap - s.nr));  // 0: nothing left to rank
  s.nc = s.nr + s.ntop;
  s.nm = clampi(k_marg[b], 0, min(s.n - s.nc, km_cap));
  return s;
}

// exp(x), x <= 0: k = rne(x * fl(1/ln 2)); r = x - k*ln2 in two FMAs with ln2
// split into a 16-bit head and a tail; e^r from the Taylor polynomial of
// degree 7 by Horner's rule (coefficients 1/n! rounded to fp32); the result
// scaled by 2^k exactly.  0 below -80, so no result is subnormal.
__device__ __forceinline__ float cw_exp(float x) {
#pragma clang fp contract(off)
  if (!(x >= -80.0f)) return 0.0f;
  const float k = __builtin_rintf(__fmul_rn(x, 0x1.715476p+0f));
  float r = __builtin_fmaf(-k, 0x1.62e4p-1f, x);
  r = __builtin_fmaf(-k, 0x1.7f7d1cp-20f, r);
  float p = 0x1.a01a02p-13f;
  p = __builtin_fmaf(p, r, 0x1.6c16c2p-10f);
  p = __builtin_fmaf(p, r, 0x1.111112p-7f);
  p = __builtin_fmaf(p, r, 0x1.555556p-5f);
  p = __builtin_fmaf(p, r, 0x1.555556p-3f);
  p = __builtin_fmaf(p, r, 0.5f);
  p = __builtin_fmaf(p, r, 1.0f);
  p = __builtin_fmaf(p, r, 1.0f);
  return ldexpf(p, (int)k);
}

// Order-preserving uint32 key of an fp32 logit; -0 and +0 share a key.
__device__ __forceinline__ uint32_t logit_key(float s) {
  uint32_t u = __float_as_uint(s == 0.0f ? 0.0f : s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace smallkv
