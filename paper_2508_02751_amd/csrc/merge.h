// Log-sum-exp combine of stage 1's per-chunk partials for one small head,
// shared by the standalone merge kernel and the fused merge+partition kernel.
#pragma once

#include "common.h"

namespace smallkv {

// Partials of one (unit, chunk): for each padded head i < GP the record
// [max, sum, acc[0..D)] (acc relative to that chunk's max).
struct MergeIn {
  const float *part;  // head i's record of chunk 0 of its unit
  int64_t stride;     // floats between consecutive chunks' records (GP*(D+2))
  int nv;             // chunks that hold tokens (ceil(N / chunk))
};

// Upper bound of chunks per unit (n_cap / smallest tile).
constexpr int kMaxChunks = 4096;

// Executed by a whole workgroup of NT threads (NT a multiple of 64 and of
// the head dim d, which is 64 or 128).  Thread (c, grp) combines the records
// s = grp, grp + NT/d, ... of output dim c online (one round trip of loads),
// then the groups are combined through LDS.  lds_red: at least 3*NT + 2
// floats.  Returns M and Z to every thread and hands out[c] = O_c / Z to
// `store` (called by threads c < d).
template <int NT, typename Store>
__device__ __forceinline__ void merge_head(const MergeIn &in, int d, float *lds_red, float &M,
                                           float &Z, Store store) {
  const int tid = threadIdx.x;
  const int ng = NT / d, c = tid % d, grp = tid / d;
  float mx = -INFINITY, z = 0.0f, o = 0.0f;
  for (int s0 = grp; s0 < in.nv; s0 += 4 * ng) {
    float ms[4], zs[4], os[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int s = s0 + k * ng;
      const float *p = in.part + (int64_t)s * in.stride;
      const bool ok = s < in.nv;
      ms[k] = ok ? p[0] : -INFINITY;
      zs[k] = ok ? p[1] : 0.0f;
      os[k] = ok ? p[2 + c] : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (ms[k] == -INFINITY) continue;
      const float mn = fmaxf(mx, ms[k]);
      const float a = __expf(mx - mn), b = __expf(ms[k] - mn);
      z = z * a + zs[k] * b;
      o = o * a + os[k] * b;
      mx = mn;
    }
  }
  float *rm = lds_red, *rz = lds_red + NT, *ro = lds_red + 2 * NT;
  rm[tid] = mx;
  rz[tid] = z;
  ro[tid] = o;
  __syncthreads();
  if (tid < d) {
    float Mx = -INFINITY;
    for (int g = 0; g < ng; ++g) Mx = fmaxf(Mx, rm[g * d + tid]);
    float Zt = 0.0f, Ot = 0.0f;
    for (int g = 0; g < ng; ++g) {
      const float w = rm[g * d + tid] == -INFINITY ? 0.0f : __expf(rm[g * d + tid] - Mx);
      Zt += rz[g * d + tid] * w;
      Ot += ro[g * d + tid] * w;
    }
    store(tid, Ot / Zt);
    if (tid == 0) {
      lds_red[3 * NT] = Mx;
      lds_red[3 * NT + 1] = Zt;
    }
  }
  __syncthreads();
  M = lds_red[3 * NT];
  Z = lds_red[3 * NT + 1];
}

}  // namespace smallkv
