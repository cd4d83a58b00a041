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
// the head dim d, which is 64 or 128).  lds_w: at least nv floats; lds_red:
// at least NT/64 + NT floats.  Returns M and Z to every thread and hands
// out[c] = O_c / Z to `store` (called by threads c < d).
template <int NT, typename Store>
__device__ __forceinline__ void merge_head(const MergeIn &in, int d, float *lds_w, float *lds_red,
                                           float &M, float &Z, Store store) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int NW = NT / 64;
  float mx = -INFINITY;
  for (int s = tid; s < in.nv; s += NT) mx = fmaxf(mx, in.part[s * in.stride]);
  mx = wave_max(mx);
  if (lane == 0) lds_red[wave] = mx;
  __syncthreads();
  M = lds_red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) M = fmaxf(M, lds_red[w]);
  __syncthreads();
  float zl = 0.0f;
  for (int s = tid; s < in.nv; s += NT) {
    const float w = __expf(in.part[s * in.stride] - M);
    lds_w[s] = w;
    zl = __builtin_fmaf(in.part[s * in.stride + 1], w, zl);
  }
  zl = wave_sum(zl);
  if (lane == 0) lds_red[wave] = zl;
  __syncthreads();
  Z = 0.0f;
#pragma unroll
  for (int w = 0; w < NW; ++w) Z += lds_red[w];
  // O: thread (c, group) sums chunks s = group, group + ng, ...
  const int ng = NT / d, c = tid % d, grp = tid / d;
  float o = 0.0f;
  for (int s = grp; s < in.nv; s += ng) o = __builtin_fmaf(in.part[s * in.stride + 2 + c], lds_w[s], o);
  float *red = lds_red + NW;
  red[grp * d + c] = o;
  __syncthreads();
  if (tid < d) {
    float t = 0.0f;
    for (int g = 0; g < ng; ++g) t += red[g * d + tid];
    store(tid, t / Z);
  }
  __syncthreads();  // lds_w / lds_red may be reused by the caller
}

}  // namespace smallkv
