// Stage 1: the small model's full decode attention over its uncompressed
// cache (Algorithm 1, decode branch; the full small cache C^s_all of the
// "Saliency Shift Compensation" paragraph).
//
// small_attn_split: one workgroup per (sequence, layer, kv head, token chunk).
//   Pass 1 stages K tiles through LDS with coalesced 16-byte loads; each
//   thread then owns one token and evaluates the logit of every query head
//   of the GQA group as a sequential fp32 FMA chain (the bit-exact key), and
//   writes it out.  Pass 2 stages V tiles, turns the thread's own logits into
//   exp(s - chunk max) and accumulates P.V with threads laid over
//   (dim group, token stripe).  Output: per chunk and head (max, sum, P.V).
// small_attn_merge: log-sum-exp combine of the chunks of one small head into
//   row_max, row_sum and the head's output.
#include "common.h"
#include "launch.h"

namespace smallkv {
namespace {

constexpr int kThreads = 256;

template <typename T, int D>
struct SmallCfg {
  static constexpr int ROWB = D * (int)sizeof(T);                   // bytes per K/V row
  static constexpr int TILE = 32768 / ROWB < 256 ? 32768 / ROWB : 256;  // rows per LDS tile
  static constexpr int ROWS = ROWB + 16;                            // padded LDS row stride
  static constexpr int V16 = ROWB / 16;                             // 16-byte vectors per row
  static constexpr int VD = 4;                                      // dims per thread in P.V
  static constexpr int NDG = D / VD;                                // dim groups
  static constexpr int NTP = kThreads / NDG;                        // token stripes
};

struct SmallArgs {
  int n_cap, layers, hq, hkv, g, chunk, n_split;
  float scale;
  const int32_t *seq_len;
  const void *q, *k, *v;
  void *out;
  float *logits, *row_max, *row_sum, *part;
};

template <typename T, int D>
__device__ __forceinline__ void stage_rows(unsigned char *tile, const unsigned char *src, int nr) {
  using C = SmallCfg<T, D>;
  for (int x = threadIdx.x; x < nr * C::V16; x += kThreads) {
    const int r = x / C::V16, w = x % C::V16;
    const uint4 v = *reinterpret_cast<const uint4 *>(src + (int64_t)r * C::ROWB + w * 16);
    *reinterpret_cast<uint4 *>(tile + r * C::ROWS + w * 16) = v;
  }
}

template <typename T>
__device__ __forceinline__ void load4(const unsigned char *p, float *o);
template <>
__device__ __forceinline__ void load4<float>(const unsigned char *p, float *o) {
  const uint4 v = *reinterpret_cast<const uint4 *>(p);
  elem<float>::unpack(v, o);
}
template <>
__device__ __forceinline__ void load4<bf16_t>(const unsigned char *p, float *o) {
  const uint2 v = *reinterpret_cast<const uint2 *>(p);
  o[0] = bf16_lo(v.x);
  o[1] = bf16_hi(v.x);
  o[2] = bf16_lo(v.y);
  o[3] = bf16_hi(v.y);
}

template <typename T, int D, int GP>
__global__ __launch_bounds__(kThreads) void small_attn_split(SmallArgs a) {
  using C = SmallCfg<T, D>;
  __shared__ __align__(16) unsigned char tile[C::TILE * C::ROWS];
  __shared__ __align__(16) float sq[GP * D];
  __shared__ __align__(16) float sp[C::TILE * GP];
  __shared__ float red[4 * GP];
  __shared__ float redz[4 * GP];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int unit = blockIdx.x / a.n_split, split = blockIdx.x % a.n_split;
  const int kvh = unit % a.hkv, bl = unit / a.hkv, layer = bl % a.layers, b = bl / a.layers;
  const int n = clampi(a.seq_len[b], 1, a.n_cap);
  const int t0 = split * a.chunk;
  if (t0 >= n) return;
  const int t1 = min(t0 + a.chunk, n);
  const int g = a.g;
  const int64_t head0 = ((int64_t)b * a.layers + layer) * a.hq + (int64_t)kvh * g;  // q row of head 0

  for (int x = tid; x < GP * D; x += kThreads) {
    const int i = x / D, c = x % D;
    sq[x] = i < g ? elem<T>::load1(a.q, (head0 + i) * D + c) : 0.0f;
  }
  const int64_t row0 = (int64_t)unit * a.n_cap;  // K/V row of token 0 of this unit
  const unsigned char *kb = reinterpret_cast<const unsigned char *>(a.k) + row0 * C::ROWB;
  const unsigned char *vb = reinterpret_cast<const unsigned char *>(a.v) + row0 * C::ROWB;
  float *lrow = a.logits + head0 * a.n_cap;  // logits [b][j][n_cap], j = layer*hq + kvh*g + i

  // ---- pass 1: logits (the ranking key) and the chunk max -------------
  float mx[GP];
#pragma unroll
  for (int i = 0; i < GP; ++i) mx[i] = -INFINITY;
  for (int tb = t0; tb < t1; tb += C::TILE) {
    const int nr = min(C::TILE, t1 - tb);
    stage_rows<T, D>(tile, kb + (int64_t)tb * C::ROWB, nr);
    __syncthreads();
    if (tid < nr) {
      float kr[D];
#pragma unroll
      for (int w = 0; w < C::V16; ++w) {
        const uint4 v = *reinterpret_cast<const uint4 *>(tile + tid * C::ROWS + w * 16);
        elem<T>::unpack(v, kr + w * elem<T>::per16);
      }
#pragma unroll
      for (int i = 0; i < GP; ++i) {
        if (i < g) {
          float acc = 0.0f;
#pragma unroll
          for (int c = 0; c < D; ++c) acc = __builtin_fmaf(sq[i * D + c], kr[c], acc);
          float s = acc * a.scale;
          s = (s == 0.0f) ? 0.0f : s;
          lrow[(int64_t)i * a.n_cap + tb + tid] = s;
          mx[i] = fmaxf(mx[i], s);
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < GP; ++i) {
    const float v = wave_max(mx[i]);
    if (lane == 0) red[wave * GP + i] = v;
  }
  __syncthreads();
  float m[GP];
#pragma unroll
  for (int i = 0; i < GP; ++i)
    m[i] = fmaxf(fmaxf(red[i], red[GP + i]), fmaxf(red[2 * GP + i], red[3 * GP + i]));

  // ---- pass 2: exp(s - m) and P.V --------------------------------------
  const int dg = tid % C::NDG, tp = tid / C::NDG;
  float acc[GP][C::VD];
  float zl[GP];
#pragma unroll
  for (int i = 0; i < GP; ++i) {
    zl[i] = 0.0f;
#pragma unroll
    for (int c = 0; c < C::VD; ++c) acc[i][c] = 0.0f;
  }
  for (int tb = t0; tb < t1; tb += C::TILE) {
    const int nr = min(C::TILE, t1 - tb);
    stage_rows<T, D>(tile, vb + (int64_t)tb * C::ROWB, nr);
    if (tid < nr) {
#pragma unroll
      for (int i = 0; i < GP; ++i) {
        float e = 0.0f;
        if (i < g) {
          e = __expf(lrow[(int64_t)i * a.n_cap + tb + tid] - m[i]);
          zl[i] += e;
        }
        sp[tid * GP + i] = e;
      }
    }
    __syncthreads();
    for (int t = tp; t < nr; t += C::NTP) {
      float vv[C::VD];
      load4<T>(tile + t * C::ROWS + dg * C::VD * (int)sizeof(T), vv);
      float p[GP];
#pragma unroll
      for (int i = 0; i < GP; i += 4) {
        const float4 w = *reinterpret_cast<const float4 *>(sp + t * GP + i);
        p[i] = w.x;
        p[i + 1] = w.y;
        p[i + 2] = w.z;
        p[i + 3] = w.w;
      }
#pragma unroll
      for (int i = 0; i < GP; ++i)
        if (i < g) {
#pragma unroll
          for (int c = 0; c < C::VD; ++c) acc[i][c] = __builtin_fmaf(p[i], vv[c], acc[i][c]);
        }
    }
    __syncthreads();
  }

  // ---- reductions: z over all threads, P.V over token stripes -----------
#pragma unroll
  for (int i = 0; i < GP; ++i) {
    const float v = wave_sum(zl[i]);
    if (lane == 0) redz[wave * GP + i] = v;
  }
  // stripes inside one wave first
#pragma unroll
  for (int o = C::NDG; o < kWave; o <<= 1)
#pragma unroll
    for (int i = 0; i < GP; ++i)
#pragma unroll
      for (int c = 0; c < C::VD; ++c) acc[i][c] += __shfl_xor(acc[i][c], o, kWave);
  float *buf = reinterpret_cast<float *>(tile);  // [4 waves][GP][D]; tile is free now
  if (lane < C::NDG) {
#pragma unroll
    for (int i = 0; i < GP; ++i)
#pragma unroll
      for (int c = 0; c < C::VD; ++c) buf[(wave * GP + i) * D + dg * C::VD + c] = acc[i][c];
  }
  __syncthreads();
  float *part = a.part + (int64_t)blockIdx.x * GP * (D + 2);
  for (int x = tid; x < g * D; x += kThreads) {
    const int i = x / D, c = x % D;
    part[i * (D + 2) + 2 + c] = buf[i * D + c] + buf[(GP + i) * D + c] +
                                buf[(2 * GP + i) * D + c] + buf[(3 * GP + i) * D + c];
  }
  if (tid == 0) {
#pragma unroll
    for (int i = 0; i < GP; ++i)
      if (i < g) {
        part[i * (D + 2)] = m[i];
        part[i * (D + 2) + 1] = redz[i] + redz[GP + i] + redz[2 * GP + i] + redz[3 * GP + i];
      }
  }
}

// One workgroup of D threads per small head: combine its chunks.
template <typename T, int D, int GP>
__global__ __launch_bounds__(D) void small_attn_merge(SmallArgs a) {
  const int row = blockIdx.x;  // = b * (layers*hq) + layer*hq + h
  const int h = row % a.hq, bl = row / a.hq, layer = bl % a.layers, b = bl / a.layers;
  const int unit = (b * a.layers + layer) * a.hkv + h / a.g, i = h % a.g;
  const int n = clampi(a.seq_len[b], 1, a.n_cap);
  const int nv = (n + a.chunk - 1) / a.chunk;
  const float *p = a.part + (int64_t)unit * a.n_split * GP * (D + 2) + i * (D + 2);
  const int64_t stride = (int64_t)GP * (D + 2);
  float M = -INFINITY;
  for (int s = 0; s < nv; ++s) M = fmaxf(M, p[s * stride]);
  float Z = 0.0f, o = 0.0f;
  const int c = threadIdx.x;
  for (int s = 0; s < nv; ++s) {
    const float w = __expf(p[s * stride] - M);
    Z = __builtin_fmaf(p[s * stride + 1], w, Z);
    o = __builtin_fmaf(p[s * stride + 2 + c], w, o);
  }
  if (c == 0) {
    a.row_max[row] = M;
    a.row_sum[row] = Z;
  }
  elem<T>::store1(a.out, (int64_t)row * D + c, o / Z);
}

template <typename T, int D, int GP>
hipError_t launch_t(const SmallArgs &a, int units, hipStream_t st) {
  hipLaunchKernelGGL((small_attn_split<T, D, GP>), dim3(units * a.n_split), dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rows = units / a.hkv * a.hq;
  hipLaunchKernelGGL((small_attn_merge<T, D, GP>), dim3(rows), dim3(D), 0, st, a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_gp(const SmallArgs &a, int units, int gp, hipStream_t st) {
  if (gp == 4) return launch_t<T, D, 4>(a, units, st);
  if (gp == 8) return launch_t<T, D, 8>(a, units, st);
  return launch_t<T, D, 16>(a, units, st);
}

}  // namespace

SmallPlan plan_small(const smallkv_batch_t &b, const smallkv_model_t &m) {
  SmallPlan p{};
  const int esz = m.dtype == SMALLKV_F32 ? 4 : 2;
  const int rowb = m.head_dim * esz;
  p.tile = 32768 / rowb < 256 ? 32768 / rowb : 256;
  const int64_t units = (int64_t)b.batch * m.n_layers * m.n_kv_heads;
  const int max_split = (b.n_cap + p.tile - 1) / p.tile;
  int want = (int)((4096 + units - 1) / units);
  int ns = want < 1 ? 1 : (want > max_split ? max_split : want);
  const int per = (b.n_cap + ns - 1) / ns;
  p.chunk = (per + p.tile - 1) / p.tile * p.tile;
  p.n_split = (b.n_cap + p.chunk - 1) / p.chunk;
  const int g = m.n_q_heads / m.n_kv_heads;
  p.gp = g <= 4 ? 4 : (g <= 8 ? 8 : 16);
  p.ws_bytes = (size_t)units * p.n_split * p.gp * (m.head_dim + 2) * sizeof(float);
  return p;
}

hipError_t launch_small_attn(const smallkv_batch_t &b, const smallkv_model_t &m, float *logits,
                             float *row_max, float *row_sum, float *ws, const SmallPlan &p,
                             hipStream_t st) {
  SmallArgs a;
  a.n_cap = b.n_cap;
  a.layers = m.n_layers;
  a.hq = m.n_q_heads;
  a.hkv = m.n_kv_heads;
  a.g = m.n_q_heads / m.n_kv_heads;
  a.chunk = p.chunk;
  a.n_split = p.n_split;
  a.scale = m.scale;
  a.seq_len = b.seq_len;
  a.q = m.q;
  a.k = m.k;
  a.v = m.v;
  a.out = m.out;
  a.logits = logits;
  a.row_max = row_max;
  a.row_sum = row_sum;
  a.part = ws;
  const int units = b.batch * m.n_layers * m.n_kv_heads;
  if (m.dtype == SMALLKV_F32)
    return m.head_dim == 64 ? launch_gp<float, 64>(a, units, p.gp, st)
                            : launch_gp<float, 128>(a, units, p.gp, st);
  return m.head_dim == 64 ? launch_gp<bf16_t, 64>(a, units, p.gp, st)
                          : launch_gp<bf16_t, 128>(a, units, p.gp, st);
}

}  // namespace smallkv
