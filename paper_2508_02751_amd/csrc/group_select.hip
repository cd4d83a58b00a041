// Group selection: the query heads of one large-model kv head share one
// critical and one marginal set (the KV cache is stored per kv head), ranked
// by the sum of their small heads' attention probabilities -- the summed
// selection of the implementation pseudocode (Appendix D, `.sum.topk`).
//
// The sum decides integers, so it has one defined evaluation (smallkv.h):
//   e_j(t) = cw_exp(s_j(t) - m_j)                        (fp32)
//   Zq_j   = sum_t floor(e_j(t) * 2^40), an exact integer (any order)
//   Z_j    = fp32(Zq_j) * 2^-40
//   F(t)   = ((e_j0/Z_j0 + e_j1/Z_j1) + ...)               (fp32, heads ascending)
// Kernels, between stage 1 (logits and exact row maxima) and stage 3:
//   group_zq      -- per small head and 2048-token chunk: the chunk's part
//                    of Zq_j as a 64-bit integer (the readers add the parts:
//                    exact, integer addition is associative); it also zeroes
//                    the row maxima that group_scores raises atomically;
//   group_scores  -- per (sequence, large layer, kv head) and 1024-token
//                    chunk: F(t) for every token, the row's largest F by an
//                    atomic max on its bits;
//   (the partition kernel then ranks F, its bins read as log2 of the key)
//   group_weights -- one workgroup per large query head: its own small
//                    head's p' = exp(s - m) / Z (stage 1's statistics) on the
//                    group's marginal list, and its masses S'_C, S'_M.
#include "common.h"
#include "launch.h"

#pragma clang fp contract(off)

namespace smallkv {
namespace {

constexpr int kGT = 256;

struct GroupSelArgs {
  int n_cap, nsh, L, hq, hkv, gq, kc_cap, km_cap;
  const int32_t *seq_len, *k_crit, *k_marg, *k_recent, *head_map;
  const float *logits, *row_max, *row_sum;
  uint64_t *zq_int;        // [B][nsh][nzc]: the exact integer sums per token chunk
  int nzc;                 // token chunks of group_zq per row
  int n_keymax;            // entries of key_max, zeroed by group_zq
  float *keys, *key_max;   // [B][L*hkv][n_cap], [B][L*hkv]
  const int32_t *crit, *marg;  // group lists [B][L*hkv][cap]
  float *marg_prob, *mass;     // per large head [B][L*hq][km_cap], [B][L*hq][2]
  // accumulated-score selection: per small head, acc [B][nsh][n_cap] (the
  // running score, updated in place); lists and weights per small head
  int accum;
  float *acc;
};

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, o, kWave);
    const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), o, kWave);
    v += ((uint64_t)hi << 32) | lo;
  }
  return v;
}

constexpr int kZqTok = 8 * kGT;     // tokens per group_zq workgroup (8 per thread)
constexpr int kScoreTok = 4 * kGT;  // tokens per group_scores workgroup (4 per thread)

// blockIdx.x: small head row; blockIdx.y: a chunk of kZqTok tokens, whose
// integer sum it writes (0 past the row's end): integer addition is
// associative, so the readers' sum of the chunks is the exact sum.  The
// workgroups also zero key_max, which group_scores / accum_scores then
// raise with atomic maxima.
__global__ __launch_bounds__(kGT) void group_zq(GroupSelArgs a) {
  __shared__ uint64_t part[kGT / kWave];
  const int wg = blockIdx.x * gridDim.y + blockIdx.y, nwg = gridDim.x * gridDim.y;
  for (int i = wg * kGT + threadIdx.x; i < a.n_keymax; i += nwg * kGT) a.key_max[i] = 0.0f;
  const int row = blockIdx.x, b = row / a.nsh;
  const int n = clampi(a.seq_len[b], 1, a.n_cap);
  const int t0 = blockIdx.y * kZqTok;
  const float m = a.row_max[row];
  const float *lg = a.logits + (int64_t)row * a.n_cap;
  uint64_t z = 0;
#pragma unroll
  for (int q = 0; q < kZqTok / kGT; ++q) {
    const int t = t0 + q * kGT + threadIdx.x;
    if (t < n) {
      const float e = cw_exp(__fsub_rn(lg[t], m));
      z += (uint64_t)__float2ull_rz(__fmul_rn(e, 0x1p40f));  // exact scaling, truncation
    }
  }
  z = wave_sum_u64(z);
  if ((threadIdx.x & (kWave - 1)) == 0) part[threadIdx.x / kWave] = z;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t s = 0;
    for (int w = 0; w < kGT / kWave; ++w) s += part[w];
    a.zq_int[(int64_t)row * a.nzc + blockIdx.y] = s;
  }
}

// Z of a small head row: the chunks' exact integer sums added, rounded once
// to fp32 and scaled by 2^-40.
__device__ __forceinline__ float zq_of(const GroupSelArgs &a, int64_t row) {
  uint64_t z = 0;
  for (int c = 0; c < a.nzc; ++c) z += a.zq_int[row * a.nzc + c];
  return __fmul_rn(__ull2float_rn(z), 0x1p-40f);
}

// blockIdx.x: group row (b, layer, kv head); blockIdx.y: a chunk of
// kScoreTok tokens.  The row's largest key by an atomic max on its bits
// (exact: keys are non-negative).
__global__ __launch_bounds__(kGT) void group_scores(GroupSelArgs a) {
  constexpr int kMaxGQ = 16;
  constexpr int kQ = kScoreTok / kGT;
  __shared__ const float *lrow[kMaxGQ];
  __shared__ float lm[kMaxGQ], lz[kMaxGQ], wmax[kGT / kWave];
  const int grow = blockIdx.x;
  const int per = a.L * a.hkv, b = grow / per, layer = (grow % per) / a.hkv, kvh = grow % a.hkv;
  const int n = clampi(a.seq_len[b], 1, a.n_cap);
  const int t0 = blockIdx.y * kScoreTok;
  if (t0 >= n) return;
  if ((int)threadIdx.x < a.gq) {
    const int h = threadIdx.x;
    const int j = clampi(a.head_map[layer * a.hq + kvh * a.gq + h], 0, a.nsh - 1);
    const int64_t row = (int64_t)b * a.nsh + j;
    lrow[h] = a.logits + row * a.n_cap;
    lm[h] = a.row_max[row];
    lz[h] = zq_of(a, row);
  }
  __syncthreads();
  float f[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) f[q] = 0.0f;
  for (int h = 0; h < a.gq; ++h) {
    const float *lg = lrow[h];
    const float m = lm[h], z = lz[h];
#pragma unroll
    for (int q = 0; q < kQ; ++q) {  // kQ independent chains; heads in ascending order
      const int t = t0 + q * kGT + threadIdx.x;
      if (t < n) f[q] = __fadd_rn(f[q], __fdiv_rn(cw_exp(__fsub_rn(lg[t], m)), z));
    }
  }
  float *out = a.keys + (int64_t)grow * a.n_cap;
  float fmx = 0.0f;
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    const int t = t0 + q * kGT + threadIdx.x;
    if (t < n) {
      out[t] = f[q];
      fmx = fmaxf(fmx, f[q]);
    }
  }
  fmx = wave_max(fmx);
  if ((threadIdx.x & (kWave - 1)) == 0) wmax[threadIdx.x / kWave] = fmx;
  __syncthreads();
  if (threadIdx.x == 0) {
    float x = wmax[0];
    for (int w = 1; w < kGT / kWave; ++w) x = fmaxf(x, wmax[w]);
    atomicMax(reinterpret_cast<unsigned int *>(&a.key_max[grow]), __float_as_uint(x));
  }
}

// Accumulated scores: blockIdx.x a small head row, blockIdx.y a chunk of
// kScoreTok tokens.  acc[t] += e(t) / Z in place; the row's largest score by
// an atomic max on its bits.
__global__ __launch_bounds__(kGT) void accum_scores(GroupSelArgs a) {
  constexpr int kQ = kScoreTok / kGT;
  __shared__ float wmax[kGT / kWave];
  const int row = blockIdx.x, b = row / a.nsh;
  const int n = clampi(a.seq_len[b], 1, a.n_cap);
  const int t0 = blockIdx.y * kScoreTok;
  if (t0 >= n) return;
  const float m = a.row_max[row];
  const float z = zq_of(a, row);
  const float *lg = a.logits + (int64_t)row * a.n_cap;
  float *acc = a.acc + (int64_t)row * a.n_cap;
  float fmx = 0.0f;
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    const int t = t0 + q * kGT + threadIdx.x;
    if (t < n) {
      const float f = __fadd_rn(acc[t], __fdiv_rn(cw_exp(__fsub_rn(lg[t], m)), z));
      acc[t] = f;
      fmx = fmaxf(fmx, f);
    }
  }
  fmx = wave_max(fmx);
  if ((threadIdx.x & (kWave - 1)) == 0) wmax[threadIdx.x / kWave] = fmx;
  __syncthreads();
  if (threadIdx.x == 0) {
    float x = wmax[0];
    for (int w = 1; w < kGT / kWave; ++w) x = fmaxf(x, wmax[w]);
    atomicMax(reinterpret_cast<unsigned int *>(&a.key_max[row]), __float_as_uint(x));
  }
}

__global__ __launch_bounds__(kGT) void group_weights(GroupSelArgs a) {
  __shared__ float red[2][kGT / kWave];
  // group selection: one workgroup per large query head (b, layer, h), lists
  // of its group; accumulated scores: one per small head, its own lists
  const int prow = blockIdx.x;
  int b, j;
  int64_t grow;
  if (a.accum) {
    b = prow / a.nsh;
    j = prow % a.nsh;
    grow = prow;
  } else {
    const int perq = a.L * a.hq, layer = (prow % perq) / a.hq, h = prow % a.hq;
    b = prow / perq;
    grow = ((int64_t)b * a.L + layer) * a.hkv + h / a.gq;
    j = clampi(a.head_map[layer * a.hq + h], 0, a.nsh - 1);
  }
  const Sizes sz = set_sizes(a.seq_len, a.k_crit, a.k_marg, a.k_recent, b, a.n_cap, a.kc_cap,
                             a.km_cap);
  const int64_t row = (int64_t)b * a.nsh + j;
  const float m = a.row_max[row], zinv = 1.0f / a.row_sum[row];
  const float *lg = a.logits + row * a.n_cap;
  const int32_t *crit = a.crit + grow * a.kc_cap, *marg = a.marg + grow * a.km_cap;
  const int last = sz.n - 1;
  // four entries per thread per pass: their list loads, then their logit
  // loads, are in flight together (each thread still adds in k order)
  constexpr int kB = 4;
  float sc = 0.0f, sm = 0.0f;
  for (int k0 = threadIdx.x; k0 < sz.nc; k0 += kB * kGT) {
    int t[kB];
    float v[kB];
#pragma unroll
    for (int q = 0; q < kB; ++q) {
      const int k = k0 + q * kGT;
      t[q] = k < sz.nc ? clampi(crit[k], 0, last) : -1;
    }
#pragma unroll
    for (int q = 0; q < kB; ++q) v[q] = t[q] >= 0 ? lg[t[q]] : 0.0f;
#pragma unroll
    for (int q = 0; q < kB; ++q)
      if (t[q] >= 0) sc += __expf(v[q] - m) * zinv;
  }
  float *mp = a.marg_prob + (int64_t)prow * a.km_cap;
  for (int k0 = threadIdx.x; k0 < a.km_cap; k0 += kB * kGT) {
    int t[kB];
    float v[kB];
#pragma unroll
    for (int q = 0; q < kB; ++q) {
      const int k = k0 + q * kGT;
      t[q] = k < sz.nm ? clampi(marg[k], 0, last) : -1;
    }
#pragma unroll
    for (int q = 0; q < kB; ++q) v[q] = t[q] >= 0 ? lg[t[q]] : 0.0f;
#pragma unroll
    for (int q = 0; q < kB; ++q) {
      const int k = k0 + q * kGT;
      if (k < a.km_cap) {
        const float p = t[q] >= 0 ? __expf(v[q] - m) * zinv : 0.0f;
        mp[k] = p;
        sm += p;
      }
    }
  }
  sc = wave_sum(sc);
  sm = wave_sum(sm);
  if ((threadIdx.x & (kWave - 1)) == 0) {
    red[0][threadIdx.x / kWave] = sc;
    red[1][threadIdx.x / kWave] = sm;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float x = 0.0f, y = 0.0f;
    for (int w = 0; w < kGT / kWave; ++w) {
      x += red[0][w];
      y += red[1][w];
    }
    a.mass[2 * (int64_t)prow] = x;
    a.mass[2 * (int64_t)prow + 1] = y;
  }
}

GroupSelArgs group_args(const smallkv_batch_t &b, const smallkv_model_t &small,
                        const smallkv_model_t &large, const int32_t *head_map,
                        const float *logits, const float *row_max, const float *row_sum) {
  GroupSelArgs a{};
  a.n_cap = b.n_cap;
  a.nsh = small.n_layers * small.n_q_heads;
  a.L = large.n_layers;
  a.hq = large.n_q_heads;
  a.hkv = large.n_kv_heads;
  a.gq = large.n_q_heads / large.n_kv_heads;
  a.kc_cap = b.kc_cap;
  a.km_cap = b.km_cap;
  a.seq_len = b.seq_len;
  a.k_crit = b.k_crit;
  a.k_marg = b.k_marg;
  a.k_recent = b.k_recent;
  a.head_map = head_map;
  a.logits = logits;
  a.row_max = row_max;
  a.row_sum = row_sum;
  return a;
}

}  // namespace

GroupLayout group_layout(const smallkv_batch_t &b, const smallkv_model_t &small,
                         const smallkv_model_t &large, size_t offset, bool accum) {
  auto r256 = [](size_t x) { return (x + 255) / 256 * 256; };
  const size_t nsh = (size_t)small.n_layers * small.n_q_heads;
  // rows ranked: groups, or small heads for accumulated scores (whose
  // scores are the caller's state: no key buffer)
  const size_t grows = accum ? (size_t)b.batch * nsh
                             : (size_t)b.batch * large.n_layers * large.n_kv_heads;
  GroupLayout l{};
  l.zq = r256(offset);
  const size_t nzc = (size_t)(b.n_cap + kZqTok - 1) / kZqTok;
  l.keys = l.zq + r256((size_t)b.batch * nsh * nzc * sizeof(uint64_t));
  l.key_max = l.keys + (accum ? 0 : r256(grows * b.n_cap * sizeof(float)));
  l.part_mp = l.key_max + r256(grows * sizeof(float));
  l.part_mass = l.part_mp + r256(grows * (b.km_cap > 0 ? b.km_cap : 1) * sizeof(float));
  l.end = l.part_mass + r256(grows * 2 * sizeof(float));
  return l;
}

hipError_t launch_group_select(const smallkv_batch_t &b, const smallkv_model_t &small,
                               const smallkv_model_t &large, const int32_t *head_map,
                               const float *logits, const float *row_max, const float *row_sum,
                               int32_t *crit, int32_t *marg, float *marg_prob, float *mass,
                               void *ws, const GroupLayout &lay, hipStream_t st) {
  char *w = static_cast<char *>(ws);
  GroupSelArgs a = group_args(b, small, large, head_map, logits, row_max, row_sum);
  a.zq_int = reinterpret_cast<uint64_t *>(w + lay.zq);
  a.keys = reinterpret_cast<float *>(w + lay.keys);
  a.key_max = reinterpret_cast<float *>(w + lay.key_max);
  a.crit = crit;
  a.marg = marg;
  a.marg_prob = marg_prob;
  a.mass = mass;
  const int nsh = small.n_layers * small.n_q_heads;
  const int grows_per = large.n_layers * large.n_kv_heads;
  const int zrows = b.batch * nsh, grows = b.batch * grows_per;
  a.nzc = (b.n_cap + kZqTok - 1) / kZqTok;
  a.n_keymax = grows;
  hipLaunchKernelGGL(group_zq, dim3(zrows, a.nzc), dim3(kGT), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(group_scores, dim3(grows, (b.n_cap + kScoreTok - 1) / kScoreTok), dim3(kGT), 0,
                     st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // (64 bins per binade for the summed probabilities: 32 and 128 were slower)
  e = launch_group_partition(b, grows_per, a.keys, a.key_max, crit, marg,
                             reinterpret_cast<float *>(w + lay.part_mp),
                             reinterpret_cast<float *>(w + lay.part_mass), 64, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(group_weights, dim3(b.batch * large.n_layers * large.n_q_heads), dim3(kGT), 0,
                     st, a);
  return hipGetLastError();
}

}  // namespace smallkv

namespace smallkv {

hipError_t launch_accum_select(const smallkv_batch_t &b, const smallkv_model_t &small,
                               const float *logits, const float *row_max, const float *row_sum,
                               float *acc, int32_t *crit, int32_t *marg, float *marg_prob,
                               float *mass, void *ws, const GroupLayout &lay, hipStream_t st) {
  char *w = static_cast<char *>(ws);
  GroupSelArgs a = group_args(b, small, small, nullptr, logits, row_max, row_sum);
  a.accum = 1;
  a.acc = acc;
  a.zq_int = reinterpret_cast<uint64_t *>(w + lay.zq);
  a.key_max = reinterpret_cast<float *>(w + lay.key_max);
  a.crit = crit;
  a.marg = marg;
  a.marg_prob = marg_prob;
  a.mass = mass;
  const int nsh = small.n_layers * small.n_q_heads, rows = b.batch * nsh;
  a.nzc = (b.n_cap + kZqTok - 1) / kZqTok;
  a.n_keymax = rows;
  hipLaunchKernelGGL(group_zq, dim3(rows, a.nzc), dim3(kGT), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accum_scores, dim3(rows, (b.n_cap + kScoreTok - 1) / kScoreTok), dim3(kGT), 0,
                     st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // (32 bins per binade for the running scores: 64 was slower)
  e = launch_group_partition(b, nsh, acc, a.key_max, crit, marg,
                             reinterpret_cast<float *>(w + lay.part_mp),
                             reinterpret_cast<float *>(w + lay.part_mass), 32, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(group_weights, dim3(rows), dim3(kGT), 0, st, a);
  return hipGetLastError();
}

}  // namespace smallkv
