// Stage 2: the top-k partition of each small head's tokens into critical,
// marginal and evicted sets (Eq. 4 read as "keep the top-scored tokens";
// Eq. 6: TopK is critical, Top(P-K) -- the next P-K of the same order -- is
// marginal).  Tokens are ordered by (logit descending, index ascending).
//
// One workgroup per (sequence, small head) row.  For the |C|-th and the
// (|C|+|M|)-th token of the order ("targets"):
//   1. a 2048-bin histogram of a monotone bin of the logit -- its distance
//      to the row max in steps of 1/64 -- locates each target's bin without
//      the atomic pile-up that raw key bits give (logits share their top
//      bits);
//   2. the keys of each target's bin are gathered into LDS and an exact
//      11+11+10-bit radix select among them gives the target key T and how
//      many tokens equal to T it takes (the lowest indices); a bin too full
//      for LDS is selected from the whole row instead;
//   3. one ordered pass compacts C and M in ascending token order with
//      workgroup prefix sums, computes p' for marginal tokens and the masses
//      S'_C, S'_M.
// Rows up to 16384 tokens are read once, 4 consecutive logits per thread
// per 2048-token chunk, and kept in registers for all passes; longer rows
// are re-read per pass, four chunks in flight at a time.  The fused variants first combine stage 1's per-chunk
// partials of their head (row max, row sum, the head's output), so a step
// needs no separate merge launch.  Deterministic.
#include "common.h"
#include "launch.h"
#include "merge.h"

namespace smallkv {
namespace {

constexpr int kPT = 512;  // threads per row
constexpr int kWaves = kPT / kWave;
constexpr int kBins = 2048;
constexpr int kCap = 4096;  // candidate keys per target kept in LDS
constexpr int kChunk = 4 * kPT;  // tokens per register chunk

struct PartArgs {
  int n_cap, nsh, kc_cap, km_cap;
  const int32_t *seq_len, *k_crit, *k_marg;
  const float *logits;
  float *row_max, *row_sum;  // read (standalone) or written (fused)
  int32_t *crit, *marg;
  float *marg_prob, *mass;
  // fused merge of stage 1
  const float *part;
  void *small_out;
  int layers, hq, hkv, g, chunk, n_split, d, gp, out_bf16;
};

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Monotone non-decreasing bin of a logit below the row max M: 2047 for the
// top 1/64 of a logit unit, one bin per further 1/64, 0 for everything more
// than 32 below.  Explicitly rounded ops so every pass computes the same bin.
__device__ __forceinline__ int logit_bin(float s, float M) {
  float d = __fmul_rn(__fsub_rn(M, s), 64.0f);
  d = fminf(fmaxf(d, 0.0f), 2047.0f);
  return 2047 - (int)d;
}

// One wave: find the bin of hist[0..NB) (scanned from the top) holding the
// rr-th element (1-based); returns the bin and the count strictly above it.
// Each lane owns NB/64 consecutive bins (lane 0 the highest) and scans them
// in registers.
template <int NB>
__device__ __forceinline__ void find_digit(const uint32_t *hist, uint32_t rr, int &digit,
                                           uint32_t &above) {
  constexpr int PER = NB / kWave;
  const int lane = threadIdx.x & 63;
  const int lo = NB - (lane + 1) * PER;  // this lane's bins: lo .. lo+PER-1
  uint32_t hv[PER];
#pragma unroll
  for (int k = 0; k < PER; k += 4) {
    const uint4 v = *reinterpret_cast<const uint4 *>(hist + lo + k);
    hv[k] = v.x;
    hv[k + 1] = v.y;
    hv[k + 2] = v.z;
    hv[k + 3] = v.w;
  }
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) s += hv[k];
  uint32_t inc = s;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(inc, o, kWave);
    if (lane >= o) inc += y;
  }
  const uint32_t exc = inc - s;  // elements in the bins above this lane's
  const uint64_t who = __ballot(exc < rr && rr <= inc);
  const int src = who ? __ffsll((unsigned long long)who) - 1 : 0;
  // every lane scans its own bins from the top; lane src's answer is used
  uint32_t cum = exc, ab = exc;
  int dsel = lo;
  bool found = false;
#pragma unroll
  for (int k = PER - 1; k >= 0; --k) {
    const bool hit = !found && cum + hv[k] >= rr;
    dsel = hit ? lo + k : dsel;
    ab = hit ? cum : ab;
    found = found || hit;
    cum += hv[k];
  }
  digit = __shfl(dsel, src, kWave);
  above = __shfl(ab, src, kWave);
}

// Inclusive prefix sum over the wave (64 lanes).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(v, o, kWave);
    if (lane >= o) v += y;
  }
  return v;
}

struct alignas(16) PartShared {
  uint32_t hist[2][kBins];
  union {  // the merge's chunk weights are dead before candidates are gathered
    uint32_t cand[2][kCap];
    float mw[kMaxChunks];
  };
  uint32_t sel[2][4];  // per target: prefix, mask, remaining rank, bin
  uint32_t res[2][2];  // per target selected by counting: key, ties taken
  uint32_t ncand[2];
  uint32_t wtot[2][2][kWaves];
  float wsum[2][kWaves];
  float mred[kWaves + kPT];
};
static_assert(sizeof(float) * kMaxChunks <= sizeof(uint32_t) * 2 * kCap, "mw fits in cand");

struct RowCtx {
  int row, n, nc, nm;
  const float *lg;
  int32_t *crit, *marg;
  float *mp;
  float M, Z;
};

template <bool kMerge>
__device__ __forceinline__ void row_setup(const PartArgs &a, PartShared &sh, RowCtx &r) {
  r.row = blockIdx.x;
  const int b = r.row / a.nsh;
  const Sizes sz = set_sizes(a.seq_len, a.k_crit, a.k_marg, b, a.n_cap, a.kc_cap, a.km_cap);
  r.n = sz.n;
  r.nc = sz.nc;
  r.nm = sz.nm;
  r.lg = a.logits + (int64_t)r.row * a.n_cap;
  r.crit = a.crit + (int64_t)r.row * a.kc_cap;
  r.marg = a.marg + (int64_t)r.row * a.km_cap;
  r.mp = a.marg_prob + (int64_t)r.row * a.km_cap;
  if constexpr (kMerge) {
    const int j = r.row % a.nsh, layer = j / a.hq, h = j % a.hq;
    const int unit = (b * a.layers + layer) * a.hkv + h / a.g, i = h % a.g;
    MergeIn in;
    in.stride = (int64_t)a.gp * (a.d + 2);
    in.part = a.part + (int64_t)unit * a.n_split * in.stride + i * (a.d + 2);
    in.nv = (r.n + a.chunk - 1) / a.chunk;
    void *out = a.small_out;
    const int64_t o0 = (int64_t)r.row * a.d;
    const bool bf = a.out_bf16;
    merge_head<kPT>(in, a.d, sh.mw, sh.mred, r.M, r.Z, [&](int c, float v) {
      if (bf)
        elem<bf16_t>::store1(out, o0 + c, v);
      else
        elem<float>::store1(out, o0 + c, v);
    });
    if (threadIdx.x == 0) {
      a.row_max[r.row] = r.M;
      a.row_sum[r.row] = r.Z;
    }
  } else {
    r.M = a.row_max[r.row];
    r.Z = a.row_sum[r.row];
  }
}

// The row as seen by the passes: chunk k holds tokens [k*kChunk, (k+1)*kChunk),
// 4 consecutive tokens per thread (token of value e = k*kChunk + 4*tid + e).
// R > 0: the row sits in R registers per thread, read from memory once.
// R == 0: every pass reads it from memory, four chunks in flight at a time.
template <int R>
struct Row {
  float s[R > 0 ? R : 4];
  const float *lg;
  int n;

  bool aligned;  // 16-byte aligned row: whole chunks load as one float4

  __device__ __forceinline__ float4 fetch(int k) const {
    const int t = k * kChunk + 4 * (int)threadIdx.x;
    float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (aligned && t + 3 < n) {
      v = *reinterpret_cast<const float4 *>(lg + t);
    } else {
      if (t < n) v.x = lg[t];
      if (t + 1 < n) v.y = lg[t + 1];
      if (t + 2 < n) v.z = lg[t + 2];
      if (t + 3 < n) v.w = lg[t + 3];
    }
    return v;
  }
  __device__ __forceinline__ void load() {
    if constexpr (R > 0) {
#pragma unroll
      for (int k = 0; k < R / 4; ++k) {
        const float4 v = fetch(k);
        s[4 * k] = v.x;
        s[4 * k + 1] = v.y;
        s[4 * k + 2] = v.z;
        s[4 * k + 3] = v.w;
      }
    }
  }
  __device__ __forceinline__ float4 chunk(int k) const {
    if constexpr (R > 0)
      return make_float4(s[4 * k], s[4 * k + 1], s[4 * k + 2], s[4 * k + 3]);
    else
      return fetch(k);
  }
  __device__ __forceinline__ int chunks() const { return (n + kChunk - 1) / kChunk; }
  __device__ __forceinline__ bool valid(int k, int e) const {
    return k * kChunk + 4 * (int)threadIdx.x + e < n;
  }
  // f(value, valid) for every slot of every chunk, with the wave converged
  template <typename F>
  __device__ __forceinline__ void each(F f) const {
    if constexpr (R > 0) {
#pragma unroll
      for (int k = 0; k < R / 4; ++k) {
        if (k * kChunk >= n) break;
#pragma unroll
        for (int e = 0; e < 4; ++e) f(s[4 * k + e], valid(k, e));
      }
    } else {
      const int nk = chunks();
      for (int k0 = 0; k0 < nk; k0 += 4) {
        float4 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = k0 + j < nk ? fetch(k0 + j) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          f(v[j].x, valid(k0 + j, 0));
          f(v[j].y, valid(k0 + j, 1));
          f(v[j].z, valid(k0 + j, 2));
          f(v[j].w, valid(k0 + j, 3));
        }
      }
    }
  }
};

// Steps 1 and 2: the two target keys and the ties each takes.
template <typename Row>
__device__ __forceinline__ void select_targets(PartShared &sh, const RowCtx &r, const Row &row,
                                               uint32_t &TC, uint32_t &TP, uint32_t &needC,
                                               uint32_t &needP) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float M = r.M;
  for (int x = tid; x < kBins; x += kPT) sh.hist[0][x] = 0;
  if (tid < 2) {
    sh.sel[tid][0] = 0;
    sh.sel[tid][1] = 0;
    sh.sel[tid][2] = (uint32_t)(tid == 0 ? r.nc : r.nc + r.nm);
    sh.ncand[tid] = 0;
  }
  __syncthreads();
  row.each([&](float s, bool valid) {
    if (valid) atomicAdd(&sh.hist[0][logit_bin(s, M)], 1u);
  });
  __syncthreads();
  if (wave < 2) {
    int bin;
    uint32_t above;
    find_digit<kBins>(sh.hist[0], sh.sel[wave][2], bin, above);
    if (lane == 0) {
      sh.sel[wave][2] -= above;
      sh.sel[wave][3] = (uint32_t)bin;
    }
  }
  __syncthreads();
  const int bin0 = (int)sh.sel[0][3], bin1 = (int)sh.sel[1][3];
  const bool lds0 = sh.hist[0][bin0] <= (uint32_t)kCap, lds1 = sh.hist[0][bin1] <= (uint32_t)kCap;
  if (lds0 || lds1) {
    // gather the candidate keys (order inside a bin does not matter here)
    const uint64_t lt = lanemask_lt();
    row.each([&](float s, bool valid) {
      const int bn = valid ? logit_bin(s, M) : -1;
      const uint32_t u = logit_key(s);
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const bool take = (x == 0 ? lds0 : lds1) && bn == (x == 0 ? bin0 : bin1);
        const uint64_t bal = __ballot(take);
        if (bal) {  // one LDS atomic per wave
          uint32_t off = 0;
          if (lane == 0) off = atomicAdd(&sh.ncand[x], (uint32_t)__popcll(bal));
          off = __shfl(off, 0, kWave);
          if (take) sh.cand[x][off + __popcll(bal & lt)] = u;
        }
      }
    });
  }
  __syncthreads();  // candidates and their counts visible
  // few candidates: rank each one by counting (all pairs), no radix passes
  const uint32_t nc0 = lds0 ? sh.ncand[0] : 0u, nc1 = lds1 ? sh.ncand[1] : 0u;
  const bool cnt0 = lds0 && nc0 <= (uint32_t)kPT, cnt1 = lds1 && nc1 <= (uint32_t)kPT;
#pragma unroll
  for (int x = 0; x < 2; ++x) {
    const bool cnt = x == 0 ? cnt0 : cnt1;
    const uint32_t nx = x == 0 ? nc0 : nc1;
    if (cnt && (uint32_t)tid < nx) {
      const uint32_t key = sh.cand[x][tid];
      uint32_t gt = 0, eq = 0;
      for (uint32_t c = 0; c < nx; ++c) {
        const uint32_t v = sh.cand[x][c];
        gt += v > key ? 1u : 0u;
        eq += v == key ? 1u : 0u;
      }
      const uint32_t rr = sh.sel[x][2];
      if (gt < rr && rr <= gt + eq) {  // every tie of the target writes the same values
        sh.res[x][0] = key;
        sh.res[x][1] = rr - gt;
      }
    }
  }
  const bool lds0r = lds0 && !cnt0, lds1r = lds1 && !cnt1;  // radix over LDS candidates
  const bool need_radix = !cnt0 || !cnt1;
  for (int pass = 0; need_radix && pass < 3; ++pass) {  // digits of 11, 11 and 10 bits
    const int shf = pass == 0 ? 21 : (pass == 1 ? 10 : 0), nb = pass < 2 ? 2048 : 1024;
    const uint32_t dmask = (uint32_t)nb - 1u;
    __syncthreads();  // candidates / previous selection visible; hist free
    for (int x = tid; x < 2 * kBins; x += kPT) (&sh.hist[0][0])[x] = 0;
    __syncthreads();
    const uint32_t p0 = sh.sel[0][0], m0 = sh.sel[0][1], p1 = sh.sel[1][0], m1 = sh.sel[1][1];
    if (lds0r)
      for (int k = tid; k < (int)sh.ncand[0]; k += kPT) {
        const uint32_t u = sh.cand[0][k];
        if ((u & m0) == p0) atomicAdd(&sh.hist[0][(u >> shf) & dmask], 1u);
      }
    if (lds1r)
      for (int k = tid; k < (int)sh.ncand[1]; k += kPT) {
        const uint32_t u = sh.cand[1][k];
        if ((u & m1) == p1) atomicAdd(&sh.hist[1][(u >> shf) & dmask], 1u);
      }
    if (!lds0 || !lds1)  // a bin too full for LDS: select it from the row
      row.each([&](float s, bool valid) {
        const int bn = valid ? logit_bin(s, M) : -1;
        const uint32_t u = logit_key(s);
        if (!lds0 && bn == bin0 && (u & m0) == p0) atomicAdd(&sh.hist[0][(u >> shf) & dmask], 1u);
        if (!lds1 && bn == bin1 && (u & m1) == p1) atomicAdd(&sh.hist[1][(u >> shf) & dmask], 1u);
      });
    __syncthreads();
    if (wave < 2) {
      int digit;
      uint32_t above;
      if (pass < 2)
        find_digit<2048>(sh.hist[wave], sh.sel[wave][2], digit, above);
      else
        find_digit<1024>(sh.hist[wave], sh.sel[wave][2], digit, above);
      if (lane == 0) {
        sh.sel[wave][0] |= (uint32_t)digit << shf;
        sh.sel[wave][1] |= dmask << shf;
        sh.sel[wave][2] -= above;
      }
    }
  }
  __syncthreads();
  TC = cnt0 ? sh.res[0][0] : sh.sel[0][0];
  TP = cnt1 ? sh.res[1][0] : sh.sel[1][0];
  needC = cnt0 ? sh.res[0][1] : sh.sel[0][2];
  needP = cnt1 ? sh.res[1][1] : sh.sel[1][2];
}

// Workgroup exclusive prefix of a packed pair of 16-bit counts (per chunk
// totals stay below 65536); returns this thread's offset and the total.
__device__ __forceinline__ void block_scan2(PartShared &sh, int par, int slot, uint32_t v,
                                            uint32_t &excl, uint32_t &total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t inc = wave_incl_scan(v);
  if (lane == 63) sh.wtot[par][slot][wave] = inc;
  __syncthreads();
  uint32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t x = sh.wtot[par][slot][w];
    off += w < wave ? x : 0u;
    tot += x;
  }
  excl = off + inc - v;
  total = tot;
}

__device__ __forceinline__ void finish_row(const PartArgs &a, PartShared &sh, const RowCtx &r,
                                           float sc, float sm) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = r.nc + tid; i < a.kc_cap; i += kPT) r.crit[i] = -1;
  for (int i = r.nm + tid; i < a.km_cap; i += kPT) {
    r.marg[i] = -1;
    r.mp[i] = 0.0f;
  }
  sc = wave_sum(sc);
  sm = wave_sum(sm);
  if (lane == 0) {
    sh.wsum[0][wave] = sc;
    sh.wsum[1][wave] = sm;
  }
  __syncthreads();
  if (tid == 0) {
    float x = 0.0f, y = 0.0f;
    for (int w = 0; w < kWaves; ++w) {
      x += sh.wsum[0][w];
      y += sh.wsum[1][w];
    }
    a.mass[2 * (int64_t)r.row] = x;
    a.mass[2 * (int64_t)r.row + 1] = y;
  }
}

// ---------------------------------------------------------------- kernel --

template <bool kMerge, int R>
__global__ __launch_bounds__(kPT) void partition_kernel(PartArgs a) {
  __shared__ PartShared sh;
  RowCtx r;
  row_setup<kMerge>(a, sh, r);
  const int tid = threadIdx.x;
  Row<R> row;
  row.lg = r.lg;
  row.n = r.n;
  row.aligned = (reinterpret_cast<uintptr_t>(r.lg) & 15) == 0;
  row.load();
  uint32_t TC, TP, needC, needP;
  select_targets(sh, r, row, TC, TP, needC, needP);

  // ordered compaction, one chunk at a time
  const float Zinv = 1.0f / r.Z;
  uint32_t carry_eqC = 0, carry_eqP = 0, carry_c = 0, carry_m = 0;
  float sc = 0.0f, sm = 0.0f;
  const int nk = row.chunks();
  auto compact = [&](int k, const float4 cur) {
    const float sv[4] = {cur.x, cur.y, cur.z, cur.w};
    const int par = k & 1;
    const int t0 = k * kChunk + 4 * tid;
    uint32_t u[4];
    bool eqC[4], eqP[4];
    uint32_t cnt = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool valid = t0 + e < r.n;
      u[e] = logit_key(sv[e]);
      eqC[e] = valid && u[e] == TC;
      eqP[e] = valid && u[e] == TP;
      cnt += (eqC[e] ? 1u : 0u) + (eqP[e] ? 0x10000u : 0u);
    }
    uint32_t ex, tot;
    block_scan2(sh, par, 0, cnt, ex, tot);
    uint32_t rC = carry_eqC + (ex & 0xffffu), rP = carry_eqP + (ex >> 16);
    bool inC[4], inM[4];
    uint32_t cm = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool valid = t0 + e < r.n;
      inC[e] = valid && (u[e] > TC || (eqC[e] && rC < needC));
      const bool inP = valid && (u[e] > TP || (eqP[e] && rP < needP));
      inM[e] = inP && !inC[e];
      rC += eqC[e] ? 1u : 0u;
      rP += eqP[e] ? 1u : 0u;
      cm += (inC[e] ? 1u : 0u) + (inM[e] ? 0x10000u : 0u);
    }
    carry_eqC += tot & 0xffffu;
    carry_eqP += tot >> 16;
    block_scan2(sh, par, 1, cm, ex, tot);
    uint32_t pc = carry_c + (ex & 0xffffu), pm = carry_m + (ex >> 16);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float p = (inC[e] || inM[e]) ? __expf(sv[e] - r.M) * Zinv : 0.0f;
      sc += inC[e] ? p : 0.0f;
      sm += inM[e] ? p : 0.0f;
      // the guards only matter if the select were wrong: never write past a row
      if (inC[e] && pc < (uint32_t)r.nc) r.crit[pc] = t0 + e;
      if (inM[e] && pm < (uint32_t)r.nm) {
        r.marg[pm] = t0 + e;
        r.mp[pm] = p;
      }
      pc += inC[e] ? 1u : 0u;
      pm += inM[e] ? 1u : 0u;
    }
    carry_c += tot & 0xffffu;
    carry_m += tot >> 16;
  };
  if constexpr (R > 0) {
#pragma unroll
    for (int k = 0; k < R / 4; ++k) {
      if (k >= nk) break;
      compact(k, row.chunk(k));
    }
  } else {
    float4 nxt = row.chunk(0);
    for (int k = 0; k < nk; ++k) {
      const float4 cur = nxt;
      if (k + 1 < nk) nxt = row.chunk(k + 1);  // in flight during this chunk's scans
      compact(k, cur);
    }
  }
  finish_row(a, sh, r, sc, sm);
}

PartArgs base_args(const smallkv_batch_t &b, int n_small_heads, const float *logits,
                   float *row_max, float *row_sum, int32_t *crit, int32_t *marg,
                   float *marg_prob, float *mass) {
  PartArgs a{};
  a.n_cap = b.n_cap;
  a.nsh = n_small_heads;
  a.kc_cap = b.kc_cap;
  a.km_cap = b.km_cap;
  a.seq_len = b.seq_len;
  a.k_crit = b.k_crit;
  a.k_marg = b.k_marg;
  a.logits = logits;
  a.row_max = row_max;
  a.row_sum = row_sum;
  a.crit = crit;
  a.marg = marg;
  a.marg_prob = marg_prob;
  a.mass = mass;
  return a;
}

template <bool kMerge>
hipError_t launch_rows(const PartArgs &a, int rows, hipStream_t st) {
  const dim3 grid(rows), block(kPT);
  const int n = a.n_cap;
  if (n <= 4 * kPT)
    hipLaunchKernelGGL((partition_kernel<kMerge, 4>), grid, block, 0, st, a);
  else if (n <= 8 * kPT)
    hipLaunchKernelGGL((partition_kernel<kMerge, 8>), grid, block, 0, st, a);
  else if (n <= 16 * kPT)
    hipLaunchKernelGGL((partition_kernel<kMerge, 16>), grid, block, 0, st, a);
  else if (n <= 32 * kPT)
    hipLaunchKernelGGL((partition_kernel<kMerge, 32>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((partition_kernel<kMerge, 0>), grid, block, 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_partition(const smallkv_batch_t &b, int n_small_heads, const float *logits,
                            const float *row_max, const float *row_sum, int32_t *crit,
                            int32_t *marg, float *marg_prob, float *mass, hipStream_t st) {
  const PartArgs a = base_args(b, n_small_heads, logits, const_cast<float *>(row_max),
                               const_cast<float *>(row_sum), crit, marg, marg_prob, mass);
  return launch_rows<false>(a, b.batch * n_small_heads, st);
}

hipError_t launch_merge_partition(const smallkv_batch_t &b, const smallkv_model_t &m,
                                  const SmallPlan &p, const float *ws, const float *logits,
                                  float *row_max, float *row_sum, int32_t *crit, int32_t *marg,
                                  float *marg_prob, float *mass, hipStream_t st) {
  const int nsh = m.n_layers * m.n_q_heads;
  PartArgs a = base_args(b, nsh, logits, row_max, row_sum, crit, marg, marg_prob, mass);
  a.part = ws;
  a.small_out = m.out;
  a.layers = m.n_layers;
  a.hq = m.n_q_heads;
  a.hkv = m.n_kv_heads;
  a.g = m.n_q_heads / m.n_kv_heads;
  a.chunk = p.chunk;
  a.n_split = p.n_split;
  a.d = m.head_dim;
  a.gp = p.gp;
  a.out_bf16 = m.dtype == SMALLKV_BF16;
  return launch_rows<true>(a, b.batch * nsh, st);
}

}  // namespace smallkv
