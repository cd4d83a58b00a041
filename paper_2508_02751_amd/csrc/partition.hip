// Stage 2: the top-k partition of each small head's tokens into critical,
// marginal and evicted sets (Eq. 4 read as "keep the top-scored tokens";
// Eq. 6: TopK is critical, Top(P-K) -- the next P-K of the same order -- is
// marginal).  Tokens are ordered by (logit descending, index ascending).
//
// One workgroup per (sequence, small head) row:
//   1. radix select on order-preserving uint32 keys, 11+11+10 bits, finds the
//      key T_C of the |C|-th token and T_P of the (|C|+|M|)-th token, and how
//      many tokens equal to each threshold are taken (lowest indices first);
//   2. one ordered pass compacts C and M in ascending token order with
//      wave ballots and a workgroup prefix, computes p' for marginal tokens
//      and the masses S'_C, S'_M.
// The result depends only on the logits, so it is deterministic.
#include "common.h"
#include "launch.h"

namespace smallkv {
namespace {

constexpr int kPT = 512;            // threads per row
constexpr int kWaves = kPT / kWave;
constexpr int kBins = 2048;         // largest digit: 11 bits

struct PartArgs {
  int n_cap, nsh, kc_cap, km_cap;
  const int32_t *seq_len, *k_crit, *k_marg;
  const float *logits, *row_max, *row_sum;
  int32_t *crit, *marg;
  float *marg_prob, *mass;
};

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Find, in a descending scan of hist[0..nb), the digit holding the rr-th
// element (1-based); returns the digit and the count strictly above it.
// Executed by one whole wave.
__device__ __forceinline__ void find_digit(const uint32_t *hist, int nb, uint32_t rr, int &digit,
                                           uint32_t &above) {
  const int lane = threadIdx.x & 63;
  const int per = nb / kWave;  // bins per lane; lane 0 owns the highest bins
  const int hi = nb - 1 - lane * per;
  uint32_t s = 0;
  for (int k = 0; k < per; ++k) s += hist[hi - k];
  // inclusive prefix over lanes
  uint32_t inc = s;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(inc, o, kWave);
    if (lane >= o) inc += y;
  }
  const uint32_t exc = inc - s;
  const bool mine = exc < rr && rr <= inc;
  const uint64_t who = __ballot(mine);
  const int src = who ? __ffsll((unsigned long long)who) - 1 : 0;
  int dsel = 0;
  uint32_t ab = 0;
  if (lane == src) {
    uint32_t cum = exc;
    for (int k = 0; k < per; ++k) {
      const uint32_t h = hist[hi - k];
      if (cum + h >= rr) {
        dsel = hi - k;
        break;
      }
      cum += h;
    }
    ab = cum;
  }
  digit = __shfl(dsel, src, kWave);
  above = __shfl(ab, src, kWave);
}

__global__ __launch_bounds__(kPT) void partition_kernel(PartArgs a) {
  __shared__ uint32_t hist[2][kBins];
  __shared__ uint32_t sel[2][3];     // per target: prefix, mask, remaining rank
  __shared__ uint32_t wtot[2][4][kWaves];
  __shared__ float wsum[2][kWaves];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = blockIdx.x, b = row / a.nsh;
  const Sizes sz = set_sizes(a.seq_len, a.k_crit, a.k_marg, b, a.n_cap, a.kc_cap, a.km_cap);
  const int n = sz.n, nc = sz.nc, nm = sz.nm;
  const float *lg = a.logits + (int64_t)row * a.n_cap;
  int32_t *crit = a.crit + (int64_t)row * a.kc_cap;
  int32_t *marg = a.marg + (int64_t)row * a.km_cap;
  float *mp = a.marg_prob + (int64_t)row * a.km_cap;

  if (tid < 2) {
    sel[tid][0] = 0;
    sel[tid][1] = 0;
    sel[tid][2] = (uint32_t)(tid == 0 ? nc : nc + nm);
  }
  // ---- radix select: digits of 11, 11 and 10 bits -----------------------
  const int shifts[3] = {21, 10, 0};
  const int nbits[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = shifts[pass], nb = 1 << nbits[pass];
    const uint32_t dmask = (uint32_t)nb - 1u;
    for (int x = tid; x < 2 * kBins; x += kPT) (&hist[0][0])[x] = 0;
    __syncthreads();
    const uint32_t p0 = sel[0][0], m0 = sel[0][1], p1 = sel[1][0], m1 = sel[1][1];
    for (int t = tid; t < n; t += kPT) {
      const uint32_t u = logit_key(lg[t]);
      const uint32_t dg = (u >> sh) & dmask;
      if ((u & m0) == p0) atomicAdd(&hist[0][dg], 1u);
      if ((u & m1) == p1) atomicAdd(&hist[1][dg], 1u);
    }
    __syncthreads();
    if (wave < 2) {
      int digit;
      uint32_t above;
      find_digit(hist[wave], nb, sel[wave][2], digit, above);
      if (lane == 0) {
        sel[wave][0] |= (uint32_t)digit << sh;
        sel[wave][1] |= dmask << sh;
        sel[wave][2] -= above;
      }
    }
    __syncthreads();
  }
  const uint32_t TC = sel[0][0], TP = sel[1][0];
  const uint32_t needC = sel[0][2], needP = sel[1][2];  // ties taken at each threshold

  // ---- ordered compaction -----------------------------------------------
  const float M = a.row_max[row];
  const float Zinv = 1.0f / a.row_sum[row];
  uint32_t carry_eqC = 0, carry_eqP = 0, carry_c = 0, carry_m = 0;
  float sc = 0.0f, sm = 0.0f;
  const uint64_t lt = lanemask_lt();
  int par = 0;
  for (int base = 0; base < n; base += kPT, par ^= 1) {
    const int t = base + tid;
    const bool valid = t < n;
    const float s = valid ? lg[t] : 0.0f;
    const uint32_t u = logit_key(s);
    const bool eqC = valid && u == TC, eqP = valid && u == TP;
    const uint64_t bC = __ballot(eqC), bP = __ballot(eqP);
    if (lane == 0) {
      wtot[par][0][wave] = __popcll(bC);
      wtot[par][1][wave] = __popcll(bP);
    }
    __syncthreads();
    uint32_t offC = carry_eqC, offP = carry_eqP, totC = 0, totP = 0;
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t xc = wtot[par][0][w], xp = wtot[par][1][w];
      if (w < wave) {
        offC += xc;
        offP += xp;
      }
      totC += xc;
      totP += xp;
    }
    const uint32_t rC = offC + __popcll(bC & lt), rP = offP + __popcll(bP & lt);
    const bool inC = valid && (u > TC || (eqC && rC < needC));
    const bool inP = valid && (u > TP || (eqP && rP < needP));
    const bool inM = inP && !inC;
    const uint64_t cC = __ballot(inC), cM = __ballot(inM);
    if (lane == 0) {
      wtot[par][2][wave] = __popcll(cC);
      wtot[par][3][wave] = __popcll(cM);
    }
    __syncthreads();
    uint32_t posC = carry_c, posM = carry_m, nC = 0, nM = 0;
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t xc = wtot[par][2][w], xm = wtot[par][3][w];
      if (w < wave) {
        posC += xc;
        posM += xm;
      }
      nC += xc;
      nM += xm;
    }
    if (inC || inM) {
      const float p = __expf(s - M) * Zinv;
      // the guards only matter if the select were wrong: never write past a row
      if (inC) {
        const uint32_t k = posC + __popcll(cC & lt);
        if (k < (uint32_t)nc) crit[k] = t;
        sc += p;
      } else {
        const uint32_t k = posM + __popcll(cM & lt);
        if (k < (uint32_t)nm) {
          marg[k] = t;
          mp[k] = p;
        }
        sm += p;
      }
    }
    carry_eqC += totC;
    carry_eqP += totP;
    carry_c += nC;
    carry_m += nM;
  }
  for (int i = nc + tid; i < a.kc_cap; i += kPT) crit[i] = -1;
  for (int i = nm + tid; i < a.km_cap; i += kPT) {
    marg[i] = -1;
    mp[i] = 0.0f;
  }
  sc = wave_sum(sc);
  sm = wave_sum(sm);
  if (lane == 0) {
    wsum[0][wave] = sc;
    wsum[1][wave] = sm;
  }
  __syncthreads();
  if (tid == 0) {
    float x = 0.0f, y = 0.0f;
    for (int w = 0; w < kWaves; ++w) {
      x += wsum[0][w];
      y += wsum[1][w];
    }
    a.mass[2 * (int64_t)row] = x;
    a.mass[2 * (int64_t)row + 1] = y;
  }
}

}  // namespace

hipError_t launch_partition(const smallkv_batch_t &b, int n_small_heads, const float *logits,
                            const float *row_max, const float *row_sum, int32_t *crit,
                            int32_t *marg, float *marg_prob, float *mass, hipStream_t st) {
  PartArgs a;
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
  hipLaunchKernelGGL(partition_kernel, dim3(b.batch * n_small_heads), dim3(kPT), 0, st, a);
  return hipGetLastError();
}

}  // namespace smallkv
