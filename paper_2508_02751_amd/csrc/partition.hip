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
//   2. the keys of each target's bin are gathered into LDS and ranked
//      exactly: by counting all pairs when the bin is small, else by an
//      11+11+10-bit radix select (over LDS, or over the row when the bin
//      exceeds the LDS buffer).  This gives the target key T, how many
//      tokens equal to T the set takes (the lowest indices) and how many
//      tokens equal T in all;
//   3. one ordered pass compacts C and M in ascending token order with
//      workgroup prefix sums (DPP wave scans), computes p' for marginal
//      tokens and the masses S'_C, S'_M.  Tie ranks are scanned only when a
//      threshold's ties are split between two sets.
// Rows of up to 16 (20 with 256 threads) logits per thread are read once,
// 4 consecutive logits per thread per chunk, and kept in registers; their
// compaction needs a single barrier.  Longer rows are re-read per pass, four
// chunks in flight.  Many rows (several per CU) get 256 threads each, so
// that more rows are resident; few rows get 512.  The fused variant first
// combines stage 1's per-chunk records of its head (row max, row sum, the
// head's output), so a step needs no separate merge launch.
// The result depends only on the logits: deterministic.
#include "common.h"
#include "launch.h"
#include "merge.h"

namespace smallkv {
namespace {

// PT: threads per row (a template parameter: 256 when many rows share the
// GPU, 512 or 1024 when a few rows must finish fast)
constexpr int kBins = 2048;
// With 512 or more threads per row, histograms keep 16 bytes of padding
// after every 32 bins: find_digit's lanes each read 32 consecutive bins, and
// the 144-byte stride between lanes puts the 16 lanes of an access on
// distinct banks (a 128-byte stride piles them 8 deep on the same ones).
// Narrow rows are bound by their per-logit passes instead, where the padded
// index costs two instructions per logit.
template <int PT>
struct Hist {
  static constexpr bool pad = PT >= 512;
  static constexpr int size = pad ? kBins + kBins / 8 : kBins;
  static __device__ __forceinline__ int idx(int b) { return pad ? b + (b >> 5) * 4 : b; }
};
constexpr int kCap = 2048;       // candidate keys per target kept in LDS
constexpr int kMaxNK = 5;        // chunks of a register-cached row
template <int PT>
struct PC {
  static constexpr int waves = PT / kWave;
  static constexpr int chunk = 4 * PT;  // tokens per chunk (4 per thread)
};

struct PartArgs {
  int n_cap, nsh, kc_cap, km_cap;
  const int32_t *seq_len, *k_crit, *k_marg, *k_recent;
  const float *logits;
  float *row_max, *row_sum;  // read (standalone) or written (fused)
  int32_t *crit, *marg;
  float *marg_prob, *mass;
  // fused merge of stage 1
  const float *part;
  void *small_out;
  int layers, hq, hkv, g, chunk, n_split, d, gp, out_bf16;
  // optional list offsets, [rows][nblk]: (critical, marginal) entries before
  // each 256-token boundary of the row (written when not null)
  int2 *tab;
  int nblk;
  // optional (fused only): the small model's held rows -> token positions,
  // [B][layers][hkv][n_cap] (n_cap = rows per kv head here), clamped below
  // tok_len[b]
  const int32_t *row_pos, *tok_len;
  int tok_cap;
  float pscale;  // probability keys: the bin scale (see plog2)
};

// Raw buffer views: an access at an offset at or past the view's size reads
// zero / writes nothing, without touching memory, so masked lanes need no
// branch (exec-mask regions around every conditional store cost more than
// the stores).
constexpr uint32_t kOOB = 0x80000000u;
constexpr int kBufWord3 = 0x00020000;  // gfx9 raw buffer descriptor word 3 (32-bit data)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, (int)bytes, kBufWord3);
}

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

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_shift(uint32_t v) {
  // lanes without a source (or outside ROW_MASK) read 0
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xf, false);
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP: shifts of 1, 2,
// 4, 8 inside each 16-lane row, then the row ends broadcast to the next rows.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += dpp_shift<0x111, 0xf>(v);  // row_shr:1
  v += dpp_shift<0x112, 0xf>(v);  // row_shr:2
  v += dpp_shift<0x114, 0xf>(v);  // row_shr:4
  v += dpp_shift<0x118, 0xf>(v);  // row_shr:8
  v += dpp_shift<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
  v += dpp_shift<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3
  return v;
}

// One wave: find the bin of hist[0..NB) (scanned from the top) holding the
// rr-th element (1-based); returns the bin and the count strictly above it.
// Each lane owns NB/64 consecutive bins (lane 0 the highest) in registers.
template <int NB, int PT>
__device__ __forceinline__ void find_digit(const uint32_t *hist, uint32_t rr, int &digit,
                                           uint32_t &above) {
  constexpr int PER = NB / kWave;
  const int lane = threadIdx.x & 63;
  const int lo = NB - (lane + 1) * PER;  // this lane's bins: lo .. lo+PER-1
  uint32_t hv[PER];
#pragma unroll
  for (int k = 0; k < PER; k += 4) {
    const uint4 v = *reinterpret_cast<const uint4 *>(hist + Hist<PT>::idx(lo) + k);  // inside one 32-bin group
    hv[k] = v.x;
    hv[k + 1] = v.y;
    hv[k + 2] = v.z;
    hv[k + 3] = v.w;
  }
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) s += hv[k];
  const uint32_t inc = wave_incl_scan(s);
  const uint32_t exc = inc - s;  // elements in the bins above this lane's
  const uint64_t who = __ballot(exc < rr && rr <= inc);
  const int src = who ? __ffsll((unsigned long long)who) - 1 : 0;
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

template <int PT>
struct alignas(16) PartShared {
  uint32_t hist[2][Hist<PT>::size];  // bin b at Hist<PT>::idx(b)
  uint32_t cand[2][kCap];
  uint32_t sel[2][4];  // radix: prefix, mask, remaining rank, count of T
  uint32_t res[2][4];  // counting: key, ties taken, ties in all
  uint32_t ncand[2];
  uint32_t wt[4][kMaxNK][PC<PT>::waves];  // wave totals of the block scans
  float wsum[2][PC<PT>::waves];
  float mred[3 * PT + 2];
};

struct RowCtx {
  int row, n, nc, nm;
  int ntop, older;  // top-ranked critical count; tokens ranked (the rest are recent)
  const float *lg;
  int32_t *crit, *marg;
  float *mp;
  float M, Z;
  const int32_t *pos;  // row -> token position (null: row = token)
  int last;            // largest position a list may name
};

__device__ __forceinline__ void row_setup(const PartArgs &a, RowCtx &r) {
  r.row = blockIdx.x;
  const int b = r.row / a.nsh;
  const Sizes sz = set_sizes(a.seq_len, a.k_crit, a.k_marg, a.k_recent, b, a.n_cap, a.kc_cap,
                             a.km_cap);
  r.n = sz.n;
  r.nc = sz.nc;
  r.nm = sz.nm;
  r.ntop = sz.ntop;
  r.older = sz.n - sz.nr;
  r.lg = a.logits + (int64_t)r.row * a.n_cap;
  r.crit = a.crit + (int64_t)r.row * a.kc_cap;
  r.marg = a.marg + (int64_t)r.row * a.km_cap;
  r.mp = a.marg_prob + (int64_t)r.row * a.km_cap;
  r.pos = nullptr;
  r.last = 0;
  if (a.row_pos) {
    const int j = r.row % a.nsh, layer = j / a.hq, h = j % a.hq;
    const int64_t unit = ((int64_t)b * a.layers + layer) * a.hkv + h / a.g;
    r.pos = a.row_pos + unit * a.n_cap;
    r.last = clampi(a.tok_len[b], 1, a.tok_cap) - 1;
  }
}

// Row max and sum: combined from stage 1's chunk records (fused; also writes
// the head's output) or read back.
template <bool kMerge, int PT>
__device__ __forceinline__ void row_stats(const PartArgs &a, PartShared<PT> &sh, RowCtx &r) {
  if constexpr (kMerge) {
    const int b = r.row / a.nsh, j = r.row % a.nsh, layer = j / a.hq, h = j % a.hq;
    const int unit = (b * a.layers + layer) * a.hkv + h / a.g, i = h % a.g;
    MergeIn in;
    in.stride = (int64_t)a.gp * (a.d + 2);
    in.part = a.part + (int64_t)unit * a.n_split * in.stride + i * (a.d + 2);
    in.nv = (r.n + a.chunk - 1) / a.chunk;
    void *out = a.small_out;
    const int64_t o0 = (int64_t)r.row * a.d;
    const bool bf = a.out_bf16;
    merge_head<PT>(in, a.d, sh.mred, r.M, r.Z, [&](int c, float v) {
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
// kRecent: the row may end in recent tokens (kept unranked); without them
// every token is ranked and the kernel carries no test for it.
// Bin of a non-negative key that is a probability (or a sum of them) rather
// than a logit: its bit pattern read as exponent + mantissa fraction, a
// monotone stand-in for log2, in bins of a set fraction of a binade.  Exact (integer below
// 2^24, power-of-2 scaling).
// pscale = bins per binade / (64 * 2^15): key bits >> 8 count 2^15 steps per
// binade and logit_bin takes 64 bins per unit (2048 bins below the key).
__device__ __forceinline__ float plog2(float x, float pscale) {
  return (float)(__float_as_uint(x) >> 8) * pscale;
}

template <int R, int PT, bool kRecent, bool kProb = false>
struct Row {
  static constexpr int kChunk = PC<PT>::chunk;
  // histogram bin of a key below the row's largest key M
  __device__ __forceinline__ int bin(float s, float M) const {
    if constexpr (kProb) return logit_bin(plog2(s, pscale), plog2(M, pscale));
    return logit_bin(s, M);
  }
  float pscale;  // kProb: key bits >> 8 to bins of 1/64 (see plog2)
  float s[R > 0 ? R : 4];
  const float *lg;
  int n;
  int nrank;     // tokens ranked: the first nrank (the rest, recent, are kept unranked)
  bool aligned;  // 16-byte aligned row of a multiple of 4 entries: whole chunks
                 // load as one float4 through `buf`
  __amdgpu_buffer_rsrc_t buf;  // the row's whole allocation (entries past n read
                               // as whatever is there and are never ranked)

  __device__ __forceinline__ float4 fetch(int k) const {
    const int t = k * kChunk + 4 * (int)threadIdx.x;
    float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (aligned) {
      v = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(buf, (uint32_t)t * 4u, 0, 0));
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
  __device__ __forceinline__ bool ranked(int k, int e) const {
    if constexpr (!kRecent) return valid(k, e);
    return k * kChunk + 4 * (int)threadIdx.x + e < nrank;
  }
  // f(value, ranked) for every slot of every chunk holding ranked tokens,
  // with the wave converged
  template <typename F>
  __device__ __forceinline__ void each(F f) const {
    if constexpr (R > 0) {
#pragma unroll
      for (int k = 0; k < R / 4; ++k) {
        if (k * kChunk >= (kRecent ? nrank : n)) break;
#pragma unroll
        for (int e = 0; e < 4; ++e) f(s[4 * k + e], ranked(k, e));
      }
    } else {
      const int nk = ((kRecent ? nrank : n) + kChunk - 1) / kChunk;
      float4 nx[4];  // the next four chunks, in flight while these are used
#pragma unroll
      for (int j = 0; j < 4; ++j) nx[j] = j < nk ? fetch(j) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      for (int k0 = 0; k0 < nk; k0 += 4) {
        float4 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = nx[j];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (k0 + 4 + j < nk) nx[j] = fetch(k0 + 4 + j);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          f(v[j].x, ranked(k0 + j, 0));
          f(v[j].y, ranked(k0 + j, 1));
          f(v[j].z, ranked(k0 + j, 2));
          f(v[j].w, ranked(k0 + j, 3));
        }
      }
    }
  }
};

struct Targets {
  uint32_t T[2];     // key of the |C|-th / (|C|+|M|)-th token
  uint32_t need[2];  // tokens equal to T that the set takes
  uint32_t eq[2];    // tokens equal to T in the row
};

// Steps 1 and 2.
template <int PT, typename Row>
__device__ __forceinline__ Targets select_targets(PartShared<PT> &sh, const RowCtx &r, const Row &row) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // The targets' ranks count ranked (older) tokens only.  Rank 0 -- no
  // ranked token in the set -- is resolved as rank 1 and then replaced by a
  // key above every logit's.
  if (r.ntop + r.nm == 0) return Targets{{~0u, ~0u}, {0u, 0u}, {0u, 0u}};
  const float M = r.M;
  for (int x = tid; x < Hist<PT>::size; x += PT) sh.hist[0][x] = 0;
  if (tid < 2) sh.ncand[tid] = 0;
  __syncthreads();
  row.each([&](float s, bool valid) {
    if (valid) atomicAdd(&sh.hist[0][Hist<PT>::idx(row.bin(s, M))], 1u);
  });
  __syncthreads();
  // every wave finds both targets' bins itself: no broadcast needed
  uint32_t rr[2] = {(uint32_t)max(r.ntop, 1), (uint32_t)(r.ntop + r.nm)};
  int bin[2];
  uint32_t cnt[2];
#pragma unroll
  for (int x = 0; x < 2; ++x) {
    uint32_t above;
    find_digit<kBins, PT>(sh.hist[0], rr[x], bin[x], above);
    rr[x] -= above;
    cnt[x] = sh.hist[0][Hist<PT>::idx(bin[x])];
  }
  // 0: rank by counting, 1: radix over LDS candidates, 2: radix over the row
  int mode[2];
#pragma unroll
  for (int x = 0; x < 2; ++x) mode[x] = cnt[x] <= (uint32_t)PT ? 0 : (cnt[x] <= (uint32_t)kCap ? 1 : 2);
  if (mode[0] < 2 || mode[1] < 2) {
    const uint64_t lt = lanemask_lt();
    const int gb0 = mode[0] < 2 ? bin[0] : -2, gb1 = mode[1] < 2 ? bin[1] : -2;  // bins gathered
    row.each([&](float s, bool valid) {
      const int bn = valid ? row.bin(s, M) : -1;
      // one ballot for both targets: most waves hold no candidate of either
      if (__ballot((bn == gb0) | (bn == gb1))) {
        const uint32_t u = logit_key(s);
#pragma unroll
        for (int x = 0; x < 2; ++x) {
          const bool take = bn == (x ? gb1 : gb0);
          const uint64_t bal = __ballot(take);
          if (bal) {  // one LDS atomic per wave
            uint32_t off = 0;
            if (lane == 0) off = atomicAdd(&sh.ncand[x], (uint32_t)__popcll(bal));
            off = __shfl(off, 0, kWave);
            if (take) sh.cand[x][off + __popcll(bal & lt)] = u;
          }
        }
      }
    });
  }
  if (tid < 2) {
    sh.sel[tid][0] = 0;
    sh.sel[tid][1] = 0;
    sh.sel[tid][2] = rr[tid];
  }
  __syncthreads();  // candidates visible
#pragma unroll
  for (int x = 0; x < 2; ++x) {
    if (mode[x] == 0 && (uint32_t)tid < cnt[x]) {
      const uint32_t key = sh.cand[x][tid];
      uint32_t gt = 0, eq = 0;
      for (uint32_t c0 = 0; c0 < cnt[x]; c0 += 8) {  // 8 keys per step, two 16-byte reads
        const uint4 a = *reinterpret_cast<const uint4 *>(&sh.cand[x][c0]);
        const uint4 b = *reinterpret_cast<const uint4 *>(&sh.cand[x][c0 + 4]);
        const uint32_t vs[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bool ok = c0 + e < cnt[x];
          gt += ok && vs[e] > key ? 1u : 0u;
          eq += ok && vs[e] == key ? 1u : 0u;
        }
      }
      if (gt < rr[x] && rr[x] <= gt + eq) {  // every tie of the target writes the same
        sh.res[x][0] = key;
        sh.res[x][1] = rr[x] - gt;
        sh.res[x][2] = eq;
      }
    }
  }
  if (mode[0] != 0 || mode[1] != 0) {
    for (int pass = 0; pass < 3; ++pass) {  // digits of 11, 11 and 10 bits
      const int shf = pass == 0 ? 21 : (pass == 1 ? 10 : 0), nb = pass < 2 ? 2048 : 1024;
      const uint32_t dmask = (uint32_t)nb - 1u;
      __syncthreads();  // previous selection visible; hist free
      for (int x = tid; x < 2 * Hist<PT>::size; x += PT) (&sh.hist[0][0])[x] = 0;
      __syncthreads();
      const uint32_t p0 = sh.sel[0][0], m0 = sh.sel[0][1], p1 = sh.sel[1][0], m1 = sh.sel[1][1];
      if (mode[0] == 1)
        for (int k = tid; k < (int)cnt[0]; k += PT) {
          const uint32_t u = sh.cand[0][k];
          if ((u & m0) == p0) atomicAdd(&sh.hist[0][Hist<PT>::idx((u >> shf) & dmask)], 1u);
        }
      if (mode[1] == 1)
        for (int k = tid; k < (int)cnt[1]; k += PT) {
          const uint32_t u = sh.cand[1][k];
          if ((u & m1) == p1) atomicAdd(&sh.hist[1][Hist<PT>::idx((u >> shf) & dmask)], 1u);
        }
      if (mode[0] == 2 || mode[1] == 2)
        row.each([&](float s, bool valid) {
          const int bn = valid ? row.bin(s, M) : -1;
          const uint32_t u = logit_key(s);
          if (mode[0] == 2 && bn == bin[0] && (u & m0) == p0) atomicAdd(&sh.hist[0][Hist<PT>::idx((u >> shf) & dmask)], 1u);
          if (mode[1] == 2 && bn == bin[1] && (u & m1) == p1) atomicAdd(&sh.hist[1][Hist<PT>::idx((u >> shf) & dmask)], 1u);
        });
      __syncthreads();
      if (wave < 2 && mode[wave] != 0) {
        int digit;
        uint32_t above;
        if (pass < 2)
          find_digit<2048, PT>(sh.hist[wave], sh.sel[wave][2], digit, above);
        else
          find_digit<1024, PT>(sh.hist[wave], sh.sel[wave][2], digit, above);
        if (lane == 0) {
          sh.sel[wave][0] |= (uint32_t)digit << shf;
          sh.sel[wave][1] |= dmask << shf;
          sh.sel[wave][2] -= above;
          sh.sel[wave][3] = sh.hist[wave][Hist<PT>::idx(digit)];  // after the last pass: count of T
        }
      }
    }
  }
  __syncthreads();
  Targets t;
#pragma unroll
  for (int x = 0; x < 2; ++x) {
    const bool c = mode[x] == 0;
    t.T[x] = c ? sh.res[x][0] : sh.sel[x][0];
    t.need[x] = c ? sh.res[x][1] : sh.sel[x][2];
    t.eq[x] = c ? sh.res[x][2] : sh.sel[x][3];
  }
  if (r.ntop == 0) {
    t.T[0] = ~0u;
    t.need[0] = 0u;
    t.eq[0] = 0u;
  }
  return t;
}

// Workgroup exclusive prefix of NK packed values (two 16-bit counts each;
// per-chunk totals stay below 65536) with one barrier.
template <int NK, int PT>
__device__ __forceinline__ void block_scan(PartShared<PT> &sh, int slot, const uint32_t *v,
                                           uint32_t *excl, uint32_t *total) {
  constexpr int kWaves = PC<PT>::waves;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc[NK];
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    inc[k] = wave_incl_scan(v[k]);
    if (lane == 63) sh.wt[slot][k][wave] = inc[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t x = sh.wt[slot][k][w];
      off += w < wave ? x : 0u;
      tot += x;
    }
    excl[k] = off + inc[k] - v[k];
    total[k] = tot;
  }
}

template <int PT>
__device__ __forceinline__ void finish_row(const PartArgs &a, PartShared<PT> &sh, const RowCtx &r,
                                           float sc, float sm) {
  constexpr int kWaves = PC<PT>::waves;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = r.nc + tid; i < a.kc_cap; i += PT) r.crit[i] = -1;
  for (int i = r.nm + tid; i < a.km_cap; i += PT) {
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

// Step 3 helpers: membership of one value and its output.
struct Compactor {
  const RowCtx &r;
  Targets t;
  float Zinv;
  // the row's lists as raw buffers of exactly |C| and |M| entries: a store
  // past them (or of a non-member, at kOOB) is dropped
  __amdgpu_buffer_rsrc_t cbuf, mbuf, pbuf;
  float sc = 0.0f, sm = 0.0f;

  // the thresholds as the logits they are the keys of (the key above every
  // logit's, of an empty set, becomes a NaN, which no logit reaches)
  float Tf[2];

  __device__ static float key_value(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
  }

  __device__ Compactor(const RowCtx &rc, const Targets &tg, float zinv)
      : r(rc), t(tg), Zinv(zinv), cbuf(buffer_of(rc.crit, 4u * (uint32_t)rc.nc)),
        mbuf(buffer_of(rc.marg, 4u * (uint32_t)rc.nm)),
        pbuf(buffer_of(rc.mp, 4u * (uint32_t)rc.nm)) {
    Tf[0] = key_value(tg.T[0]);
    Tf[1] = key_value(tg.T[1]);
  }

  // Membership when no threshold's ties are split between two sets (every
  // token equal to a threshold is in its set): plain float compares, which
  // order logits as their keys do (-0 equals +0).
  __device__ __forceinline__ void classify_unsplit(float s, bool ranked, bool recent, bool &inC,
                                                   bool &inM) const {
    inC = recent | (ranked & (s >= Tf[0]));
    inM = ranked & (s >= Tf[1]) & !inC;
  }

  // rC / rP: the value's rank (0-based, token order) among the row's ties at
  // T; recent tokens are critical whatever their key
  // s compared with the thresholds' logits orders as its key would (-0
  // equals +0; the NaN of an empty set's threshold is never reached), so no
  // key is formed.  Bitwise, not short-circuit: every operand is cheap, and
  // && / || would let the compiler branch around them.
  __device__ __forceinline__ void classify(float s, bool ranked, bool recent, uint32_t rC,
                                           uint32_t rP, bool &inC, bool &inM) const {
    inC = recent | (ranked & ((s > Tf[0]) | ((s == Tf[0]) & (rC < t.need[0]))));
    const bool inP = ranked & ((s > Tf[1]) | ((s == Tf[1]) & (rP < t.need[1])));
    inM = inP & !inC;
  }
  __device__ __forceinline__ void emit(float s, int tok, bool inC, bool inM, uint32_t &pc,
                                       uint32_t &pm) {
    const float p = __expf(s - r.M) * Zinv;
    sc += inC ? p : 0.0f;
    sm += inM ? p : 0.0f;
    // the small model's held rows name their token positions
    if (r.pos && (inC || inM)) tok = clampi(r.pos[tok], 0, r.last);
    // stores past a list (only if the select were wrong) are dropped by the
    // buffer views, as are those of non-members
    __builtin_amdgcn_raw_buffer_store_b32((uint32_t)tok, cbuf, inC ? pc * 4u : kOOB, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b32((uint32_t)tok, mbuf, inM ? pm * 4u : kOOB, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(p), pbuf, inM ? pm * 4u : kOOB, 0, 0);
    pc += inC ? 1u : 0u;
    pm += inM ? 1u : 0u;
  }
};

// The list offsets at a 256-token boundary: the thread whose first token
// starts the block (lane 0 of its wave: 64 threads x 4 tokens) records the
// list positions it is about to write.
__device__ __forceinline__ void offsets(const PartArgs &a, const RowCtx &r, int tok0, uint32_t pc,
                                        uint32_t pm) {
  if (a.tab && (threadIdx.x & 63) == 0 && tok0 < r.n)
    a.tab[(int64_t)r.row * a.nblk + (tok0 >> 8)] = make_int2((int)pc, (int)pm);
}

// ---------------------------------------------------------------- kernel --

template <bool kMerge, int R, int PT, bool kRecent, bool kProb = false>
__global__ __launch_bounds__(PT) __attribute__((amdgpu_waves_per_eu(4)))
void partition_kernel(PartArgs a) {
  constexpr int kChunk = PC<PT>::chunk;
  __shared__ PartShared<PT> sh;
  RowCtx r;
  row_setup(a, r);
  const int tid = threadIdx.x;
  Row<R, PT, kRecent, kProb> row;
  row.lg = r.lg;
  row.n = r.n;
  row.nrank = r.older;
  row.pscale = a.pscale;
  row.aligned = (reinterpret_cast<uintptr_t>(r.lg) & 15) == 0 && (a.n_cap & 3) == 0;
  row.buf = buffer_of(r.lg, 4u * (uint32_t)a.n_cap);
  row.load();  // in flight while the row's statistics arrive
  row_stats<kMerge>(a, sh, r);
  Compactor cp(r, select_targets(sh, r, row), 1.0f / r.Z);
  // ties at a threshold split between two sets need their ranks in token order
  const bool split = cp.t.need[0] < cp.t.eq[0] || cp.t.need[1] < cp.t.eq[1];

  if constexpr (R > 0) {
    constexpr int NK = R / 4;
    static_assert(NK <= kMaxNK, "register row too long");
    uint32_t rank_base[NK];  // tie ranks (C low, P high) before this thread's values
#pragma unroll
    for (int k = 0; k < NK; ++k) rank_base[k] = 0;
    if (split) {
      uint32_t v[NK], ex[NK], tot[NK];
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        v[k] = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool ok = row.ranked(k, e);
          const uint32_t u = logit_key(row.s[4 * k + e]);
          v[k] += ((ok & (u == cp.t.T[0])) ? 1u : 0u) + ((ok & (u == cp.t.T[1])) ? 0x10000u : 0u);
        }
      }
      block_scan<NK>(sh, 0, v, ex, tot);
      uint32_t carry = 0;
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        rank_base[k] = carry + ex[k];
        carry += tot[k];
      }
    }
    bool inC[R], inM[R];
    uint32_t v[NK], ex[NK], tot[NK];
#pragma unroll
    for (int k = 0; k < NK; ++k) {
      uint32_t rC = rank_base[k] & 0xffffu, rP = rank_base[k] >> 16;
      v[k] = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = 4 * k + e;
        const bool ok = row.ranked(k, e);
        const float x = row.s[i];
        cp.classify(x, ok, kRecent & row.valid(k, e) & !ok, rC, rP, inC[i], inM[i]);
        rC += (ok & (x == cp.Tf[0])) ? 1u : 0u;
        rP += (ok & (x == cp.Tf[1])) ? 1u : 0u;
        v[k] += (inC[i] ? 1u : 0u) + (inM[i] ? 0x10000u : 0u);
      }
    }
    block_scan<NK>(sh, 1, v, ex, tot);
    uint32_t carry_c = 0, carry_m = 0;
#pragma unroll
    for (int k = 0; k < NK; ++k) {
      uint32_t pc = carry_c + (ex[k] & 0xffffu), pm = carry_m + (ex[k] >> 16);
      if constexpr (kMerge) offsets(a, r, k * kChunk + 4 * tid, pc, pm);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        cp.emit(row.s[4 * k + e], k * kChunk + 4 * tid + e, inC[4 * k + e], inM[4 * k + e], pc, pm);
      carry_c += tot[k] & 0xffffu;
      carry_m += tot[k] >> 16;
    }
  } else {
    // Long rows: one workgroup scan per NG chunks, the next NG in flight.
    constexpr int NG = 3;
    static_assert(NG <= kMaxNK, "scan slots");
    const int nk = row.chunks();
    // tie ranks before the group, one 32-bit count per threshold: a row may
    // hold more than 65535 ties (only a group's own counts are packed)
    uint32_t carry_eq_c = 0, carry_eq_p = 0, carry_c = 0, carry_m = 0;
    float4 nxt[NG];
#pragma unroll
    for (int j = 0; j < NG; ++j) nxt[j] = j < nk ? row.chunk(j) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int k0 = 0, it = 0; k0 < nk; k0 += NG, ++it) {
      float sv[NG][4];
#pragma unroll
      for (int j = 0; j < NG; ++j) {
        sv[j][0] = nxt[j].x;
        sv[j][1] = nxt[j].y;
        sv[j][2] = nxt[j].z;
        sv[j][3] = nxt[j].w;
      }
#pragma unroll
      for (int j = 0; j < NG; ++j)
        if (k0 + NG + j < nk) nxt[j] = row.chunk(k0 + NG + j);
      const int par = 2 * (it & 1);
      uint32_t rank[NG];  // keys are recomputed where used: fewer live registers
#pragma unroll
      for (int j = 0; j < NG; ++j) rank[j] = 0;
      uint32_t group_eq = 0;  // the group's ties of T[0] (low half) and T[1] (high half)
      if (split) {
        uint32_t v[NG], ex[NG], tot[NG];
#pragma unroll
        for (int j = 0; j < NG; ++j) {
          v[j] = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e)
          {
            const bool ok = row.ranked(k0 + j, e);
            const uint32_t u = logit_key(sv[j][e]);
            v[j] += ((ok & (u == cp.t.T[0])) ? 1u : 0u) + ((ok & (u == cp.t.T[1])) ? 0x10000u : 0u);
          }
        }
        block_scan<NG>(sh, par, v, ex, tot);
        uint32_t in_group = 0;  // ties of the group's earlier chunks (packed, < 2^16 each)
#pragma unroll
        for (int j = 0; j < NG; ++j) {
          rank[j] = in_group + ex[j];
          in_group += tot[j];
        }
        group_eq = in_group;
      }
      bool inC[NG][4], inM[NG][4];
      uint32_t v[NG], ex[NG], tot[NG];
      if (split) {
#pragma unroll
        for (int j = 0; j < NG; ++j) {
          uint32_t rC = carry_eq_c + (rank[j] & 0xffffu), rP = carry_eq_p + (rank[j] >> 16);
          v[j] = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool ok = row.ranked(k0 + j, e);
            const float x = sv[j][e];
            cp.classify(x, ok, kRecent & row.valid(k0 + j, e) & !ok, rC, rP, inC[j][e], inM[j][e]);
            rC += (ok & (x == cp.Tf[0])) ? 1u : 0u;
            rP += (ok & (x == cp.Tf[1])) ? 1u : 0u;
            v[j] += (inC[j][e] ? 1u : 0u) + (inM[j][e] ? 0x10000u : 0u);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < NG; ++j) {
          v[j] = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool ok = row.ranked(k0 + j, e);
            cp.classify_unsplit(sv[j][e], ok, kRecent & row.valid(k0 + j, e) & !ok, inC[j][e],
                                inM[j][e]);
            v[j] += (inC[j][e] ? 1u : 0u) + (inM[j][e] ? 0x10000u : 0u);
          }
        }
      }
      block_scan<NG>(sh, par + 1, v, ex, tot);
#pragma unroll
      for (int j = 0; j < NG; ++j) {
        uint32_t pc = carry_c + (ex[j] & 0xffffu), pm = carry_m + (ex[j] >> 16);
        if constexpr (kMerge) offsets(a, r, (k0 + j) * kChunk + 4 * tid, pc, pm);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          cp.emit(sv[j][e], (k0 + j) * kChunk + 4 * tid + e, inC[j][e], inM[j][e], pc, pm);
        carry_c += tot[j] & 0xffffu;
        carry_m += tot[j] >> 16;
      }
      carry_eq_c += group_eq & 0xffffu;
      carry_eq_p += group_eq >> 16;
    }
  }
  finish_row(a, sh, r, cp.sc, cp.sm);
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
  a.k_recent = b.k_recent;
  a.logits = logits;
  a.row_max = row_max;
  a.row_sum = row_sum;
  a.crit = crit;
  a.marg = marg;
  a.marg_prob = marg_prob;
  a.mass = mass;
  return a;
}

// Rows of 1024 threads (16 waves, so at most 128 VGPRs per thread) exist
// only with up to 8 logits per thread in registers: the 16-logit and
// memory-path rows need more and would spill to scratch at that width.
constexpr int kWideMaxR = 8;

template <bool kMerge, int PT, bool kRecent, bool kProb>
hipError_t launch_pt(const PartArgs &a, int rows, hipStream_t st) {
  const dim3 grid(rows), block(PT);
  const int n = a.n_cap;
  if (n <= 4 * PT)
    hipLaunchKernelGGL((partition_kernel<kMerge, 4, PT, kRecent, kProb>), grid, block, 0, st, a);
  else if (n <= 8 * PT)
    hipLaunchKernelGGL((partition_kernel<kMerge, 8, PT, kRecent, kProb>), grid, block, 0, st, a);
  else if constexpr (PT == 1024)
    return hipErrorInvalidValue;  // the caller picks 1024 threads only for n <= 8 * 1024
  else if (n <= 16 * PT)
    hipLaunchKernelGGL((partition_kernel<kMerge, 16, PT, kRecent, kProb>), grid, block, 0, st, a);
  else if (PT == 256 && n <= 20 * PT)  // narrow rows: one more register chunk
    hipLaunchKernelGGL((partition_kernel<kMerge, PT == 256 ? 20 : 16, PT, kRecent, kProb>), grid,
                       block, 0, st, a);
  else
    hipLaunchKernelGGL((partition_kernel<kMerge, 0, PT, kRecent, kProb>), grid, block, 0, st, a);
  return hipGetLastError();
}

// Many rows (several per CU): 256 threads each, so that more rows are
// resident at once; few rows: 512 threads, so that each finishes sooner;
// at most one row per CU: 1024.
constexpr int kManyRows = 4 * 256;

template <bool kMerge, bool kProb = false>
hipError_t launch_rows(const PartArgs &a, int rows, hipStream_t st) {
  if (a.k_recent) {
    if (rows >= kManyRows) return launch_pt<kMerge, 256, true, kProb>(a, rows, st);
    return launch_pt<kMerge, 512, true, kProb>(a, rows, st);
  }
  if (rows >= kManyRows) return launch_pt<kMerge, 256, false, kProb>(a, rows, st);
  // at most one row per CU: 1024 threads shorten each row's passes
  // (with more rows some CUs would run two of them in turn)
  if (rows <= 256 && a.n_cap <= kWideMaxR * 1024)
    return launch_pt<kMerge, 1024, false, kProb>(a, rows, st);
  return launch_pt<kMerge, 512, false, kProb>(a, rows, st);
}

}  // namespace

hipError_t launch_partition(const smallkv_batch_t &b, int n_small_heads, const float *logits,
                            const float *row_max, const float *row_sum, int32_t *crit,
                            int32_t *marg, float *marg_prob, float *mass,
                            const smallkv_model_t *held, const int32_t *tok_len, int tok_cap,
                            hipStream_t st) {
  PartArgs a = base_args(b, n_small_heads, logits, const_cast<float *>(row_max),
                         const_cast<float *>(row_sum), crit, marg, marg_prob, mass);
  if (held) {
    a.layers = held->n_layers;
    a.hq = held->n_q_heads;
    a.hkv = held->n_kv_heads;
    a.g = held->n_q_heads / held->n_kv_heads;
    a.row_pos = held->row_pos;
    a.tok_len = tok_len;
    a.tok_cap = tok_cap;
  }
  return launch_rows<false>(a, b.batch * n_small_heads, st);
}

hipError_t launch_merge_partition(const smallkv_batch_t &b, const smallkv_model_t &m,
                                  const SmallPlan &p, const float *ws, const float *logits,
                                  float *row_max, float *row_sum, int32_t *crit, int32_t *marg,
                                  float *marg_prob, float *mass, int2 *tab,
                                  const int32_t *tok_len, int tok_cap, hipStream_t st) {
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
  a.tab = tab;
  a.nblk = list_blocks(b);
  a.row_pos = m.row_pos;
  a.tok_len = tok_len;
  a.tok_cap = tok_cap;
  return launch_rows<true>(a, b.batch * nsh, st);
}

}  // namespace smallkv

namespace smallkv {

hipError_t launch_group_partition(const smallkv_batch_t &b, int group_rows, const float *keys,
                                  const float *key_max, int32_t *crit, int32_t *marg,
                                  float *marg_prob, float *mass, int bins_per_binade,
                                  hipStream_t st) {
  // keys are sums of probabilities: the row's largest key stands in for both
  // the row max and the normaliser (the p' this writes are not used)
  PartArgs a = base_args(b, group_rows, keys, const_cast<float *>(key_max),
                         const_cast<float *>(key_max), crit, marg, marg_prob, mass);
  // key bits >> 8 hold 15 mantissa bits per binade; logit_bin takes 64 steps
  // per unit, so a unit of 64 / bins_per_binade binades
  a.pscale = (float)bins_per_binade / (64.0f * 32768.0f);
  return launch_rows<false, true>(a, b.batch * group_rows, st);
}

}  // namespace smallkv
