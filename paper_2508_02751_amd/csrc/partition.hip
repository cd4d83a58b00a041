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
//   3. one ordered pass compacts C and M in ascending token order and
//      computes p' for marginal tokens and the masses S'_C, S'_M.  The row
//      is read in slots of PT consecutive tokens, one per thread, so a wave
//      holds 64 consecutive tokens of a slot: its members are lane masks
//      (ballots of single compares, combined on the scalar unit), and their
//      list positions are the wave's base plus a masked bit count (mbcnt);
//      one workgroup exchange of per-(wave, slot) counts per group of slots
//      gives the bases.  Tie ranks (also mbcnt over a ballot) are counted
//      only when a threshold's ties are split between two sets.
// Rows of up to 16 (20 with 256 threads) slots are read once and kept in
// registers (one exchange); longer rows are re-read per pass, 16 slots in
// flight, the candidate gather from the row's end (it starts on what the
// histogram pass read last).  Many rows (several per CU) get 256 threads
// each, so that more rows are resident (six re-read rows per CU); few rows
// get 512, or 1024 when there is at most one per CU.  The fused variant
// first combines stage 1's per-chunk records of its head (row max, row sum,
// the head's output), so a step needs no separate merge launch.
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
template <int PT>
struct PC {
  static constexpr int waves = PT / kWave;
};
// Rows resident per CU: six for the long 256-thread rows (the many-row
// launches, where more rows in flight hide the passes' latency: 80 VGPRs),
// four otherwise (the register rows need up to 128 VGPRs).
template <int R, int PT>
constexpr int rows_per_cu() { return R == 0 && PT == 256 ? 6 : 4; }
// Candidate keys per target kept in LDS: 512 in the long 256-thread rows,
// so that six of them fit a CU's LDS, else 2048.
template <int R, int PT>
constexpr int cand_cap() { return R == 0 && PT == 256 ? 512 : 2048; }
// Slots of a long row per workgroup exchange (and in flight while a group is
// compacted)
constexpr int kGroup = 16;
// Slots per exchange at most: a register row's R, or kGroup
constexpr int kMaxSlots = 20;

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

// The lanes where p holds, straight from the compare that made p (HIP's
// __ballot takes an int, which costs a select and a compare per use)
__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }
// This lane's bit of a wave-uniform lane mask, used as a lane predicate
// without leaving the scalar unit
__device__ __forceinline__ bool lane_in(uint64_t m) { return __builtin_amdgcn_inverse_ballot_w64(m); }

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Distance of a key s below the row's largest key M in steps of 1/64 (M64 =
// 64 M), clamped to 0..2047: the histogram bin 2047 - i holds the keys at
// distance i, so the top 1/64 of a unit is bin 2047 and everything more than
// 32 below is bin 0.  One correctly rounded fma: monotone in s, and the same
// in every pass, which is all the select needs of it.
__device__ __forceinline__ int bin_index(float s, float M64) {
  float d = __fmaf_rn(s, -64.0f, M64);
  d = fminf(fmaxf(d, 0.0f), 2047.0f);
  return (int)d;
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

template <int PT, int CAP>
struct alignas(16) PartShared {
  static constexpr int cap = CAP;
  uint32_t hist[2][Hist<PT>::size];  // bin b at Hist<PT>::idx(b)
  uint32_t cand[2][CAP];
  uint32_t sel[2][4];  // radix: prefix, mask, remaining rank, count of T
  uint32_t res[2][4];  // counting: key, ties taken, ties in all
  uint32_t ncand[2];
  uint32_t cnt[4][PC<PT>::waves][kMaxSlots];  // per-(wave, slot) counts of the exchanges
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
template <bool kMerge, int PT, int CAP>
__device__ __forceinline__ void row_stats(const PartArgs &a, PartShared<PT, CAP> &sh, RowCtx &r) {
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

// The row as seen by the passes: slot q holds tokens [q*PT, (q+1)*PT), token
// q*PT + tid in thread tid, so a wave holds 64 consecutive tokens of it.
// R > 0: the row sits in R registers per thread (slots 0..R-1), read from
// memory once.  R == 0: every pass reads it from memory, kGroup slots in
// flight.  kRecent: the row may end in recent tokens (kept unranked); without
// them every token is ranked and the kernel carries no test for it.
// Bin of a non-negative key that is a probability (or a sum of them) rather
// than a logit: its bit pattern read as exponent + mantissa fraction, a
// monotone stand-in for log2, in bins of a set fraction of a binade.  Exact (integer below
// 2^24, power-of-2 scaling).
// pscale = bins per binade / (64 * 2^15): key bits >> 8 count 2^15 steps per
// binade and a bin is 1/64 of a unit (2048 bins below the key).
__device__ __forceinline__ float plog2(float x, float pscale) {
  return (float)(__float_as_uint(x) >> 8) * pscale;
}

// A long row's next slots are requested at a raised wave priority, so that
// the loads leave before the other rows' arithmetic (LLaMA stage 2 -2%).
__device__ __forceinline__ void prio_hi() { __builtin_amdgcn_s_setprio(2); }
__device__ __forceinline__ void prio_lo() { __builtin_amdgcn_s_setprio(0); }

template <int R, int PT, bool kRecent, bool kProb = false>
struct Row {
  float pscale;  // kProb: key bits >> 8 to bins of 1/64 (see plog2)
  float M64;     // 64 x the row's largest key as the bins see it
  float s[R > 0 ? R : 1];
  int n;
  int nrank;     // tokens ranked: the first nrank (the rest, recent, are kept unranked)
  __amdgpu_buffer_rsrc_t buf;  // the row's n tokens: slots past them read zero
                               // without a memory access (a short row of a
                               // wide variant reads only its own tokens)

  __device__ __forceinline__ void set_max(float M) {
    if constexpr (kProb) M64 = 64.0f * plog2(M, pscale);
    else M64 = 64.0f * M;
  }
  // distance index of a key (0: the top bin; histogram bin 2047 - index)
  __device__ __forceinline__ int bin_of(float s) const {
    if constexpr (kProb) return bin_index(plog2(s, pscale), M64);
    return bin_index(s, M64);
  }
  __device__ __forceinline__ int tok(int q) const { return q * PT + (int)threadIdx.x; }
  // slots past the row's tokens read zero (raw buffer view)
  __device__ __forceinline__ float fetch(int q) const {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(buf, (uint32_t)tok(q) * 4u, 0, 0));
  }
  __device__ __forceinline__ void load() {
    if constexpr (R > 0) {
#pragma unroll
      for (int q = 0; q < R; ++q) s[q] = fetch(q);
    }
  }
  __device__ __forceinline__ int slots() const { return (n + PT - 1) / PT; }
  __device__ __forceinline__ bool valid(int q) const { return tok(q) < n; }
  __device__ __forceinline__ bool ranked(int q) const {
    if constexpr (!kRecent) return valid(q);
    return tok(q) < nrank;
  }
  // f(value, ranked) for every slot holding ranked tokens, with the wave
  // converged.  kRev: from the row's end to its start, so that a pass that
  // follows a forward one starts on what that one read last, which is still
  // in L2 (order-free passes only).
  template <bool kRev = false, typename F>
  __device__ __forceinline__ void each(F f) const {
    const int nq = ((kRecent ? nrank : n) + PT - 1) / PT;
    if constexpr (R > 0) {
#pragma unroll
      for (int q = 0; q < R; ++q)  // a fixed count (a break would keep s[] in memory)
        if (q < nq) f(s[q], ranked(q));
    } else {
      // the next slots, in flight while these are used (past the row's end
      // too: they read zero, and are not used)
      float nx[kGroup];
      if constexpr (kRev) {
        const int last = (nq - 1) / kGroup * kGroup;  // first slot of the last group
#pragma unroll
        for (int j = 0; j < kGroup; ++j) nx[j] = fetch(last + j);
        for (int q0 = last; q0 >= 0; q0 -= kGroup) {
          float v[kGroup];
#pragma unroll
          for (int j = 0; j < kGroup; ++j) v[j] = nx[j];
          prio_hi();
          if (q0 >= kGroup)
#pragma unroll
            for (int j = 0; j < kGroup; ++j) nx[j] = fetch(q0 - kGroup + j);
          prio_lo();
#pragma unroll
          for (int j = kGroup - 1; j >= 0; --j)
            if (q0 + j < nq) f(v[j], ranked(q0 + j));
        }
      } else {
#pragma unroll
        for (int j = 0; j < kGroup; ++j) nx[j] = fetch(j);
        for (int q0 = 0; q0 < nq; q0 += kGroup) {
          float v[kGroup];
#pragma unroll
          for (int j = 0; j < kGroup; ++j) v[j] = nx[j];
          prio_hi();
#pragma unroll
          for (int j = 0; j < kGroup; ++j) nx[j] = fetch(q0 + kGroup + j);
          prio_lo();
#pragma unroll
          for (int j = 0; j < kGroup; ++j)
            if (q0 + j < nq) f(v[j], ranked(q0 + j));
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
template <int PT, int CAP, typename Row>
__device__ __forceinline__ Targets select_targets(PartShared<PT, CAP> &sh, const RowCtx &r, const Row &row) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // The targets' ranks count ranked (older) tokens only.  Rank 0 -- no
  // ranked token in the set -- is resolved as rank 1 and then replaced by a
  // key above every logit's.
  if (r.ntop + r.nm == 0) return Targets{{~0u, ~0u}, {0u, 0u}, {0u, 0u}};
  for (int x = tid; x < Hist<PT>::size; x += PT) sh.hist[0][x] = 0;
  if (tid < 2) sh.ncand[tid] = 0;
  __syncthreads();
  row.each([&](float s, bool valid) {
    if (valid) atomicAdd(&sh.hist[0][Hist<PT>::idx(2047 - row.bin_of(s))], 1u);
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
  for (int x = 0; x < 2; ++x) mode[x] = cnt[x] <= (uint32_t)PT ? 0 : (cnt[x] <= (uint32_t)CAP ? 1 : 2);
  if (mode[0] < 2 || mode[1] < 2) {
    const uint64_t lt = lanemask_lt();
    // distance indices of the bins gathered (-1: none)
    const int gb0 = mode[0] < 2 ? 2047 - bin[0] : -1, gb1 = mode[1] < 2 ? 2047 - bin[1] : -1;
    // backwards: the histogram pass read the row forwards
    row.template each<true>([&](float s, bool valid) {
      const int bn = row.bin_of(s);
      const uint64_t ok = ballot(valid);
      const uint64_t h[2] = {ok & ballot(bn == gb0), ok & ballot(bn == gb1)};
      // most waves hold no candidate of either target
      if (h[0] | h[1]) {
        const uint32_t u = logit_key(s);
#pragma unroll
        for (int x = 0; x < 2; ++x) {
          const uint64_t bal = h[x];
          const bool take = lane_in(bal);
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
  // Counting: key k of target x's bin against all n of the bin's keys.
  auto count = [&](int x, uint32_t k, uint32_t n, uint32_t rank) {
    const uint32_t key = sh.cand[x][k];
    uint32_t gt = 0, eq = 0;
    for (uint32_t c0 = 0; c0 < n; c0 += 8) {  // 8 keys per step, two 16-byte reads
      const uint4 a = *reinterpret_cast<const uint4 *>(&sh.cand[x][c0]);
      const uint4 b = *reinterpret_cast<const uint4 *>(&sh.cand[x][c0 + 4]);
      const uint32_t vs[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool ok = c0 + e < n;
        gt += ok && vs[e] > key ? 1u : 0u;
        eq += ok && vs[e] == key ? 1u : 0u;
      }
    }
    if (gt < rank && rank <= gt + eq) {  // every tie of the target writes the same
      sh.res[x][0] = key;
      sh.res[x][1] = rank - gt;
      sh.res[x][2] = eq;
    }
  };
  if (mode[0] == 0 && mode[1] == 0 && cnt[0] + cnt[1] <= (uint32_t)PT) {
    // both targets at once: target 1's keys on the threads after target 0's
    const bool second = (uint32_t)tid >= cnt[0];
    const uint32_t k = second ? (uint32_t)tid - cnt[0] : (uint32_t)tid;
    const uint32_t n = second ? cnt[1] : cnt[0];
    if (k < n) count(second ? 1 : 0, k, n, second ? rr[1] : rr[0]);
  } else {
#pragma unroll
    for (int x = 0; x < 2; ++x)
      if (mode[x] == 0 && (uint32_t)tid < cnt[x]) count(x, tid, cnt[x], rr[x]);
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
          const int bn = valid ? 2047 - row.bin_of(s) : -1;
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

// One exchange of a group of G slots: each wave's count for each slot
// (packed, two 16-bit counts; a group's totals stay below 65536) gives, in
// lane j, the counts before (slot j, this wave) within the group (read back
// per slot with readlane), and the group's totals.  Lane j sums slot j over
// the waves; one wave scan orders the slots.  One barrier; `buf` alternates
// so that the next exchange can write while slow waves still read this one.
template <int G, int PT, int CAP>
__device__ __forceinline__ uint32_t exchange(PartShared<PT, CAP> &sh, int buf, const uint32_t *cnt,
                                             uint32_t &total) {
  constexpr int kWaves = PC<PT>::waves;
  static_assert(G <= kMaxSlots && G <= kWave, "slots per exchange");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0)
#pragma unroll
    for (int j = 0; j < G; ++j) sh.cnt[buf][wave][j] = cnt[j];
  __syncthreads();
  uint32_t tot = 0, part = 0;
  if (lane < G)
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t v = sh.cnt[buf][w][lane];
      tot += v;
      part += w < wave ? v : 0u;
    }
  const uint32_t inc = wave_incl_scan(tot);
  total = __builtin_amdgcn_readlane(inc, G - 1);
  return inc - tot + part;
}

// Positions of the set lanes of m below this lane, plus base
__device__ __forceinline__ uint32_t mbcnt(uint64_t m, uint32_t base) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, base));
}

template <int PT, int CAP>
__device__ __forceinline__ void finish_row(const PartArgs &a, PartShared<PT, CAP> &sh, const RowCtx &r,
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

// Step 3: the thresholds as logits, and the output of a wave's members.
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

  // Writes the members of a wave's 64 consecutive tokens (lane masks mC,
  // mM; the wave's first entries go to list positions bc, bm) and adds their
  // p' to the masses.  Stores past a list (only if the select were wrong)
  // are dropped by the buffer views, as are those of non-members.
  template <bool kHeld>
  __device__ __forceinline__ void emit(float s, int tok, uint64_t mC, uint64_t mM, uint32_t bc,
                                       uint32_t bm) {
    const bool inC = lane_in(mC), inM = lane_in(mM);
    const float p = __expf(s - r.M) * Zinv;
    sc += inC ? p : 0.0f;
    sm += inM ? p : 0.0f;
    // the small model's held rows name their token positions
    if constexpr (kHeld)
      if (lane_in(mC | mM)) tok = clampi(r.pos[tok], 0, r.last);
    const uint32_t pc = mbcnt(mC, bc), pm = mbcnt(mM, bm);
    __builtin_amdgcn_raw_buffer_store_b32((uint32_t)tok, cbuf, inC ? pc * 4u : kOOB, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b32((uint32_t)tok, mbuf, inM ? pm * 4u : kOOB, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(p), pbuf, inM ? pm * 4u : kOOB, 0, 0);
  }
};

// The list offsets at 256-token boundaries, for a group of G slots from q0:
// in every fourth wave (64 tokens each, so its first token starts a block),
// lane j records the list positions before the wave's tokens of slot j.
template <int G, int PT>
__device__ __forceinline__ void offsets(const PartArgs &a, const RowCtx &r, int q0, uint32_t pc,
                                        uint32_t pm) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tok0 = (q0 + lane) * PT + kWave * wave;
  if ((wave & 3) == 0 && lane < G && tok0 < r.n)
    a.tab[(int64_t)r.row * a.nblk + (tok0 >> 8)] = make_int2((int)pc, (int)pm);
}

// ---------------------------------------------------------------- kernel --

// Step 3 over a group of G slots x[0..G) starting at slot q0: membership,
// one exchange of the per-wave counts (two with split ties: their ranks
// first), then each wave writes its members at its base + mbcnt.
template <int R, int PT, bool kRecent, bool kProb, bool kSplit, bool kHeld>
struct Step3 {
  PartShared<PT, cand_cap<R, PT>()> &sh;
  const PartArgs &a;
  const RowCtx &r;
  const Row<R, PT, kRecent, kProb> &row;
  Compactor &cp;
  bool offs;  // record the list offsets (a.tab)
  // entries before the group: C, M, and the ties of T[0] / T[1]
  uint32_t carry_c = 0, carry_m = 0, carry_eq_c = 0, carry_eq_p = 0;

  // Lane masks of the critical and marginal members among slot q0 + j's
  // tokens: C = recent | (ranked & at or above the critical threshold), M =
  // ranked & at or above the marginal one, minus C.  Each mask is a ballot
  // of one compare; the set algebra runs on the scalar unit.  Where a
  // threshold's ties are split between two sets, a token equal to it is in
  // the set only if its rank among the row's ties (token order) is below
  // the set's share of them.
  template <int G>
  __device__ __forceinline__ void members(const float (&x)[G], int q0, int j, uint32_t tb,
                                          uint64_t &mC, uint64_t &mM) const {
    const int tid = threadIdx.x, q = q0 + j;
    const uint64_t ok = ballot(tid < (kRecent ? row.nrank : row.n) - q * PT);
    uint64_t rec = 0;
    if constexpr (kRecent) rec = ballot(tid < row.n - q * PT) & ~ok;
    if constexpr (kSplit) {
      const uint32_t t = __builtin_amdgcn_readlane(tb, j);
      const uint64_t e0 = ok & ballot(x[j] == cp.Tf[0]), e1 = ok & ballot(x[j] == cp.Tf[1]);
      const uint64_t r0 = ballot(mbcnt(e0, carry_eq_c + (t & 0xffffu)) < cp.t.need[0]);
      const uint64_t r1 = ballot(mbcnt(e1, carry_eq_p + (t >> 16)) < cp.t.need[1]);
      mC = rec | (ok & ballot(x[j] > cp.Tf[0])) | (e0 & r0);
      mM = ((ok & ballot(x[j] > cp.Tf[1])) | (e1 & r1)) & ~mC;
    } else {
      mC = rec | (ok & ballot(x[j] >= cp.Tf[0]));
      mM = ok & ballot(x[j] >= cp.Tf[1]) & ~mC;
    }
  }

  template <int G>
  __device__ __forceinline__ void group(const float (&x)[G], int q0, int par) {
    const int nq = min(G, row.slots() - q0);  // slots holding tokens
    uint32_t tb = 0;  // lane j: ties (packed) before (slot j, this wave) within the group
    uint32_t ttot = 0;
    if constexpr (kSplit) {
      uint32_t tc[G];
#pragma unroll
      for (int j = 0; j < G; ++j) {
        tc[j] = 0;
        if (j >= nq) continue;
        const uint64_t ok = ballot((int)threadIdx.x < (kRecent ? row.nrank : row.n) - (q0 + j) * PT);
        tc[j] = (uint32_t)__popcll(ok & ballot(x[j] == cp.Tf[0])) +
                ((uint32_t)__popcll(ok & ballot(x[j] == cp.Tf[1])) << 16);
      }
      tb = exchange<G>(sh, par, tc, ttot);
    }
    uint32_t mc[G], mtot;
#pragma unroll
    for (int j = 0; j < G; ++j) {
      mc[j] = 0;
      if (j >= nq) continue;
      uint64_t mC, mM;
      members(x, q0, j, tb, mC, mM);
      mc[j] = (uint32_t)__popcll(mC) + ((uint32_t)__popcll(mM) << 16);
    }
    const uint32_t mb = exchange<G>(sh, par + 1, mc, mtot);
    if (offs) offsets<G, PT>(a, r, q0, carry_c + (mb & 0xffffu), carry_m + (mb >> 16));
#pragma unroll
    for (int j = 0; j < G; ++j) {
      if (j >= nq) continue;
      uint64_t mC, mM;
      members(x, q0, j, tb, mC, mM);
      const uint32_t m = __builtin_amdgcn_readlane(mb, j);
      cp.template emit<kHeld>(x[j], row.tok(q0 + j), mC, mM, carry_c + (m & 0xffffu),
                              carry_m + (m >> 16));
    }
    carry_c += mtot & 0xffffu;
    carry_m += mtot >> 16;
    carry_eq_c += ttot & 0xffffu;
    carry_eq_p += ttot >> 16;
  }

  __device__ __forceinline__ void run() {
    if constexpr (R > 0) {
      group<R>(row.s, 0, 0);
    } else {
      // long rows: one exchange per kGroup slots, the next kGroup in flight
      const int nq = row.slots();
      // (slots past the row's end are read too: they read zero, and no
      // pass uses them)
      float nx[kGroup];
#pragma unroll
      for (int j = 0; j < kGroup; ++j) nx[j] = row.fetch(j);
      for (int q0 = 0, gi = 0; q0 < nq; q0 += kGroup, ++gi) {
        float v[kGroup];
#pragma unroll
        for (int j = 0; j < kGroup; ++j) v[j] = nx[j];
        prio_hi();
#pragma unroll
        for (int j = 0; j < kGroup; ++j) nx[j] = row.fetch(q0 + kGroup + j);
        prio_lo();
        group<kGroup>(v, q0, 2 * (gi & 1));
      }
    }
  }
};

template <bool kMerge, int R, int PT, bool kRecent, bool kProb = false>
__global__ __launch_bounds__(PT) __attribute__((amdgpu_waves_per_eu(rows_per_cu<R, PT>())))
void partition_kernel(PartArgs a) {
  __shared__ PartShared<PT, cand_cap<R, PT>()> sh;
  RowCtx r;
  row_setup(a, r);
  Row<R, PT, kRecent, kProb> row;
  row.n = r.n;
  row.nrank = r.older;
  row.pscale = a.pscale;
  row.buf = buffer_of(r.lg, 4u * (uint32_t)r.n);
  row.load();  // in flight while the row's statistics arrive
  row_stats<kMerge>(a, sh, r);
  row.set_max(r.M);
  Compactor cp(r, select_targets(sh, r, row), 1.0f / r.Z);
  // ties at a threshold split between two sets need their ranks in token order
  const bool split = cp.t.need[0] < cp.t.eq[0] || cp.t.need[1] < cp.t.eq[1];
  const bool offs = kMerge && a.tab;
  if (r.pos) {
    if (split)
      Step3<R, PT, kRecent, kProb, true, true>{sh, a, r, row, cp, offs}.run();
    else
      Step3<R, PT, kRecent, kProb, false, true>{sh, a, r, row, cp, offs}.run();
  } else if (split) {
    Step3<R, PT, kRecent, kProb, true, false>{sh, a, r, row, cp, offs}.run();
  } else {
    Step3<R, PT, kRecent, kProb, false, false>{sh, a, r, row, cp, offs}.run();
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
  // many rows, or rows long enough to be re-read per pass even at 256
  // threads (six of them per CU) and enough of them to fill the CUs that way
  // (the 672 rows of 65536 tokens of the Qwen2-72B step: 0.147 -> 0.143 ms)
  if (rows >= kManyRows || (rows >= 512 && a.n_cap > 20 * 256))
    return launch_pt<kMerge, 256, false, kProb>(a, rows, st);
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
  // key bits >> 8 hold 15 mantissa bits per binade; a bin is 1/64 of a unit,
  // per unit, so a unit of 64 / bins_per_binade binades
  a.pscale = (float)bins_per_binade / (64.0f * 32768.0f);
  return launch_rows<false, true>(a, b.batch * group_rows, st);
}

}  // namespace smallkv
