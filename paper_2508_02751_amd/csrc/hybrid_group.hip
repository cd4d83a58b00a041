// Stage 3 for a whole GQA group at once: bf16, head_dim 128, up to 8 query
// heads per kv head (Eq. 6; Algorithm 1, "O_c of critical tokens ... O_m of
// marginal tokens ... O_c + O_m").
//
// The query heads that share a kv head read different small heads (Eq. 3),
// so their critical and marginal sets differ but overlap heavily.  Reading
// the rows head by head fetches every shared row once per head; here one
// workgroup serves the whole group over a range of tokens and reads each
// row of the union once:
//   * per window of kWin tokens, the group's 2g sorted index lists (C and M
//     of each head) are scanned from per-list cursors into 16 LDS membership
//     bits per token (bit h: critical for head h, bit 8+h: marginal), which
//     are compacted into the ascending list of union rows;
//   * each wave streams blocks of 32 union rows.  QK runs on MFMA
//     (v_mfma_f32_16x16x32_bf16) with the K rows loaded straight from HBM as
//     the A operand (M = 16 rows, K = 32 dims) and the group's queries as B
//     (N = heads); K rows that no head holds critical are not read.  An
//     online softmax per head masks the logits by the critical bits;
//   * P.V runs on MFMA too: the rows of P are the 8 heads' critical weights
//     exp(s - m) and their marginal probabilities p' (taken from the marginal
//     lists by rank), split into bf16 hi + lo; V is transposed in
//     registers (v_perm) into a per-wave LDS tile;
//   * the waves' states merge in LDS; with one split the workgroup writes
//     the output, otherwise a (max, sum, O_C, O_M) record per head that
//     hybrid_group_merge combines.
// The workgroups of one kv head's splits share an XCD, so the index lists
// they all scan stay in that XCD's L2.
#include <limits.h>

#include <algorithm>

#include "common.h"
#include "launch.h"

namespace smallkv {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;

constexpr int kGT = 256;                 // threads per workgroup
constexpr int kGW = kGT / kWave;         // waves
constexpr int kD = 128;                  // head dim
constexpr int kRowB = kD * 2;            // bytes per bf16 K/V row
constexpr int kWin = 4096;               // tokens per membership window
constexpr int kPosBits = 12;             // log2(kWin)
constexpr int kBR = 32;                  // union rows per wave block
constexpr int kVTS = kBR * 2 + 16;       // V^T row stride in LDS (bytes)
// V^T byte offset of (dim, 8-row group): every 8 dims shift by 16 bytes more,
// so that the 16 lanes writing dims 8c + d (c = 0..15) and the 16 lanes
// reading dims 16nb + 0..15 each spread over all banks (2-way, the minimum
// for 16-byte accesses) instead of piling 16-deep on one.
__device__ __forceinline__ int vt_off(int dim, int rg) { return dim * kVTS + (dim >> 3) * 16 + rg * 16; }
constexpr int kVTBytes = 128 * kVTS + 16 * 16;
constexpr int kPS = kBR + 4;             // P row stride (floats)
constexpr int kMaxG = 8;
constexpr int kXcd = 8;
constexpr int kRec = 2 * kD + 2;         // floats per (split, head) record
constexpr int kTargetWgs = 512;          // two resident workgroups per CU
constexpr int kMaxSplit = 32;            // token ranges per kv head (one per 256 tokens at most)
constexpr int64_t kSetupTok = 384;       // per-workgroup setup, in streamed-token time
// Raw buffer loads: an offset at or past the resource's size returns zero
// without touching memory, so masked lanes need no branch.
constexpr uint32_t kOOB = 0x80000000u;
constexpr int kBufWord3 = 0x00020000;    // gfx9 raw buffer descriptor word 3
constexpr int64_t kMaxBuf = 0x7fffffff;

struct GroupArgs {
  int n_cap, layers, hq, hkv, g, nsh, kc_cap, km_cap, mode, units, n_split, span;
  int layer0, nl;  // the large layers this launch runs: [layer0, layer0 + nl) of `layers`
  int mp_bytes;  // size of marg_prob in bytes (< 2^31)
  int64_t n_rows;
  float scale;
  const int32_t *seq_len, *k_crit, *k_marg, *k_recent, *head_map;
  const void *q, *k, *v;
  const int32_t *k_slot, *v_slot;
  const int32_t *crit, *marg;
  const float *marg_prob, *mass;
  float *rec;
  void *out;
  const int2 *tab;  // the partition's list offsets ([rows][nblk]), or null
  int nblk;
  int group_sel;    // lists per (b, layer, kv head), marg_prob/mass per query head
};

struct WaveTiles {
  unsigned char vt[kVTBytes];   // V^T of the block (dims x rows), later the wave's O
  float p[16][kPS];             // P: slot (C head h / M head 8+h) x row
  float alpha[16];              // per-slot rescale of the accumulators
};

struct GroupShared {
  uint32_t mem[kWin / 2];       // membership bits of window positions 2i (low half), 2i+1
  uint32_t uni[kWin];           // union rows: (bits << kPosBits) | position
  WaveTiles w[kGW];
  int cur[2 * kMaxG];           // list cursors (first entry not yet consumed)
  int cend[2 * kMaxG];          // with list offsets: each list's end of the token range
  int mstart[kMaxG];            // M-list cursor at the window start
  int wcnt[kGW][kMaxG];         // marginal entries per head in each wave's rows
  int64_t hrow[kMaxG];          // row of each head's lists: small head (b, j), or its group
  int64_t prow[kMaxG];          // row of each head's marg_prob and mass
  float ac[kMaxG], am[kMaxG];
};

__device__ __forceinline__ void alphas(int mode, float sc, float sm, float &ac, float &am) {
  switch (mode) {
    case SMALLKV_NORM_NONE:
      ac = 1.0f;
      am = 1.0f;
      break;
    case SMALLKV_NORM_SLM_CRIT:
      ac = sc;
      am = 1.0f;
      break;
    case SMALLKV_NORM_RETAINED:
      ac = sc / (sc + sm);
      am = 1.0f / (sc + sm);
      break;
    case SMALLKV_NORM_MARG_FILL:
      ac = sc;
      am = sm > 0.0f ? (1.0f - sc) / sm : 0.0f;
      break;
    default:
      ac = 1.0f - sm;
      am = 1.0f;
      break;
  }
}

// Orders the wave's own LDS writes before its later reads (and reads before
// later writes): a wave's LDS instructions execute in order, so only the
// compiler has to be kept from moving them.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Max with the lane 32 (then 16) positions away.
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ uint4 load16(const unsigned char *p) { return *reinterpret_cast<const uint4 *>(p); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void *p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, bytes, kBufWord3);
}
__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
// The same, non-temporal and past the first-level cache (cache policy
// SC0 | NT): for the V rows, which each instruction reads whole and nothing
// reads again, so that they do not evict lines still in use.  (The K rows
// are read half a line per instruction, the other half by the next: those
// stay cached.)
constexpr int kCpolNT = 3;
__device__ __forceinline__ uint4 bload16_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCpolNT));
}

// The list a wave owns in slot i: L = wave + kGW * i; L < g is head L's
// critical list, g <= L < 2g head (L - g)'s marginal list.
struct ListRef {
  const int32_t *p;
  int len;
  uint32_t bit;
  bool on;
};

__device__ __forceinline__ ListRef list_ref(const GroupArgs &a, const GroupShared &sh, int L, int nc, int nm) {
  ListRef r;
  r.on = L < 2 * a.g;
  r.p = a.crit;
  r.len = 0;
  r.bit = 0;
  if (!r.on) return r;
  if (L < a.g) {
    r.p = a.crit + sh.hrow[L] * a.kc_cap;
    r.len = nc;
    r.bit = 1u << L;
  } else {
    r.p = a.marg + sh.hrow[L - a.g] * a.km_cap;
    r.len = nm;
    r.bit = 1u << (8 + L - a.g);
  }
  return r;
}

// First position of every list holding a token >= target (the lists are
// ascending).  The wave runs one 64-way search per list, all lists in
// lockstep so that their loads overlap: probes split [lo, hi) into 64
// pieces, the ballot of "entry < target" picks the piece.
constexpr int kLPW = 2 * kMaxG / kGW;  // lists per wave
__device__ __forceinline__ void lower_bounds(const ListRef (&l)[kLPW], int target, int (&res)[kLPW]) {
  const int lane = threadIdx.x & 63;
  int lo[kLPW], hi[kLPW];
#pragma unroll
  for (int i = 0; i < kLPW; ++i) {
    lo[i] = 0;
    hi[i] = (l[i].on && target > 0) ? l[i].len : 0;
  }
  for (;;) {
    bool more = false;
#pragma unroll
    for (int i = 0; i < kLPW; ++i) more |= hi[i] - lo[i] > kWave;
    if (!more) break;
    int v[kLPW];
#pragma unroll
    for (int i = 0; i < kLPW; ++i) {
      const int span = hi[i] - lo[i];
      v[i] = INT_MAX;
      if (span > kWave) v[i] = l[i].p[lo[i] + (int)(((int64_t)lane * span) >> 6)];
    }
#pragma unroll
    for (int i = 0; i < kLPW; ++i) {
      const int span = hi[i] - lo[i];
      if (span > kWave) {
        const int c = __popcll(__ballot(v[i] < target));
        const int nlo = c > 0 ? lo[i] + (int)(((int64_t)(c - 1) * span) >> 6) + 1 : lo[i];
        const int nhi = c < kWave ? lo[i] + (int)(((int64_t)c * span) >> 6) : hi[i];
        lo[i] = nlo;
        hi[i] = nhi;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < kLPW; ++i) {
    const int q = lo[i] + lane;
    const int v = q < hi[i] ? l[i].p[q] : INT_MAX;
    res[i] = lo[i] + __popcll(__ballot(v < target));
  }
}

// kResolved: slot maps into a store of at most 65536 rows (see below)
template <bool kResolved>
__global__ __launch_bounds__(kGT) __attribute__((amdgpu_waves_per_eu(2))) void hybrid_group_kernel(GroupArgs a) {
  __shared__ __align__(16) GroupShared sh;
  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index, known to the compiler as wave-uniform: everything derived
  // from it (the owned lists, their pointers and bits) stays in SGPRs
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // XCD-aware numbering: x = ((u / 8) * n_split + sp) * 8 + u % 8
  const int x = blockIdx.x;
  const int rest = x / kXcd;
  const int u = (rest / a.n_split) * kXcd + x % kXcd, sp = rest % a.n_split;
  if (u >= a.units) return;
  const int kvh = u % a.hkv, bl = u / a.hkv, layer = a.layer0 + bl % a.nl, b = bl / a.nl;
  // the (sequence, layer, kv head) in the whole stack's layout
  const int64_t ua = ((int64_t)b * a.layers + layer) * a.hkv + kvh;
  const int g = a.g;
  // the heads' small heads, requested before the sequence's sizes arrive
  // (the index is valid whatever they are)
  const int hm = tid < g ? a.head_map[layer * a.hq + kvh * g + tid] : 0;
  const Sizes sz = set_sizes(a.seq_len, a.k_crit, a.k_marg, a.k_recent, b, a.n_cap, a.kc_cap, a.km_cap);
  const int t_begin = sp * a.span;
  if (t_begin >= sz.n) return;
  const int t_end = min(t_begin + a.span, sz.n);
  // With the partition's list offsets at both ends of a range of one window,
  // every list's entries in it are known before any is read: they are
  // loaded in one round instead of a scan that reads on until it passes the
  // window's end.
  const bool flat = a.tab && t_end - t_begin <= kWin;
  const int hc = lane & 15, lq = lane >> 4;  // MFMA column (head / slot) and lane quarter
  WaveTiles &wt = sh.w[wave];

  if (tid < g) {
    const int j = clampi(hm, 0, a.nsh - 1);
    const int64_t row = (int64_t)b * a.nsh + j;
    const int64_t qrow = ((int64_t)b * a.layers + layer) * a.hq + (int64_t)kvh * g + tid;
    const int64_t hrow = a.group_sel ? ua : row;
    sh.hrow[tid] = hrow;
    if (a.tab) {
      // the partition's offsets at the range's ends (multiples of 256 tokens,
      // or the sequence's end): entries of each list below t_begin / t_end;
      // clamped: no table content can move a cursor outside its list
      const int2 *tb = a.tab + hrow * a.nblk;
      const int2 v0 = tb[t_begin >> 8];
      const int2 v1 = t_end < sz.n ? tb[t_end >> 8] : make_int2(sz.nc, sz.nm);
      const int c0 = clampi(v0.x, 0, sz.nc), m0 = clampi(v0.y, 0, sz.nm);
      sh.cur[tid] = c0;
      sh.cur[g + tid] = m0;
      sh.cend[tid] = clampi(v1.x, c0, sz.nc);
      sh.cend[g + tid] = clampi(v1.y, m0, sz.nm);
    }
    const int64_t prow = a.group_sel ? qrow : row;
    sh.prow[tid] = prow;
    float ac, am;
    alphas(a.mode, a.mass[2 * prow], a.mass[2 * prow + 1], ac, am);
    sh.ac[tid] = ac;
    sh.am[tid] = am;
  } else if (tid < kMaxG) {
    sh.hrow[tid] = 0;
    sh.prow[tid] = 0;
    sh.ac[tid] = 0.0f;
    sh.am[tid] = 0.0f;
  }
  // P slots no head writes stay zero; slots 8..15 (marginal) never rescale
  for (int i = lane; i < 16 * kPS; i += kWave) (&wt.p[0][0])[i] = 0.0f;
  if (lane < 16) wt.alpha[lane] = 1.0f;
  for (int i = tid; i < kWin / 2; i += kGT) sh.mem[i] = 0u;  // each window's compaction clears it again
  __syncthreads();

  ListRef lists[kLPW];
#pragma unroll
  for (int i = 0; i < kLPW; ++i) lists[i] = list_ref(a, sh, wave + kGW * i, sz.nc, sz.nm);
  if (!a.tab) {  // (with offsets the cursors are set above)
    int res[kLPW];
    lower_bounds(lists, t_begin, res);
    if (lane == 0)
#pragma unroll
      for (int i = 0; i < kLPW; ++i)
        if (lists[i].on) sh.cur[wave + kGW * i] = res[i];
  }

  if (flat) {
    // membership of the range's one window: each owned list's entries of
    // the range, kF per lane per round, all lists' loads in flight together
    // (before the queries and accumulators hold registers)
    constexpr int kF = 8;
    int c0[kLPW], ne[kLPW];
#pragma unroll
    for (int i = 0; i < kLPW; ++i) {
      const int L = wave + kGW * i;
      c0[i] = lists[i].on ? sh.cur[L] : 0;
      ne[i] = lists[i].on ? sh.cend[L] - c0[i] : 0;
      if (lists[i].on && L >= g && lane == 0) sh.mstart[L - g] = c0[i];
    }
    for (int k0 = 0;; k0 += kF * kWave) {
      bool any = false;
#pragma unroll
      for (int i = 0; i < kLPW; ++i) any |= k0 < ne[i];
      if (!any) break;
      int e[kLPW][kF];
#pragma unroll
      for (int i = 0; i < kLPW; ++i)
#pragma unroll
        for (int k = 0; k < kF; ++k) {
          const int pos = k0 + lane + kWave * k;
          e[i][k] = pos < ne[i] ? lists[i].p[c0[i] + pos] : -1;
        }
#pragma unroll
      for (int i = 0; i < kLPW; ++i)
#pragma unroll
        for (int k = 0; k < kF; ++k) {
          // (an entry outside the window could come only from wrong offsets)
          const int p = e[i][k] - t_begin;
          if ((unsigned)p < (unsigned)(t_end - t_begin)) atomicOr(&sh.mem[p >> 1], lists[i].bit << (16 * (p & 1)));
        }
    }
  }

  // the group's queries as the B operand of QK: lane holds head hc, dims 32ks + 8lq .. +7
  const int64_t qrow0 = ((int64_t)b * a.layers + layer) * a.hq + (int64_t)kvh * g;
  uint4 qb[kD / 32];
#pragma unroll
  for (int ks = 0; ks < kD / 32; ++ks)
    qb[ks] = hc < g ? load16(reinterpret_cast<const unsigned char *>(a.q) + ((qrow0 + hc) * kD + ks * 32 + lq * 8) * 2)
                    : make_uint4(0u, 0u, 0u, 0u);

  const int64_t rowb = kRowB;
  const unsigned char *kb = reinterpret_cast<const unsigned char *>(a.k) + ua * a.n_rows * rowb;
  const unsigned char *vb = reinterpret_cast<const unsigned char *>(a.v) + ua * a.n_rows * rowb;
  const __amdgpu_buffer_rsrc_t kbuf = buffer_of(kb, (int)(a.n_rows * rowb));
  const __amdgpu_buffer_rsrc_t vbuf = buffer_of(vb, (int)(a.n_rows * rowb));
  const __amdgpu_buffer_rsrc_t mbuf = buffer_of(a.marg_prob, a.mp_bytes);
  const int32_t *ksl = a.k_slot ? a.k_slot + ua * a.n_cap : nullptr;
  const int32_t *vsl = a.v_slot ? a.v_slot + ua * a.n_cap : nullptr;
  const int last_row = (int)(a.n_rows - 1);
  // With slot maps into a store of at most 65536 rows, each window's union
  // rows are looked up before the rows stream: the K row replaces the
  // position in the row's entry (membership bits above it), the V row goes
  // to a 16-bit table in the membership words, so the streaming loop reads
  // both from LDS instead of waiting on two dependent loads per block.
  constexpr bool resolved = kResolved;
  constexpr int bit0 = resolved ? 16 : kPosBits;  // membership bits' position in an entry
  uint16_t *const vrow = reinterpret_cast<uint16_t *>(sh.mem);

  f32x4_t acc[kD / 16];
#pragma unroll
  for (int nb = 0; nb < kD / 16; ++nb) acc[nb] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  float m_run = -INFINITY, z_lane = 0.0f;  // per column hc (a head for hc < g)

  for (int ws = t_begin; ws < t_end; ws += kWin) {
    const int we = min(ws + kWin, t_end);

    // ---- membership (a single window with list offsets: above) -----------
    if (!flat) {
      // scan each owned list from its cursor up to we
      int c[kLPW];
      bool act[kLPW];
#pragma unroll
      for (int i = 0; i < kLPW; ++i) {
        act[i] = lists[i].on;
        c[i] = act[i] ? sh.cur[wave + kGW * i] : 0;
        const int L = wave + kGW * i;
        if (act[i] && L >= g && lane == 0) sh.mstart[L - g] = c[i];
      }
      for (;;) {
        bool any = false;
#pragma unroll
        for (int i = 0; i < kLPW; ++i) any |= act[i];
        if (!any) break;
        int e[kLPW][4];
#pragma unroll
        for (int i = 0; i < kLPW; ++i)
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int pos = c[i] + lane + kWave * k;
            e[i][k] = (act[i] && pos < lists[i].len) ? lists[i].p[pos] : INT_MAX;
          }
#pragma unroll
        for (int i = 0; i < kLPW; ++i) {
          if (!act[i]) continue;
          int cnt = 0;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const bool in = e[i][k] < we;
            if (in && e[i][k] >= ws) {
              const int p = e[i][k] - ws;
              atomicOr(&sh.mem[p >> 1], lists[i].bit << (16 * (p & 1)));
            }
            cnt += __popcll(__ballot(in));
          }
          c[i] += cnt;
          if (cnt < 4 * kWave) act[i] = false;
        }
      }
      if (lane == 0)
#pragma unroll
        for (int i = 0; i < kLPW; ++i)
          if (lists[i].on) sh.cur[wave + kGW * i] = c[i];
    }
    __syncthreads();

    // ---- compaction into ascending union rows ---------------------------
    // Thread t takes pc consecutive positions, so wave w's rows are those
    // of positions [w * 64 * pc, (w + 1) * 64 * pc): it streams exactly the
    // rows its own threads compact, and counts their marginal bits here.
    // Thread t takes positions t*pc .. +pc-1: the membership words from
    // word t*pc/2 on, shifted by half a word when t*pc is odd, so that
    // mw[k] holds positions 2k and 2k+1 of the thread.
    constexpr int PW = kWin / kGT / 2;  // most membership words per thread
    const int pc = (we - ws + kGT - 1) / kGT;
    const int w0 = (tid * pc) >> 1, odd = (tid * pc) & 1;
    // (loops over words and positions stop at the window's pc: wave-uniform)
    uint32_t mw[PW];
    if ((pc & 1) == 0) {  // every thread starts on a word boundary
#pragma unroll
      for (int k = 0; k < PW; ++k) mw[k] = 2 * k < pc ? sh.mem[w0 + k] : 0u;
    } else {
      uint32_t nx = 0u;
#pragma unroll
      for (int k = PW; k >= 0; --k) {
        uint32_t x = 0u;
        if (2 * k <= pc && 2 * k < pc + odd && w0 + k < kWin / 2) x = sh.mem[w0 + k];
        if (k < PW) {
          mw[k] = odd ? __builtin_amdgcn_alignbit(nx, x, 16) : x;
          if (2 * k + 1 >= pc) mw[k] &= 2 * k < pc ? 0xffffu : 0u;  // past the thread's last position
        }
        nx = x;
      }
    }
    int cnt = 0;
#pragma unroll
    for (int k = 0; k < PW; ++k) cnt += ((mw[k] & 0xffffu) != 0u) + ((mw[k] >> 16) != 0u);
    int inc = cnt;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int y = __shfl_up(inc, o, kWave);
      if (lane >= o) inc += y;
    }
    // each wave's union rows go to its own range of uni, from wave*64*pc on
    const int r0 = wave * kWave * pc;
    const int r1 = r0 + __builtin_amdgcn_readlane(inc, kWave - 1);
    for (int h = 0; h < g; ++h) {
      int c = 0;
#pragma unroll
      for (int k = 0; k < PW; ++k) {
        if (2 * k >= pc) break;
        c += __popcll(__ballot((mw[k] >> (8 + h)) & 1u)) + __popcll(__ballot((mw[k] >> (24 + h)) & 1u));
      }
      if (lane == 0) sh.wcnt[wave][h] = c;
    }
    __syncthreads();  // every thread has read its words (a word may be shared by two): clear them
#pragma unroll
    for (int k = 0; k <= PW; ++k)
      if (2 * k <= pc && 2 * k < pc + odd) sh.mem[w0 + k] = 0u;
    {
      int o = r0 + inc - cnt;
#pragma unroll
      for (int k = 0; k < 2 * PW; ++k) {
        if (k >= pc) break;
        const uint32_t m = (mw[k >> 1] >> (16 * (k & 1))) & 0xffffu;
        if (m) sh.uni[o++] = (m << kPosBits) | (uint32_t)(tid * pc + k);
      }
    }
    if constexpr (resolved) {
      // this wave's own rows (written by its own threads above); the
      // membership words of its positions were cleared above, and no other
      // wave touches them until the window's end
      wave_lds_fence();
      for (int i0 = r0; i0 < r1; i0 += 4 * kWave) {
        uint32_t e[4];
        int rk[4], rv[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int i = i0 + j * kWave + lane;
          e[j] = i < r1 ? sh.uni[i] : 0u;
          const int tok = ws + (int)(e[j] & (kWin - 1));
          rk[j] = i < r1 ? ksl[tok] : 0;
          rv[j] = i < r1 ? vsl[tok] : 0;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int i = i0 + j * kWave + lane;
          if (i < r1) {
            sh.uni[i] = ((e[j] >> kPosBits) << 16) | (uint32_t)clampi(rk[j], 0, last_row);
            vrow[i] = (uint16_t)clampi(rv[j], 0, last_row);
          }
        }
      }
      wave_lds_fence();
    }
    // element index in marg_prob of the next marginal entry of each head
    // (wave-uniform: kept in SGPRs)
    int mpos[kMaxG];
#pragma unroll
    for (int h = 0; h < kMaxG; ++h) {
      int p = 0;
      if (h < g) {
        p = (int)(sh.prow[h] * a.km_cap) + sh.mstart[h];
        for (int w = 0; w < wave; ++w) p += sh.wcnt[w][h];
      }
      mpos[h] = __builtin_amdgcn_readfirstlane(p);
    }
    __syncthreads();

    // ---- stream the rows: QK, online softmax, P.V -----------------------
    // Software pipeline: the next block's K rows and marginal weights are
    // requested as soon as this block's QK has consumed its K registers, its
    // V rows as soon as this block's V is in LDS, so the gathers of block
    // i + 1 overlap the arithmetic of block i.
    uint4 kr[2][kD / 32];  // K rows (A operand of QK): row h*16 + hc, dims 32ks + 8lq .. +7
    uint4 vr[8];           // V rows: dims 8hc .. +7 of rows 8lq .. 8lq+7
    float wm[kMaxG];       // p' of the rows' marginal heads (lanes < 32 own the rows)
    auto rows_of = [&](int rb, int &rk, int &rv, uint32_t &bits) {
      const int own = rb + (lane & 31);
      const bool valid = own < r1;
      const uint32_t e = valid ? sh.uni[own] : 0u;
      if constexpr (resolved) {
        bits = e >> 16;
        rk = (int)(e & 0xffffu);
        rv = valid ? (int)vrow[own] : 0;
        return;
      }
      bits = e >> kPosBits;
      const int tok = ws + (int)(e & (kWin - 1));
      rk = tok;
      rv = tok;
      if (valid && ksl) {
        rk = ksl[tok];
        rv = vsl[tok];
      }
      rk = clampi(rk, 0, last_row);
      rv = clampi(rv, 0, last_row);
    };
    // rows no head holds critical are not read: their offset is out of range
    auto issue_k = [&](int rk, uint32_t bits) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int src = h * 16 + hc;
        const int row = __shfl(rk, src, kWave);
        const bool crit = (__shfl((int)bits, src, kWave) & 0xff) != 0;
        const uint32_t off = crit ? (uint32_t)row * kRowB + lq * 16 : kOOB;
#pragma unroll
        for (int ks = 0; ks < kD / 32; ++ks) kr[h][ks] = bload16(kbuf, off + ks * 64);
      }
    };
    // marginal weights p', taken from each head's list by rank (one load per
    // head slot, out of range where the row is not marginal for that head);
    // lanes 32..63 mirror lanes 0..31
    auto issue_m = [&](uint32_t bits) {
      const uint32_t below = (1u << (lane & 31)) - 1u;
#pragma unroll
      for (int h = 0; h < kMaxG; ++h) {
        const bool mb = (bits >> (8 + h)) & 1u;
        const uint32_t mask = (uint32_t)__ballot(mb);
        const int rank = __popc(mask & below);
        const uint32_t off = mb ? (uint32_t)(mpos[h] + rank) * 4u : kOOB;
        wm[h] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(mbuf, off, 0, 0));
        mpos[h] += __popc(mask);
      }
    };
    auto issue_v = [&](int rb, int rv) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int src = lq * 8 + k;
        const int row = __shfl(rv, src, kWave);
        vr[k] = bload16_stream(vbuf, rb + src < r1 ? (uint32_t)row * kRowB + hc * 16 : kOOB);
      }
    };
    if (r0 < r1) {
      int rk, rv;
      uint32_t bits;
      rows_of(r0, rk, rv, bits);
      issue_k(rk, bits);
      issue_m(bits);
      issue_v(r0, rv);
    }
    for (int r = r0; r < r1; r += kBR) {
      const int rn = r + kBR;
      const bool more = rn < r1;

      // QK: S^T[row][head], lane holds rows h*16 + 4lq + i of head hc
      f32x4_t s[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) s[h] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int ks = 0; ks < kD / 32; ++ks)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kr[h][ks]),
                                                         __builtin_bit_cast(bf16x8_t, qb[ks]), s[h], 0, 0, 0);
      // this block's marginal weights into P (frees wm; alpha_M is applied
      // per head at the end), then the next block's K rows and weights go out
#pragma unroll
      for (int h = 0; h < kMaxG; ++h) wt.p[8 + h][lane & 31] = wm[h];
      int rvn = 0;
      if (more) {
        // the next block's requests at a raised wave priority, so that they
        // leave before the other waves' arithmetic (LLaMA stage 3 -1%)
        int rkn;
        uint32_t bitsn;
        __builtin_amdgcn_s_setprio(2);
        rows_of(rn, rkn, rvn, bitsn);
        issue_k(rkn, bitsn);
        issue_m(bitsn);
        __builtin_amdgcn_s_setprio(0);
      }
      float sv[2][4];
      float bmax = -INFINITY;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int rr = r + h * 16 + lq * 4;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t uu = sh.uni[min(rr + i, kWin - 1)];
          const bool cb = hc < g && rr + i < r1 && ((uu >> (bit0 + hc)) & 1u);
          sv[h][i] = cb ? s[h][i] * a.scale : -INFINITY;
          bmax = fmaxf(bmax, sv[h][i]);
        }
      }
      bmax = max_xor16(max_xor32(bmax));
      const float mn = fmaxf(m_run, bmax);
      const float alpha = mn == -INFINITY ? 1.0f : __expf(m_run - mn);
      m_run = mn;
      z_lane *= alpha;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float ev[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ev[i] = sv[h][i] == -INFINITY ? 0.0f : __expf(sv[h][i] - mn);
          z_lane += ev[i];
        }
        if (hc < 8)
          *reinterpret_cast<float4 *>(&wt.p[hc][h * 16 + lq * 4]) = make_float4(ev[0], ev[1], ev[2], ev[3]);
      }
      if (lane < 8) wt.alpha[lane] = alpha;

      // V^T into LDS: 8 dims x 8 rows per lane through v_perm
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        const uint32_t sel = (d & 1) ? 0x07060302u : 0x05040100u;
        uint32_t w4[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const uint32_t x0 = (&vr[2 * p].x)[d >> 1], x1 = (&vr[2 * p + 1].x)[d >> 1];
          w4[p] = __builtin_amdgcn_perm(x1, x0, sel);
        }
        *reinterpret_cast<uint4 *>(wt.vt + vt_off(hc * 8 + d, lq)) = make_uint4(w4[0], w4[1], w4[2], w4[3]);
      }
      if (more) {
        __builtin_amdgcn_s_setprio(2);
        issue_v(rn, rvn);
        __builtin_amdgcn_s_setprio(0);
      }
      wave_lds_fence();

      // P.V: O[slot][dim] += P[slot][rows] V[rows][dim]
      if (__ballot(alpha != 1.0f)) {  // some head's max moved
        const float4 al = *reinterpret_cast<const float4 *>(&wt.alpha[lq * 4]);
#pragma unroll
        for (int nb = 0; nb < kD / 16; ++nb) {
          acc[nb][0] *= al.x;
          acc[nb][1] *= al.y;
          acc[nb][2] *= al.z;
          acc[nb][3] *= al.w;
        }
      }
      const float4 p0 = *reinterpret_cast<const float4 *>(&wt.p[hc][lq * 8]);
      const float4 p1 = *reinterpret_cast<const float4 *>(&wt.p[hc][lq * 8 + 4]);
      const float pf[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
      bf16x8_t ph, pl;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const __bf16 hi = (__bf16)pf[i];
        ph[i] = hi;
        pl[i] = (__bf16)(pf[i] - (float)hi);
      }
      // four dim blocks at a time: hi for each, then lo, so that no
      // accumulator feeds the very next MFMA
#pragma unroll
      for (int nq = 0; nq < kD / 16; nq += 4) {
        bf16x8_t B[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          B[i] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4 *>(wt.vt + vt_off((nq + i) * 16 + hc, lq)));
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[nq + i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, B[i], acc[nq + i], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[nq + i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, B[i], acc[nq + i], 0, 0, 0);
      }
      wave_lds_fence();
    }
    if (resolved && we < t_end) {
      // the next window's membership goes into the words the V rows used:
      // each wave clears its own (only it reads them), then all wait, so
      // that no wave's membership writes meet another's clearing
      for (int i = (r0 >> 1) + lane; i < (r1 + 1) >> 1; i += kWave) sh.mem[i] = 0u;
      __syncthreads();
    }
  }

  // ---- merge the waves, then write the output or this split's record ----
  const float z_col = sum_xor16(sum_xor32(z_lane));
  __syncthreads();  // the V^T tiles are free
  static_assert(16 * kD * 4 <= kVTBytes, "the wave's O fits the V^T tile");
  float *wo = reinterpret_cast<float *>(wt.vt);  // [16 slots][kD]
#pragma unroll
  for (int nb = 0; nb < kD / 16; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) wo[(lq * 4 + i) * kD + nb * 16 + hc] = acc[nb][i];
  if (lane < 16) {
    wt.p[0][lane] = m_run;
    wt.p[1][lane] = z_col;
  }
  __syncthreads();
  for (int idx = tid; idx < g * kD; idx += kGT) {
    const int h = idx / kD, d = idx % kD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kGW; ++w) M = fmaxf(M, sh.w[w].p[0][h]);
    float Z = 0.0f, oc = 0.0f, om = 0.0f;
#pragma unroll
    for (int w = 0; w < kGW; ++w) {
      const float mw = sh.w[w].p[0][h];
      const float f = mw == -INFINITY ? 0.0f : __expf(mw - M);
      const float *o = reinterpret_cast<const float *>(sh.w[w].vt);
      Z = __builtin_fmaf(sh.w[w].p[1][h], f, Z);
      oc = __builtin_fmaf(o[h * kD + d], f, oc);
      om += o[(8 + h) * kD + d];
    }
    om *= sh.am[h];
    if (a.n_split == 1) {
      const float o = (Z > 0.0f ? sh.ac[h] * (oc / Z) : 0.0f) + om;
      elem<bf16_t>::store1(a.out, (qrow0 + h) * kD + d, o);
    } else {
      float *rec = a.rec + (((int64_t)u * a.n_split + sp) * g + h) * kRec;
      if (d == 0) {
        rec[0] = M;
        rec[1] = Z;
      }
      rec[2 + d] = oc;
      rec[2 + kD + d] = om;
    }
  }
}

// Combine the split records of one (sequence, layer, kv head, query head):
// log-sum-exp over the critical parts, plain sum over the marginal parts.
// One workgroup per query head, one thread per dim.
__global__ __launch_bounds__(kD) void hybrid_group_merge(GroupArgs a) {
  const int u = blockIdx.x / a.g, h = blockIdx.x % a.g, d = threadIdx.x;
  const int kvh = u % a.hkv, bl = u / a.hkv, layer = a.layer0 + bl % a.nl, b = bl / a.nl;
  const int n = clampi(a.seq_len[b], 1, a.n_cap);
  const int ns = clampi((n + a.span - 1) / a.span, 1, min(a.n_split, kMaxSplit));
  const int g = a.g;
  const int64_t qrow = ((int64_t)b * a.layers + layer) * a.hq + (int64_t)kvh * g + h;
  const int j = clampi(a.head_map[layer * a.hq + kvh * g + h], 0, a.nsh - 1);
  const int64_t row = a.group_sel ? qrow : (int64_t)b * a.nsh + j;
  float ac, am;
  alphas(a.mode, a.mass[2 * row], a.mass[2 * row + 1], ac, am);
  const float *rec0 = a.rec + ((int64_t)u * a.n_split * g + h) * kRec;
  const int64_t sstride = (int64_t)g * kRec;
  // the records eight at a time, all eight in flight at once (past ns the
  // last record is re-read and weighted 0), combined online
  constexpr int kGroup = 8;
  float M = -INFINITY, Z = 0.0f, oc = 0.0f, om = 0.0f;
  for (int s0 = 0; s0 < ns; s0 += kGroup) {
    float ms[kGroup], zs[kGroup], os[kGroup], oms[kGroup];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const float *r = rec0 + min(s0 + i, ns - 1) * sstride;
      ms[i] = r[0];
      zs[i] = r[1];
      os[i] = r[2 + d];
      oms[i] = r[2 + kD + d];
    }
    float mg = M;
#pragma unroll
    for (int i = 0; i < kGroup; ++i) mg = s0 + i < ns ? fmaxf(mg, ms[i]) : mg;
    if (mg != M) {  // (uniform) rescale what the earlier groups added
      const float f = M == -INFINITY ? 0.0f : __expf(M - mg);
      Z *= f;
      oc *= f;
      M = mg;
    }
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const bool ok = s0 + i < ns;
      const float f = (!ok || ms[i] == -INFINITY) ? 0.0f : __expf(ms[i] - M);
      Z = __builtin_fmaf(zs[i], f, Z);
      oc = __builtin_fmaf(os[i], f, oc);
      om += ok ? oms[i] : 0.0f;
    }
  }
  const float o = (Z > 0.0f ? ac * (oc / Z) : 0.0f) + om;
  elem<bf16_t>::store1(a.out, qrow * kD + d, o);
}

}  // namespace

GroupPlan plan_group(const smallkv_batch_t &b, const smallkv_model_t &m, int n_small_heads,
                     int n_run) {
  GroupPlan p{};
  if (n_run < 0) n_run = m.n_layers;
  const int g = m.n_q_heads / m.n_kv_heads;
  p.use = m.dtype == SMALLKV_BF16 && m.head_dim == kD && g <= kMaxG &&
          m.n_rows * kRowB <= kMaxBuf &&
          (int64_t)b.batch * std::max<int64_t>(n_small_heads, (int64_t)m.n_layers * m.n_q_heads) *
                  b.km_cap * (int64_t)sizeof(float) <= kMaxBuf;  // marg_prob of either selection
  if (!p.use) return p;
  const int64_t units = (int64_t)b.batch * n_run * m.n_kv_heads;
  // splits per kv head: the fewest token-equivalents on the critical path,
  // rounds of resident workgroups (a partial last round costs a whole one) x
  // (span + the fixed per-workgroup setup); ties go to fewer splits
  const int64_t max_s = (b.n_cap + 255) / 256;  // at least 256 tokens per split
  auto cost = [&](int64_t c) {
    return (units * c + kTargetWgs - 1) / kTargetWgs * ((b.n_cap + c - 1) / c + kSetupTok);
  };
  int64_t s = 1;
  for (int64_t c = 2; c <= kMaxSplit && c <= max_s; ++c)
    if (cost(c) < cost(s)) s = c;
  p.span = (int)(((b.n_cap + s - 1) / s + 255) / 256 * 256);  // range starts on list-offset blocks
  p.n_split = (int)((b.n_cap + p.span - 1) / p.span);
  p.ws_bytes = p.n_split > 1 ? (size_t)units * p.n_split * g * kRec * sizeof(float) : 0;
  return p;
}

hipError_t launch_hybrid_group(const smallkv_batch_t &b, const smallkv_model_t &m,
                               const int32_t *head_map, int n_small_heads, const int32_t *crit,
                               const int32_t *marg, const float *marg_prob, const float *mass,
                               int mode, const GroupPlan &p, float *ws, const int2 *tab,
                               bool group_sel, int layer0, int nl, hipStream_t st) {
  GroupArgs a;
  a.layer0 = layer0;
  a.nl = nl;
  a.n_cap = b.n_cap;
  a.layers = m.n_layers;
  a.hq = m.n_q_heads;
  a.hkv = m.n_kv_heads;
  a.g = m.n_q_heads / m.n_kv_heads;
  a.nsh = n_small_heads;
  a.kc_cap = b.kc_cap;
  a.km_cap = b.km_cap;
  a.mode = mode;
  a.units = b.batch * nl * m.n_kv_heads;
  a.n_split = p.n_split;
  a.span = p.span;
  const int64_t prows = group_sel ? (int64_t)m.n_layers * m.n_q_heads : n_small_heads;
  a.mp_bytes = (int)((int64_t)b.batch * prows * b.km_cap * (int64_t)sizeof(float));
  a.n_rows = m.n_rows;
  a.scale = m.scale;
  a.seq_len = b.seq_len;
  a.k_crit = b.k_crit;
  a.k_marg = b.k_marg;
  a.k_recent = b.k_recent;
  a.head_map = head_map;
  a.q = m.q;
  a.k = m.k;
  a.v = m.v;
  a.k_slot = m.k_slot;
  a.v_slot = m.v_slot;
  a.crit = crit;
  a.marg = marg;
  a.marg_prob = marg_prob;
  a.mass = mass;
  a.group_sel = group_sel ? 1 : 0;
  a.rec = ws;
  a.tab = tab;
  a.nblk = list_blocks(b);
  a.out = m.out;
  const int groups = (a.units + kXcd - 1) / kXcd;
  if (m.k_slot && m.n_rows <= 65536)
    hipLaunchKernelGGL(hybrid_group_kernel<true>, dim3(groups * kXcd * a.n_split), dim3(kGT), 0, st, a);
  else
    hipLaunchKernelGGL(hybrid_group_kernel<false>, dim3(groups * kXcd * a.n_split), dim3(kGT), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_split == 1) return e;
  hipLaunchKernelGGL(hybrid_group_merge, dim3(a.units * a.g), dim3(kD), 0, st, a);
  return hipGetLastError();
}

}  // namespace smallkv
