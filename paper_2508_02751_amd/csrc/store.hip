// Maintenance of the large model's compact store after a step's selection:
// the critical tokens keep K and V, the marginal tokens V (Algorithm 1; the
// paper migrates these rows between host and device memory in parallel with
// the large model's forward).  For every (sequence, large layer, kv head):
// U_K = the union of the critical lists of the query heads it serves, U_V =
// U_K and their marginal lists; row r of the new store holds the r-th token
// of the union in ascending order, the slot maps name each token's row (or
// -1).  A row the previous store already holds (its old slot map) is copied
// from there; only the others are read from the full store, which may live
// in host memory.
//
//   store_index -- one workgroup per kv head: membership bits of both unions
//                  in LDS (atomic ORs from the lists, eight list entries in
//                  flight per thread), ranks by a popcount scan over the
//                  bitmap words, both slot maps for t < N_b, the union sizes,
//                  and per union row its source: a row of the old store, or
//                  the token's row of the full store;
//   store_copy  -- the rows as a flat array of 16-byte pieces (a wave reads
//                  1 KB of consecutive rows), one piece per thread per pass,
//                  128 workgroups per kv head and union; one load of the
//                  row's source stands between a piece and its data.
#include "common.h"
#include "launch.h"

namespace smallkv {
namespace {

constexpr int kIT = 1024;  // store_index threads
constexpr int kCT = 256;   // store_copy threads

struct StoreArgs {
  int n_cap, layers, hq, hkv, g, nsh, kc_cap, km_cap, select, words;
  int64_t rows;
  int row_bytes;  // head_dim * element size
  const int32_t *seq_len, *head_map, *crit, *marg;
  const unsigned char *full_k, *full_v, *old_k, *old_v;
  const int32_t *old_k_slot, *old_v_slot;
  unsigned char *new_k, *new_v;
  int32_t *k_slot, *v_slot, *counts;
  // [units][rows] per union, in row order: the old store's row (>= 0) or
  // -(t + 1) for token t's row of the full store
  int32_t *src_k, *src_v;
};

// Exclusive scan of one value per thread over the workgroup.
__device__ __forceinline__ int block_exscan(int v, int *red, int &total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  int x = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  if (lane == kWave - 1) red[wave] = x;
  __syncthreads();
  int base = 0;
  total = 0;
  for (int w = 0; w < kIT / kWave; ++w) {
    if (w < wave) base += red[w];
    total += red[w];
  }
  __syncthreads();
  return base + x - v;
}

// The source code of token t's row in a union: its row in the old store
// when the old slot map holds it, else its row of the full store.
__device__ __forceinline__ int32_t row_source(const int32_t *old_slot, int64_t sbase, int t,
                                              int64_t rows) {
  const int os = old_slot ? old_slot[sbase + t] : -1;
  return (os >= 0 && os < rows) ? os : -(t + 1);
}

__global__ __launch_bounds__(kIT) void store_index(StoreArgs a) {
  extern __shared__ uint32_t smem[];  // bits K [words], bits V [words], word ranks K, V
  uint32_t *bk = smem, *bv = smem + a.words;
  int *rk = reinterpret_cast<int *>(smem + 2 * a.words), *rv = rk + a.words;
  __shared__ int red[kIT / kWave];
  const int unit = blockIdx.x;
  const int kvh = unit % a.hkv, bl = unit / a.hkv, layer = bl % a.layers, b = bl / a.layers;
  const int n = clampi(a.seq_len[b], 1, a.n_cap);
  const int nw = (n + 31) / 32;
  for (int w = threadIdx.x; w < nw; w += kIT) bk[w] = bv[w] = 0u;
  __syncthreads();
  // membership from the lists of the group's query heads (one shared set
  // per kv head with group selection); -1 padding and anything outside
  // [0, n) ignored.  Entry e of the flat walk: head e / per, then its
  // critical list, then its marginal list.
  const int heads = a.select ? 1 : a.g;
  const int per = a.kc_cap + a.km_cap;
  const int total = heads * per;
  constexpr int kBatch = 8;
  for (int e0 = threadIdx.x; e0 < total; e0 += kBatch * kIT) {
    int tok[kBatch];
    bool crit[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {  // every load issued before any use
      const int e = e0 + k * kIT;
      tok[k] = -1;
      crit[k] = false;
      if (e < total) {
        const int h = e / per, i = e - h * per;
        int64_t row;
        if (a.select) {
          row = unit;
        } else {
          const int j = clampi(a.head_map[layer * a.hq + kvh * a.g + h], 0, a.nsh - 1);
          row = (int64_t)b * a.nsh + j;
        }
        crit[k] = i < a.kc_cap;
        tok[k] = crit[k] ? a.crit[row * a.kc_cap + i] : a.marg[row * a.km_cap + (i - a.kc_cap)];
      }
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int t = tok[k];
      if (t >= 0 && t < n) {
        if (crit[k]) atomicOr(&bk[t >> 5], 1u << (t & 31));
        atomicOr(&bv[t >> 5], 1u << (t & 31));
      }
    }
  }
  __syncthreads();
  // word ranks: each thread scans a run of consecutive words
  const int wper = (nw + kIT - 1) / kIT, w0 = threadIdx.x * wper, w1 = min(w0 + wper, nw);
  int ck = 0, cv = 0;
  for (int w = w0; w < w1; ++w) {
    ck += __popc(bk[w]);
    cv += __popc(bv[w]);
  }
  int tk, tv;
  int ok = block_exscan(ck, red, tk);
  int ov = block_exscan(cv, red, tv);
  for (int w = w0; w < w1; ++w) {
    rk[w] = ok;
    rv[w] = ov;
    ok += __popc(bk[w]);
    ov += __popc(bv[w]);
  }
  __syncthreads();
  // slot maps and the rows' sources
  const int64_t sbase = (int64_t)unit * a.n_cap, ubase = (int64_t)unit * a.rows;
  for (int t = threadIdx.x; t < n; t += kIT) {
    const uint32_t below = (1u << (t & 31)) - 1u;
    const uint32_t wk = bk[t >> 5], wv = bv[t >> 5];
    int sk = -1, sv = -1;
    if (wk >> (t & 31) & 1u) {
      const int r = rk[t >> 5] + __popc(wk & below);
      if (r < a.rows) {
        sk = r;
        a.src_k[ubase + r] = row_source(a.old_k ? a.old_k_slot : nullptr, sbase, t, a.rows);
      }
    }
    if (wv >> (t & 31) & 1u) {
      const int r = rv[t >> 5] + __popc(wv & below);
      if (r < a.rows) {
        sv = r;
        a.src_v[ubase + r] = row_source(a.old_v ? a.old_v_slot : nullptr, sbase, t, a.rows);
      }
    }
    a.k_slot[sbase + t] = sk;
    a.v_slot[sbase + t] = sv;
  }
  if (threadIdx.x == 0) {
    a.counts[2 * (int64_t)unit] = tk;
    a.counts[2 * (int64_t)unit + 1] = tv;
  }
}

// blockIdx.x: kv head unit; blockIdx.y: one of kCopySplit interleaved
// shares of the union's pieces; blockIdx.z: K (0) or V (1).  Piece q of the
// flat array is piece q % pieces of row q / pieces.  One piece per thread
// per pass: many workgroups each walking nearby rows keep the DRAM pages
// they touch few (eight pieces in flight per thread, 128 rows apart, ran
// the rebuild 60% slower).
constexpr int kCopySplit = 128;

typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;

__global__ __launch_bounds__(kCT) void store_copy(StoreArgs a) {
  constexpr int kStride = kCopySplit * kCT;
  const int unit = blockIdx.x, isv = blockIdx.z;
  const int lim = (int)min<int64_t>((int64_t)a.counts[2 * (int64_t)unit + isv], a.rows);
  // a power of two (8, 16 or 32); a union has at most n_cap <= 131072 rows,
  // so piece indices fit 32 bits
  const int pieces = a.row_bytes / 16, psh = __ffs(pieces) - 1;
  const int items = lim * pieces;
  const int32_t *src = (isv ? a.src_v : a.src_k) + (int64_t)unit * a.rows;
  const unsigned char *full = (isv ? a.full_v : a.full_k) + (int64_t)unit * a.n_cap * a.row_bytes;
  const unsigned char *old = isv ? a.old_v : a.old_k;
  if (old) old += (int64_t)unit * a.rows * a.row_bytes;
  uint4 *dst = reinterpret_cast<uint4 *>((isv ? a.new_v : a.new_k) + (int64_t)unit * a.rows * a.row_bytes);
  for (int q = blockIdx.y * kCT + threadIdx.x; q < items; q += kStride) {
    const int c = src[q >> psh];
    const unsigned char *row =
        (c >= 0 && old) ? old + (int64_t)c * a.row_bytes
                        : full + (int64_t)clampi(c >= 0 ? 0 : -c - 1, 0, a.n_cap - 1) * a.row_bytes;
    // each piece is read once and written once, and the store is read only
    // by the next step: non-temporal both ways (the rebuild after a Qwen2-7B
    // step 111 -> 104 us)
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(row) + (q & (pieces - 1)));
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t *>(dst) + q);
  }
}

}  // namespace

size_t store_index_lds(int n_cap) {
  const size_t words = (size_t)(n_cap + 31) / 32;
  return words * 4 * sizeof(uint32_t);
}

size_t store_workspace(const smallkv_store_t &s) {
  const size_t units = (size_t)s.batch.batch * s.n_layers * s.n_kv_heads;
  return 2 * units * (size_t)s.rows * sizeof(int32_t) + 2 * units * sizeof(int32_t);
}

hipError_t launch_store_update(const smallkv_store_t &s, void *ws, hipStream_t st) {
  StoreArgs a{};
  a.n_cap = s.batch.n_cap;
  a.layers = s.n_layers;
  a.hq = s.n_q_heads;
  a.hkv = s.n_kv_heads;
  a.g = s.n_q_heads / s.n_kv_heads;
  a.nsh = s.n_small_heads;
  a.kc_cap = s.batch.kc_cap;
  a.km_cap = s.batch.km_cap;
  a.select = s.select == SMALLKV_SELECT_GROUP ? 1 : 0;
  a.words = (s.batch.n_cap + 31) / 32;
  a.rows = s.rows;
  a.row_bytes = s.head_dim * (s.dtype == SMALLKV_F32 ? 4 : 2);
  a.seq_len = s.batch.seq_len;
  a.head_map = s.head_map;
  a.crit = s.crit_idx;
  a.marg = s.marg_idx;
  a.full_k = static_cast<const unsigned char *>(s.full_k);
  a.full_v = static_cast<const unsigned char *>(s.full_v);
  a.old_k = static_cast<const unsigned char *>(s.old_k);
  a.old_v = static_cast<const unsigned char *>(s.old_v);
  a.old_k_slot = s.old_k_slot;
  a.old_v_slot = s.old_v_slot;
  a.new_k = static_cast<unsigned char *>(s.new_k);
  a.new_v = static_cast<unsigned char *>(s.new_v);
  a.k_slot = s.k_slot;
  a.v_slot = s.v_slot;
  const int units = s.batch.batch * s.n_layers * s.n_kv_heads;
  int32_t *w = static_cast<int32_t *>(ws);
  a.src_k = w;
  a.src_v = w + (size_t)units * s.rows;
  a.counts = s.counts ? s.counts : w + 2 * (size_t)units * s.rows;
  hipLaunchKernelGGL(store_index, dim3(units), dim3(kIT), store_index_lds(s.batch.n_cap), st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(store_copy, dim3(units, kCopySplit, 2), dim3(kCT), 0, st, a);
  return hipGetLastError();
}

}  // namespace smallkv
