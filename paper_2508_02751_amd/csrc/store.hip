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
//                  in LDS (atomic ORs from the lists), ranks by a popcount
//                  scan over the bitmap words, both slot maps for t < N_b,
//                  the unions' token lists (workspace) and their sizes;
//   store_copy  -- 16 lanes per row, 16 bytes each, four rows in flight,
//                  eight workgroups per kv head and union: every row from the
//                  old store or the full one.
#include "common.h"
#include "launch.h"

namespace smallkv {
namespace {

constexpr int kST = 256;

struct StoreArgs {
  int n_cap, layers, hq, hkv, g, nsh, kc_cap, km_cap, select, words;
  int64_t rows;
  int row_bytes;  // head_dim * element size
  const int32_t *seq_len, *head_map, *crit, *marg;
  const unsigned char *full_k, *full_v, *old_k, *old_v;
  const int32_t *old_k_slot, *old_v_slot;
  unsigned char *new_k, *new_v;
  int32_t *k_slot, *v_slot, *counts;
  int32_t *uk, *uv;  // [units][rows]: the unions' tokens in row order
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
  for (int w = 0; w < kST / kWave; ++w) {
    if (w < wave) base += red[w];
    total += red[w];
  }
  __syncthreads();
  return base + x - v;
}

__global__ __launch_bounds__(kST) void store_index(StoreArgs a) {
  extern __shared__ uint32_t smem[];  // bits K [words], bits V [words], word ranks K, V
  uint32_t *bk = smem, *bv = smem + a.words;
  int *rk = reinterpret_cast<int *>(smem + 2 * a.words), *rv = rk + a.words;
  __shared__ int red[kST / kWave];
  const int unit = blockIdx.x;
  const int kvh = unit % a.hkv, bl = unit / a.hkv, layer = bl % a.layers, b = bl / a.layers;
  const int n = clampi(a.seq_len[b], 1, a.n_cap);
  const int nw = (n + 31) / 32;
  for (int w = threadIdx.x; w < nw; w += kST) bk[w] = bv[w] = 0u;
  __syncthreads();
  // membership from the lists of the group's query heads (-1 padding and
  // anything outside [0, n) ignored)
  for (int h = 0; h < a.g; ++h) {
    int64_t row;
    if (a.select) {
      row = unit;
    } else {
      const int j = clampi(a.head_map[layer * a.hq + kvh * a.g + h], 0, a.nsh - 1);
      row = (int64_t)b * a.nsh + j;
    }
    const int32_t *c = a.crit + row * a.kc_cap, *m = a.marg + row * a.km_cap;
    for (int i = threadIdx.x; i < a.kc_cap; i += kST) {
      const int t = c[i];
      if (t >= 0 && t < n) {
        atomicOr(&bk[t >> 5], 1u << (t & 31));
        atomicOr(&bv[t >> 5], 1u << (t & 31));
      }
    }
    for (int i = threadIdx.x; i < a.km_cap; i += kST) {
      const int t = m[i];
      if (t >= 0 && t < n) atomicOr(&bv[t >> 5], 1u << (t & 31));
    }
  }
  __syncthreads();
  // word ranks: each thread scans a run of consecutive words
  const int per = (nw + kST - 1) / kST, w0 = threadIdx.x * per, w1 = min(w0 + per, nw);
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
  // slot maps and the unions' token lists
  const int64_t sbase = (int64_t)unit * a.n_cap, ubase = (int64_t)unit * a.rows;
  for (int t = threadIdx.x; t < n; t += kST) {
    const uint32_t below = (1u << (t & 31)) - 1u;
    const uint32_t wk = bk[t >> 5], wv = bv[t >> 5];
    int sk = -1, sv = -1;
    if (wk >> (t & 31) & 1u) {
      const int r = rk[t >> 5] + __popc(wk & below);
      if (r < a.rows) {
        sk = r;
        a.uk[ubase + r] = t;
      }
    }
    if (wv >> (t & 31) & 1u) {
      const int r = rv[t >> 5] + __popc(wv & below);
      if (r < a.rows) {
        sv = r;
        a.uv[ubase + r] = t;
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
// shares of its rows; blockIdx.z: K (0) or V (1).  Each group of 16 lanes
// copies one row at a time in 16-byte pieces, four rows in flight; a row is
// one of the union's, from the old store when its old slot map holds the
// token, else from the full store.
constexpr int kCopySplit = 8;

__global__ __launch_bounds__(kST) void store_copy(StoreArgs a) {
  constexpr int kGroups = kST / 16, kStride = kCopySplit * kGroups, kInFlight = 4;
  const int unit = blockIdx.x, isv = blockIdx.z;
  const int lim = (int)min<int64_t>((int64_t)a.counts[2 * (int64_t)unit + isv], a.rows);
  const int lane16 = threadIdx.x & 15;
  const int first = blockIdx.y * kGroups + (threadIdx.x >> 4);
  const int32_t *u = (isv ? a.uv : a.uk) + (int64_t)unit * a.rows;
  const int32_t *old_slot = isv ? a.old_v_slot : a.old_k_slot;
  const unsigned char *full = isv ? a.full_v : a.full_k;
  const unsigned char *old = isv ? a.old_v : a.old_k;
  unsigned char *dst = isv ? a.new_v : a.new_k;
  const int pieces = a.row_bytes / 16;  // 4 .. 32
  for (int p = lane16; p < pieces; p += 16)
    for (int r0 = first; r0 < lim; r0 += kInFlight * kStride) {
      uint4 v[kInFlight];
#pragma unroll
      for (int k = 0; k < kInFlight; ++k) {
        const int r = r0 + k * kStride;
        if (r < lim) {
          const int t = clampi(u[r], 0, a.n_cap - 1);
          const int os = old_slot ? old_slot[(int64_t)unit * a.n_cap + t] : -1;
          const unsigned char *src =
              (old && os >= 0 && os < a.rows)
                  ? old + ((int64_t)unit * a.rows + os) * a.row_bytes
                  : full + ((int64_t)unit * a.n_cap + t) * a.row_bytes;
          v[k] = reinterpret_cast<const uint4 *>(src)[p];
        }
      }
#pragma unroll
      for (int k = 0; k < kInFlight; ++k) {
        const int r = r0 + k * kStride;
        if (r < lim)
          reinterpret_cast<uint4 *>(dst + ((int64_t)unit * a.rows + r) * a.row_bytes)[p] = v[k];
      }
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
  a.uk = w;
  a.uv = w + (size_t)units * s.rows;
  a.counts = s.counts ? s.counts : w + 2 * (size_t)units * s.rows;
  hipLaunchKernelGGL(store_index, dim3(units), dim3(kST), store_index_lds(s.batch.n_cap), st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(store_copy, dim3(units, kCopySplit, 2), dim3(kST), 0, st, a);
  return hipGetLastError();
}

}  // namespace smallkv
