// Prefill similarity matching (Method section, "Similarity Matching",
// Eqs. 1-3): over a window of the prompt, the accumulative attention score F
// of every head of both models (Eq. 1), each head's TopK token set, and for
// every large head the small head whose TopK set has the largest Jaccard
// similarity (Eqs. 2-3).
//
// The TopK sets and the argmax are integer decisions taken on fp32 sums, so
// every value feeding them has one defined evaluation, the one smallkv.h
// states: logits as sequential fp32 FMA chains; an exp by Cody-Waite
// reduction and a degree-7 Taylor polynomial; row sums and column sums taken
// one term at a time in ascending token order.  The result is bit-exact
// against any implementation of that definition.
//
// Four kernels:
//   match_logits -- the causal logit matrix S of each head, one wave per
//                   64x64 tile, 8x8 independent FMA chains per lane over Q
//                   and K slices staged in LDS as fp32 (one LDS byte read per
//                   FMA), and each row's maximum over the tile;
//   match_rowsum -- one thread per pair of rows (u, w-1-u) of every head, so
//                   that the lanes of a wave do equal work: each row's max
//                   from the tile maxima and its sum Z_u, v ascending;
//   match_scores -- one workgroup per head, one thread per token: the column
//                   sum F_v, u ascending (a wave's lanes read each row of S
//                   together), then the TopK set by counting, for each token,
//                   the tokens ranked above it;
//   match_map    -- one wave per large head: Jaccard ratios against every
//                   small head from TopK bitsets (popcounts), the argmax by
//                   exact cross-multiplication, ties to the lowest small head.
#include "common.h"
#include "launch.h"

#pragma clang fp contract(off)

namespace smallkv {
namespace {

constexpr int kTile = 64;     // tokens per side of a logit tile
constexpr int kMatchThreads = 256;

struct LogitArgs {
  const void *q, *k;  // [B][layers][hq][w_cap][D], [B][layers][hkv][w_cap][D]
  int layers, hq, hkv, w_cap, ld, nt;  // ld: row pitch of S
  float scale;
  const int32_t *win_len;
  float *S;           // [B][H][w_cap][ld], entries v <= u < w written
  float *pmax;        // [B][H][w_cap][nt]: max of row u over tile column V
  int H, head0;       // heads per sequence (both models); this model's first
};

constexpr int kChunk = 32;            // head-dim slice staged per step
constexpr int kPitch = kChunk + 4;    // LDS row pitch (floats)

// Stage dims [c0, c0+kChunk) of 64 rows of one head's operand, from token r0,
// into LDS as fp32; rows at or past the window are zero.  Every load of the
// slice is issued before the first is used.
// A 64-row x kChunk-dim slice in two steps: its 16-byte pieces into
// registers (issued a chunk ahead of their use), then into LDS as fp32.
template <typename T>
struct Slice {
  static constexpr int per = elem<T>::per16;
  static constexpr int vpr = kChunk / per;       // 16-byte vectors per row slice
  static constexpr int n = kTile * vpr / kWave;  // vectors per lane
};

template <typename T, int D>
__device__ __forceinline__ void load_chunk(uint4 (&v)[Slice<T>::n], const T *src, int r0, int w, int c0) {
  constexpr int per = Slice<T>::per, vpr = Slice<T>::vpr, n = Slice<T>::n;
#pragma unroll
  for (int q = 0; q < n; ++q) {
    const int e = q * kWave + threadIdx.x, r = e / vpr, c = (e % vpr) * per;
    v[q] = r0 + r < w ? *reinterpret_cast<const uint4 *>(src + (int64_t)(r0 + r) * D + c0 + c)
                      : make_uint4(0u, 0u, 0u, 0u);
  }
}

template <typename T>
__device__ __forceinline__ void store_chunk(float *dst, const uint4 (&v)[Slice<T>::n]) {
  constexpr int per = Slice<T>::per, vpr = Slice<T>::vpr, n = Slice<T>::n;
#pragma unroll
  for (int q = 0; q < n; ++q) {
    const int e = q * kWave + threadIdx.x, r = e / vpr, c = (e % vpr) * per;
    float o[per];
    elem<T>::unpack(v[q], o);
#pragma unroll
    for (int i = 0; i < per; i += 4)
      *reinterpret_cast<float4 *>(dst + r * kPitch + c + i) =
          make_float4(o[i], o[i + 1], o[i + 2], o[i + 3]);
  }
}

// 8x8 FMA chains of one lane over one staged slice: rows ty + 8i of Qs,
// columns tx + 8j of Ks, dims ascending.  kFull: all 64 rows and columns of
// the tile are in the window (no bounds in the loop body).
template <bool kFull>
__device__ __forceinline__ void chains(float (&acc)[8][8], const float *Qs, const float *Ks, int ty,
                                       int tx, int imax, int jmax) {
#pragma unroll 1
  for (int c = 0; c < kChunk; c += 4) {
    float4 qa[8], kb[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (kFull || i < imax) qa[i] = *reinterpret_cast<const float4 *>(Qs + (ty + 8 * i) * kPitch + c);
#pragma unroll
    for (int jj = 0; jj < 8; ++jj)
      if (kFull || jj < jmax) kb[jj] = *reinterpret_cast<const float4 *>(Ks + (tx + 8 * jj) * kPitch + c);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (!kFull && i >= imax) break;  // rows past the window (uniform)
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        if (!kFull && jj >= jmax) break;
        float s = acc[i][jj];
        s = __builtin_fmaf(qa[i].x, kb[jj].x, s);
        s = __builtin_fmaf(qa[i].y, kb[jj].y, s);
        s = __builtin_fmaf(qa[i].z, kb[jj].z, s);
        s = __builtin_fmaf(qa[i].w, kb[jj].w, s);
        acc[i][jj] = s;
      }
    }
  }
}

// One wave per 64x64 tile (U, V) of the lower triangle.  Lane (ty, tx) owns
// rows ty + 8i and columns tx + 8j (i, j < 8): 64 independent FMA chains,
// each over the head dimension in ascending order.  kFull: the tile lies
// wholly inside the window; otherwise it is in the window's last, partial
// tile row, whose rows and columns past the window are skipped 8 at a time.
template <typename T, int D, bool kFull>
__device__ __forceinline__ void logits_tile(const LogitArgs &a, float *Qs, float *Ks, int U, int V,
                                            int j, int b, int w) {
  const int imax = min(8, (w - U * kTile + 7) / 8);
  const int jmax = min(8, (w - V * kTile + 7) / 8);
  const int layer = j / a.hq, h = j % a.hq, g = h / (a.hq / a.hkv);
  const T *Q = static_cast<const T *>(a.q) + ((((int64_t)b * a.layers + layer) * a.hq + h) * a.w_cap) * D;
  const T *K = static_cast<const T *>(a.k) + ((((int64_t)b * a.layers + layer) * a.hkv + g) * a.w_cap) * D;
  const int lane = threadIdx.x, ty = lane >> 3, tx = lane & 7;
  float acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) acc[i][jj] = 0.0f;
  uint4 qv[Slice<T>::n], kv[Slice<T>::n];
  load_chunk<T, D>(qv, Q, U * kTile, w, 0);
  load_chunk<T, D>(kv, K, V * kTile, w, 0);
  for (int c0 = 0; c0 < D; c0 += kChunk) {
    store_chunk<T>(Qs, qv);
    store_chunk<T>(Ks, kv);
    __syncthreads();
    if (c0 + kChunk < D) {  // the next slice arrives while this one is used
      load_chunk<T, D>(qv, Q, U * kTile, w, c0 + kChunk);
      load_chunk<T, D>(kv, K, V * kTile, w, c0 + kChunk);
    }
    chains<kFull>(acc, Qs, Ks, ty, tx, imax, jmax);
    __syncthreads();
  }
  const int64_t hrow = (int64_t)b * a.H + a.head0 + j;
  float *S = a.S + hrow * a.w_cap * a.ld;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (i >= imax) continue;
    const int u = U * kTile + ty + 8 * i;
    float m = -INFINITY;
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      if (jj >= jmax) continue;
      const int v = V * kTile + tx + 8 * jj;
      float s = __fmul_rn(acc[i][jj], a.scale);
      if (s == 0.0f) s = 0.0f;  // -0 -> +0
      if (u < w && v <= u) {
        S[(int64_t)u * a.ld + v] = s;
        m = s > m ? s : m;
      }
    }
    // max over the 8 lanes of this row group
#pragma unroll
    for (int o = 1; o < 8; o <<= 1) {
      const float x = __shfl_xor(m, o, kWave);
      m = x > m ? x : m;
    }
    if (tx == 0 && u < w) a.pmax[(hrow * a.w_cap + u) * a.nt + V] = m;
  }
}

// blockIdx.x < nt*(nt+1)/2 enumerates the lower triangle of tiles (those
// wholly inside the window are computed); the next nt blocks are the tile
// columns of the window's last tile row when the window is not a multiple of
// 64 tokens.  Both kinds run in one launch.
template <typename T, int D>
__global__ __launch_bounds__(kWave) void match_logits(LogitArgs a) {
  __shared__ float Qs[kTile * kPitch];
  __shared__ float Ks[kTile * kPitch];
  const int j = blockIdx.y, b = blockIdx.z;
  const int w = clampi(a.win_len[b], 1, a.w_cap);
  const int tri = a.nt * (a.nt + 1) / 2;
  if ((int)blockIdx.x < tri) {
    int U = 0;
    while ((U + 1) * (U + 2) / 2 <= (int)blockIdx.x) ++U;
    const int V = (int)blockIdx.x - U * (U + 1) / 2;
    if ((U + 1) * kTile > w) return;
    logits_tile<T, D, true>(a, Qs, Ks, U, V, j, b, w);
  } else {
    const int U = (w - 1) / kTile, V = (int)blockIdx.x - tri;
    if ((U + 1) * kTile == w || V > U) return;
    logits_tile<T, D, false>(a, Qs, Ks, U, V, j, b, w);
  }
}

struct ScoreArgs {
  const float *S, *pmax;
  float2 *mz;               // [B][H][w_cap]: (m_u, Z_u)
  int w_cap, ld, nt, H, nw; // nw: 64-token words per TopK bitset
  const int32_t *win_len, *top_k;
  uint64_t *bits;           // [B][H][nw]
  float *scores;            // optional [B][H][w_cap]
  uint64_t *top_bits;       // optional copy of bits
};

constexpr int kInFlight = 8;  // loads each thread issues before using them

// Row statistics: one thread per row u of every head (blockIdx.x covers 256
// rows, blockIdx.y the head, blockIdx.z the sequence).  m_u from the tile
// maxima; Z_u = e[u][0] + ... + e[u][u], one term at a time, v ascending.
// Row u's max (from the tile maxima) and its sum Z_u, v ascending.
__device__ __forceinline__ void row_sum(const ScoreArgs &a, int64_t hrow, int u) {
  const float *pm = a.pmax + (hrow * a.w_cap + u) * a.nt;
  float m = pm[0];
  for (int V = 1; V <= u / kTile; ++V) m = pm[V] > m ? pm[V] : m;
  const float4 *row = reinterpret_cast<const float4 *>(a.S + (hrow * a.w_cap + u) * a.ld);
  const int n4 = u / 4 + 1;  // float4s holding v = 0 .. u
  float z = 0.0f;
  for (int i0 = 0; i0 < n4; i0 += kInFlight) {
    float4 x[kInFlight];
#pragma unroll
    for (int q = 0; q < kInFlight; ++q) x[q] = i0 + q < n4 ? row[i0 + q] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int q = 0; q < kInFlight; ++q) {
      const int v = 4 * (i0 + q);
      if (v <= u) z = __fadd_rn(z, cw_exp(__fsub_rn(x[q].x, m)));
      if (v + 1 <= u) z = __fadd_rn(z, cw_exp(__fsub_rn(x[q].y, m)));
      if (v + 2 <= u) z = __fadd_rn(z, cw_exp(__fsub_rn(x[q].z, m)));
      if (v + 3 <= u) z = __fadd_rn(z, cw_exp(__fsub_rn(x[q].w, m)));
    }
  }
  a.mz[hrow * a.w_cap + u] = make_float2(m, z);
}

// Thread p sums rows p and w-1-p (once when they coincide), so that every
// lane of a wave adds about w terms whatever its rows.
__global__ __launch_bounds__(kMatchThreads) void match_rowsum(ScoreArgs a) {
  const int p = blockIdx.x * kMatchThreads + threadIdx.x, head = blockIdx.y, b = blockIdx.z;
  const int w = clampi(a.win_len[b], 1, a.w_cap);
  if (p >= (w + 1) / 2) return;
  const int64_t hrow = (int64_t)b * a.H + head;
  row_sum(a, hrow, p);
  if (w - 1 - p != p) row_sum(a, hrow, w - 1 - p);
}

// Column sums and the TopK set: one workgroup per head, thread v adds
// e[u][v] / Z_u for u = v, v+1, ..., w-1, one term at a time (the threads of
// a wave read one row of S together).
__global__ __launch_bounds__(kMatchThreads) void match_scores(ScoreArgs a) {
  __shared__ float2 smz[kMatchThreads];
  __shared__ float sf[kMatchThreads];
  const int head = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
  const int w = clampi(a.win_len[b], 1, a.w_cap);
  const int k = clampi(a.top_k[b], 1, w);
  const int64_t hrow = (int64_t)b * a.H + head;
  if (t < w) smz[t] = a.mz[hrow * a.w_cap + t];
  __syncthreads();
  float f = 0.0f;
  if (t < w) {
    const float *col = a.S + hrow * a.w_cap * a.ld + t;
    // rows from the wave's first column, so that the lanes read each row together
    for (int u0 = t & ~(kWave - 1); u0 < w; u0 += kInFlight) {
      float x[kInFlight];
#pragma unroll
      for (int q = 0; q < kInFlight; ++q) {
        const int u = u0 + q;
        x[q] = (u < w && u >= t) ? col[(int64_t)u * a.ld] : 0.0f;
      }
#pragma unroll
      for (int q = 0; q < kInFlight; ++q) {
        const int u = u0 + q;
        if (u < w && u >= t) {
          const float2 mz = smz[u];
          f = __fadd_rn(f, __fdiv_rn(cw_exp(__fsub_rn(x[q], mz.x)), mz.y));
        }
      }
    }
    sf[t] = f;
  }
  __syncthreads();
  // TopK: ranked first by larger F, then by lower token index
  bool in = false;
  if (t < w) {
    int above = 0;
    for (int u = 0; u < w; ++u) {
      const float x = sf[u];
      above += (x > f || (x == f && u < t)) ? 1 : 0;
    }
    in = above < k;
  }
  const uint64_t word = __ballot(in);
  const int wv = t / kWave;
  if ((t & (kWave - 1)) == 0 && wv < a.nw) {
    a.bits[hrow * a.nw + wv] = word;
    if (a.top_bits) a.top_bits[hrow * a.nw + wv] = word;
  }
  if (a.scores && t < w) a.scores[hrow * a.w_cap + t] = f;
}

struct MapArgs {
  const uint64_t *bits;
  int H, nl, ns, nw;
  int32_t *head_map;  // [B][nl]
};

// a/b > c/d for b, d > 0 (a may be -1 as "no candidate")
__device__ __forceinline__ bool ratio_gt(int a, int b, int c, int d) { return a * d > c * b; }

__global__ __launch_bounds__(kMatchThreads) void match_map(MapArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int i = blockIdx.x * (kMatchThreads / kWave) + threadIdx.x / kWave;
  const int b = blockIdx.y;
  if (i >= a.nl) return;  // whole waves; no barrier follows
  const uint64_t *Ti = a.bits + ((int64_t)b * a.H + i) * a.nw;
  uint64_t ti[4];
  int ci = 0;
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    ti[x] = x < a.nw ? Ti[x] : 0ull;
    ci += __popcll(ti[x]);
  }
  int bn = -1, bd = 1, bj = 0x7fffffff;
  for (int j = lane; j < a.ns; j += kWave) {
    const uint64_t *Tj = a.bits + ((int64_t)b * a.H + a.nl + j) * a.nw;
    int in = 0, cj = 0;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const uint64_t tj = x < a.nw ? Tj[x] : 0ull;
      in += __popcll(ti[x] & tj);
      cj += __popcll(tj);
    }
    const int un = ci + cj - in;
    if (ratio_gt(in, un, bn, bd)) {  // j rises: a tie keeps the lower one
      bn = in;
      bd = un;
      bj = j;
    }
  }
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) {
    const int n2 = __shfl_xor(bn, o, kWave), d2 = __shfl_xor(bd, o, kWave);
    const int j2 = __shfl_xor(bj, o, kWave);
    if (ratio_gt(n2, d2, bn, bd) || (n2 * bd == bn * d2 && j2 < bj)) {
      bn = n2;
      bd = d2;
      bj = j2;
    }
  }
  if (lane == 0) a.head_map[(int64_t)b * a.nl + i] = bj;
}

template <typename T, int D>
hipError_t launch_logits_t(const LogitArgs &la, int tiles, int heads, int batch, hipStream_t st) {
  hipLaunchKernelGGL((match_logits<T, D>), dim3(tiles + la.nt, heads, batch), dim3(kWave), 0, st, la);
  return hipGetLastError();
}

hipError_t launch_logits(const smallkv_window_t &m, int batch, int w_cap, const int32_t *win_len,
                         float *S, float *pmax, int H, int head0, hipStream_t st) {
  LogitArgs la{};
  la.q = m.q;
  la.k = m.k;
  la.layers = m.n_layers;
  la.hq = m.n_q_heads;
  la.hkv = m.n_kv_heads;
  la.w_cap = w_cap;
  la.scale = m.scale;
  la.win_len = win_len;
  const int nt = (w_cap + kTile - 1) / kTile;
  la.nt = nt;
  la.ld = (w_cap + 3) / 4 * 4;
  la.S = S;
  la.pmax = pmax;
  la.H = H;
  la.head0 = head0;
  const int tiles = nt * (nt + 1) / 2;
  const int heads = m.n_layers * m.n_q_heads;
  const bool bf = m.dtype == SMALLKV_BF16;
  if (m.head_dim == 64)
    return bf ? launch_logits_t<bf16_t, 64>(la, tiles, heads, batch, st)
              : launch_logits_t<float, 64>(la, tiles, heads, batch, st);
  return bf ? launch_logits_t<bf16_t, 128>(la, tiles, heads, batch, st)
            : launch_logits_t<float, 128>(la, tiles, heads, batch, st);
}

}  // namespace

MatchLayout match_layout(const smallkv_match_t &m) {
  MatchLayout l{};
  const int64_t H = (int64_t)m.large.n_layers * m.large.n_q_heads +
                    (int64_t)m.small.n_layers * m.small.n_q_heads;
  l.nw = (m.w_cap + kWave - 1) / kWave;
  l.nt = (m.w_cap + kTile - 1) / kTile;
  l.ld = (m.w_cap + 3) / 4 * 4;
  auto round256 = [](size_t x) { return (x + 255) / 256 * 256; };
  const size_t mat = (size_t)m.batch * H * m.w_cap * l.ld * sizeof(float);
  l.pmax_offset = round256(mat);
  l.mz_offset = l.pmax_offset + round256((size_t)m.batch * H * m.w_cap * l.nt * sizeof(float));
  l.bits_offset = l.mz_offset + round256((size_t)m.batch * H * m.w_cap * sizeof(float2));
  l.total = l.bits_offset + (size_t)m.batch * H * l.nw * sizeof(uint64_t);
  return l;
}

hipError_t launch_match(const smallkv_match_t &m, void *ws, hipStream_t st) {
  const MatchLayout lay = match_layout(m);
  char *base = static_cast<char *>(ws);
  float *S = reinterpret_cast<float *>(base);
  float *pmax = reinterpret_cast<float *>(base + lay.pmax_offset);
  float2 *mz = reinterpret_cast<float2 *>(base + lay.mz_offset);
  uint64_t *bits = reinterpret_cast<uint64_t *>(base + lay.bits_offset);
  const int nl = m.large.n_layers * m.large.n_q_heads;
  const int ns = m.small.n_layers * m.small.n_q_heads;
  const int H = nl + ns;
  hipError_t e = launch_logits(m.large, m.batch, m.w_cap, m.win_len, S, pmax, H, 0, st);
  if (e != hipSuccess) return e;
  e = launch_logits(m.small, m.batch, m.w_cap, m.win_len, S, pmax, H, nl, st);
  if (e != hipSuccess) return e;
  ScoreArgs sa{S, pmax, mz, m.w_cap, lay.ld, lay.nt, H, lay.nw, m.win_len, m.top_k, bits,
               m.scores, m.top_bits};
  hipLaunchKernelGGL(match_rowsum, dim3(((m.w_cap + 1) / 2 + kMatchThreads - 1) / kMatchThreads, H, m.batch),
                     dim3(kMatchThreads), 0, st, sa);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(match_scores, dim3(H, m.batch), dim3(kMatchThreads), 0, st, sa);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  MapArgs ma{bits, H, nl, ns, lay.nw, m.head_map};
  const int waves = kMatchThreads / kWave;
  hipLaunchKernelGGL(match_map, dim3((nl + waves - 1) / waves, m.batch), dim3(kMatchThreads), 0, st,
                     ma);
  return hipGetLastError();
}

}  // namespace smallkv
