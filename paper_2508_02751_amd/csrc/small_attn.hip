// Stage 1: the small model's full decode attention over its uncompressed
// cache (Algorithm 1, decode branch; the full small cache C^s_all of the
// "Saliency Shift Compensation" paragraph).
//
// One workgroup per (sequence, layer, kv head, token chunk); the chunk is
// walked in LDS tiles with an online softmax, and the workgroup emits one
// partial record per query head of the GQA group: (chunk max, sum, P.V).
//
// bf16 kernel (small_attn_mfma), per tile:
//   * K rows are staged in LDS with coalesced 16-byte loads; the V rows of
//     the tile are loaded into registers at the same time, 8 consecutive
//     tokens x 8 dims per thread, so their latency hides behind QK;
//   * each thread owns one token and evaluates the logit of every query head
//     of the group as a sequential fp32 FMA chain over the head dimension
//     (the bit-exact ranking key), and writes it out;
//   * P = exp(s - running max) is split into bf16 hi + lo parts and V is
//     transposed in registers (v_perm) into a token-contiguous LDS tile, so
//     P.V runs on MFMA (v_mfma_f32_16x16x32_bf16): M = query heads (padded
//     to 16), N = 16 dims per wave, K = 32 tokens per instruction, twice
//     (hi, lo), which keeps ~16 bits of P.
// fp32 kernel (small_attn_valu): the same tiling with P.V on fp32 FMA.
// small_attn_merge: log-sum-exp combine of a head's chunk records.
#include "common.h"
#include "launch.h"
#include "merge.h"

namespace smallkv {
namespace {

constexpr int kThreads = 256;

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

template <typename T, int D>
struct SmallCfg {
  static constexpr int ROWB = D * (int)sizeof(T);                       // bytes per K/V row
  static constexpr int TILE = 32768 / ROWB < 256 ? 32768 / ROWB : 256;  // tokens per tile
  static constexpr int ROWS = ROWB + 16;                                // padded K row stride
  static constexpr int V16 = ROWB / 16;                                 // 16-byte vectors per row
};

struct SmallArgs {
  int n_cap, layers, hq, hkv, g, chunk, n_split;
  float scale;
  const int32_t *seq_len;
  const void *q, *k, *v;
  void *out;
  float *logits, *row_max, *row_sum, *part;
};

struct UnitPos {
  int unit, split, b, layer, kvh, n, t0, t1;
  int64_t head0;  // q row (and logits row) of the group's first query head
};

__device__ __forceinline__ bool unit_pos(const SmallArgs &a, UnitPos &u) {
  u.unit = blockIdx.x / a.n_split;
  u.split = blockIdx.x % a.n_split;
  u.kvh = u.unit % a.hkv;
  const int bl = u.unit / a.hkv;
  u.layer = bl % a.layers;
  u.b = bl / a.layers;
  u.n = clampi(a.seq_len[u.b], 1, a.n_cap);
  u.t0 = u.split * a.chunk;
  u.t1 = min(u.t0 + a.chunk, u.n);
  u.head0 = ((int64_t)u.b * a.layers + u.layer) * a.hq + (int64_t)u.kvh * a.g;
  return u.t0 < u.n;
}

// Sequential fp32 FMA chain over the head dimension, then one multiply by
// the scale; -0 becomes +0.  This is the bit-exact ranking key.
template <int D>
__device__ __forceinline__ float chain_logit(const float *q, const float *k, float scale) {
  float acc = 0.0f;
#pragma unroll
  for (int c = 0; c < D; ++c) acc = __builtin_fmaf(q[c], k[c], acc);
  const float s = acc * scale;
  return s == 0.0f ? 0.0f : s;
}

// The same chain with q read as bf16 pairs through the constant address
// space: wave-uniform scalar loads, so every FMA takes q from an SGPR and the
// query costs no LDS traffic.  Bit-identical to chain_logit.
typedef const __attribute__((address_space(4))) uint32_t *const_u32_ptr;
template <int D>
__device__ __forceinline__ float chain_logit_sq(const_u32_ptr qw, const float *k, float scale) {
  float acc = 0.0f;
#pragma unroll
  for (int c = 0; c < D; c += 2) {
    const uint32_t w = qw[c / 2];
    acc = __builtin_fmaf(bf16_lo(w), k[c], acc);
    acc = __builtin_fmaf(bf16_hi(w), k[c + 1], acc);
  }
  const float s = acc * scale;
  return s == 0.0f ? 0.0f : s;
}

// Max (or sum) over the wave of GP per-head values at once.  Halving
// exchanges hand every lane group one head (head = lane >> (6 - log2 GP)):
// across lane halves with v_permlane32_swap, across row pairs with
// v_permlane16_swap, inside a row with DPP; then each group reduces alone
// with DPP.  No LDS traffic and no per-lane selects above the row level.
template <bool kMax>
__device__ __forceinline__ float red_op(float x, float y) {
  return kMax ? fmaxf(x, y) : x + y;
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}

template <int GP, bool kMax>
__device__ __forceinline__ float wave_reduce_heads(float (&v)[GP]) {
  const int lane = threadIdx.x & 63;
  int n = GP;
  if (n >= 2) {  // lanes 0-31 keep heads [0, n/2), lanes 32-63 the rest
#pragma unroll
    for (int i = 0; i < GP / 2; ++i) {
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[i]), __float_as_uint(v[i + GP / 2]),
                                                      false, false);
      v[i] = red_op<kMax>(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    n >>= 1;
  }
  if (n >= 2) {  // even rows keep the lower half of the heads, odd rows the upper
#pragma unroll
    for (int i = 0; i < GP / 4; ++i) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[i]), __float_as_uint(v[i + GP / 4]),
                                                      false, false);
      v[i] = red_op<kMax>(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    n >>= 1;
  }
  if (n >= 2) {  // row halves: lane i pairs with i ^ 8 (row_ror:8)
    const bool upper = (lane & 8) != 0;
#pragma unroll
    for (int i = 0; i < GP / 8; ++i) {
      const float keep = upper ? v[i + GP / 8] : v[i];
      const float send = upper ? v[i] : v[i + GP / 8];
      v[i] = red_op<kMax>(keep, dpp<0x128>(send));
    }
    n >>= 1;
  }
  if (n >= 2) {  // 8-lane halves: lane i pairs with 7 - i (row_half_mirror)
    const bool upper = (lane & 4) != 0;
#pragma unroll
    for (int i = 0; i < GP / 16; ++i) {
      const float keep = upper ? v[i + GP / 16] : v[i];
      const float send = upper ? v[i] : v[i + GP / 16];
      v[i] = red_op<kMax>(keep, dpp<0x141>(send));
    }
    n >>= 1;
  }
  // the group of 64 / GP lanes now shares one head: reduce it
  float x = v[0];
  x = red_op<kMax>(x, dpp<0xB1>(x));                    // lane ^ 1
  x = red_op<kMax>(x, dpp<0x4E>(x));                    // lane ^ 2
  if (GP <= 8) x = red_op<kMax>(x, dpp<0x141>(x));      // 8-lane mirror
  if (GP <= 4) x = red_op<kMax>(x, dpp<0x140>(x));      // 16-lane mirror
  return x;  // the reduction of head (lane >> (6 - log2 GP))
}

template <int GP>
constexpr int head_shift() {
  return GP == 4 ? 4 : (GP == 8 ? 3 : 2);
}

// A 16-byte piece of the small cache, which a step reads exactly once:
// loaded non-temporally, so that streaming 17 GB of K and V through the
// caches does not evict the logits this kernel writes for the partition
// (LLaMA step: stage 1 3.73 -> 3.49 ms with the same pages).
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;
__device__ __forceinline__ uint4 stream16(const unsigned char *p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

template <typename T, int D>
__device__ __forceinline__ void stage_k(unsigned char *tile, const unsigned char *src, int nr) {
  using C = SmallCfg<T, D>;
#pragma unroll
  for (int r = 0; r < C::TILE * C::V16 / kThreads; ++r) {
    const int x = threadIdx.x + r * kThreads;
    const int row = x / C::V16, w = x % C::V16;
    if (row < nr)
      *reinterpret_cast<uint4 *>(tile + row * C::ROWS + w * 16) = stream16(src + (int64_t)row * C::ROWB + w * 16);
  }
}

// ------------------------------------------------------------ bf16 / MFMA --

// G: the query-group size when known at compile time (0: runtime a.g, the
// padded heads then run on zero queries instead of behind branches).
// kPre: the chunk has several tiles; the next tile's K rows travel into
// registers while this tile computes (costs registers, so single-tile chunks
// go without).
template <int D, int GP, int G, bool kPre>
__global__ __launch_bounds__(kThreads) void small_attn_mfma(SmallArgs a) {
  using C = SmallCfg<bf16_t, D>;
  constexpr int TILE = C::TILE;
  constexpr int DC = D / 8;                   // 8-dim chunks per row
  constexpr int TB = kThreads / DC;           // 8-token blocks per V load pass
  static_assert(TB * 8 == TILE, "one V pass covers the tile");
  constexpr int VTS = (TILE + 8) * 2;         // V^T and P row stride (bytes)
  constexpr int NB = D / 16;                  // 16-dim MFMA blocks
  constexpr int NBW = NB / 4;                 // blocks per wave
  // V^T rows of 8-dim group c start 16*c bytes further, so that the lanes
  // writing dims 8c + d for different c do not share a bank
  constexpr int VTB = D * VTS + (D / 8) * 16;
  constexpr int TB_BYTES = C::TILE * C::ROWS > VTB ? C::TILE * C::ROWS : VTB;

  __shared__ __align__(16) unsigned char tile[TB_BYTES];  // K tile, then V^T
  __shared__ __align__(16) unsigned char pt[2][GP * VTS];  // P hi, P lo (bf16)
  __shared__ float red[4 * GP];
  __shared__ float salpha[16];

  UnitPos u;
  if (!unit_pos(a, u)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = G > 0 ? G : a.g;
  constexpr int GC = G > 0 ? G : GP;  // heads the chains run on
  const int64_t row0 = (int64_t)u.unit * a.n_cap;
  const unsigned char *kb = reinterpret_cast<const unsigned char *>(a.k) + row0 * C::ROWB;
  const unsigned char *vb = reinterpret_cast<const unsigned char *>(a.v) + row0 * C::ROWB;
  float *lrow = a.logits + u.head0 * a.n_cap;
  const int tb8 = tid / DC, dc = tid % DC;  // V: token block and dim chunk of this thread

  float m_run[GP], z_thr[GP];
#pragma unroll
  for (int i = 0; i < GP; ++i) {
    m_run[i] = -INFINITY;
    z_thr[i] = 0.0f;
  }
  f32x4_t acc[NBW];
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb) acc[nb] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

  constexpr int KR = C::TILE * C::V16 / kThreads;  // 16-byte K pieces per thread
  uint4 kpre[kPre ? KR : 1];
  auto load_k = [&](int t, int n) {
#pragma unroll
    for (int r = 0; r < KR; ++r) {
      const int x = tid + r * kThreads;
      const int row = x / C::V16, w = x % C::V16;
      kpre[r] = row < n ? stream16(kb + (int64_t)(t + row) * C::ROWB + w * 16)
                        : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  auto store_k = [&]() {
#pragma unroll
    for (int r = 0; r < KR; ++r) {
      const int x = tid + r * kThreads;
      const int row = x / C::V16, w = x % C::V16;
      *reinterpret_cast<uint4 *>(tile + row * C::ROWS + w * 16) = kpre[r];
    }
  };
  if constexpr (kPre) {
    load_k(u.t0, min(TILE, u.t1 - u.t0));
    store_k();
  }

  for (int tb = u.t0; tb < u.t1; tb += TILE) {
    const int nr = min(TILE, u.t1 - tb);
    const int tn = tb + TILE;
    if constexpr (kPre) {
      __syncthreads();  // this tile's K is in LDS
      if (tn < u.t1) load_k(tn, min(TILE, u.t1 - tn));
    } else {
      stage_k<bf16_t, D>(tile, kb + (int64_t)tb * C::ROWB, nr);
      __syncthreads();
    }

    // ---- logits: one token per thread, sequential FMA chains ------------
    // The chain of each head runs over dims 0..D-1 in order; the K row is
    // unpacked half a row at a time to keep registers low.
    float s[GP];
#pragma unroll
    for (int i = 0; i < GP; ++i) s[i] = 0.0f;
    if (tid < nr) {
      const_u32_ptr qw = (const_u32_ptr)(reinterpret_cast<uintptr_t>(a.q)) + u.head0 * (D / 2);
      // q of one (half, head) step: QW words in SGPRs.  Scalar loads return
      // out of order, so any use of one waits for all in flight: each step
      // first touches its own q (one FMA, which waits), then requests the
      // next step's q, then runs the rest of its chain while those arrive.
      constexpr int QW = D / 4;
      constexpr int NSTEP = 2 * GC;
      auto q_at = [&](int st) { return qw + (st % GC) * (D / 2) + (st / GC) * QW; };
      uint32_t qc[QW], qn[QW];
#pragma unroll
      for (int w = 0; w < QW; ++w) qc[w] = q_at(0)[w];
      float kr[D / 2];
#pragma unroll
      for (int st = 0; st < NSTEP; ++st) {
        const int i = st % GC, half = st / GC;
        if (G == 0 && i >= g) {  // padded head slot of a runtime group size
          if (st + 1 < NSTEP)
#pragma unroll
            for (int w = 0; w < QW; ++w) qc[w] = q_at(st + 1)[w];
          continue;
        }
        if (i == 0) {  // this half of the K row, unpacked
#pragma unroll
          for (int w = 0; w < C::V16 / 2; ++w) {
            const uint4 v = *reinterpret_cast<const uint4 *>(tile + tid * C::ROWS + (half * C::V16 / 2 + w) * 16);
            elem<bf16_t>::unpack(v, kr + w * 8);
          }
        }
        s[i] = __builtin_fmaf(bf16_lo(qc[0]), kr[0], s[i]);
        __builtin_amdgcn_sched_barrier(0);
        if (st + 1 < NSTEP)
#pragma unroll
          for (int w = 0; w < QW; ++w) qn[w] = q_at(st + 1)[w];
        __builtin_amdgcn_sched_barrier(0);
        s[i] = __builtin_fmaf(bf16_hi(qc[0]), kr[1], s[i]);
#pragma unroll
        for (int c = 2; c < D / 2; c += 2) {
          s[i] = __builtin_fmaf(bf16_lo(qc[c / 2]), kr[c], s[i]);
          s[i] = __builtin_fmaf(bf16_hi(qc[c / 2]), kr[c + 1], s[i]);
        }
#pragma unroll
        for (int w = 0; w < QW; ++w) qc[w] = qn[w];
      }
#pragma unroll
      for (int i = 0; i < GP; ++i) {
        if (i < g) {
          float x = s[i] * a.scale;
          x = x == 0.0f ? 0.0f : x;
          lrow[(int64_t)i * a.n_cap + tb + tid] = x;
          s[i] = x;
        } else {
          s[i] = -INFINITY;
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < GP; ++i) s[i] = -INFINITY;
    }
    {
      float t[GP];
#pragma unroll
      for (int i = 0; i < GP; ++i) t[i] = s[i];
      const float mx = wave_reduce_heads<GP, true>(t);
      constexpr int sh = head_shift<GP>();
      if ((lane & ((1 << sh) - 1)) == 0) red[wave * GP + (lane >> sh)] = mx;
    }
    // V rows of 8 consecutive tokens x one 8-dim chunk, into registers
    uint4 vr[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int tok = tb8 * 8 + k;
      vr[k] = tok < nr ? stream16(vb + (int64_t)(tb + tok) * C::ROWB + dc * 16)
                       : make_uint4(0u, 0u, 0u, 0u);
    }
    __syncthreads();  // K tile no longer read; red visible

    // ---- online softmax, P hi/lo and V^T into LDS -----------------------
    float alpha[GP];
#pragma unroll
    for (int i = 0; i < GP; ++i) {
      const float mt = fmaxf(fmaxf(red[i], red[GP + i]), fmaxf(red[2 * GP + i], red[3 * GP + i]));
      const float mn = fmaxf(m_run[i], mt);
      alpha[i] = i < g ? __expf(m_run[i] - mn) : 1.0f;  // 0 on the first tile
      m_run[i] = mn;
      const float e = (i < g && tid < nr) ? __expf(s[i] - mn) : 0.0f;
      z_thr[i] = __builtin_fmaf(z_thr[i], alpha[i], e);
      const __bf16 hi = (__bf16)e;  // v_cvt_pk_bf16_f32, round to nearest even
      const __bf16 lo = (__bf16)(e - (float)hi);
      if (tid < TILE) {
        *reinterpret_cast<__bf16 *>(pt[0] + i * VTS + tid * 2) = hi;
        *reinterpret_cast<__bf16 *>(pt[1] + i * VTS + tid * 2) = lo;
      }
    }
    if (tid < 16) {
      float al = 1.0f;
#pragma unroll
      for (int i = 0; i < GP; ++i)
        if (i == tid) al = alpha[i];
      salpha[tid] = al;
    }
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      const uint32_t sel = (d & 1) ? 0x07060302u : 0x05040100u;
      uint32_t w[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const uint32_t x0 = (&vr[2 * p].x)[d >> 1], x1 = (&vr[2 * p + 1].x)[d >> 1];
        w[p] = __builtin_amdgcn_perm(x1, x0, sel);
      }
      *reinterpret_cast<uint4 *>(tile + (dc * 8 + d) * VTS + dc * 16 + tb8 * 16) = make_uint4(w[0], w[1], w[2], w[3]);
    }
    __syncthreads();

    // ---- P.V on MFMA --------------------------------------------------------
    const int mrow = lane & 15, kq = lane >> 4;
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[nb][r] *= salpha[kq * 4 + r];
#pragma unroll
    for (int ks = 0; ks < TILE / 32; ++ks) {
      const int tok = ks * 32 + kq * 8;
      uint4 ah = make_uint4(0u, 0u, 0u, 0u), al = ah;
      if (mrow < GP) {
        ah = *reinterpret_cast<const uint4 *>(pt[0] + mrow * VTS + tok * 2);
        al = *reinterpret_cast<const uint4 *>(pt[1] + mrow * VTS + tok * 2);
      }
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) {
        const int dim = (wave + 4 * nb) * 16 + mrow;
        const uint4 bv = *reinterpret_cast<const uint4 *>(tile + dim * VTS + (dim >> 3) * 16 + tok * 2);
        const bf16x8_t B = __builtin_bit_cast(bf16x8_t, bv);
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ah), B, acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, al), B, acc[nb], 0, 0, 0);
      }
    }
    __syncthreads();  // before the next tile overwrites the K/V^T and P tiles
    if constexpr (kPre)
      if (tn < u.t1) store_k();
  }

  // ---- chunk record: max, sum and P.V per query head ----------------------
  {
    const float zs = wave_reduce_heads<GP, false>(z_thr);
    constexpr int sh = head_shift<GP>();
    if ((lane & ((1 << sh) - 1)) == 0) red[wave * GP + (lane >> sh)] = zs;
  }
  __syncthreads();
  float *part = a.part + (int64_t)blockIdx.x * GP * (D + 2);
  const int kq = lane >> 4, ncol = lane & 15;
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int head = kq * 4 + r, dim = (wave + 4 * nb) * 16 + ncol;
      if (head < g) part[head * (D + 2) + 2 + dim] = acc[nb][r];
    }
  if (tid == 0) {
#pragma unroll
    for (int i = 0; i < GP; ++i)
      if (i < g) {
        part[i * (D + 2)] = m_run[i];
        part[i * (D + 2) + 1] = red[i] + red[GP + i] + red[2 * GP + i] + red[3 * GP + i];
      }
  }
}

// ---------------------------------------------------------------- fp32 --

template <int D, int GP>
__global__ __launch_bounds__(kThreads) void small_attn_valu(SmallArgs a) {
  using C = SmallCfg<float, D>;
  constexpr int TILE = C::TILE;
  constexpr int VD = 4;              // dims per thread in P.V
  constexpr int NDG = D / VD;        // dim groups
  constexpr int NTP = kThreads / NDG;  // token stripes
  __shared__ __align__(16) unsigned char tile[TILE * C::ROWS];
  __shared__ __align__(16) float sq[GP * D];
  __shared__ __align__(16) float sp[TILE * GP];
  __shared__ float red[4 * GP];

  UnitPos u;
  if (!unit_pos(a, u)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = a.g;
  for (int x = tid; x < GP * D; x += kThreads) {
    const int i = x / D, c = x % D;
    sq[x] = i < g ? elem<float>::load1(a.q, (u.head0 + i) * D + c) : 0.0f;
  }
  const int64_t row0 = (int64_t)u.unit * a.n_cap;
  const unsigned char *kb = reinterpret_cast<const unsigned char *>(a.k) + row0 * C::ROWB;
  const unsigned char *vb = reinterpret_cast<const unsigned char *>(a.v) + row0 * C::ROWB;
  float *lrow = a.logits + u.head0 * a.n_cap;
  const int dg = tid % NDG, tp = tid / NDG;

  float m_run[GP], z_thr[GP], acc[GP][VD];
#pragma unroll
  for (int i = 0; i < GP; ++i) {
    m_run[i] = -INFINITY;
    z_thr[i] = 0.0f;
#pragma unroll
    for (int c = 0; c < VD; ++c) acc[i][c] = 0.0f;
  }
  for (int tb = u.t0; tb < u.t1; tb += TILE) {
    const int nr = min(TILE, u.t1 - tb);
    stage_k<float, D>(tile, kb + (int64_t)tb * C::ROWB, nr);
    __syncthreads();
    float s[GP];
#pragma unroll
    for (int i = 0; i < GP; ++i) s[i] = -INFINITY;
    if (tid < nr) {
      float kr[D];
#pragma unroll
      for (int w = 0; w < C::V16; ++w) {
        const uint4 v = *reinterpret_cast<const uint4 *>(tile + tid * C::ROWS + w * 16);
        elem<float>::unpack(v, kr + w * 4);
      }
#pragma unroll
      for (int i = 0; i < GP; ++i)
        if (i < g) {
          s[i] = chain_logit<D>(sq + i * D, kr, a.scale);
          lrow[(int64_t)i * a.n_cap + tb + tid] = s[i];
        }
    }
#pragma unroll
    for (int i = 0; i < GP; ++i) {
      const float v = wave_max(s[i]);
      if (lane == 0) red[wave * GP + i] = v;
    }
    __syncthreads();
    float alpha[GP];
#pragma unroll
    for (int i = 0; i < GP; ++i) {
      const float mt = fmaxf(fmaxf(red[i], red[GP + i]), fmaxf(red[2 * GP + i], red[3 * GP + i]));
      const float mn = fmaxf(m_run[i], mt);
      alpha[i] = i < g ? __expf(m_run[i] - mn) : 1.0f;
      m_run[i] = mn;
      const float e = (i < g && tid < nr) ? __expf(s[i] - mn) : 0.0f;
      z_thr[i] = __builtin_fmaf(z_thr[i], alpha[i], e);
      if (tid < TILE) sp[tid * GP + i] = e;
#pragma unroll
      for (int c = 0; c < VD; ++c) acc[i][c] *= alpha[i];
    }
    // V tile replaces the K tile
    stage_k<float, D>(tile, vb + (int64_t)tb * C::ROWB, nr);
    __syncthreads();
    for (int t = tp; t < nr; t += NTP) {
      float vv[VD];
      elem<float>::unpack(*reinterpret_cast<const uint4 *>(tile + t * C::ROWS + dg * VD * 4), vv);
#pragma unroll
      for (int i = 0; i < GP; ++i)
        if (i < g) {
          const float p = sp[t * GP + i];
#pragma unroll
          for (int c = 0; c < VD; ++c) acc[i][c] = __builtin_fmaf(p, vv[c], acc[i][c]);
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < GP; ++i) {
    const float v = wave_sum(z_thr[i]);
    if (lane == 0) red[wave * GP + i] = v;
  }
#pragma unroll
  for (int o = NDG; o < kWave; o <<= 1)
#pragma unroll
    for (int i = 0; i < GP; ++i)
#pragma unroll
      for (int c = 0; c < VD; ++c) acc[i][c] += __shfl_xor(acc[i][c], o, kWave);
  float *buf = reinterpret_cast<float *>(tile);  // [4 waves][GP][D]
  static_assert(4 * GP * D * 4 <= TILE * C::ROWS, "reduction buffer fits the tile");
  if (lane < NDG) {
#pragma unroll
    for (int i = 0; i < GP; ++i)
#pragma unroll
      for (int c = 0; c < VD; ++c) buf[(wave * GP + i) * D + dg * VD + c] = acc[i][c];
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
        part[i * (D + 2)] = m_run[i];
        part[i * (D + 2) + 1] = red[i] + red[GP + i] + red[2 * GP + i] + red[3 * GP + i];
      }
  }
}

// ------------------------------------------------------------- merge --

// Same workgroup shape as the merge fused into the partition kernel, so the
// two entry points combine the records in the same order (bit-identical).
constexpr int kMergeThreads = 512;

template <typename T, int D, int GP>
__global__ __launch_bounds__(kMergeThreads) void small_attn_merge(SmallArgs a) {
  __shared__ float mred[3 * kMergeThreads + 2];
  const int row = blockIdx.x;  // = b * (layers*hq) + layer*hq + h
  const int h = row % a.hq, bl = row / a.hq, layer = bl % a.layers, b = bl / a.layers;
  const int unit = (b * a.layers + layer) * a.hkv + h / a.g, i = h % a.g;
  const int n = clampi(a.seq_len[b], 1, a.n_cap);
  MergeIn in;
  in.stride = (int64_t)GP * (D + 2);
  in.part = a.part + (int64_t)unit * a.n_split * in.stride + i * (D + 2);
  in.nv = (n + a.chunk - 1) / a.chunk;
  float M, Z;
  void *out = a.out;
  merge_head<kMergeThreads>(in, D, mred, M, Z,
                          [&](int c, float v) { elem<T>::store1(out, (int64_t)row * D + c, v); });
  if (threadIdx.x == 0) {
    a.row_max[row] = M;
    a.row_sum[row] = Z;
  }
}

template <int D, int GP, int G>
void launch_mfma(const SmallArgs &a, int units, hipStream_t st) {
  if (a.chunk > SmallCfg<bf16_t, D>::TILE)
    hipLaunchKernelGGL((small_attn_mfma<D, GP, G, true>), dim3(units * a.n_split), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((small_attn_mfma<D, GP, G, false>), dim3(units * a.n_split), dim3(kThreads), 0, st, a);
}

template <int D, int GP>
hipError_t launch_split_t(const SmallArgs &a, int units, bool f32, hipStream_t st) {
  if (f32) {
    hipLaunchKernelGGL((small_attn_valu<D, GP>), dim3(units * a.n_split), dim3(kThreads), 0, st, a);
  } else if constexpr (GP == 4) {
    if (a.g == 4) launch_mfma<D, 4, 4>(a, units, st);
    else launch_mfma<D, 4, 0>(a, units, st);
  } else if constexpr (GP == 8) {
    if (a.g == 7) launch_mfma<D, 8, 7>(a, units, st);
    else if (a.g == 8) launch_mfma<D, 8, 8>(a, units, st);
    else launch_mfma<D, 8, 0>(a, units, st);
  } else {
    if (a.g == 16) launch_mfma<D, 16, 16>(a, units, st);
    else launch_mfma<D, 16, 0>(a, units, st);
  }
  return hipGetLastError();
}

template <int D>
hipError_t launch_split_gp(const SmallArgs &a, int units, int gp, bool f32, hipStream_t st) {
  if (gp == 4) return launch_split_t<D, 4>(a, units, f32, st);
  if (gp == 8) return launch_split_t<D, 8>(a, units, f32, st);
  return launch_split_t<D, 16>(a, units, f32, st);
}

template <typename T, int D>
hipError_t launch_merge_gp(const SmallArgs &a, int rows, int gp, hipStream_t st) {
  if (gp == 4)
    hipLaunchKernelGGL((small_attn_merge<T, D, 4>), dim3(rows), dim3(kMergeThreads), 0, st, a);
  else if (gp == 8)
    hipLaunchKernelGGL((small_attn_merge<T, D, 8>), dim3(rows), dim3(kMergeThreads), 0, st, a);
  else
    hipLaunchKernelGGL((small_attn_merge<T, D, 16>), dim3(rows), dim3(kMergeThreads), 0, st, a);
  return hipGetLastError();
}

SmallArgs make_args(const smallkv_batch_t &b, const smallkv_model_t &m, float *logits,
                    float *row_max, float *row_sum, float *ws, const SmallPlan &p) {
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
  return a;
}

}  // namespace

SmallPlan plan_small(const smallkv_batch_t &b, const smallkv_model_t &m) {
  SmallPlan p{};
  const int esz = m.dtype == SMALLKV_F32 ? 4 : 2;
  const int rowb = m.head_dim * esz;
  p.tile = 32768 / rowb < 256 ? 32768 / rowb : 256;
  const int64_t units = (int64_t)b.batch * m.n_layers * m.n_kv_heads;
  const int max_split = (b.n_cap + p.tile - 1) / p.tile;
  // about two rounds of resident workgroups (three per CU): fewer, longer
  // chunks pipeline their tiles, more of them only add merge records; at
  // least four tiles per chunk when that still gives every CU a workgroup,
  // so that the next tile's K loads overlap the current tile's arithmetic
  // (a one-tile chunk loads, then computes); and rows of more than 32 tiles
  // in chunks of at most 16, so that long rows give enough workgroups that
  // the last round of them is a small part of the launch (rows of up to 17
  // tiles, as in a batch of many short sequences, are fastest unsplit)
  const int want = (int)((1536 + units - 1) / units);
  int ns = want < 1 ? 1 : (want > max_split ? max_split : want);
  const int four = max_split / 4 < 1 ? 1 : max_split / 4;
  if (units * four >= 256 && ns > four) ns = four;
  const int least = max_split > 32 ? (max_split + 15) / 16 : 1;
  if (ns < least) ns = least;
  if (ns > kMaxChunks) ns = kMaxChunks;
  const int per = (b.n_cap + ns - 1) / ns;
  p.chunk = (per + p.tile - 1) / p.tile * p.tile;
  p.n_split = (b.n_cap + p.chunk - 1) / p.chunk;
  const int g = m.n_q_heads / m.n_kv_heads;
  p.gp = g <= 4 ? 4 : (g <= 8 ? 8 : 16);
  p.ws_bytes = (size_t)units * p.n_split * p.gp * (m.head_dim + 2) * sizeof(float);
  return p;
}

hipError_t launch_small_split(const smallkv_batch_t &b, const smallkv_model_t &m, float *logits,
                              float *ws, const SmallPlan &p, hipStream_t st) {
  const SmallArgs a = make_args(b, m, logits, nullptr, nullptr, ws, p);
  const int units = b.batch * m.n_layers * m.n_kv_heads;
  const bool f32 = m.dtype == SMALLKV_F32;
  return m.head_dim == 64 ? launch_split_gp<64>(a, units, p.gp, f32, st)
                          : launch_split_gp<128>(a, units, p.gp, f32, st);
}

hipError_t launch_small_attn(const smallkv_batch_t &b, const smallkv_model_t &m, float *logits,
                             float *row_max, float *row_sum, float *ws, const SmallPlan &p,
                             hipStream_t st) {
  hipError_t e = launch_small_split(b, m, logits, ws, p, st);
  if (e != hipSuccess) return e;
  const SmallArgs a = make_args(b, m, logits, row_max, row_sum, ws, p);
  const int rows = b.batch * m.n_layers * m.n_q_heads;
  if (m.dtype == SMALLKV_F32)
    return m.head_dim == 64 ? launch_merge_gp<float, 64>(a, rows, p.gp, st)
                            : launch_merge_gp<float, 128>(a, rows, p.gp, st);
  return m.head_dim == 64 ? launch_merge_gp<bf16_t, 64>(a, rows, p.gp, st)
                          : launch_merge_gp<bf16_t, 128>(a, rows, p.gp, st);
}

}  // namespace smallkv
