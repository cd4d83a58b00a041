// Stage 3: the large model's hybrid decode attention (Eq. 6; Algorithm 1,
// "Calculate attention output O_c of critical tokens ... O_m of marginal
// tokens ... Attention Output by O_c + O_m").
//
// One workgroup per (sequence, layer, large query head); large head i reads
// the partition of small head f(i) through head_map.
//   Phase 1: the K rows of the critical tokens are gathered, LPR lanes per
//            row and 16 bytes per lane; each wave takes a block of entries,
//            loads their indices with one coalesced load, hands them out
//            with lane shuffles and keeps a whole block of row loads in
//            flight; the row's lanes reduce their partial dots with DPP and
//            the logits go to LDS.
//   Phase 2: softmax over the critical logits (workgroup max and sum), then
//            one gather of V rows for critical and marginal tokens, weights
//            alpha_C*e_t/Z_C and alpha_M*p'_t, into one accumulator.
// Workgroups are numbered so that the query heads sharing a kv head land on
// the same XCD back to back: their gathered rows overlap and hit in that
// XCD's L2.
#include "common.h"
#include "launch.h"

namespace smallkv {
namespace {

constexpr int kHT = 256;
constexpr int kNW = kHT / kWave;
constexpr int kXcd = 8;

struct HybArgs {
  int n_cap, layers, hq, hkv, g, nsh, kc_cap, km_cap, mode, units;
  int layer0, nl;  // the large layers this launch runs: [layer0, layer0 + nl) of `layers`
  int64_t n_rows;
  float scale;
  const int32_t *seq_len, *k_crit, *k_marg, *k_recent, *head_map;
  const void *q, *k, *v;
  const int32_t *k_slot, *v_slot;
  const int32_t *crit, *marg;
  const float *marg_prob, *mass;
  void *out;
  int group_sel;  // lists per (b, layer, kv head), marg_prob/mass per query head
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

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, false));
}

// Sum over the LPR consecutive lanes that hold one row; every lane of the
// group ends with the sum.  DPP inside 16-lane rows, one shuffle beyond.
template <int LPR>
__device__ __forceinline__ float row_reduce(float x) {
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]: lane ^ 1
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]: lane ^ 2
  x += dpp<0x141>(x);  // row_half_mirror: lane i <-> 7-i inside 8
  if constexpr (LPR >= 16) x += dpp<0x140>(x);  // row_mirror: lane i <-> 15-i inside 16
  if constexpr (LPR >= 32) x += __shfl_xor(x, 16, kWave);
  return x;
}

template <typename T, int D>
__global__ __launch_bounds__(kHT) void hybrid_kernel(HybArgs a) {
  constexpr int EPL = elem<T>::per16;            // elements per lane (one 16-byte load)
  constexpr int LPR = D / EPL;                   // lanes per row
  constexpr int RPW = kWave / LPR;               // rows per wave instruction
  constexpr int NSUB = 16;                       // row loads in flight per lane
  constexpr int BE = RPW * NSUB < kWave ? RPW * NSUB : kWave;  // entries per wave block
  constexpr int NS = BE / RPW;                   // sub-steps per block
  static_assert(LPR >= 8 && LPR <= 32, "lane group size");
  extern __shared__ float s_crit[];  // [kc_cap] logits, then exp weights
  __shared__ float red[kNW];
  __shared__ float accbuf[kNW][D];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane % LPR, rg = lane / LPR;
  // XCD-aware numbering: x = ((u / 8) * g + hh) * 8 + u % 8
  const int x = blockIdx.x;
  const int rest = x / kXcd;
  const int u = (rest / a.g) * kXcd + x % kXcd, hh = rest % a.g;
  if (u >= a.units) return;
  const int kvh = u % a.hkv, bl = u / a.hkv, layer = a.layer0 + bl % a.nl, b = bl / a.nl;
  // the (sequence, layer, kv head) in the whole stack's layout
  const int64_t ua = ((int64_t)b * a.layers + layer) * a.hkv + kvh;
  const int h = kvh * a.g + hh;
  const int j = clampi(a.head_map[layer * a.hq + h], 0, a.nsh - 1);
  const int64_t qrow = ((int64_t)b * a.layers + layer) * a.hq + h;
  // lists of the small head f(i), or of the group; weights of f(i), or of the head
  const int64_t lrow = a.group_sel ? ua : (int64_t)b * a.nsh + j;
  const int64_t row = a.group_sel ? qrow : lrow;
  const Sizes sz = set_sizes(a.seq_len, a.k_crit, a.k_marg, a.k_recent, b, a.n_cap, a.kc_cap, a.km_cap);
  const int nc = sz.nc, nm = sz.nm, ntot = sz.nc + sz.nm;
  const int32_t *crit = a.crit + lrow * a.kc_cap;
  const int32_t *marg = a.marg + lrow * a.km_cap;
  const float *mp = a.marg_prob + row * a.km_cap;

  float qv[EPL];
  elem<T>::unpack(*reinterpret_cast<const uint4 *>(reinterpret_cast<const unsigned char *>(a.q) +
                                                   (qrow * D + sub * EPL) * (int64_t)sizeof(T)),
                  qv);
  const int64_t rowb = D * (int64_t)sizeof(T);
  const unsigned char *kb = reinterpret_cast<const unsigned char *>(a.k) + ua * a.n_rows * rowb + sub * 16;
  const unsigned char *vb = reinterpret_cast<const unsigned char *>(a.v) + ua * a.n_rows * rowb + sub * 16;
  const int32_t *ks = a.k_slot ? a.k_slot + ua * a.n_cap : nullptr;
  const int32_t *vs = a.v_slot ? a.v_slot + ua * a.n_cap : nullptr;
  const int last_row = (int)(a.n_rows - 1);

  // ---- phase 1: critical logits -----------------------------------------
  float lmax = -INFINITY;
  for (int base = wave * BE; base < nc; base += kNW * BE) {
    const int my = base + lane;
    int r = 0;
    if (lane < BE && my < nc) {
      const int t = clampi(crit[my], 0, a.n_cap - 1);
      r = clampi(ks ? ks[t] : t, 0, last_row);
    }
    uint4 w[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int rk = __shfl(r, k * RPW + rg, kWave);
      w[k] = *reinterpret_cast<const uint4 *>(kb + rk * rowb);
    }
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      float kv[EPL];
      elem<T>::unpack(w[k], kv);
      float d = 0.0f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) d = __builtin_fmaf(qv[e], kv[e], d);
      d = row_reduce<LPR>(d);
      const int i = base + k * RPW + rg;
      if (i < nc) {
        const float s = d * a.scale;
        if (sub == 0) s_crit[i] = s;
        lmax = fmaxf(lmax, s);
      }
    }
  }
  lmax = wave_max(lmax);
  if (lane == 0) red[wave] = lmax;
  __syncthreads();
  float m = red[0];
#pragma unroll
  for (int w = 1; w < kNW; ++w) m = fmaxf(m, red[w]);
  __syncthreads();
  float zl = 0.0f;
  for (int i = tid; i < nc; i += kHT) {
    const float e = __expf(s_crit[i] - m);
    s_crit[i] = e;
    zl += e;
  }
  zl = wave_sum(zl);
  if (lane == 0) red[wave] = zl;
  __syncthreads();
  float z = 0.0f;
#pragma unroll
  for (int w = 0; w < kNW; ++w) z += red[w];
  float ac, am;
  alphas(a.mode, a.mass[2 * row], a.mass[2 * row + 1], ac, am);
  const float wc = ac / z;

  // ---- phase 2: one weighted gather of V rows -----------------------------
  float acc[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc[e] = 0.0f;
  for (int base = wave * BE; base < ntot; base += kNW * BE) {
    const int my = base + lane;
    int r = 0;
    float wt = 0.0f;
    if (lane < BE && my < ntot) {
      int t;
      if (my < nc) {
        t = crit[my];
        wt = s_crit[my] * wc;
      } else {
        t = marg[my - nc];
        wt = mp[my - nc] * am;
      }
      t = clampi(t, 0, a.n_cap - 1);
      r = clampi(vs ? vs[t] : t, 0, last_row);
    }
    uint4 w[NS];
    float wk[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int src = k * RPW + rg;
      const int rk = __shfl(r, src, kWave);
      wk[k] = __shfl(wt, src, kWave);
      w[k] = *reinterpret_cast<const uint4 *>(vb + rk * rowb);
    }
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      float vv[EPL];
      elem<T>::unpack(w[k], vv);
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = __builtin_fmaf(wk[k], vv[e], acc[e]);
    }
  }
#pragma unroll
  for (int o = LPR; o < kWave; o <<= 1)
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] += __shfl_xor(acc[e], o, kWave);
  if (lane < LPR) {
#pragma unroll
    for (int e = 0; e < EPL; ++e) accbuf[wave][sub * EPL + e] = acc[e];
  }
  __syncthreads();
  if (tid < D) {
    float o = 0.0f;
#pragma unroll
    for (int w = 0; w < kNW; ++w) o += accbuf[w][tid];
    elem<T>::store1(a.out, qrow * D + tid, o);
  }
}

}  // namespace

hipError_t launch_hybrid(const smallkv_batch_t &b, const smallkv_model_t &m,
                         const int32_t *head_map, int n_small_heads, const int32_t *crit,
                         const int32_t *marg, const float *marg_prob, const float *mass,
                         int mode, bool group_sel, int layer0, int nl, hipStream_t st) {
  HybArgs a;
  a.layer0 = layer0;
  a.nl = nl;
  a.group_sel = group_sel ? 1 : 0;
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
  a.out = m.out;
  const int groups = (a.units + kXcd - 1) / kXcd;
  const dim3 grid(groups * kXcd * a.g);
  const size_t shm = (size_t)b.kc_cap * sizeof(float);
  if (m.dtype == SMALLKV_F32) {
    if (m.head_dim == 64)
      hipLaunchKernelGGL((hybrid_kernel<float, 64>), grid, dim3(kHT), shm, st, a);
    else
      hipLaunchKernelGGL((hybrid_kernel<float, 128>), grid, dim3(kHT), shm, st, a);
  } else {
    if (m.head_dim == 64)
      hipLaunchKernelGGL((hybrid_kernel<bf16_t, 64>), grid, dim3(kHT), shm, st, a);
    else
      hipLaunchKernelGGL((hybrid_kernel<bf16_t, 128>), grid, dim3(kHT), shm, st, a);
  }
  return hipGetLastError();
}

}  // namespace smallkv
