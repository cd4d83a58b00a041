// The C ABI of include/smallkv.h: host-side validation, workspace planning
// and launches.  Nothing here touches device memory or synchronises.
#include <hip/hip_runtime.h>

#include <mutex>

#include "launch.h"
#include "smallkv.h"

using namespace smallkv;

namespace {

bool model_ok(const smallkv_model_t *m) {
  if (!m || !m->q || !m->k || !m->v || !m->out) return false;
  if (m->n_layers < 1 || m->n_q_heads < 1 || m->n_kv_heads < 1) return false;
  if (m->n_q_heads % m->n_kv_heads) return false;
  if (m->dtype != SMALLKV_F32 && m->dtype != SMALLKV_BF16) return false;
  if (m->n_rows < 1) return false;
  if (!(m->scale == m->scale)) return false;  // NaN scale
  return true;
}

bool batch_ok(const smallkv_batch_t *b) {
  return b && b->batch >= 1 && b->n_cap >= 1 && b->seq_len && b->k_crit && b->k_marg &&
         b->kc_cap >= 1 && b->km_cap >= 0;
}

bool dim_supported(const smallkv_model_t *m) { return m->head_dim == 64 || m->head_dim == 128; }

int check_small(const smallkv_batch_t *b, const smallkv_model_t *s) {
  if (!batch_ok(b) || !model_ok(s)) return SMALLKV_EINVAL;
  if (s->k_slot || s->v_slot) return SMALLKV_EINVAL;
  if (!s->held != !s->row_pos) return SMALLKV_EINVAL;  // both or neither
  if (s->held ? (s->n_rows < 1 || s->n_rows > b->n_cap) : s->n_rows != b->n_cap)
    return SMALLKV_EINVAL;
  if (!dim_supported(s)) return SMALLKV_EUNSUPPORTED;
  if (s->n_q_heads / s->n_kv_heads > 16) return SMALLKV_EUNSUPPORTED;
  if ((int64_t)b->batch * s->n_layers * s->n_q_heads > INT32_MAX / 2) return SMALLKV_EUNSUPPORTED;
  return SMALLKV_OK;
}

int check_large(const smallkv_batch_t *b, const smallkv_model_t *l, const int32_t *head_map,
                int n_small_heads) {
  if (!batch_ok(b) || !model_ok(l) || !head_map || n_small_heads < 1) return SMALLKV_EINVAL;
  if (!l->k_slot != !l->v_slot) return SMALLKV_EINVAL;  // both maps or neither
  if (l->held || l->row_pos) return SMALLKV_EINVAL;      // small model only
  if (!l->k_slot && l->n_rows != b->n_cap) return SMALLKV_EINVAL;
  if (l->n_rows > INT32_MAX) return SMALLKV_EUNSUPPORTED;
  if (!dim_supported(l)) return SMALLKV_EUNSUPPORTED;
  if (!plan_group(*b, *l, n_small_heads).use && b->kc_cap > kHybridMaxCrit) return SMALLKV_EUNSUPPORTED;
  if ((int64_t)b->batch * l->n_layers * l->n_q_heads > INT32_MAX / 2) return SMALLKV_EUNSUPPORTED;
  return SMALLKV_OK;
}

int check_mode(int mode) {
  return (mode >= SMALLKV_NORM_REMAINING && mode <= SMALLKV_NORM_MARG_FILL) ? SMALLKV_OK
                                                                            : SMALLKV_EINVAL;
}

int status_of(hipError_t e) { return e == hipSuccess ? SMALLKV_OK : SMALLKV_EDEVICE; }

size_t max_sz(size_t x, size_t y) { return x > y ? x : y; }

// The batch as stages 1-2 see it: with the small model's own eviction they
// run over its held rows (lengths held[b], n_rows rows per kv head).
smallkv_batch_t small_view(const smallkv_batch_t &b, const smallkv_model_t &s) {
  smallkv_batch_t v = b;
  if (s.held) {
    v.seq_len = s.held;
    v.n_cap = (int32_t)s.n_rows;
  }
  return v;
}

// Workspace of a whole step: stage 1's chunk records, then (reused) stage
// 3's split records, and after both the partition's list offsets, which
// stage 2 writes while it reads stage 1's records and stage 3 reads while it
// writes its own (grouped stage 3 only).
// With group selection the group intermediates also start at offset 0:
// they are written after stage 1's merge and read before stage 3.
struct StepLayout {
  size_t tab_offset, tab_bytes, total;
};
StepLayout step_layout(const smallkv_batch_t &b, const smallkv_model_t &small,
                       const smallkv_model_t &large, int nsh, int select) {
  const SmallPlan p = plan_small(small_view(b, small), small);
  const GroupPlan gp = plan_group(b, large, nsh);
  StepLayout l{};
  if (select == SMALLKV_SELECT_GROUP || select == SMALLKV_SELECT_ACCUM) {
    l.total = max_sz(max_sz(p.ws_bytes, gp.use ? gp.ws_bytes : 0),
                     group_layout(b, small, large, 0, select == SMALLKV_SELECT_ACCUM).end);
    return l;
  }
  l.tab_offset = (max_sz(p.ws_bytes, gp.use ? gp.ws_bytes : 0) + 255) / 256 * 256;
  // (with one token range per kv head every cursor starts at 0: no offsets;
  // the partition writes them in row order, so not with held rows either)
  l.tab_bytes = gp.use && gp.n_split > 1 && !small.held ? list_offsets_bytes(b, nsh) : 0;
  l.total = l.tab_bytes ? l.tab_offset + l.tab_bytes : max_sz(p.ws_bytes, gp.use ? gp.ws_bytes : 0);
  return l;
}

// Stage 3: the grouped kernel where it applies, the per-head kernel otherwise.
// Layers [layer0, layer0 + nl) of l (all of them by default).
hipError_t launch_stage3(const smallkv_batch_t &b, const smallkv_model_t &l, const int32_t *head_map,
                         int nsh, const int32_t *crit, const int32_t *marg, const float *marg_prob,
                         const float *mass, int mode, void *ws, const int2 *tab, bool group_sel,
                         hipStream_t st, int layer0 = 0, int nl = -1) {
  if (nl < 0) nl = l.n_layers;
  const GroupPlan gp = plan_group(b, l, nsh, nl);
  if (gp.use)
    return launch_hybrid_group(b, l, head_map, nsh, crit, marg, marg_prob, mass, mode, gp,
                               static_cast<float *>(ws), tab, group_sel, layer0, nl, st);
  return launch_hybrid(b, l, head_map, nsh, crit, marg, marg_prob, mass, mode, group_sel, layer0,
                       nl, st);
}

// Host checks of a stage-3 call (whole stack or a layer range).
int check_stage3(const smallkv_batch_t *batch, const smallkv_model_t *large,
                 const int32_t *head_map, int32_t n_small_heads, const int32_t *crit_idx,
                 const int32_t *marg_idx, const float *marg_prob, const float *mass, int32_t mode,
                 int32_t select) {
  int rc = check_large(batch, large, head_map, n_small_heads);
  if (rc) return rc;
  if ((rc = check_mode(mode))) return rc;
  if (select != SMALLKV_SELECT_HEAD && select != SMALLKV_SELECT_GROUP) return SMALLKV_EINVAL;
  if (!crit_idx || !mass) return SMALLKV_EINVAL;
  if (batch->km_cap > 0 && (!marg_idx || !marg_prob)) return SMALLKV_EINVAL;
  return SMALLKV_OK;
}

// Workspace of a stage-3 call over `nl` layers.
size_t stage3_workspace(const smallkv_batch_t &b, const smallkv_model_t &l, int nsh, int nl) {
  const GroupPlan gp = plan_group(b, l, nsh, nl);
  return gp.use ? gp.ws_bytes : 0;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int check_window(const smallkv_window_t &m) {
  if (!m.q || !m.k || m.n_layers < 1 || m.n_q_heads < 1 || m.n_kv_heads < 1) return SMALLKV_EINVAL;
  if (m.n_q_heads % m.n_kv_heads) return SMALLKV_EINVAL;
  if (m.dtype != SMALLKV_F32 && m.dtype != SMALLKV_BF16) return SMALLKV_EINVAL;
  if (!(m.scale == m.scale)) return SMALLKV_EINVAL;
  if (!aligned16(m.q) || !aligned16(m.k)) return SMALLKV_EINVAL;
  if (m.head_dim != 64 && m.head_dim != 128) return SMALLKV_EUNSUPPORTED;
  if ((int64_t)m.n_layers * m.n_q_heads > 65535) return SMALLKV_EUNSUPPORTED;
  return SMALLKV_OK;
}

int check_store(const smallkv_store_t *s) {
  if (!s || !batch_ok(&s->batch)) return SMALLKV_EINVAL;
  if (s->n_layers < 1 || s->n_q_heads < 1 || s->n_kv_heads < 1 || s->n_q_heads % s->n_kv_heads)
    return SMALLKV_EINVAL;
  if (s->dtype != SMALLKV_F32 && s->dtype != SMALLKV_BF16) return SMALLKV_EINVAL;
  if (s->select < SMALLKV_SELECT_HEAD || s->select > SMALLKV_SELECT_ACCUM) return SMALLKV_EINVAL;
  if (!s->head_map || s->n_small_heads < 1 || !s->crit_idx || s->rows < 1) return SMALLKV_EINVAL;
  if (s->batch.km_cap > 0 && !s->marg_idx) return SMALLKV_EINVAL;
  if (!s->full_k || !s->full_v || !s->new_k || !s->new_v || !s->k_slot || !s->v_slot)
    return SMALLKV_EINVAL;
  const bool any_old = s->old_k || s->old_v || s->old_k_slot || s->old_v_slot;
  const bool all_old = s->old_k && s->old_v && s->old_k_slot && s->old_v_slot;
  if (any_old && !all_old) return SMALLKV_EINVAL;
  if (all_old && (s->old_k == s->new_k || s->old_v == s->new_v)) return SMALLKV_EINVAL;
  const void *ptrs[] = {s->full_k, s->full_v, s->new_k, s->new_v, s->old_k, s->old_v};
  for (const void *p : ptrs)
    if (p && !aligned16(p)) return SMALLKV_EINVAL;
  if (s->head_dim != 64 && s->head_dim != 128) return SMALLKV_EUNSUPPORTED;
  if (s->batch.n_cap > 131072 || s->rows > INT32_MAX / 2) return SMALLKV_EUNSUPPORTED;
  return SMALLKV_OK;
}

int check_match(const smallkv_match_t *m) {
  if (!m || !m->win_len || !m->top_k || !m->head_map) return SMALLKV_EINVAL;
  if (m->batch < 1 || m->w_cap < 1) return SMALLKV_EINVAL;
  if (m->batch > 65535 || m->w_cap > 256) return SMALLKV_EUNSUPPORTED;
  int rc = check_window(m->large);
  if (rc) return rc;
  if ((rc = check_window(m->small))) return rc;
  const int64_t H = (int64_t)m->large.n_layers * m->large.n_q_heads +
                    (int64_t)m->small.n_layers * m->small.n_q_heads;
  if (H > 65535) return SMALLKV_EUNSUPPORTED;
  return SMALLKV_OK;
}

// The address the kernels read `p` at: device memory as it is; pinned host
// memory (hipHostMalloc, mapped into the device's address space) at the
// device address the runtime reports for it.  Pageable or unknown host
// memory is rejected before anything is enqueued.
int device_view(const void *p, const void **out) {
  hipPointerAttribute_t at{};
  if (hipPointerGetAttributes(&at, p) != hipSuccess) {
    (void)hipGetLastError();
    return SMALLKV_EINVAL;
  }
  if (at.type == hipMemoryTypeDevice || at.type == hipMemoryTypeManaged ||
      at.type == hipMemoryTypeUnified) {
    *out = p;
    return SMALLKV_OK;
  }
  if (at.type == hipMemoryTypeHost && at.devicePointer && at.hostPointer) {
    // both attributes name the same byte of the allocation, so the
    // distance from either to `p` is the same
    *out = static_cast<const char *>(at.devicePointer) +
           (static_cast<const char *>(p) - static_cast<const char *>(at.hostPointer));
    return aligned16(*out) ? SMALLKV_OK : SMALLKV_EINVAL;
  }
  return SMALLKV_EINVAL;
}

int check_step(const smallkv_step_t *s);
int run_step(const smallkv_step_t *s, void *ws, size_t ws_bytes, void *stream,
             void *const *events);

}  // namespace

// Workspace of smallkv_step_noalloc: one copy per GPU, held from the
// library's load until the process ends.  Host code never passes this name
// to a kernel or a copy (on the host it stands for no device address): it
// uses the address hipGetSymbolAddress reports for the device.
static __device__ __align__(256) unsigned char scratch[SMALLKV_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // scratch's device address per device, once looked up

// The scratch address on the device `stream` belongs to (the current device
// for the null stream), looked up once per device with that device current.
int device_scratch(hipStream_t stream, void **out) {
  int dev = -1;
  if ((stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev)) != hipSuccess) {
    (void)hipGetLastError();
    return SMALLKV_EDEVICE;
  }
  if (dev < 0 || dev >= kMaxDevices) return SMALLKV_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SMALLKV_EDEVICE;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return SMALLKV_EDEVICE;
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return SMALLKV_EDEVICE;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SMALLKV_OK;
}

}  // namespace

extern "C" {

int smallkv_abi_version(void) { return SMALLKV_ABI_VERSION; }

const char *smallkv_status_string(int status) {
  switch (status) {
    case SMALLKV_OK:
      return "ok";
    case SMALLKV_EINVAL:
      return "invalid argument";
    case SMALLKV_EUNSUPPORTED:
      return "unsupported shape or type";
    case SMALLKV_EWORKSPACE:
      return "workspace too small";
    case SMALLKV_EDEVICE:
      return "HIP launch error";
    default:
      return "unknown status";
  }
}

int smallkv_workspace_size(const smallkv_step_t *step, size_t *bytes) {
  if (!step || !bytes) return SMALLKV_EINVAL;
  int rc = check_small(&step->batch, &step->small);
  if (rc) return rc;
  const int nsh = step->small.n_layers * step->small.n_q_heads;
  if ((rc = check_large(&step->batch, &step->large, step->head_map, nsh))) return rc;
  if (step->select < SMALLKV_SELECT_HEAD || step->select > SMALLKV_SELECT_ACCUM)
    return SMALLKV_EINVAL;
  *bytes = step_layout(step->batch, step->small, step->large, nsh, step->select).total;
  return SMALLKV_OK;
}

int smallkv_small_attn(const smallkv_batch_t *batch, const smallkv_model_t *small, float *logits,
                       float *row_max, float *row_sum, void *ws, size_t ws_bytes, void *stream) {
  int rc = check_small(batch, small);
  if (rc) return rc;
  if (!logits || !row_max || !row_sum) return SMALLKV_EINVAL;
  const smallkv_batch_t sb = small_view(*batch, *small);
  const SmallPlan p = plan_small(sb, *small);
  if (p.ws_bytes && (!ws || ws_bytes < p.ws_bytes)) return SMALLKV_EWORKSPACE;
  return status_of(launch_small_attn(sb, *small, logits, row_max, row_sum,
                                     static_cast<float *>(ws), p,
                                     static_cast<hipStream_t>(stream)));
}

int smallkv_partition(const smallkv_batch_t *batch, const smallkv_model_t *small,
                      int32_t n_small_heads, const float *logits, const float *row_max,
                      const float *row_sum, int32_t *crit_idx, int32_t *marg_idx,
                      float *marg_prob, float *mass, void *ws, size_t ws_bytes, void *stream) {
  (void)ws;
  (void)ws_bytes;
  if (!batch_ok(batch) || n_small_heads < 1) return SMALLKV_EINVAL;
  if (!logits || !row_max || !row_sum || !crit_idx || !mass) return SMALLKV_EINVAL;
  if (batch->km_cap > 0 && (!marg_idx || !marg_prob)) return SMALLKV_EINVAL;
  if ((int64_t)batch->batch * n_small_heads > INT32_MAX / 2) return SMALLKV_EUNSUPPORTED;
  const bool held = small && small->held;
  if (held) {
    const int rc = check_small(batch, small);
    if (rc) return rc;
    if (n_small_heads != small->n_layers * small->n_q_heads) return SMALLKV_EINVAL;
  }
  return status_of(launch_partition(held ? small_view(*batch, *small) : *batch, n_small_heads,
                                    logits, row_max, row_sum, crit_idx, marg_idx, marg_prob, mass,
                                    held ? small : nullptr, batch->seq_len, batch->n_cap,
                                    static_cast<hipStream_t>(stream)));
}

int smallkv_hybrid_attn(const smallkv_batch_t *batch, const smallkv_model_t *large,
                        const int32_t *head_map, int32_t n_small_heads, const int32_t *crit_idx,
                        const int32_t *marg_idx, const float *marg_prob, const float *mass,
                        int32_t mode, int32_t select, void *ws, size_t ws_bytes, void *stream) {
  if (!large) return SMALLKV_EINVAL;
  return smallkv_hybrid_attn_layers(batch, large, 0, large->n_layers, head_map, n_small_heads,
                                    crit_idx, marg_idx, marg_prob, mass, mode, select, ws,
                                    ws_bytes, stream);
}

int smallkv_hybrid_attn_workspace_size(const smallkv_batch_t *batch,
                                       const smallkv_model_t *large, int32_t layer_count,
                                       int32_t n_small_heads, size_t *bytes) {
  if (!bytes || !batch || !large) return SMALLKV_EINVAL;
  if (!batch_ok(batch) || !model_ok(large) || n_small_heads < 1) return SMALLKV_EINVAL;
  if (layer_count < 1 || layer_count > large->n_layers) return SMALLKV_EINVAL;
  *bytes = stage3_workspace(*batch, *large, n_small_heads, layer_count);
  return SMALLKV_OK;
}

int smallkv_hybrid_attn_layers(const smallkv_batch_t *batch, const smallkv_model_t *large,
                               int32_t layer_begin, int32_t layer_count, const int32_t *head_map,
                               int32_t n_small_heads, const int32_t *crit_idx,
                               const int32_t *marg_idx, const float *marg_prob,
                               const float *mass, int32_t mode, int32_t select, void *ws,
                               size_t ws_bytes, void *stream) {
  const int rc = check_stage3(batch, large, head_map, n_small_heads, crit_idx, marg_idx,
                              marg_prob, mass, mode, select);
  if (rc) return rc;
  if (layer_begin < 0 || layer_count < 1 || layer_begin > large->n_layers - layer_count)
    return SMALLKV_EINVAL;
  const size_t need = stage3_workspace(*batch, *large, n_small_heads, layer_count);
  if (need && (!ws || ws_bytes < need)) return SMALLKV_EWORKSPACE;
  return status_of(launch_stage3(*batch, *large, head_map, n_small_heads, crit_idx, marg_idx,
                                 marg_prob, mass, mode, ws, nullptr,
                                 select == SMALLKV_SELECT_GROUP,
                                 static_cast<hipStream_t>(stream), layer_begin, layer_count));
}

int smallkv_accum_select_workspace_size(const smallkv_batch_t *batch,
                                        const smallkv_model_t *small, size_t *bytes) {
  if (!bytes) return SMALLKV_EINVAL;
  const int rc = check_small(batch, small);
  if (rc) return rc;
  *bytes = group_layout(*batch, *small, *small, 0, true).end;
  return SMALLKV_OK;
}

int smallkv_accum_select(const smallkv_batch_t *batch, const smallkv_model_t *small,
                         const float *logits, const float *row_max, const float *row_sum,
                         float *acc_score, int32_t *crit_idx, int32_t *marg_idx,
                         float *marg_prob, float *mass, void *ws, size_t ws_bytes, void *stream) {
  const int rc = check_small(batch, small);
  if (rc) return rc;
  if (small->held) return SMALLKV_EUNSUPPORTED;
  if (!logits || !row_max || !row_sum || !acc_score || !crit_idx || !mass) return SMALLKV_EINVAL;
  if (batch->km_cap > 0 && (!marg_idx || !marg_prob)) return SMALLKV_EINVAL;
  const GroupLayout lay = group_layout(*batch, *small, *small, 0, true);
  if (!ws || ws_bytes < lay.end) return SMALLKV_EWORKSPACE;
  return status_of(launch_accum_select(*batch, *small, logits, row_max, row_sum, acc_score,
                                       crit_idx, marg_idx, marg_prob, mass, ws, lay,
                                       static_cast<hipStream_t>(stream)));
}

int smallkv_group_select_workspace_size(const smallkv_batch_t *batch,
                                        const smallkv_model_t *small,
                                        const smallkv_model_t *large, size_t *bytes) {
  if (!bytes || !large) return SMALLKV_EINVAL;
  int rc = check_small(batch, small);
  if (rc) return rc;
  if (!model_ok(large)) return SMALLKV_EINVAL;
  *bytes = group_layout(*batch, *small, *large, 0).end;
  return SMALLKV_OK;
}

int smallkv_group_select(const smallkv_batch_t *batch, const smallkv_model_t *small,
                         const smallkv_model_t *large, const int32_t *head_map,
                         const float *logits, const float *row_max, const float *row_sum,
                         int32_t *crit_idx, int32_t *marg_idx, float *marg_prob, float *mass,
                         void *ws, size_t ws_bytes, void *stream) {
  int rc = check_small(batch, small);
  if (rc) return rc;
  const int nsh = small->n_layers * small->n_q_heads;
  if ((rc = check_large(batch, large, head_map, nsh))) return rc;
  if (small->held || large->n_q_heads / large->n_kv_heads > 16) return SMALLKV_EUNSUPPORTED;
  if (!logits || !row_max || !row_sum || !crit_idx || !mass) return SMALLKV_EINVAL;
  if (batch->km_cap > 0 && (!marg_idx || !marg_prob)) return SMALLKV_EINVAL;
  const GroupLayout lay = group_layout(*batch, *small, *large, 0);
  if (!ws || ws_bytes < lay.end) return SMALLKV_EWORKSPACE;
  return status_of(launch_group_select(*batch, *small, *large, head_map, logits, row_max, row_sum,
                                       crit_idx, marg_idx, marg_prob, mass, ws, lay,
                                       static_cast<hipStream_t>(stream)));
}

int smallkv_store_workspace_size(const smallkv_store_t *s, size_t *bytes) {
  if (!bytes) return SMALLKV_EINVAL;
  const int rc = check_store(s);
  if (rc) return rc;
  *bytes = store_workspace(*s);
  return SMALLKV_OK;
}

int smallkv_store_update(const smallkv_store_t *s, void *ws, size_t ws_bytes, void *stream) {
  const int rc = check_store(s);
  if (rc) return rc;
  if (!ws || ws_bytes < store_workspace(*s)) return SMALLKV_EWORKSPACE;
  smallkv_store_t d = *s;
  if (device_view(s->full_k, &d.full_k) || device_view(s->full_v, &d.full_v))
    return SMALLKV_EINVAL;
  return status_of(launch_store_update(d, ws, static_cast<hipStream_t>(stream)));
}

int smallkv_match_workspace_size(const smallkv_match_t *m, size_t *bytes) {
  if (!bytes) return SMALLKV_EINVAL;
  const int rc = check_match(m);
  if (rc) return rc;
  *bytes = match_layout(*m).total;
  return SMALLKV_OK;
}

int smallkv_match(const smallkv_match_t *m, void *ws, size_t ws_bytes, void *stream) {
  const int rc = check_match(m);
  if (rc) return rc;
  if (!ws || ws_bytes < match_layout(*m).total) return SMALLKV_EWORKSPACE;
  return status_of(launch_match(*m, ws, static_cast<hipStream_t>(stream)));
}

int smallkv_step(const smallkv_step_t *s, void *ws, size_t ws_bytes, void *stream) {
  return run_step(s, ws, ws_bytes, stream, nullptr);
}

int smallkv_step_events(const smallkv_step_t *s, void *ws, size_t ws_bytes, void *stream,
                        void *const *events) {
  return run_step(s, ws, ws_bytes, stream, events);
}

int smallkv_step_noalloc(const smallkv_step_t *s, void *stream) {
  int rc = check_step(s);
  if (rc) return rc;
  size_t need = 0;
  if ((rc = smallkv_workspace_size(s, &need))) return rc;
  if (need > SMALLKV_NOALLOC_SCRATCH_BYTES) return SMALLKV_EWORKSPACE;
  void *ws = nullptr;
  if ((rc = device_scratch(static_cast<hipStream_t>(stream), &ws))) return rc;
  return run_step(s, ws, SMALLKV_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}

}  // extern "C"

namespace {

// Every host-visible check of a whole step, before anything is enqueued.
int check_step(const smallkv_step_t *s) {
  if (!s) return SMALLKV_EINVAL;
  const int nsh = s->small.n_layers * s->small.n_q_heads;
  int rc = check_small(&s->batch, &s->small);
  if (rc) return rc;
  if ((rc = check_large(&s->batch, &s->large, s->head_map, nsh))) return rc;
  if ((rc = check_mode(s->mode))) return rc;
  if (!s->logits || !s->row_max || !s->row_sum || !s->crit_idx || !s->mass) return SMALLKV_EINVAL;
  if (s->batch.km_cap > 0 && (!s->marg_idx || !s->marg_prob)) return SMALLKV_EINVAL;
  const bool group = s->select == SMALLKV_SELECT_GROUP;
  const bool accum = s->select == SMALLKV_SELECT_ACCUM;
  if (!group && !accum && s->select != SMALLKV_SELECT_HEAD) return SMALLKV_EINVAL;
  if (accum && !s->acc_score) return SMALLKV_EINVAL;
  if ((group || accum) && s->small.held) return SMALLKV_EUNSUPPORTED;
  if (group && s->large.n_q_heads / s->large.n_kv_heads > 16) return SMALLKV_EUNSUPPORTED;
  return SMALLKV_OK;
}

// events (optional, entries may be null): recorded on the stream before
// stage 1, after stage 1's chunk kernel (after its merge too with group or
// accumulated selection), after stage 2 and after stage 3.
int run_step(const smallkv_step_t *s, void *ws, size_t ws_bytes, void *stream,
             void *const *events) {
  const int rc = check_step(s);
  if (rc) return rc;
  const int nsh = s->small.n_layers * s->small.n_q_heads;
  const bool group = s->select == SMALLKV_SELECT_GROUP;
  const bool accum = s->select == SMALLKV_SELECT_ACCUM;
  const smallkv_batch_t sb = small_view(s->batch, s->small);
  const SmallPlan p = plan_small(sb, s->small);
  const StepLayout lay = step_layout(s->batch, s->small, s->large, nsh, s->select);
  if (lay.total && (!ws || ws_bytes < lay.total)) return SMALLKV_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  auto mark = [&](int i) {
    return events && events[i] ? hipEventRecord(static_cast<hipEvent_t>(events[i]), st)
                               : hipSuccess;
  };
  if (mark(0) != hipSuccess) return SMALLKV_EDEVICE;
  hipError_t e;
  if (accum || group) {
    // stage 1 with its own merge, the selection (accumulated scores and
    // their partition, or the group sets), stage 3 on its lists
    e = launch_small_attn(sb, s->small, s->logits, s->row_max, s->row_sum,
                          static_cast<float *>(ws), p, st);
    if (e != hipSuccess || mark(1) != hipSuccess) return SMALLKV_EDEVICE;
    if (accum)
      e = launch_accum_select(s->batch, s->small, s->logits, s->row_max, s->row_sum,
                              s->acc_score, s->crit_idx, s->marg_idx, s->marg_prob, s->mass, ws,
                              group_layout(s->batch, s->small, s->large, 0, true), st);
    else
      e = launch_group_select(s->batch, s->small, s->large, s->head_map, s->logits, s->row_max,
                              s->row_sum, s->crit_idx, s->marg_idx, s->marg_prob, s->mass, ws,
                              group_layout(s->batch, s->small, s->large, 0), st);
    if (e != hipSuccess || mark(2) != hipSuccess) return SMALLKV_EDEVICE;
    e = launch_stage3(s->batch, s->large, s->head_map, nsh, s->crit_idx, s->marg_idx,
                      s->marg_prob, s->mass, s->mode, ws, nullptr, group, st);
    if (e != hipSuccess || mark(3) != hipSuccess) return SMALLKV_EDEVICE;
    return SMALLKV_OK;
  }
  int2 *tab = lay.tab_bytes ? reinterpret_cast<int2 *>(static_cast<char *>(ws) + lay.tab_offset)
                            : nullptr;
  e = launch_small_split(sb, s->small, s->logits, static_cast<float *>(ws), p, st);
  if (e != hipSuccess || mark(1) != hipSuccess) return SMALLKV_EDEVICE;
  e = launch_merge_partition(sb, s->small, p, static_cast<const float *>(ws), s->logits,
                             s->row_max, s->row_sum, s->crit_idx, s->marg_idx, s->marg_prob,
                             s->mass, tab, s->batch.seq_len, s->batch.n_cap, st);
  if (e != hipSuccess || mark(2) != hipSuccess) return SMALLKV_EDEVICE;
  // stage 1's records are consumed by now: stage 3 reuses the workspace
  // below the list offsets
  e = launch_stage3(s->batch, s->large, s->head_map, nsh, s->crit_idx, s->marg_idx, s->marg_prob,
                    s->mass, s->mode, ws, tab, false, st);
  if (e != hipSuccess || mark(3) != hipSuccess) return SMALLKV_EDEVICE;
  return SMALLKV_OK;
}

}  // namespace
