"""Python binding of libsmallkv.so (include/smallkv.h).

Argument marshalling only: torch tensors are used for device memory and the
current HIP stream, their pointers and shapes go through ctypes to the C ABI,
and every step of the computation runs in the library's HIP kernels.  There
is no fallback: if the library is not built, or a call fails, this module
raises.

Entry points mirror the C names: smallkv_small_attn, smallkv_partition,
smallkv_hybrid_attn, smallkv_step, smallkv_workspace_size, and the prefill
matching smallkv_match, smallkv_match_workspace_size.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsmallkv.so")

F32, BF16 = 0, 1
NORM_REMAINING, NORM_NONE, NORM_SLM_CRIT, NORM_RETAINED, NORM_MARG_FILL = range(5)
SELECT_HEAD, SELECT_GROUP, SELECT_ACCUM = 0, 1, 2
OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EDEVICE = 0, -1, -2, -3, -4


class Batch(C.Structure):
    _fields_ = [("batch", C.c_int32), ("n_cap", C.c_int32),
                ("seq_len", C.c_void_p), ("k_crit", C.c_void_p), ("k_marg", C.c_void_p),
                ("k_recent", C.c_void_p), ("kc_cap", C.c_int32), ("km_cap", C.c_int32)]


class Model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("dtype", C.c_int32), ("scale", C.c_float),
                ("q", C.c_void_p), ("k", C.c_void_p), ("v", C.c_void_p),
                ("n_rows", C.c_int64), ("k_slot", C.c_void_p), ("v_slot", C.c_void_p),
                ("out", C.c_void_p), ("held", C.c_void_p), ("row_pos", C.c_void_p)]


class Step(C.Structure):
    _fields_ = [("batch", Batch), ("small", Model), ("large", Model),
                ("head_map", C.c_void_p), ("mode", C.c_int32),
                ("logits", C.c_void_p), ("row_max", C.c_void_p), ("row_sum", C.c_void_p),
                ("crit_idx", C.c_void_p), ("marg_idx", C.c_void_p),
                ("marg_prob", C.c_void_p), ("mass", C.c_void_p), ("select", C.c_int32),
                ("acc_score", C.c_void_p)]


class Window(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("dtype", C.c_int32), ("scale", C.c_float),
                ("q", C.c_void_p), ("k", C.c_void_p)]


class Match(C.Structure):
    _fields_ = [("batch", C.c_int32), ("w_cap", C.c_int32), ("win_len", C.c_void_p),
                ("top_k", C.c_void_p), ("large", Window), ("small", Window),
                ("head_map", C.c_void_p), ("scores", C.c_void_p), ("top_bits", C.c_void_p)]


class Store(C.Structure):
    _fields_ = [("batch", Batch), ("n_layers", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("dtype", C.c_int32),
                ("head_map", C.c_void_p), ("n_small_heads", C.c_int32), ("select", C.c_int32),
                ("crit_idx", C.c_void_p), ("marg_idx", C.c_void_p), ("full_k", C.c_void_p),
                ("full_v", C.c_void_p), ("rows", C.c_int64), ("old_k", C.c_void_p),
                ("old_v", C.c_void_p), ("old_k_slot", C.c_void_p), ("old_v_slot", C.c_void_p),
                ("new_k", C.c_void_p), ("new_v", C.c_void_p), ("k_slot", C.c_void_p),
                ("v_slot", C.c_void_p), ("counts", C.c_void_p)]


EXPORTS = ("smallkv_small_attn", "smallkv_partition", "smallkv_hybrid_attn", "smallkv_step",
           "smallkv_step_noalloc", "smallkv_step_events", "smallkv_hybrid_attn_layers",
           "smallkv_hybrid_attn_workspace_size", "smallkv_workspace_size", "smallkv_match", "smallkv_match_workspace_size",
           "smallkv_group_select", "smallkv_group_select_workspace_size",
           "smallkv_accum_select", "smallkv_accum_select_workspace_size",
           "smallkv_store_update", "smallkv_store_workspace_size",
           "smallkv_status_string", "smallkv_abi_version")

_lib = None


def lib():
    """Load libsmallkv.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_2508_02751_amd.build`")
        L = C.CDLL(LIB_PATH)
        P = C.POINTER
        L.smallkv_small_attn.argtypes = [P(Batch), P(Model), C.c_void_p, C.c_void_p, C.c_void_p,
                                         C.c_void_p, C.c_size_t, C.c_void_p]
        L.smallkv_partition.argtypes = [P(Batch), P(Model), C.c_int32, C.c_void_p, C.c_void_p,
                                        C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                        C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
        L.smallkv_hybrid_attn.argtypes = [P(Batch), P(Model), C.c_void_p, C.c_int32, C.c_void_p,
                                          C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32,
                                          C.c_int32, C.c_void_p, C.c_size_t, C.c_void_p]
        L.smallkv_group_select.argtypes = [P(Batch), P(Model), P(Model), C.c_void_p, C.c_void_p,
                                           C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                           C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                                           C.c_void_p]
        L.smallkv_group_select_workspace_size.argtypes = [P(Batch), P(Model), P(Model),
                                                          P(C.c_size_t)]
        L.smallkv_accum_select.argtypes = [P(Batch), P(Model), C.c_void_p, C.c_void_p,
                                           C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                           C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                                           C.c_void_p]
        L.smallkv_accum_select_workspace_size.argtypes = [P(Batch), P(Model), P(C.c_size_t)]
        L.smallkv_store_update.argtypes = [P(Store), C.c_void_p, C.c_size_t, C.c_void_p]
        L.smallkv_store_workspace_size.argtypes = [P(Store), P(C.c_size_t)]
        L.smallkv_step.argtypes = [P(Step), C.c_void_p, C.c_size_t, C.c_void_p]
        L.smallkv_step_noalloc.argtypes = [P(Step), C.c_void_p]
        L.smallkv_step_events.argtypes = [P(Step), C.c_void_p, C.c_size_t, C.c_void_p,
                                          P(C.c_void_p)]
        L.smallkv_hybrid_attn_layers.argtypes = [P(Batch), P(Model), C.c_int32, C.c_int32,
                                                 C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                                                 C.c_void_p, C.c_void_p, C.c_int32, C.c_int32,
                                                 C.c_void_p, C.c_size_t, C.c_void_p]
        L.smallkv_hybrid_attn_workspace_size.argtypes = [P(Batch), P(Model), C.c_int32,
                                                         C.c_int32, P(C.c_size_t)]
        L.smallkv_workspace_size.argtypes = [P(Step), P(C.c_size_t)]
        L.smallkv_match.argtypes = [P(Match), C.c_void_p, C.c_size_t, C.c_void_p]
        L.smallkv_match_workspace_size.argtypes = [P(Match), P(C.c_size_t)]
        L.smallkv_status_string.argtypes = [C.c_int]
        L.smallkv_status_string.restype = C.c_char_p
        L.smallkv_abi_version.argtypes = []
        for f in ("smallkv_small_attn", "smallkv_partition", "smallkv_hybrid_attn",
                  "smallkv_step", "smallkv_step_noalloc", "smallkv_step_events",
                  "smallkv_hybrid_attn_layers", "smallkv_hybrid_attn_workspace_size",
                  "smallkv_workspace_size", "smallkv_abi_version",
                  "smallkv_match", "smallkv_match_workspace_size", "smallkv_group_select",
                  "smallkv_group_select_workspace_size", "smallkv_accum_select",
                  "smallkv_accum_select_workspace_size", "smallkv_store_update",
                  "smallkv_store_workspace_size"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


class SmallKVError(RuntimeError):
    def __init__(self, fn, status):
        msg = lib().smallkv_status_string(status).decode()
        super().__init__(f"{fn} failed with status {status} ({msg})")
        self.status = status


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libsmallkv must be contiguous")
    return t.data_ptr()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise ValueError(f"unsupported dtype {t.dtype}")


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


@dataclasses.dataclass
class BatchSpec:
    """Sequences and budgets: seq_len/k_crit/k_marg (and the optional recent
    budget k_recent) are int32 device tensors [B]."""
    seq_len: torch.Tensor
    k_crit: torch.Tensor
    k_marg: torch.Tensor
    n_cap: int
    kc_cap: int
    km_cap: int
    k_recent: Optional[torch.Tensor] = None

    def c(self) -> Batch:
        ts = [self.seq_len, self.k_crit, self.k_marg]
        if self.k_recent is not None:
            ts.append(self.k_recent)
        for t in ts:
            if t.dtype != torch.int32:
                raise ValueError("seq_len, k_crit, k_marg and k_recent must be int32")
        return Batch(self.seq_len.numel(), self.n_cap, _ptr(self.seq_len), _ptr(self.k_crit),
                     _ptr(self.k_marg), _ptr(self.k_recent) if self.k_recent is not None else None,
                     self.kc_cap, self.km_cap)


@dataclasses.dataclass
class ModelSpec:
    """One model's operands: q [B][L][Hq][d], k/v [B][L][Hkv][n_rows][d], out like q.
    Small model only: held [B] and row_pos [B][L][Hkv][n_rows] (int32) when its
    own cache is compressed."""
    q: torch.Tensor
    k: torch.Tensor
    v: torch.Tensor
    out: torch.Tensor
    scale: float
    k_slot: Optional[torch.Tensor] = None
    v_slot: Optional[torch.Tensor] = None
    held: Optional[torch.Tensor] = None
    row_pos: Optional[torch.Tensor] = None

    def c(self) -> Model:
        B, L, hq, d = self.q.shape
        hkv, rows = self.k.shape[2], self.k.shape[3]
        if self.k.shape != self.v.shape or self.out.shape != self.q.shape:
            raise ValueError("k/v or out shape mismatch")
        if not (self.q.dtype == self.k.dtype == self.v.dtype == self.out.dtype):
            raise ValueError("q, k, v and out must share a dtype")
        for t in (self.k_slot, self.v_slot, self.held, self.row_pos):
            if t is not None and t.dtype != torch.int32:
                raise ValueError("slot and position maps must be int32")
        return Model(L, hq, hkv, d, _dtype_code(self.q), self.scale, _ptr(self.q), _ptr(self.k),
                     _ptr(self.v), rows, _ptr(self.k_slot), _ptr(self.v_slot), _ptr(self.out),
                     _ptr(self.held), _ptr(self.row_pos))


def _check(fn, rc):
    if rc != OK:
        raise SmallKVError(fn, rc)


def _ws(ws: Optional[torch.Tensor]):
    return (None, 0) if ws is None else (_ptr(ws), ws.numel() * ws.element_size())


def smallkv_workspace_size(batch: BatchSpec, small: ModelSpec, large: ModelSpec,
                           head_map, select: int = SELECT_HEAD) -> int:
    st = Step()
    st.select = int(select)
    st.batch = batch.c()
    st.small = small.c()
    st.large = large.c()
    st.head_map = _ptr(head_map)
    n = C.c_size_t()
    _check("smallkv_workspace_size", lib().smallkv_workspace_size(C.byref(st), C.byref(n)))
    return n.value


def smallkv_small_attn(batch: BatchSpec, small: ModelSpec, logits, row_max, row_sum,
                       ws=None, stream=None):
    b, m = batch.c(), small.c()
    w, wb = _ws(ws)
    _check("smallkv_small_attn", lib().smallkv_small_attn(
        C.byref(b), C.byref(m), _ptr(logits), _ptr(row_max), _ptr(row_sum), w, wb,
        _stream(stream)))


def smallkv_partition(batch: BatchSpec, n_small_heads: int, logits, row_max, row_sum,
                      crit_idx, marg_idx, marg_prob, mass, ws=None, stream=None,
                      small: Optional[ModelSpec] = None):
    """Stage 2; `small` is needed only when the small model's own cache is
    compressed (its held rows and their positions)."""
    b = batch.c()
    m = small.c() if small is not None else None
    w, wb = _ws(ws)
    _check("smallkv_partition", lib().smallkv_partition(
        C.byref(b), C.byref(m) if m is not None else None, n_small_heads, _ptr(logits),
        _ptr(row_max), _ptr(row_sum), _ptr(crit_idx), _ptr(marg_idx), _ptr(marg_prob),
        _ptr(mass), w, wb, _stream(stream)))


def smallkv_hybrid_attn(batch: BatchSpec, large: ModelSpec, head_map, n_small_heads: int,
                        crit_idx, marg_idx, marg_prob, mass, mode=NORM_REMAINING, ws=None,
                        stream=None, select: int = SELECT_HEAD):
    b, m = batch.c(), large.c()
    w, wb = _ws(ws)
    _check("smallkv_hybrid_attn", lib().smallkv_hybrid_attn(
        C.byref(b), C.byref(m), _ptr(head_map), n_small_heads, _ptr(crit_idx), _ptr(marg_idx),
        _ptr(marg_prob), _ptr(mass), int(mode), int(select), w, wb, _stream(stream)))


def smallkv_hybrid_attn_layers(batch: BatchSpec, large: ModelSpec, layer_begin: int,
                               layer_count: int, head_map, n_small_heads: int, crit_idx,
                               marg_idx, marg_prob, mass, mode=NORM_REMAINING, ws=None,
                               stream=None, select: int = SELECT_HEAD):
    """Stage 3 over large layers [layer_begin, layer_begin + layer_count) only."""
    b, m = batch.c(), large.c()
    w, wb = _ws(ws)
    _check("smallkv_hybrid_attn_layers", lib().smallkv_hybrid_attn_layers(
        C.byref(b), C.byref(m), int(layer_begin), int(layer_count), _ptr(head_map),
        n_small_heads, _ptr(crit_idx), _ptr(marg_idx), _ptr(marg_prob), _ptr(mass), int(mode),
        int(select), w, wb, _stream(stream)))


def smallkv_hybrid_attn_workspace_size(batch: BatchSpec, large: ModelSpec, layer_count: int,
                                       n_small_heads: int) -> int:
    b, m = batch.c(), large.c()
    n = C.c_size_t()
    _check("smallkv_hybrid_attn_workspace_size", lib().smallkv_hybrid_attn_workspace_size(
        C.byref(b), C.byref(m), int(layer_count), int(n_small_heads), C.byref(n)))
    return n.value


def smallkv_group_select(batch: BatchSpec, small: ModelSpec, large: ModelSpec, head_map, logits,
                         row_max, row_sum, crit_idx, marg_idx, marg_prob, mass, ws, stream=None):
    """Stage 2 of group selection (lists per large kv head, weights per large head)."""
    b, sm, lg = batch.c(), small.c(), large.c()
    w, wb = _ws(ws)
    _check("smallkv_group_select", lib().smallkv_group_select(
        C.byref(b), C.byref(sm), C.byref(lg), _ptr(head_map), _ptr(logits), _ptr(row_max),
        _ptr(row_sum), _ptr(crit_idx), _ptr(marg_idx), _ptr(marg_prob), _ptr(mass), w, wb,
        _stream(stream)))


def make_step(batch: BatchSpec, small: ModelSpec, large: ModelSpec, head_map, mode, logits,
              row_max, row_sum, crit_idx, marg_idx, marg_prob, mass,
              select: int = SELECT_HEAD, acc_score: Optional[torch.Tensor] = None) -> Step:
    """Build the C step descriptor once (it holds raw pointers: keep the tensors alive)."""
    if acc_score is not None and acc_score.dtype != torch.float32:
        raise ValueError("acc_score must be float32")
    return Step(batch.c(), small.c(), large.c(), _ptr(head_map), int(mode), _ptr(logits),
                _ptr(row_max), _ptr(row_sum), _ptr(crit_idx), _ptr(marg_idx), _ptr(marg_prob),
                _ptr(mass), int(select), _ptr(acc_score))


def smallkv_step(step: Step, ws=None, stream=None):
    w, wb = _ws(ws)
    _check("smallkv_step", lib().smallkv_step(C.byref(step), w, wb, _stream(stream)))


def smallkv_step_events(step: Step, ws, events, stream=None):
    """smallkv_step recording the given torch.cuda.Event objects (4, or None
    entries) at the stage boundaries: before stage 1, after stage 1's chunk
    kernel, after stage 2, after stage 3."""
    w, wb = _ws(ws)
    ts = torch.cuda.current_stream() if stream is None else stream
    for e in events:
        if e is not None and not e.cuda_event:
            e.record(ts)  # torch creates its HIP event at the first record
    arr = (C.c_void_p * 4)(*[None if e is None else e.cuda_event for e in events])
    _check("smallkv_step_events", lib().smallkv_step_events(C.byref(step), w, wb, _stream(stream),
                                                            arr))


NOALLOC_SCRATCH_BYTES = 32 << 20  # SMALLKV_NOALLOC_SCRATCH_BYTES


def smallkv_step_noalloc(step: Step, stream=None):
    """smallkv_step on the library's own per-GPU scratch (no workspace, no
    allocation); calls on one GPU must not overlap."""
    _check("smallkv_step_noalloc", lib().smallkv_step_noalloc(C.byref(step), _stream(stream)))


@dataclasses.dataclass
class StepBuffers:
    """The caller-owned intermediates and outputs of one decode step."""
    logits: torch.Tensor
    row_max: torch.Tensor
    row_sum: torch.Tensor
    crit_idx: torch.Tensor
    marg_idx: torch.Tensor
    marg_prob: torch.Tensor
    mass: torch.Tensor
    small_out: torch.Tensor
    large_out: torch.Tensor
    ws: Optional[torch.Tensor]
    acc_score: Optional[torch.Tensor] = None  # accumulated-score selection state


def alloc_step_buffers(batch: BatchSpec, s_q: torch.Tensor, l_q: torch.Tensor,
                       ws_bytes: int, select: int = SELECT_HEAD,
                       l_kv_heads: Optional[int] = None) -> StepBuffers:
    """Group selection: lists per (large layer, kv head), weights per large head."""
    B, l, hqs, _ = s_q.shape
    nsh = l * hqs
    _, L, hq, _ = l_q.shape
    lrows, prows = (L * l_kv_heads, L * hq) if select == SELECT_GROUP else (nsh, nsh)
    dev = s_q.device
    return StepBuffers(
        logits=torch.empty((B, nsh, batch.n_cap), dtype=torch.float32, device=dev),
        row_max=torch.empty((B, nsh), dtype=torch.float32, device=dev),
        row_sum=torch.empty((B, nsh), dtype=torch.float32, device=dev),
        crit_idx=torch.empty((B, lrows, batch.kc_cap), dtype=torch.int32, device=dev),
        marg_idx=torch.empty((B, lrows, max(batch.km_cap, 1)), dtype=torch.int32, device=dev),
        marg_prob=torch.empty((B, prows, max(batch.km_cap, 1)), dtype=torch.float32, device=dev),
        mass=torch.empty((B, prows, 2), dtype=torch.float32, device=dev),
        small_out=torch.empty_like(s_q),
        large_out=torch.empty_like(l_q),
        ws=torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev) if ws_bytes else None,
    )


# ------------------------------------------------------- prefill matching --

def window_spec(q: torch.Tensor, k: torch.Tensor, scale: float) -> Window:
    """One model's window operands: q [B][layers][Hq][w_cap][d], k [B][layers][Hkv][w_cap][d]."""
    if q.dim() != 5 or k.dim() != 5 or q.dtype != k.dtype:
        raise ValueError("window q/k must be 5-d tensors of one dtype")
    _, layers, hq, _, d = q.shape
    return Window(layers, hq, k.shape[2], d, _dtype_code(q), scale, _ptr(q), _ptr(k))


@dataclasses.dataclass
class MatchCall:
    """A prepared smallkv_match descriptor and the tensors it points at."""
    desc: Match
    head_map: torch.Tensor          # [B][L*Hq] int32
    scores: Optional[torch.Tensor]  # [B][H][w_cap] fp32
    top_bits: Optional[torch.Tensor]  # [B][H][nw] int64 (bit patterns of uint64 words)
    ws: torch.Tensor
    keep: tuple

    def run(self, stream=None):
        smallkv_match(self.desc, self.ws, stream)


def prepare_match(win_len: torch.Tensor, top_k: torch.Tensor, l_q, l_k, l_scale, s_q, s_k,
                  s_scale, scores=True, top_bits=True) -> MatchCall:
    """Descriptor, outputs and workspace for smallkv_match over the given windows."""
    for t in (win_len, top_k):
        if t.dtype != torch.int32:
            raise ValueError("win_len and top_k must be int32")
    B, L, hq, w_cap, _ = l_q.shape
    H = L * hq + s_q.shape[1] * s_q.shape[2]
    dev = l_q.device
    hm = torch.empty((B, L * hq), dtype=torch.int32, device=dev)
    sc = torch.zeros((B, H, w_cap), dtype=torch.float32, device=dev) if scores else None
    nw = (w_cap + 63) // 64
    tb = torch.zeros((B, H, nw), dtype=torch.int64, device=dev) if top_bits else None
    d = Match(B, w_cap, _ptr(win_len), _ptr(top_k), window_spec(l_q, l_k, l_scale),
              window_spec(s_q, s_k, s_scale), _ptr(hm), _ptr(sc), _ptr(tb))
    n = C.c_size_t()
    _check("smallkv_match_workspace_size", lib().smallkv_match_workspace_size(C.byref(d), C.byref(n)))
    ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device=dev)
    return MatchCall(d, hm, sc, tb, ws, (win_len, top_k, l_q, l_k, s_q, s_k))


def smallkv_match(desc: Match, ws, stream=None):
    w, wb = _ws(ws)
    _check("smallkv_match", lib().smallkv_match(C.byref(desc), w, wb, _stream(stream)))


def smallkv_accum_select(batch: BatchSpec, small: ModelSpec, logits, row_max, row_sum, acc_score,
                         crit_idx, marg_idx, marg_prob, mass, ws, stream=None):
    """Stage 2 of accumulated-score selection (acc_score updated in place)."""
    b, sm = batch.c(), small.c()
    w, wb = _ws(ws)
    _check("smallkv_accum_select", lib().smallkv_accum_select(
        C.byref(b), C.byref(sm), _ptr(logits), _ptr(row_max), _ptr(row_sum), _ptr(acc_score),
        _ptr(crit_idx), _ptr(marg_idx), _ptr(marg_prob), _ptr(mass), w, wb, _stream(stream)))


@dataclasses.dataclass
class StoreCall:
    """A prepared smallkv_store_update and the tensors it writes."""
    desc: Store
    new_k: torch.Tensor
    new_v: torch.Tensor
    k_slot: torch.Tensor
    v_slot: torch.Tensor
    counts: torch.Tensor
    ws: torch.Tensor
    keep: tuple

    def run(self, stream=None):
        smallkv_store_update(self.desc, self.ws, stream)


def prepare_store(batch: BatchSpec, head_map, n_small_heads: int, crit_idx, marg_idx,
                  full_k: torch.Tensor, full_v: torch.Tensor, rows: int, select: int = SELECT_HEAD,
                  old: Optional["StoreCall"] = None) -> StoreCall:
    """The new compact store (rows per kv head) built from a step's lists;
    `old`: the previous store, whose rows are reused.  The full store may be
    on the GPU or in pinned host memory; the new store is on the GPU."""
    B, L, hk, n_cap, d = full_k.shape
    hq = head_map.numel() // L
    dev = crit_idx.device
    nk = torch.zeros((B, L, hk, rows, d), dtype=full_k.dtype, device=dev)
    nv = torch.zeros_like(nk)
    ks = torch.full((B, L, hk, n_cap), -1, dtype=torch.int32, device=dev)
    vs = torch.full_like(ks, -1)
    cnt = torch.zeros((B, L, hk, 2), dtype=torch.int32, device=dev)
    o = old
    desc = Store(batch.c(), L, hq, hk, d, _dtype_code(full_k), _ptr(head_map), n_small_heads,
                 int(select), _ptr(crit_idx), _ptr(marg_idx), _ptr(full_k), _ptr(full_v), rows,
                 _ptr(o.new_k) if o else None, _ptr(o.new_v) if o else None,
                 _ptr(o.k_slot) if o else None, _ptr(o.v_slot) if o else None,
                 _ptr(nk), _ptr(nv), _ptr(ks), _ptr(vs), _ptr(cnt))
    n = C.c_size_t()
    _check("smallkv_store_workspace_size", lib().smallkv_store_workspace_size(C.byref(desc),
                                                                              C.byref(n)))
    ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device=dev)
    return StoreCall(desc, nk, nv, ks, vs, cnt, ws, (batch, head_map, crit_idx, marg_idx, full_k,
                                                     full_v, old))


def smallkv_store_update(desc: Store, ws, stream=None):
    w, wb = _ws(ws)
    _check("smallkv_store_update", lib().smallkv_store_update(C.byref(desc), w, wb,
                                                              _stream(stream)))
