"""ctypes front end of the CPU oracle (smallkv_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, by ``__graft_entry__.smoke()``
and by the CPU-baseline leg of ``bench.py``; the product path never imports
it.  It shares nothing with the HIP library or its binding.

Every array goes in as a contiguous numpy array (float32 for inputs that the
device holds as bf16 or fp32 -- bf16 widens to fp32 exactly -- int32 for
indices) and comes out as numpy arrays; floating-point outputs other than
the fp32 logits are float64.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "smallkv_oracle.c")
SRCS = [SRC, os.path.join(HERE, "match_oracle.c")]
LIB = os.path.join(HERE, "libsmallkv_oracle.so")

NORM_REMAINING, NORM_NONE, NORM_SLM_CRIT, NORM_RETAINED, NORM_MARG_FILL = range(5)
SELECT_HEAD, SELECT_GROUP, SELECT_ACCUM = 0, 1, 2
MODES = (NORM_REMAINING, NORM_NONE, NORM_SLM_CRIT, NORM_RETAINED, NORM_MARG_FILL)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math, no fp contraction)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call([
            "gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
            "-Wall", "-Wextra", "-fPIC", "-shared", *SRCS, "-o", tmp, "-lm"])
        os.replace(tmp, LIB)
    return LIB


_lib = None
_F = C.POINTER(C.c_float)
_D = C.POINTER(C.c_double)
_I = C.POINTER(C.c_int32)
_U8 = C.POINTER(C.c_uint8)


class StepIn(C.Structure):
    _fields_ = [
        ("batch", C.c_int32), ("n_cap", C.c_int32), ("kc_cap", C.c_int32), ("km_cap", C.c_int32),
        ("seq_len", _I), ("k_crit", _I), ("k_marg", _I), ("k_recent", _I),
        ("s_layers", C.c_int32), ("s_q_heads", C.c_int32), ("s_kv_heads", C.c_int32), ("s_dim", C.c_int32),
        ("s_scale", C.c_float),
        ("s_q", _F), ("s_k", _F), ("s_v", _F),
        ("s_rows", C.c_int64), ("s_held", _I), ("s_row_pos", _I),
        ("l_layers", C.c_int32), ("l_q_heads", C.c_int32), ("l_kv_heads", C.c_int32), ("l_dim", C.c_int32),
        ("l_scale", C.c_float),
        ("l_rows", C.c_int64),
        ("l_q", _F), ("l_k", _F), ("l_v", _F),
        ("k_slot", _I), ("v_slot", _I),
        ("head_map", _I),
        ("mode", C.c_int32),
        ("select", C.c_int32),
        ("acc", _F),
    ]


class Window(C.Structure):
    _fields_ = [("layers", C.c_int32), ("q_heads", C.c_int32), ("kv_heads", C.c_int32),
                ("dim", C.c_int32), ("scale", C.c_float), ("q", _F), ("k", _F)]


class MatchIn(C.Structure):
    _fields_ = [("batch", C.c_int32), ("w_cap", C.c_int32), ("win_len", _I), ("top_k", _I),
                ("large", Window), ("small", Window)]


class StoreIn(C.Structure):
    _fields_ = [("batch", C.c_int32), ("n_cap", C.c_int32), ("layers", C.c_int32),
                ("q_heads", C.c_int32), ("kv_heads", C.c_int32), ("dim", C.c_int32),
                ("select", C.c_int32), ("n_small_heads", C.c_int32), ("kc_cap", C.c_int32),
                ("km_cap", C.c_int32), ("rows", C.c_int64), ("seq_len", _I), ("head_map", _I),
                ("crit", _I), ("marg", _I), ("full_k", _F), ("full_v", _F), ("old_k", _F),
                ("old_v", _F), ("old_k_slot", _I), ("old_v_slot", _I)]


class StepOut(C.Structure):
    _fields_ = [
        ("logits", _F),
        ("row_max", _D), ("row_sum", _D), ("small_out", _D),
        ("crit", _I), ("marg", _I),
        ("marg_prob", _D), ("mass", _D), ("large_out", _D),
    ]


def lib():
    global _lib
    if _lib is None:
        hdr = os.path.join(HERE, "smallkv_oracle.h")
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < max(
                os.path.getmtime(f) for f in SRCS + [hdr]):
            build()
        L = C.CDLL(LIB)
        L.orc_logit.argtypes = [C.c_int, C.c_float, _F, _F]
        L.orc_logit.restype = C.c_float
        L.orc_key.argtypes = [C.c_float]
        L.orc_key.restype = C.c_uint32
        L.orc_small_head.argtypes = [C.c_int, C.c_int, C.c_float, _F, _F, _F, _F, _D, _D, _D]
        L.orc_partition.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, _F, C.c_double, C.c_double,
                                    _I, C.c_int, _I, _D, C.c_int, _D, C.POINTER(C.c_int),
                                    C.POINTER(C.c_int)]
        L.orc_hybrid_head.argtypes = [C.c_int, C.c_float, _F, _F, _F, _I, _I, C.c_int, _I,
                                      C.c_int, _I, _D, _D, C.c_int, _D]
        L.orc_step.argtypes = [C.POINTER(StepIn), C.POINTER(StepOut)]
        L.orc_exp.argtypes = [C.c_float]
        L.orc_exp.restype = C.c_float
        L.orc_exp_n.argtypes = [C.c_int, _F, _F]
        L.orc_exp_n.restype = None
        L.orc_match_scores.argtypes = [C.c_int, C.c_int, C.c_float, _F, _F, _F]
        L.orc_topk.argtypes = [C.c_int, C.c_int, _F, _U8]
        L.orc_jaccard.argtypes = [C.c_int, _U8, _U8, C.POINTER(C.c_int), C.POINTER(C.c_int)]
        L.orc_jaccard.restype = None
        L.orc_match.argtypes = [C.POINTER(MatchIn), _I, _F, _U8]
        L.orc_store_update.argtypes = [C.POINTER(StoreIn), _F, _F, _I, _I, _I]
        L.orc_store_update.restype = C.c_int
        L.orc_zq.argtypes = [C.c_int, _F, C.c_float]
        L.orc_zq.restype = C.c_float
        for f in (L.orc_small_head, L.orc_partition, L.orc_hybrid_head, L.orc_step,
                  L.orc_match_scores, L.orc_topk, L.orc_match):
            f.restype = C.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _p(a, t):
    return a.ctypes.data_as(t)


def _check(rc, what):
    if rc != 0:
        raise OracleError(f"{what} returned {rc}")


def logit(q, k, scale) -> np.float32:
    q, k = _f32(q), _f32(k)
    return np.float32(lib().orc_logit(q.size, C.c_float(scale), _p(q, _F), _p(k, _F)))


def key(s) -> int:
    return int(lib().orc_key(C.c_float(s)))


def small_head(q, K, V, scale):
    """Stage 1 for one small query head. Returns (logits f32[n], m, Z, O f64[d])."""
    q, K, V = _f32(q), _f32(K), _f32(V)
    n, d = K.shape
    logits = np.empty(n, np.float32)
    m, Z = C.c_double(), C.c_double()
    O = np.empty(d, np.float64)
    _check(lib().orc_small_head(n, d, C.c_float(scale), _p(q, _F), _p(K, _F), _p(V, _F),
                                _p(logits, _F), C.byref(m), C.byref(Z), _p(O, _D)), "orc_small_head")
    return logits, m.value, Z.value, O


def partition(logits, k_crit, k_marg, m, Z, kc_cap=None, km_cap=None, k_recent=0):
    """Stage 2 for one small head. Returns (crit, marg, marg_prob, mass) with -1 padding."""
    logits = _f32(logits)
    n = logits.size
    r_ = min(max(k_recent, 0), n)
    ntop_ = min(k_crit, n - r_)
    nc_ = ntop_ + r_
    nm_ = max(0, min(k_marg, n - nc_))
    kc_cap = nc_ if kc_cap is None else kc_cap
    km_cap = nm_ if km_cap is None else km_cap
    crit = np.empty(max(kc_cap, 1), np.int32)
    marg = np.empty(max(km_cap, 1), np.int32)
    mp = np.empty(max(km_cap, 1), np.float64)
    mass = np.empty(2, np.float64)
    nc, nm = C.c_int(), C.c_int()
    _check(lib().orc_partition(n, k_crit, k_marg, k_recent, _p(logits, _F), m, Z, _p(crit, _I), kc_cap,
                               _p(marg, _I), _p(mp, _D), km_cap, _p(mass, _D), C.byref(nc),
                               C.byref(nm)), "orc_partition")
    return crit[:kc_cap], marg[:km_cap], mp[:km_cap], mass


def hybrid_head(q, K, V, crit, marg, marg_prob, mass, scale, mode=NORM_REMAINING,
                k_slot=None, v_slot=None):
    """Stage 3 for one large query head (crit/marg may carry -1 padding)."""
    q, K, V = _f32(q), _f32(K), _f32(V)
    crit = _i32(np.asarray(crit)[np.asarray(crit) >= 0])
    marg = np.asarray(marg)
    keep = marg >= 0
    marg = _i32(marg[keep])
    mp = np.ascontiguousarray(np.asarray(marg_prob, np.float64)[keep])
    mass = np.ascontiguousarray(mass, np.float64)
    d = q.size
    O = np.empty(d, np.float64)
    ks = _i32(k_slot) if k_slot is not None else None
    vs = _i32(v_slot) if v_slot is not None else None
    _check(lib().orc_hybrid_head(d, C.c_float(scale), _p(q, _F), _p(K, _F), _p(V, _F),
                                 _p(ks, _I) if ks is not None else None,
                                 _p(vs, _I) if vs is not None else None,
                                 crit.size, _p(crit, _I), marg.size,
                                 _p(marg, _I) if marg.size else None,
                                 _p(mp, _D) if marg.size else None, _p(mass, _D), int(mode),
                                 _p(O, _D)), "orc_hybrid_head")
    return O


def step(*, seq_len, k_crit, k_marg, kc_cap, km_cap, head_map, mode,
         s_q, s_k, s_v, s_scale, l_q, l_k, l_v, l_scale, k_slot=None, v_slot=None,
         k_recent=None, s_held=None, s_row_pos=None, n_cap=None, select=SELECT_HEAD,
         acc=None):
    """A whole decode step over the library layout (see smallkv_oracle.h).

    select=SELECT_ACCUM: `acc` is a float32 array [B, l*Hqs, n_cap] (C-contiguous)
    updated in place: the running accumulated score of every small head.

    Shapes: s_q [B,l,Hqs,ds], s_k/s_v [B,l,Hks,n_cap,ds] (with the small
    model's own eviction: [B,l,Hks,s_rows,ds] plus s_held [B] and s_row_pos
    [B,l,Hks,s_rows], and n_cap given), l_q [B,L,Hq,d], l_k/l_v
    [B,L,Hk,n_rows,d], slots [B,L,Hk,n_cap] or None.
    """
    s_q, s_k, s_v, l_q, l_k, l_v = map(_f32, (s_q, s_k, s_v, l_q, l_k, l_v))
    if acc is not None and (acc.dtype != np.float32 or not acc.flags.c_contiguous):
        raise ValueError("acc must be a C-contiguous float32 array (updated in place)")
    seq_len, k_crit, k_marg, head_map = map(_i32, (seq_len, k_crit, k_marg, head_map))
    kr = _i32(k_recent) if k_recent is not None else None
    B, l, hqs, ds = s_q.shape
    hks, s_rows = s_k.shape[2], s_k.shape[3]
    held = _i32(s_held) if s_held is not None else None
    rpos = _i32(s_row_pos) if s_row_pos is not None else None
    ncap = s_rows if held is None else int(n_cap)
    _, L, hq, d = l_q.shape
    hk, nrows = l_k.shape[2], l_k.shape[3]
    ks = _i32(k_slot) if k_slot is not None else None
    vs = _i32(v_slot) if v_slot is not None else None
    nsh = l * hqs
    # group selection: lists per (large layer, kv head), weights per large head
    lrows, prows = (L * hk, L * hq) if select == SELECT_GROUP else (nsh, nsh)
    out = dict(
        logits=np.zeros((B, nsh, s_rows), np.float32),
        row_max=np.empty((B, nsh)), row_sum=np.empty((B, nsh)),
        small_out=np.empty((B, l, hqs, ds)),
        crit=np.empty((B, lrows, max(kc_cap, 1)), np.int32),
        marg=np.empty((B, lrows, max(km_cap, 1)), np.int32),
        marg_prob=np.empty((B, prows, max(km_cap, 1))),
        mass=np.empty((B, prows, 2)),
        large_out=np.empty((B, L, hq, d)),
    )
    si = StepIn(B, ncap, kc_cap, km_cap, _p(seq_len, _I), _p(k_crit, _I), _p(k_marg, _I),
                _p(kr, _I) if kr is not None else None,
                l, hqs, hks, ds, s_scale, _p(s_q, _F), _p(s_k, _F), _p(s_v, _F),
                s_rows, _p(held, _I) if held is not None else None,
                _p(rpos, _I) if rpos is not None else None,
                L, hq, hk, d, l_scale, nrows, _p(l_q, _F), _p(l_k, _F), _p(l_v, _F),
                _p(ks, _I) if ks is not None else None,
                _p(vs, _I) if vs is not None else None,
                _p(head_map, _I), int(mode), int(select),
                _p(acc, _F) if acc is not None else None)
    so = StepOut(_p(out["logits"], _F), _p(out["row_max"], _D), _p(out["row_sum"], _D),
                 _p(out["small_out"], _D), _p(out["crit"], _I), _p(out["marg"], _I),
                 _p(out["marg_prob"], _D), _p(out["mass"], _D), _p(out["large_out"], _D))
    _check(lib().orc_step(C.byref(si), C.byref(so)), "orc_step")
    out["crit"] = out["crit"][..., :kc_cap]
    out["marg"] = out["marg"][..., :km_cap]
    out["marg_prob"] = out["marg_prob"][..., :km_cap]
    return out


# ------------------------------------------------------- prefill matching --

def exp32(x):
    """orc_exp elementwise over a float32 array."""
    x = _f32(x)
    y = np.empty_like(x)
    lib().orc_exp_n(x.size, _p(x, _F), _p(y, _F))
    return y


def match_scores(Q, K, scale):
    """Eq. 1 column sums F [w] (float32) of one head's causal prefill attention."""
    Q, K = _f32(Q), _f32(K)
    w, d = Q.shape
    F = np.empty(w, np.float32)
    _check(lib().orc_match_scores(w, d, C.c_float(scale), _p(Q, _F), _p(K, _F), _p(F, _F)),
           "orc_match_scores")
    return F


def topk_set(F, k):
    """TopK of Eq. 2 as a bool array (ties to the lower index)."""
    F = _f32(F)
    t = np.empty(F.size, np.uint8)
    _check(lib().orc_topk(F.size, int(k), _p(F, _F), _p(t, _U8)), "orc_topk")
    return t.astype(bool)


def jaccard(a, b):
    """Eq. 2 as the integer pair (|A n B|, |A u B|)."""
    a = np.ascontiguousarray(a, np.uint8)
    b = np.ascontiguousarray(b, np.uint8)
    n, d = C.c_int(), C.c_int()
    lib().orc_jaccard(a.size, _p(a, _U8), _p(b, _U8), C.byref(n), C.byref(d))
    return n.value, d.value


def match(*, win_len, top_k, l_q, l_k, l_scale, s_q, s_k, s_scale):
    """Eq. 3 per sequence.  l_q [B,L,Hq,w_cap,d], l_k [B,L,Hk,w_cap,d] and the
    small model's likewise.  Returns (head_map [B,L*Hq] int32, scores
    [B,L*Hq+l*Hqs,w_cap] float32, top [B,L*Hq+l*Hqs,w_cap] bool); entries at
    or beyond a sequence's window are 0."""
    l_q, l_k, s_q, s_k = map(_f32, (l_q, l_k, s_q, s_k))
    win_len, top_k = _i32(win_len), _i32(top_k)
    B, L, hq, w_cap, d = l_q.shape
    hk = l_k.shape[2]
    _, l, hqs, _, ds = s_q.shape
    hks = s_k.shape[2]
    H = L * hq + l * hqs
    hm = np.empty((B, L * hq), np.int32)
    scores = np.zeros((B, H, w_cap), np.float32)
    top = np.zeros((B, H, w_cap), np.uint8)
    mi = MatchIn(B, w_cap, _p(win_len, _I), _p(top_k, _I),
                 Window(L, hq, hk, d, l_scale, _p(l_q, _F), _p(l_k, _F)),
                 Window(l, hqs, hks, ds, s_scale, _p(s_q, _F), _p(s_k, _F)))
    _check(lib().orc_match(C.byref(mi), _p(hm, _I), _p(scores, _F), _p(top, _U8)), "orc_match")
    return hm, scores, top.astype(bool)


def zq(logits, m) -> np.float32:
    """The group key's normaliser of one small head (orc_zq)."""
    lg = _f32(logits)
    return np.float32(lib().orc_zq(lg.size, _p(lg, _F), C.c_float(m)))


def store_update(*, seq_len, head_map, crit, marg, full_k, full_v, rows, n_small_heads,
                 select=SELECT_HEAD, old_k=None, old_v=None, old_k_slot=None, old_v_slot=None):
    """The compact store after a step (orc_store_update).  full_k/full_v
    [B,L,Hk,n_cap,d]; crit/marg as the step wrote them.  Returns (k [B,L,Hk,rows,d],
    v, k_slot [B,L,Hk,n_cap], v_slot, counts [B,L,Hk,2]); rows past a unit's
    count and slot entries at or past its sequence length are left as -1 / 0."""
    full_k, full_v = _f32(full_k), _f32(full_v)
    seq_len, head_map, crit, marg = map(_i32, (seq_len, head_map, crit, marg))
    B, L, hk, ncap, d = full_k.shape
    hq = head_map.size // L
    nk = np.zeros((B, L, hk, rows, d), np.float32)
    nv = np.zeros_like(nk)
    ks = np.full((B, L, hk, ncap), -1, np.int32)
    vs = np.full_like(ks, -1)
    cnt = np.zeros((B, L, hk, 2), np.int32)
    ok, ov = (_f32(old_k), _f32(old_v)) if old_k is not None else (None, None)
    oks, ovs = (_i32(old_k_slot), _i32(old_v_slot)) if old_k_slot is not None else (None, None)
    si = StoreIn(B, ncap, L, hq, hk, d, int(select), int(n_small_heads), crit.shape[-1],
                 marg.shape[-1], int(rows), _p(seq_len, _I), _p(head_map, _I), _p(crit, _I),
                 _p(marg, _I), _p(full_k, _F), _p(full_v, _F),
                 _p(ok, _F) if ok is not None else None, _p(ov, _F) if ov is not None else None,
                 _p(oks, _I) if oks is not None else None, _p(ovs, _I) if ovs is not None else None)
    _check(lib().orc_store_update(C.byref(si), _p(nk, _F), _p(nv, _F), _p(ks, _I), _p(vs, _I),
                                  _p(cnt, _I)), "orc_store_update")
    return nk, nv, ks, vs, cnt
