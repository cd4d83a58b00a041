"""Parity helpers: run the oracle on host copies of the exact device bytes and
compare with the library's outputs.

Tolerances (per head vector, ||gpu - ref||_inf <= tol * ||ref||_inf):
fp32 workloads 1e-5, bf16 workloads 2e-2.  Index lists and logits must be
bit-identical; row_max is exact (the max of identical fp32 logits).
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle as O

TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}


def host(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy()


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def oracle_step(x: dict, mode: int, k_slot=None, v_slot=None, l_k=None, l_v=None):
    """The oracle's whole step on host copies of the inputs in `x`."""
    from paper_2508_02751_amd.pipeline import softmax_scale
    l_k = x["l_k"] if l_k is None else l_k
    l_v = x["l_v"] if l_v is None else l_v
    return O.step(
        seq_len=host(x["seq_len"]), k_crit=host(x["k_crit"]), k_marg=host(x["k_marg"]),
        kc_cap=int(x["kc_cap"]), km_cap=int(x["km_cap"]), head_map=host(x["head_map"]),
        mode=mode, s_q=host(x["s_q"]), s_k=host(x["s_k"]), s_v=host(x["s_v"]),
        s_scale=softmax_scale(x["s_q"].shape[-1]), l_q=host(x["l_q"]), l_k=host(l_k),
        l_v=host(l_v), l_scale=softmax_scale(x["l_q"].shape[-1]),
        k_slot=None if k_slot is None else host(k_slot),
        v_slot=None if v_slot is None else host(v_slot),
        k_recent=host(x["k_recent"]) if x.get("k_recent") is not None else None,
        s_held=host(x["s_held"]) if x.get("s_held") is not None else None,
        s_row_pos=host(x["s_row_pos"]) if x.get("s_row_pos") is not None else None,
        n_cap=x.get("n_cap"), select=x.get("select", 0))


def head_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max over heads of ||got - ref||_inf / ||ref||_inf (last axis = head dim)."""
    num = np.abs(got.astype(np.float64) - ref).max(-1)
    den = np.maximum(np.abs(ref).max(-1), 1e-30)
    return float((num / den).max())


def compare_step(buf, ref: dict, x: dict, dtype, what: str = "", check_logits=True):
    """Assert parity of every output of one step; returns a dict of error figures."""
    tol = TOL[dtype]
    seq = host(x["seq_len"]).astype(np.int64)
    B = seq.size
    lg = host(buf.logits)
    if x.get("s_held") is not None:
        # stages 1-2 ran over the small model's held rows: logits rows have
        # stride n_rows and entry r is held row r
        seq = host(x["s_held"]).astype(np.int64)
        rows = ref["logits"].shape[-1]
        lg = lg.reshape(-1)[: B * lg.shape[1] * rows].reshape(B, lg.shape[1], rows)
    if check_logits:
        for b in range(B):
            n = seq[b]
            bad = (lg[b, :, :n].view(np.uint32) != ref["logits"][b, :, :n].view(np.uint32))
            assert not bad.any(), f"{what}: {int(bad.sum())} logits differ in sequence {b}"
    rm = host(buf.row_max)
    assert np.array_equal(rm, ref["row_max"].astype(np.float32)), f"{what}: row_max differs"
    rs = host(buf.row_sum)
    np.testing.assert_allclose(rs, ref["row_sum"], rtol=1e-5, err_msg=f"{what}: row_sum")
    crit = host(buf.crit_idx)[..., : ref["crit"].shape[-1]]
    assert np.array_equal(crit, ref["crit"]), f"{what}: critical index lists differ"
    km = ref["marg"].shape[-1]
    if km:
        marg = host(buf.marg_idx)[..., :km]
        assert np.array_equal(marg, ref["marg"]), f"{what}: marginal index lists differ"
        mp = host(buf.marg_prob)[..., :km]
        np.testing.assert_allclose(mp, ref["marg_prob"], rtol=2e-5, atol=1e-9,
                                   err_msg=f"{what}: marg_prob")
    np.testing.assert_allclose(host(buf.mass), ref["mass"], rtol=2e-5, atol=2e-7,
                               err_msg=f"{what}: mass")
    es = head_err(host(buf.small_out), ref["small_out"])
    el = head_err(host(buf.large_out), ref["large_out"])
    assert es <= tol, f"{what}: small-model output error {es:.3g} > {tol}"
    assert el <= tol, f"{what}: large-model output error {el:.3g} > {tol}"
    return {"small_out_err": es, "large_out_err": el}


# ------------------------------------------------- sampled (full-size) checks --

def oracle_small_row(x, b: int, j: int):
    """Oracle stages 1-2 for one small row (b, j) from host copies of its slices."""
    from paper_2508_02751_amd.pipeline import softmax_scale
    s_q, s_k, s_v = x["s_q"], x["s_k"], x["s_v"]
    hqs, hks, ds = s_q.shape[2], s_k.shape[2], s_q.shape[3]
    layer, h = divmod(j, hqs)
    g = h // (hqs // hks)
    n = int(x["seq_len"][b])
    lg, m, Z, out = O.small_head(host(s_q[b, layer, h]), host(s_k[b, layer, g, :n]),
                                 host(s_v[b, layer, g, :n]), softmax_scale(ds))
    kc, km = int(x["k_crit"][b]), int(x["k_marg"][b])
    kr = int(x["k_recent"][b]) if x.get("k_recent") is not None else 0
    crit, marg, mp, mass = O.partition(lg, kc, km, m, Z, kc_cap=int(x["kc_cap"]),
                                       km_cap=int(x["km_cap"]), k_recent=kr)
    return dict(logits=lg, m=m, Z=Z, out=out, crit=crit, marg=marg, marg_prob=mp, mass=mass)


def check_small_row(buf, x, b, j, ref, tol, what=""):
    n = int(x["seq_len"][b])
    nsh = buf.logits.shape[1]
    hqs = x["s_q"].shape[2]
    layer, h = divmod(j, hqs)
    got = host(buf.logits[b, j, :n])
    assert np.array_equal(got.view(np.uint32), ref["logits"].view(np.uint32)), f"{what}: logits ({b},{j})"
    assert np.float32(ref["m"]) == host(buf.row_max[b, j]), f"{what}: row_max ({b},{j})"
    np.testing.assert_allclose(host(buf.row_sum[b, j]), ref["Z"], rtol=1e-5)
    assert np.array_equal(host(buf.crit_idx[b, j]), ref["crit"]), f"{what}: crit ({b},{j})"
    km = ref["marg"].shape[0]
    if km:
        assert np.array_equal(host(buf.marg_idx[b, j, :km]), ref["marg"]), f"{what}: marg ({b},{j})"
        np.testing.assert_allclose(host(buf.marg_prob[b, j, :km]), ref["marg_prob"], rtol=2e-5, atol=1e-9)
    np.testing.assert_allclose(host(buf.mass[b, j]), ref["mass"], rtol=2e-5, atol=2e-7)
    e = head_err(host(buf.small_out[b, layer, h])[None], ref["out"][None])
    assert e <= tol, f"{what}: small output ({b},{j}) error {e}"
    assert nsh == x["s_q"].shape[1] * hqs


def oracle_large_head(x, b, layer, h, part, mode, l_k=None, l_v=None, k_slot=None, v_slot=None):
    """Oracle stage 3 for one large head, given the oracle's partition of its small head."""
    from paper_2508_02751_amd.pipeline import softmax_scale
    l_q = x["l_q"]
    l_k = x["l_k"] if l_k is None else l_k
    l_v = x["l_v"] if l_v is None else l_v
    hq, hk, d = l_q.shape[2], l_k.shape[2], l_q.shape[3]
    g = h // (hq // hk)
    ks = None if k_slot is None else host(k_slot[b, layer, g])
    vs = None if v_slot is None else host(v_slot[b, layer, g])
    return O.hybrid_head(host(l_q[b, layer, h]), host(l_k[b, layer, g]), host(l_v[b, layer, g]),
                         part["crit"], part["marg"], part["marg_prob"], part["mass"],
                         softmax_scale(d), mode, k_slot=ks, v_slot=vs)
