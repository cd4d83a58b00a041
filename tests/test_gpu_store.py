"""GPU parity of the retained-store maintenance (smallkv_store_update)
against the oracle: slot maps, union sizes and every stored row bit for bit."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle as O
from parity import TOL, head_err, host, log

pytestmark = pytest.mark.gpu

DEV = "cuda"


def modules():
    from paper_2508_02751_amd import smallkv as S
    from paper_2508_02751_amd import workloads as W
    from paper_2508_02751_amd.pipeline import prepare_step
    return S, W, prepare_step


def workload(name, wid, dtype="bf16", steps=1, select=0, batch=2, n=1500):
    _, W, _ = modules()
    return W.Workload(wid, name, batch, n, dtype, W.ModelShape(2, 8, 2, 64),
                      W.ModelShape(2, 8, 2, 128), ("pct", 8), ("pct", 15), ragged_min=500,
                      steps=steps, select=select)


def capacity(x, g):
    return min(x["l_k"].shape[3], g * (int(x["kc_cap"]) + int(x["km_cap"])))


def oracle_lists(x, ps, select):
    """The oracle's own step on the same inputs: its critical and marginal
    lists, which must equal the library's (the store's expected rows are
    built from the oracle's lists, not from the GPU's)."""
    from parity import oracle_step
    xs = dict(x)
    xs["select"] = select
    ref = oracle_step(xs, 0)
    crit, marg = ref["crit"], ref["marg"]
    assert np.array_equal(host(ps.buf.crit_idx)[..., : crit.shape[-1]], crit), "critical lists"
    if marg.shape[-1]:
        assert np.array_equal(host(ps.buf.marg_idx)[..., : marg.shape[-1]], marg), "marginal lists"
    return crit, marg


def oracle_store(x, ps, rows, select, old=None):
    """The oracle's store after this step: from its own lists and, when given,
    its own previous store `old` (a tuple as this function returns)."""
    crit, marg = oracle_lists(x, ps, select)
    kw = {}
    if old is not None:
        kw = dict(old_k=old[0], old_v=old[1], old_k_slot=old[2], old_v_slot=old[3])
    return O.store_update(seq_len=host(x["seq_len"]), head_map=host(x["head_map"]),
                          crit=crit, marg=marg if marg.shape[-1] else np.full(
                              crit.shape[:-1] + (1,), -1, np.int32),
                          full_k=host(x["l_k"]), full_v=host(x["l_v"]), rows=rows,
                          n_small_heads=ps.buf.logits.shape[1],
                          select=O.SELECT_GROUP if select == 1 else O.SELECT_HEAD, **kw)


def check_store(sc, ref, x, what):
    nk, nv, ks, vs, cnt = ref
    got_cnt = host(sc.counts)
    assert np.array_equal(got_cnt, cnt), f"{what}: union sizes differ"
    gks, gvs = host(sc.k_slot), host(sc.v_slot)
    gk, gv = host(sc.new_k), host(sc.new_v)
    seq = host(x["seq_len"])
    rows = nk.shape[3]
    B, L, hk = cnt.shape[:3]
    for b in range(B):
        n = int(seq[b])
        assert np.array_equal(gks[b, ..., :n], ks[b, ..., :n]), f"{what}: K slot maps differ"
        assert np.array_equal(gvs[b, ..., :n], vs[b, ..., :n]), f"{what}: V slot maps differ"
        for li in range(L):
            for g in range(hk):
                ck, cv = min(rows, cnt[b, li, g, 0]), min(rows, cnt[b, li, g, 1])
                assert np.array_equal(gk[b, li, g, :ck].view(np.uint32), nk[b, li, g, :ck].view(np.uint32))
                assert np.array_equal(gv[b, li, g, :cv].view(np.uint32), nv[b, li, g, :cv].view(np.uint32))


@pytest.mark.parametrize("select,dtype", [(0, "bf16"), (1, "bf16"), (0, "f32")])
def test_store_from_a_step(select, dtype):
    S, W, prepare_step = modules()
    w = workload(f"store{select}{dtype}", 131 + select, dtype, select=select)
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    rows = capacity(x, 4)
    sc = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                         ps.buf.marg_idx, x["l_k"], x["l_v"], rows, select)
    log(f"[store] select={select} {dtype}: {rows} rows per kv head")
    sc.run()
    torch.cuda.synchronize()
    check_store(sc, oracle_store(x, ps, rows, select), x, f"store select={select} {dtype}")


def test_store_reuses_the_previous_store_across_steps():
    """Two drifting steps; the previous store (the library's and, separately,
    the oracle's) is altered so that the source of every row (old store or
    full store) shows in the result."""
    S, W, prepare_step = modules()
    w = workload("store-steps", 134, steps=2)
    x0 = W.make_step_inputs(w, DEV, 0)
    ps = prepare_step(x0)
    ps.run()
    rows = capacity(x0, 4)
    old = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                          ps.buf.marg_idx, x0["l_k"], x0["l_v"], rows)
    old.run()
    torch.cuda.synchronize()
    ref0 = oracle_store(x0, ps, rows, 0)
    check_store(old, ref0, x0, "first store")
    old.new_k += 1.0
    old.new_v -= 1.0

    def shifted(a, by):  # the same change in the store's dtype (rounded as the library's store is)
        return (torch.from_numpy(a).to(old.new_k.dtype) + by).float().numpy()

    ref0 = (shifted(ref0[0], 1.0), shifted(ref0[1], -1.0)) + ref0[2:]
    x1 = W.make_step_inputs(w, DEV, 1)
    ps.with_query(x1["s_q"], x1["l_q"], x1["seq_len"], x1["k_crit"], x1["k_marg"])
    ps.run()
    sc = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                         ps.buf.marg_idx, x1["l_k"], x1["l_v"], rows, old=old)
    sc.run()
    torch.cuda.synchronize()
    ref = oracle_store(x1, ps, rows, 0, old=ref0)
    check_store(sc, ref, x1, "store from the previous store")
    reused = int(((ref[2] >= 0) & (ref0[2] >= 0)).sum())
    log(f"[store] {reused} K rows reused from the previous store")
    assert reused > 0


def test_store_overflow_keeps_the_first_rows():
    S, W, prepare_step = modules()
    w = workload("store-small", 135)
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    sc = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                         ps.buf.marg_idx, x["l_k"], x["l_v"], 64)
    sc.run()
    torch.cuda.synchronize()
    ref = oracle_store(x, ps, 64, 0)
    assert (ref[4][..., 1] > 64).any()
    check_store(sc, ref, x, "store past capacity")


def test_stage3_through_the_built_store_matches_the_full_cache():
    S, W, prepare_step = modules()
    w = workload("store-stage3", 136)
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    rows = capacity(x, 4)
    sc = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                         ps.buf.marg_idx, x["l_k"], x["l_v"], rows)
    sc.run()
    large = S.ModelSpec(ps.large.q, sc.new_k, sc.new_v, torch.empty_like(ps.large.out),
                        ps.large.scale, sc.k_slot, sc.v_slot)
    b = ps.buf
    S.smallkv_hybrid_attn(ps.batch, large, ps.head_map, b.logits.shape[1], b.crit_idx, b.marg_idx,
                          b.marg_prob, b.mass, ws=b.ws)
    torch.cuda.synchronize()
    err = head_err(host(large.out), host(b.large_out).astype(np.float64))
    log(f"[store] stage 3 through the store vs the full cache: {err:.3g}")
    assert err <= TOL[torch.bfloat16]
    # and against the oracle's step through the oracle's own store
    from parity import oracle_step
    nk, nv, ks, vs, _ = oracle_store(x, ps, rows, 0)
    ref = oracle_step(x, 0, k_slot=torch.from_numpy(ks), v_slot=torch.from_numpy(vs),
                      l_k=torch.from_numpy(nk), l_v=torch.from_numpy(nv))
    err = head_err(host(large.out), ref["large_out"])
    log(f"[store] stage 3 through the store vs the oracle through its store: {err:.3g}")
    assert err <= TOL[torch.bfloat16]


def test_store_from_pinned_host_memory():
    """The full store in pinned host memory: a rebuild and the update after a
    drifted step read it over the host link and equal the oracle (and the
    same calls over the full store in HBM)."""
    S, W, prepare_step = modules()
    w = workload("store-host", 137, steps=2)
    x0 = W.make_step_inputs(w, DEV, 0)
    ps = prepare_step(x0)
    ps.run()
    rows = capacity(x0, 4)
    hk, hv = x0["l_k"].cpu().pin_memory(), x0["l_v"].cpu().pin_memory()
    assert hk.is_pinned() and hv.is_pinned()
    log("[store] full store in pinned host memory: rebuild")
    old = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                          ps.buf.marg_idx, hk, hv, rows)
    old.run()
    torch.cuda.synchronize()
    assert old.new_k.is_cuda
    ref0 = oracle_store(x0, ps, rows, 0)
    check_store(old, ref0, x0, "rebuild from host memory")
    x1 = W.make_step_inputs(w, DEV, 1)
    ps.with_query(x1["s_q"], x1["l_q"], x1["seq_len"], x1["k_crit"], x1["k_marg"])
    ps.run()
    log("[store] full store in pinned host memory: update after a drifted step")
    inc = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                          ps.buf.marg_idx, hk, hv, rows, old=old)
    inc.run()
    dev_inc = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                              ps.buf.marg_idx, x1["l_k"], x1["l_v"], rows, old=old)
    dev_inc.run()
    torch.cuda.synchronize()
    check_store(inc, oracle_store(x1, ps, rows, 0, old=ref0), x1, "update from host memory")
    for a, b in ((inc.new_k, dev_inc.new_k), (inc.new_v, dev_inc.new_v),
                 (inc.k_slot, dev_inc.k_slot), (inc.v_slot, dev_inc.v_slot)):
        assert torch.equal(a, b)


def test_store_rejects_pageable_host_memory():
    S, W, prepare_step = modules()
    w = workload("store-pageable", 138)
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    torch.cuda.synchronize()
    hk, hv = x["l_k"].cpu(), x["l_v"].cpu()
    assert not hk.is_pinned()
    sc = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                         ps.buf.marg_idx, hk, hv, capacity(x, 4))
    with pytest.raises(S.SmallKVError) as e:
        sc.run()
    assert e.value.status == S.EINVAL
    assert not sc.counts.any(), "nothing may run after the rejection"


def test_steps_through_a_host_backed_store():
    """Three drifting steps, each maintaining the store from the previous one
    and the full store in pinned host memory, then running stage 3 through
    it: every step equals stage 3 over the full cache."""
    S, W, prepare_step = modules()
    w = workload("store-steps-host", 139, steps=3)
    x = W.make_step_inputs(w, DEV, 0)
    ps = prepare_step(x)
    rows = capacity(x, 4)
    hk, hv = x["l_k"].cpu().pin_memory(), x["l_v"].cpu().pin_memory()
    old = ref_old = None
    for t in range(3):
        xt = x
        if t:
            xt = W.make_step_inputs(w, DEV, t)
            ps.with_query(xt["s_q"], xt["l_q"], xt["seq_len"], xt["k_crit"], xt["k_marg"])
        ps.run()
        sc = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                             ps.buf.marg_idx, hk, hv, rows, old=old)
        sc.run()
        large = S.ModelSpec(ps.large.q, sc.new_k, sc.new_v, torch.empty_like(ps.large.out),
                            ps.large.scale, sc.k_slot, sc.v_slot)
        b = ps.buf
        S.smallkv_hybrid_attn(ps.batch, large, ps.head_map, b.logits.shape[1], b.crit_idx,
                              b.marg_idx, b.marg_prob, b.mass, ws=b.ws)
        torch.cuda.synchronize()
        err = head_err(host(large.out), host(b.large_out).astype(np.float64))
        log(f"[store] step {t}: stage 3 through the host-backed store vs the full cache: {err:.3g}")
        assert err <= TOL[torch.bfloat16]
        ref = oracle_store(xt, ps, rows, 0, old=ref_old)
        check_store(sc, ref, xt, f"host-backed store, step {t}")
        old, ref_old = sc, ref


def test_store_at_the_largest_n_cap():
    """n_cap = 131072, the largest the store accepts (the index kernel's LDS
    bitmaps and word ranks at their largest): one sequence at full length."""
    S, W, prepare_step = modules()
    w = W.Workload(140, "store-max", 1, 131072, "bf16", W.ModelShape(1, 2, 1, 64),
                   W.ModelShape(1, 8, 2, 128), ("pct", 5), ("pct", 10))
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    rows = capacity(x, 4)
    log(f"[store] n_cap 131072: {rows} rows per kv head")
    sc = S.prepare_store(ps.batch, ps.head_map, ps.buf.logits.shape[1], ps.buf.crit_idx,
                         ps.buf.marg_idx, x["l_k"], x["l_v"], rows)
    sc.run()
    torch.cuda.synchronize()
    check_store(sc, oracle_store(x, ps, rows, 0), x, "store at n_cap 131072")
