"""GPU parity: the library (through the C ABI) against the CPU oracle on the
same seeded inputs.  Index sets and logits bit-exact, outputs within the
per-dtype tolerance of tests/parity.py."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
from parity import compare_step, host, log, oracle_step
from paper_2508_02751_amd import smallkv as S
from paper_2508_02751_amd import workloads as W
from paper_2508_02751_amd.pipeline import prepare_step

pytestmark = pytest.mark.gpu

DEV = "cuda"


def run_case(w, mode=S.NORM_REMAINING, mutate=None, step=0, what=None):
    what = what or w.name
    log(f"[parity] {what} mode={mode}")
    x = W.make_step_inputs(w, DEV, step)
    if mutate is not None:
        mutate(x)
    ps = prepare_step(x, mode)
    ps.run()
    torch.cuda.synchronize()
    ref = oracle_step(x, mode)
    errs = compare_step(ps.buf, ref, x, w.torch_dtype, what)
    log(f"[parity] {what} ok {errs}")
    return ps, x, ref


def custom(name, wid, batch, n, dtype, small, large, crit, marg, **kw):
    return W.Workload(wid, name, batch, n, dtype, small, large, crit, marg, **kw)


# ---------------------------------------------------------------- configs --

@pytest.mark.parametrize("mode", O.MODES)
def test_config1_tiny_f32_all_modes(mode):
    run_case(W.WORKLOADS[1], mode)


def test_config2_qwen2_7b_full_step():
    run_case(W.WORKLOADS[2])


# ------------------------------------------------------------- edge cases --

SMALL = W.ModelShape(2, 8, 2, 64)
LARGE = W.ModelShape(3, 12, 4, 128)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ragged_lengths_and_budget_clamps(dtype):
    """Lengths from 1 to n_cap; budgets above some lengths (|C| = N, M empty)."""
    w = custom(f"ragged-{dtype}", 101, 5, 700, dtype, SMALL, LARGE, ("abs", 40), ("abs", 70),
               ragged_min=1)
    run_case(w)


def test_single_token_sequences():
    w = custom("n1", 102, 3, 1, "bf16", SMALL, LARGE, ("abs", 4), ("abs", 4))
    run_case(w)


def test_no_marginal_budget():
    w = custom("km0", 103, 2, 513, "bf16", SMALL, LARGE, ("abs", 33), ("abs", 0))
    run_case(w)


def test_everything_critical():
    w = custom("all-crit", 104, 2, 300, "f32", SMALL, LARGE, ("abs", 300), ("abs", 50))
    run_case(w)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ties_from_duplicated_keys(dtype):
    """Duplicated small-model key rows give equal logits; the lower index wins."""
    w = custom(f"ties-{dtype}", 105, 2, 1500, dtype, SMALL, LARGE, ("pct", 10), ("pct", 25))

    def dup(x):
        k = x["s_k"]
        src = torch.arange(k.shape[3], device=k.device)
        src = torch.where(src % 3 == 0, (src * 7 + 1) % k.shape[3], src)
        x["s_k"] = k[:, :, :, src].contiguous()

    run_case(w, mutate=dup)


@pytest.mark.parametrize("n", [1500, 3000])
def test_constant_logits(n):
    """Every small key equal, so every logit of a row ties: the lowest indices
    fill C, then M.  One sub-bin holds the whole row, which sends the select
    to its general path (candidates in LDS up to 2048 keys at this row
    width, else the row)."""
    w = custom(f"const-{n}", 115, 2, n, "bf16", SMALL, LARGE, ("pct", 10), ("pct", 25))
    run_case(w, mutate=flat_small_keys)


def flat_small_keys(x):
    k = x["s_k"]
    x["s_k"] = k[:, :, :, :1].expand_as(k).contiguous()


@pytest.mark.parametrize("n", [800, 3000, 6000])
def test_constant_logits_many_rows(n):
    """The same ties over 1024 rows, so 256 threads per row: register rows
    keep up to 2048 candidate keys in LDS (the whole-row bin is ranked there
    at 800 tokens, over the row at 3000), rows re-read per pass (six per CU)
    up to 512 (over the row at 6000)."""
    small = W.ModelShape(4, 16, 4, 64)
    w = custom(f"const-many-{n}", 117, 16, n, "bf16", small, LARGE, ("pct", 10), ("pct", 25))
    run_case(w, mutate=flat_small_keys)


def test_tied_block_in_long_rows():
    """Long 256-thread rows (6000 tokens, re-read per pass) where 401 tokens
    share one key: in the rows whose target falls in that tie, its bin holds
    between 256 and 512 keys and is ranked in LDS; in the others the targets
    are counted or ranked as usual."""
    small = W.ModelShape(4, 16, 4, 64)
    w = custom("tied-block-6000", 118, 16, 6000, "bf16", small, LARGE, ("pct", 10), ("pct", 25))

    def tie(x):
        k = x["s_k"].clone()
        k[:, :, :, 1:401] = k[:, :, :, :1]
        x["s_k"] = k

    run_case(w, mutate=tie)


@pytest.mark.parametrize("n", [1500, 3000])
def test_targets_far_below_the_max(n):
    """Token 0's key points along its group's queries, 20x scaled: every other
    logit is far more than 32 below the row max, so both targets sit in the
    lowest, unrefined bin."""
    w = custom(f"far-{n}", 116, 2, n, "bf16", SMALL, LARGE, ("pct", 10), ("pct", 25))

    def spike(x):
        q = x["s_q"].float()
        B, l, hq, d = q.shape
        hk = x["s_k"].shape[2]
        qg = q.view(B, l, hk, hq // hk, d).mean(3)
        k = x["s_k"].clone()
        k[:, :, :, 0] = (20.0 * qg).to(k.dtype)
        x["s_k"] = k

    run_case(w, mutate=spike)


# ------------------------------------------------------ recent tokens --
# The experimental setup's 2 : 1 : 2 split of the budget between critical,
# recent and marginal tokens: the last r tokens are critical unranked.

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_recent_window_ragged(dtype):
    """Ragged lengths from 1; sequences shorter than the recent budget keep
    every token critical and rank none."""
    w = custom(f"recent-{dtype}", 117, 5, 700, dtype, SMALL, LARGE, ("abs", 40), ("abs", 60),
               ragged_min=1, recent=("abs", 20))
    run_case(w)


def test_recent_window_qwen2_7b_full_step():
    """The Qwen2-7B + 0.5B step with the paper's 20% example budget: 10%
    critical, 5% recent, 10% marginal."""
    run_case(W.WORKLOADS[6])


def test_early_stopped_small_model_full_step():
    """The Qwen2-7B step with the small model stopped after 20 of its 24
    layers: stages 1-2 run over 20 layers and the head map ranges over their
    280 heads."""
    w = W.WORKLOADS[7]
    assert w.small.layers == 20 and int(W.head_map(w, "cpu").max()) < 20 * 14
    run_case(w)


def test_evicted_small_cache_full_step():
    """The Qwen2-7B step with the small model's own cache compressed to 40%
    of the tokens: stages 1-2 run over the held rows, the lists name their
    positions and never a token the small model dropped."""
    ps, x, ref = run_case(W.WORKLOADS[8])
    pos = host(x["s_row_pos"])
    crit = host(ps.buf.crit_idx)
    held_any = set(pos[pos >= 0].tolist())
    assert set(crit[crit >= 0].tolist()) <= held_any


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_evicted_small_cache_ragged_with_recent(dtype):
    """Ragged lengths, recent tokens and several kv heads with different
    held sets; the grouped and the per-head stage 3 both read positions."""
    w = custom("slm-evict", 121, 3, 3000, dtype, W.ModelShape(2, 8, 2, 64),
               W.ModelShape(2, 8, 2, 128), ("pct", 8), ("pct", 12), ragged_min=700,
               recent=("pct", 3), slm_keep=45)
    run_case(w)


def test_recent_window_with_ties():
    w = custom("recent-ties", 120, 2, 1500, "bf16", SMALL, LARGE, ("pct", 10), ("pct", 25),
               recent=("pct", 5))

    def dup(x):
        k = x["s_k"]
        src = torch.arange(k.shape[3], device=k.device)
        src = torch.where(src % 3 == 0, (src * 7 + 1) % k.shape[3], src)
        x["s_k"] = k[:, :, :, src].contiguous()

    run_case(w, mutate=dup)


def test_recent_window_long_rows_and_many_rows():
    """Rows re-read from memory per pass, and rows of 256 threads (1024 rows)."""
    run_case(custom("recent-long", 118, 1, 20000, "bf16", W.ModelShape(1, 4, 1, 64),
                    W.ModelShape(1, 8, 2, 128), ("pct", 5), ("pct", 15), recent=("pct", 3)))
    run_case(custom("recent-many", 119, 16, 1500, "bf16", W.ModelShape(4, 16, 4, 64),
                    W.ModelShape(2, 8, 2, 128), ("pct", 10), ("pct", 20), ragged_min=200,
                    recent=("abs", 64)))


@pytest.mark.parametrize("sd,ld", [(128, 64), (128, 128), (64, 64)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_head_dims(sd, ld, dtype):
    w = custom(f"dims-{sd}-{ld}-{dtype}", 106, 2, 600, dtype, W.ModelShape(2, 4, 1, sd),
               W.ModelShape(2, 8, 2, ld), ("abs", 50), ("abs", 120), ragged_min=200)
    run_case(w)


@pytest.mark.parametrize("g", [1, 3, 5, 16])
def test_small_group_sizes(g):
    w = custom(f"group{g}", 107, 2, 900, "bf16", W.ModelShape(2, g * 2, 2, 64),
               W.ModelShape(2, 8, 8, 128), ("abs", 90), ("abs", 100))
    run_case(w)


@pytest.mark.parametrize("mode", O.MODES)
def test_bf16_all_modes_group8(mode):
    """Every normalisation mode on the grouped bf16 stage 3 (8 query heads per kv head)."""
    w = custom("modes-g8", 111, 2, 1500, "bf16", SMALL, W.ModelShape(2, 16, 2, 128),
               ("pct", 8), ("pct", 20), ragged_min=700)
    run_case(w, mode)


@pytest.mark.parametrize("g", [2, 4, 7, 8, 16])
def test_large_group_sizes(g):
    """Large-model query groups: up to 8 share one workgroup, 16 runs per head."""
    w = custom(f"lgroup{g}", 112, 2, 1100, "bf16", SMALL, W.ModelShape(2, 2 * g, 2, 128),
               ("pct", 10), ("pct", 25), ragged_min=300)
    run_case(w)


def test_many_rows_narrow_partition():
    """1024 small-head rows: the partition runs 256 threads per row."""
    w = custom("many-rows", 113, 16, 1500, "bf16", W.ModelShape(4, 16, 4, 64),
               W.ModelShape(2, 8, 2, 128), ("pct", 10), ("pct", 20), ragged_min=200)
    run_case(w)


def test_multi_tile_chunks_prefetch():
    """1024 small kv-head units: stage 1 gives each workgroup two 256-token
    tiles and prefetches the second tile's K while the first computes."""
    w = custom("multi-tile", 114, 16, 2048, "bf16", W.ModelShape(8, 8, 8, 64),
               W.ModelShape(1, 8, 2, 128), ("pct", 10), ("pct", 20), ragged_min=700)
    run_case(w)


def test_long_rows_multi_chunk():
    """Rows long enough to need several chunks per unit and several radix bins."""
    w = custom("long", 108, 1, 40000, "bf16", W.ModelShape(1, 4, 1, 64),
               W.ModelShape(1, 8, 2, 128), ("pct", 5), ("pct", 15))
    run_case(w)


def test_long_rows_reread_per_pass():
    """Rows too long for registers, re-read from memory per pass: 256 threads
    per row (1024 rows, ragged lengths up to 7000), and 512 threads per row
    (few rows of 12 000 tokens) with every logit of a row tied, so that the
    target bins overflow the candidate buffer and the radix passes run over
    the row."""
    run_case(custom("reread-many", 121, 8, 7000, "bf16", W.ModelShape(4, 32, 4, 64),
                    W.ModelShape(2, 8, 2, 128), ("pct", 10), ("pct", 20), ragged_min=5200))

    def flat(x):
        x["s_q"].zero_()

    run_case(custom("reread-ties", 122, 2, 12000, "bf16", W.ModelShape(1, 4, 1, 64),
                    W.ModelShape(1, 8, 2, 128), ("pct", 10), ("pct", 20)), mutate=flat)


def test_more_than_65535_tied_logits():
    """A 70 000-token row whose logits all tie (zero queries): every token's
    rank among the ties is its index, past 2^16 for the last tokens, so the
    tie ranks must not be kept in 16 bits anywhere."""
    def flat(x):
        x["s_q"].zero_()

    run_case(custom("ties-70k", 123, 1, 70000, "bf16", W.ModelShape(1, 2, 1, 64),
                    W.ModelShape(1, 4, 1, 128), ("pct", 10), ("pct", 20)), mutate=flat)


def test_deterministic_repeat():
    w = W.WORKLOADS[1]
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    torch.cuda.synchronize()
    # every output buffer the step has (the running-score state exists only
    # with accumulated scores)
    first = {f.name: getattr(ps.buf, f.name).clone() for f in dataclasses.fields(ps.buf)
             if f.name != "ws" and getattr(ps.buf, f.name) is not None}
    for _ in range(3):
        ps.run()
    torch.cuda.synchronize()
    for k, v in first.items():
        assert torch.equal(v.view(torch.uint8), getattr(ps.buf, k).view(torch.uint8)), k


# --------------------------------------------------- single-stage entries --

@pytest.mark.parametrize("slm_keep", [0, 45])
def test_single_stage_calls_match_step(slm_keep):
    w = custom("stages", 109, 3, 2000, "bf16", SMALL, LARGE, ("pct", 10), ("pct", 20),
               ragged_min=500, slm_keep=slm_keep)
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    b = ps.buf
    nsh = SMALL.layers * SMALL.q_heads
    lg, rm, rs = torch.empty_like(b.logits), torch.empty_like(b.row_max), torch.empty_like(b.row_sum)
    small = S.ModelSpec(ps.small.q, ps.small.k, ps.small.v, torch.empty_like(ps.small.out),
                        ps.small.scale, held=ps.small.held, row_pos=ps.small.row_pos)
    S.smallkv_small_attn(ps.batch, small, lg, rm, rs, b.ws)
    ci, mi = torch.empty_like(b.crit_idx), torch.empty_like(b.marg_idx)
    mp, ms = torch.empty_like(b.marg_prob), torch.empty_like(b.mass)
    S.smallkv_partition(ps.batch, nsh, lg, rm, rs, ci, mi, mp, ms, small=small)
    large = S.ModelSpec(ps.large.q, ps.large.k, ps.large.v, torch.empty_like(ps.large.out),
                        ps.large.scale)
    S.smallkv_hybrid_attn(ps.batch, large, ps.head_map, nsh, ci, mi, mp, ms, ws=b.ws)
    torch.cuda.synchronize()
    if slm_keep:  # logits rows over the held rows (stride n_rows)
        held, rows = host(x["s_held"]), x["s_k"].shape[3]
        a_ = lg.view(-1)[: 3 * nsh * rows].view(3, nsh, rows)
        b_ = b.logits.view(-1)[: 3 * nsh * rows].view(3, nsh, rows)
        for bi in range(3):
            assert torch.equal(a_[bi, :, : int(held[bi])], b_[bi, :, : int(held[bi])])
    else:
        seq = host(x["seq_len"])
        for bi in range(3):
            n = int(seq[bi])
            assert torch.equal(lg[bi, :, :n], b.logits[bi, :, :n])
    for got, want in ((rm, b.row_max), (rs, b.row_sum), (ci, b.crit_idx), (mi, b.marg_idx),
                      (mp, b.marg_prob), (ms, b.mass), (small.out, b.small_out),
                      (large.out, b.large_out)):
        assert torch.equal(got, want)


# ------------------------------------------------------- compact stores --

def compact_store(x, ref):
    """Large K held for union(C) and V for union(C u M) of the query heads of
    each (sequence, layer, kv head), with token->row slot maps (test-side
    bookkeeping from the oracle's partition)."""
    l_k, l_v, hm = x["l_k"], x["l_v"], host(x["head_map"])
    B, L, hk, n_cap, d = l_k.shape
    hq = x["l_q"].shape[2]
    g = hq // hk
    ks = np.full((B, L, hk, n_cap), -1, np.int32)
    vs = np.full((B, L, hk, n_cap), -1, np.int32)
    kr, vr = [], []
    for b in range(B):
        for li in range(L):
            for kv in range(hk):
                js = [hm[li * hq + kv * g + i] for i in range(g)]
                c = sorted(set(int(t) for j in js for t in ref["crit"][b, j] if t >= 0))
                m = sorted(set(int(t) for j in js for t in ref["marg"][b, j] if t >= 0) | set(c))
                kr.append(c)
                vr.append(m)
    R = max(max(len(r) for r in kr), max(len(r) for r in vr), 1)
    ck = torch.zeros((B, L, hk, R, d), dtype=l_k.dtype, device=l_k.device)
    cv = torch.zeros_like(ck)
    u = 0
    for b in range(B):
        for li in range(L):
            for kv in range(hk):
                # rows in reverse token order so row != token
                for rows, src, dst, slot in ((kr[u], l_k, ck, ks), (vr[u], l_v, cv, vs)):
                    idx = torch.tensor(rows[::-1], dtype=torch.long, device=l_k.device)
                    dst[b, li, kv, : len(rows)] = src[b, li, kv, idx]
                    slot[b, li, kv, rows[::-1]] = np.arange(len(rows), dtype=np.int32)
                u += 1
    return ck, cv, torch.from_numpy(ks).to(l_k.device), torch.from_numpy(vs).to(l_k.device)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_compact_store_with_slot_maps(dtype):
    w = custom(f"compact-{dtype}", 110, 2, 1200, dtype, SMALL, LARGE, ("pct", 5),
               ("pct", 15), ragged_min=600)
    x = W.make_step_inputs(w, DEV)
    ref_full = oracle_step(x, S.NORM_REMAINING)
    ck, cv, ks, vs = compact_store(x, ref_full)
    log(f"[parity] compact store rows {ck.shape[3]} of {x['l_k'].shape[3]}")
    ps = prepare_step(x, k_slot=ks, v_slot=vs, l_k=ck, l_v=cv)
    ps.run()
    torch.cuda.synchronize()
    ref = oracle_step(x, S.NORM_REMAINING, k_slot=ks, v_slot=vs, l_k=ck, l_v=cv)
    np.testing.assert_array_equal(ref["large_out"], ref_full["large_out"])
    compare_step(ps.buf, ref, x, w.torch_dtype, f"compact-{dtype}")


def test_compact_store_of_more_than_65536_rows():
    """A store padded past 65536 rows per kv head: the grouped stage 3 then
    looks its slot maps up per block instead of resolving them per window
    into 16-bit LDS entries; both give the full-cache result."""
    w = custom("compact-wide", 111, 2, 1200, "bf16", SMALL, LARGE, ("pct", 5), ("pct", 15),
               ragged_min=600)
    x = W.make_step_inputs(w, DEV)
    ref_full = oracle_step(x, S.NORM_REMAINING)
    ck, cv, ks, vs = compact_store(x, ref_full)
    pad = 65600 - ck.shape[3]
    zk = torch.zeros(ck.shape[:3] + (pad, ck.shape[4]), dtype=ck.dtype, device=ck.device)
    wk, wv = torch.cat([ck, zk], 3), torch.cat([cv, zk], 3)
    log(f"[parity] compact store rows {ck.shape[3]} padded to {wk.shape[3]}")
    ps = prepare_step(x, k_slot=ks, v_slot=vs, l_k=wk, l_v=wv)
    ps.run()
    torch.cuda.synchronize()
    ref = oracle_step(x, S.NORM_REMAINING, k_slot=ks, v_slot=vs, l_k=ck, l_v=cv)
    np.testing.assert_array_equal(ref["large_out"], ref_full["large_out"])
    compare_step(ps.buf, ref, x, w.torch_dtype, "compact-wide")


# ------------------------------------------------------- group selection --

def group_sel(x):
    x["select"] = S.SELECT_GROUP


@pytest.mark.parametrize("mode", O.MODES)
def test_group_selection_tiny_f32_all_modes(mode):
    """fp32: the per-head stage 3 reads the group's lists and each head's weights."""
    run_case(W.WORKLOADS[1], mode, mutate=group_sel, what="group selection, tiny fp32")


def test_group_selection_qwen2_7b_full_step():
    """The query heads of each of the 112 large kv heads share one selection."""
    ps, x, ref = run_case(W.WORKLOADS[2], mutate=group_sel, what="group selection, Qwen2-7B")
    assert ps.buf.crit_idx.shape[1] == 28 * 4 and ps.buf.marg_prob.shape[1] == 28 * 28


@pytest.mark.parametrize("g", [2, 8, 16])
def test_group_selection_group_sizes(g):
    """Groups of 2 and 8 query heads (grouped stage 3) and 16 (per-head stage 3)."""
    w = custom(f"gsel{g}", 122, 2, 1100, "bf16", SMALL, W.ModelShape(2, 2 * g, 2, 128),
               ("pct", 10), ("pct", 25), ragged_min=300)
    run_case(w, mutate=group_sel)


def test_group_selection_ragged_with_recent_tokens():
    w = custom("gsel-recent", 123, 4, 2500, "bf16", W.ModelShape(3, 8, 2, 64),
               W.ModelShape(2, 14, 2, 128), ("pct", 8), ("pct", 15), ragged_min=50,
               recent=("pct", 4))
    run_case(w, mutate=group_sel)


def test_group_selection_repeats_bit_identically():
    x = W.make_step_inputs(W.WORKLOADS[2], DEV)
    group_sel(x)
    ps = prepare_step(x)
    ps.run()
    torch.cuda.synchronize()
    first = [t.clone() for t in (ps.buf.crit_idx, ps.buf.marg_idx, ps.buf.marg_prob, ps.buf.mass,
                                 ps.buf.large_out)]
    for _ in range(3):
        ps.run()
    torch.cuda.synchronize()
    for a_, b_ in zip(first, (ps.buf.crit_idx, ps.buf.marg_idx, ps.buf.marg_prob, ps.buf.mass,
                              ps.buf.large_out)):
        assert torch.equal(a_.view(torch.uint8), b_.view(torch.uint8))


def test_group_selection_single_stage_calls_match_step():
    w = custom("gsel-stages", 124, 2, 1800, "bf16", SMALL, LARGE, ("pct", 10), ("pct", 20),
               ragged_min=400, select=1)
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    b = ps.buf
    nsh = SMALL.layers * SMALL.q_heads
    lg, rm, rs = torch.empty_like(b.logits), torch.empty_like(b.row_max), torch.empty_like(b.row_sum)
    small = S.ModelSpec(ps.small.q, ps.small.k, ps.small.v, torch.empty_like(ps.small.out),
                        ps.small.scale)
    S.smallkv_small_attn(ps.batch, small, lg, rm, rs, b.ws)
    ci, mi = torch.empty_like(b.crit_idx), torch.empty_like(b.marg_idx)
    mp, ms = torch.empty_like(b.marg_prob), torch.empty_like(b.mass)
    S.smallkv_group_select(ps.batch, small, ps.large, ps.head_map, lg, rm, rs, ci, mi, mp, ms, b.ws)
    large = S.ModelSpec(ps.large.q, ps.large.k, ps.large.v, torch.empty_like(ps.large.out),
                        ps.large.scale)
    S.smallkv_hybrid_attn(ps.batch, large, ps.head_map, nsh, ci, mi, mp, ms, ws=b.ws,
                          select=S.SELECT_GROUP)
    torch.cuda.synchronize()
    for got, want in ((rm, b.row_max), (rs, b.row_sum), (ci, b.crit_idx), (mi, b.marg_idx),
                      (mp, b.marg_prob), (ms, b.mass), (small.out, b.small_out),
                      (large.out, b.large_out)):
        assert torch.equal(got, want)


# --------------------------------------------- accumulated scores (H2O-style) --

@pytest.mark.parametrize("dtype,recent", [("f32", None), ("bf16", ("pct", 3))])
def test_accumulated_scores_over_drifting_steps(dtype, recent):
    """Four consecutive steps of a drifting ragged batch: the running scores
    stay bit-identical to the oracle's, and so do the lists they select."""
    kw = {"recent": recent} if recent else {}
    w = custom("accum", 125, 3, 1400, dtype, W.ModelShape(2, 8, 2, 64), W.ModelShape(2, 8, 2, 128),
               ("pct", 8), ("pct", 15), ragged_min=600, steps=4, **kw)
    ps, acc_ref = None, None
    for step in range(4):
        x = W.make_step_inputs(w, DEV, step)
        x["select"] = S.SELECT_ACCUM
        if ps is None:
            ps = prepare_step(x)
            acc_ref = np.zeros(tuple(ps.buf.acc_score.shape), np.float32)
        else:
            ps.with_query(x["s_q"], x["l_q"], x["seq_len"], x["k_crit"], x["k_marg"],
                          x.get("k_recent"))
        log(f"[parity] accumulated scores, step {step}")
        ps.run()
        torch.cuda.synchronize()
        ref = O.step(seq_len=host(x["seq_len"]), k_crit=host(x["k_crit"]), k_marg=host(x["k_marg"]),
                     kc_cap=int(x["kc_cap"]), km_cap=int(x["km_cap"]), head_map=host(x["head_map"]),
                     mode=O.NORM_REMAINING, s_q=host(x["s_q"]), s_k=host(x["s_k"]), s_v=host(x["s_v"]),
                     s_scale=0.125, l_q=host(x["l_q"]), l_k=host(x["l_k"]), l_v=host(x["l_v"]),
                     l_scale=1 / np.sqrt(128.0),
                     k_recent=host(x["k_recent"]) if x.get("k_recent") is not None else None,
                     select=O.SELECT_ACCUM, acc=acc_ref)
        compare_step(ps.buf, ref, x, w.torch_dtype, f"accumulated step {step}")
        seq = host(x["seq_len"])
        got = host(ps.buf.acc_score)
        for b in range(seq.size):
            n = int(seq[b])
            assert np.array_equal(got[b, :, :n].view(np.uint32), acc_ref[b, :, :n].view(np.uint32)), \
                f"running scores differ at step {step}, sequence {b}"


def test_accumulated_single_stage_calls_match_step():
    w = custom("accum-stages", 126, 2, 1500, "bf16", SMALL, LARGE, ("pct", 10), ("pct", 20),
               ragged_min=400, select=2)
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    b = ps.buf
    nsh = SMALL.layers * SMALL.q_heads
    lg, rm, rs = torch.empty_like(b.logits), torch.empty_like(b.row_max), torch.empty_like(b.row_sum)
    small = S.ModelSpec(ps.small.q, ps.small.k, ps.small.v, torch.empty_like(ps.small.out),
                        ps.small.scale)
    S.smallkv_small_attn(ps.batch, small, lg, rm, rs, b.ws)
    acc = torch.zeros_like(b.acc_score)
    ci, mi = torch.empty_like(b.crit_idx), torch.empty_like(b.marg_idx)
    mp, ms = torch.empty_like(b.marg_prob), torch.empty_like(b.mass)
    S.smallkv_accum_select(ps.batch, small, lg, rm, rs, acc, ci, mi, mp, ms, b.ws)
    large = S.ModelSpec(ps.large.q, ps.large.k, ps.large.v, torch.empty_like(ps.large.out),
                        ps.large.scale)
    S.smallkv_hybrid_attn(ps.batch, large, ps.head_map, nsh, ci, mi, mp, ms, ws=b.ws)
    torch.cuda.synchronize()
    for got, want in ((acc, b.acc_score), (ci, b.crit_idx), (mi, b.marg_idx), (mp, b.marg_prob),
                      (ms, b.mass), (large.out, b.large_out)):
        assert torch.equal(got, want)


# ------------------------------------------- per-layer stage 3, step events --

def _layered_stage3(ps, select=S.SELECT_HEAD, per=1):
    """Stage 3 as a sequential model runs it: one smallkv_hybrid_attn_layers
    call per `per` large layers, into a fresh output."""
    b = ps.buf
    nsh = ps.buf.logits.shape[1]
    large = S.ModelSpec(ps.large.q, ps.large.k, ps.large.v, torch.empty_like(ps.large.out),
                        ps.large.scale, ps.large.k_slot, ps.large.v_slot)
    L = ps.large.q.shape[1]
    ws = torch.empty(max(1, S.smallkv_hybrid_attn_workspace_size(ps.batch, large, per, nsh)),
                     dtype=torch.uint8, device=DEV)
    for l0 in range(0, L, per):
        S.smallkv_hybrid_attn_layers(ps.batch, large, l0, min(per, L - l0), ps.head_map, nsh,
                                     b.crit_idx, b.marg_idx, b.marg_prob, b.mass, ps.mode, ws,
                                     select=select)
    torch.cuda.synchronize()
    return large.out


def _check_layered(ps, ref, dtype, select=S.SELECT_HEAD, per=1):
    """Per-layer stage 3 against the oracle (the launch over fewer kv heads
    may split their tokens into more ranges than the whole-stack launch, so
    its merge may round differently: the tolerance, not bit equality)."""
    from parity import TOL, head_err
    out = _layered_stage3(ps, select=select, per=per)
    err = head_err(host(out), ref["large_out"])
    assert err <= TOL[dtype], f"per-layer stage 3 error {err:.3g}"
    return out


@pytest.mark.parametrize("dtype,batch,per", [("bf16", 3, 1), ("bf16", 2, 2), ("f32", 3, 1)])
def test_per_layer_stage3_matches_the_oracle(dtype, batch, per):
    """One launch per large layer (grouped bf16 kernel, per-head fp32 kernel;
    several sequences, so every layer slice is strided) within the
    tolerance of the oracle; the per-head kernel does not split, so it also
    equals the whole-stack call bit for bit."""
    w = custom(f"layers-{dtype}", 121, batch, 1800, dtype, SMALL, LARGE, ("pct", 10),
               ("pct", 20), ragged_min=600)
    ps, x, ref = run_case(w)
    out = _check_layered(ps, ref, w.torch_dtype, per=per)
    if dtype == "f32":
        assert torch.equal(out.view(torch.uint8), ps.buf.large_out.view(torch.uint8))


def test_per_layer_stage3_qwen2_7b_and_group_selection():
    ps, x, ref = run_case(W.WORKLOADS[2])
    _check_layered(ps, ref, torch.bfloat16)
    w = custom("layers-group", 122, 2, 2500, "bf16", SMALL, LARGE, ("pct", 10), ("pct", 20),
               select=1)
    ps, x, ref = run_case(w)
    _check_layered(ps, ref, torch.bfloat16, select=S.SELECT_GROUP)


def test_per_layer_stage3_rejects_ranges_outside_the_stack():
    w = W.WORKLOADS[1]
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    b = ps.buf
    for l0, n in ((-1, 1), (0, 2), (1, 1), (0, 0)):
        with pytest.raises(S.SmallKVError) as ei:
            S.smallkv_hybrid_attn_layers(ps.batch, ps.large, l0, n, ps.head_map,
                                         b.logits.shape[1], b.crit_idx, b.marg_idx, b.marg_prob,
                                         b.mass, ps.mode, b.ws)
        assert ei.value.status == S.EINVAL


@pytest.mark.parametrize("select", [0, 1, 2])
def test_step_events_time_the_step_without_changing_it(select):
    w = custom(f"events-{select}", 123, 2, 3000, "bf16", SMALL, LARGE, ("pct", 10),
               ("pct", 20), ragged_min=1000, select=select)
    x = W.make_step_inputs(w, DEV)
    ps = prepare_step(x)
    ps.run()
    torch.cuda.synchronize()
    want = {f.name: getattr(ps.buf, f.name).clone() for f in dataclasses.fields(ps.buf)
            if f.name not in ("ws", "acc_score", "logits") and getattr(ps.buf, f.name) is not None}
    if select == 2:  # the running scores advance every step: start again from zero
        ps.buf.acc_score.zero_()
        ps.run()
        torch.cuda.synchronize()
        want = {k: getattr(ps.buf, k).clone() for k in want}
        ps.buf.acc_score.zero_()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    S.smallkv_step_events(ps.desc, ps.buf.ws, ev)
    torch.cuda.synchronize()
    for k, v in want.items():
        assert torch.equal(v.view(torch.uint8), getattr(ps.buf, k).view(torch.uint8)), k
    ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(3)]
    assert all(t > 0 for t in ms), ms
    # entries may be left out
    S.smallkv_step_events(ps.desc, ps.buf.ws, [None, ev[1], None, ev[3]])
    torch.cuda.synchronize()
    assert ev[1].elapsed_time(ev[3]) > 0


# ----------------------------- selection kernels at every launch width --

def test_accumulated_scores_at_the_qwen2_7b_shapes():
    """The accumulated-score selection at the Qwen2-7B + Qwen2-0.5B shapes (336
    rows of up to 8192 tokens: four Z chunks, 512-thread partition rows
    holding 16 logits per thread, 32 bins per binade) over three drifting
    steps: running scores, lists and outputs against the oracle."""
    w = custom("accum-qwen2", 127, 1, 8189, "bf16", W.QWEN2_0_5B, W.QWEN2_7B, ("pct", 10),
               ("pct", 20), ragged_min=8000, steps=3)
    assert w.n_cap == 8192
    ps, acc_ref = None, None
    for step in range(3):
        x = W.make_step_inputs(w, DEV, step)
        x["select"] = S.SELECT_ACCUM
        if ps is None:
            ps = prepare_step(x)
            acc_ref = np.zeros(tuple(ps.buf.acc_score.shape), np.float32)
        else:
            ps.with_query(x["s_q"], x["l_q"], x["seq_len"], x["k_crit"], x["k_marg"])
        log(f"[parity] accumulated scores at the Qwen2 shapes, step {step}")
        ps.run()
        torch.cuda.synchronize()
        ref = O.step(seq_len=host(x["seq_len"]), k_crit=host(x["k_crit"]), k_marg=host(x["k_marg"]),
                     kc_cap=int(x["kc_cap"]), km_cap=int(x["km_cap"]), head_map=host(x["head_map"]),
                     mode=O.NORM_REMAINING, s_q=host(x["s_q"]), s_k=host(x["s_k"]), s_v=host(x["s_v"]),
                     s_scale=0.125, l_q=host(x["l_q"]), l_k=host(x["l_k"]), l_v=host(x["l_v"]),
                     l_scale=1 / np.sqrt(128.0), select=O.SELECT_ACCUM, acc=acc_ref)
        compare_step(ps.buf, ref, x, w.torch_dtype, f"accumulated (Qwen2 shapes) step {step}")
        n = int(host(x["seq_len"])[0])
        got = host(ps.buf.acc_score)
        assert np.array_equal(got[0, :, :n].view(np.uint32), acc_ref[0, :, :n].view(np.uint32)), \
            f"running scores differ at step {step}"


@pytest.mark.parametrize("batch,n", [(22, 1500), (22, 9000), (86, 1200), (86, 5200)])
def test_group_selection_at_every_partition_width(batch, n):
    """Group rows (sequence, large layer, kv head): 264 rows run 512 threads
    each, 1032 rows 256 each; the lengths give register rows of 4 and 8
    logits per thread and the re-reading rows beyond 16 (512 threads) or 20
    (256 threads) logits per thread."""
    w = custom(f"gsel-rows{batch}-{n}", 128, batch, n, "bf16", SMALL, LARGE, ("pct", 10),
               ("pct", 20), ragged_min=n - n // 8, select=1)
    rows = batch * LARGE.layers * LARGE.kv_heads
    assert (rows > 256) and ((rows >= 1024) == (batch == 86))
    run_case(w)
