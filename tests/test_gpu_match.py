"""GPU parity of the prefill similarity matching (smallkv_match) against the
oracle: the Eq. 1 scores bit for bit, the TopK sets and the head map exactly."""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
from parity import host, log

pytestmark = pytest.mark.gpu

DEV = "cuda"


def lib_modules():
    from paper_2508_02751_amd import smallkv as S
    from paper_2508_02751_amd import workloads as W
    from paper_2508_02751_amd.pipeline import prepare_match, softmax_scale
    return S, W, prepare_match, softmax_scale


def unpack_bits(words: np.ndarray, w_cap: int) -> np.ndarray:
    """[..., nw] int64 words -> [..., w_cap] bool (bit v%64 of word v/64)."""
    u = words.astype(np.uint64)
    bits = (u[..., :, None] >> np.arange(64, dtype=np.uint64)) & np.uint64(1)
    return bits.reshape(*words.shape[:-1], -1)[..., :w_cap].astype(bool)


def oracle_match(x):
    _, _, _, softmax_scale = lib_modules()
    return O.match(win_len=host(x["win_len"]), top_k=host(x["top_k"]), l_q=host(x["l_q"]),
                   l_k=host(x["l_k"]), l_scale=softmax_scale(x["l_q"].shape[-1]),
                   s_q=host(x["s_q"]), s_k=host(x["s_k"]),
                   s_scale=softmax_scale(x["s_q"].shape[-1]))


def check_match(x, what):
    """Run both sides; return the oracle's head map after asserting the GPU's equals it."""
    _, _, prepare_match, _ = lib_modules()
    log(f"[match] {what}: GPU")
    mc = prepare_match(x)
    mc.run()
    torch.cuda.synchronize()
    log(f"[match] {what}: oracle")
    hm, sc, top = oracle_match(x)
    w_cap = x["l_q"].shape[3]
    win = host(x["win_len"]).astype(np.int64)
    g_sc = host(mc.scores)
    g_top = unpack_bits(host(mc.top_bits), w_cap)
    for b in range(win.size):
        w = int(min(max(win[b], 1), w_cap))
        bad = g_sc[b, :, :w].view(np.uint32) != sc[b, :, :w].view(np.uint32)
        assert not bad.any(), f"{what}: {int(bad.sum())} scores differ in sequence {b}"
        assert not g_sc[b, :, w:].any(), f"{what}: scores written past the window"
        assert np.array_equal(g_top[b], top[b]), f"{what}: TopK sets differ in sequence {b}"
    assert np.array_equal(host(mc.head_map), hm), f"{what}: head maps differ"
    return hm


def with_batch(w, batch, wid_offset=100):
    return dataclasses.replace(w, batch=batch, wid=w.wid + wid_offset)


def test_tiny_fp32_window_100():
    _, W, _, _ = lib_modules()
    x = W.match_inputs(W.WORKLOADS[1], 100, DEV)
    check_match(x, "tiny fp32, window 100")


@pytest.mark.parametrize("top_pct", [0, 100])
def test_tiny_fp32_max_window_extreme_budgets(top_pct):
    # window 256 (the largest supported), K = 1 or K = window
    _, W, _, _ = lib_modules()
    x = W.match_inputs(W.WORKLOADS[1], 256, DEV, top_pct=top_pct)
    hm = check_match(x, f"tiny fp32, window 256, top {top_pct}%")
    if top_pct == 100:
        assert not hm.any(), "every TopK set is the whole window: all ratios 1, lowest head"


def test_ragged_windows_bf16():
    # windows of 1, 64 (one full tile), 65 and 173 tokens in one batch, w_cap 173
    _, W, _, _ = lib_modules()
    w = dataclasses.replace(with_batch(W.WORKLOADS[1], 4), dtype="bf16")
    x = W.match_inputs(w, 173, DEV, win_len=[1, 64, 65, 173])
    check_match(x, "ragged windows 1/64/65/173 bf16")


def test_qwen2_7b_0_5b_window_200():
    _, W, _, _ = lib_modules()
    x = W.match_inputs(W.WORKLOADS[2], 200, DEV)
    hm = check_match(x, "Qwen2-7B + 0.5B, window 200")
    log(f"[match] {len(np.unique(hm))} distinct small heads among {hm.size} large heads")


def test_llama_pair_batch2_window_128():
    _, W, _, _ = lib_modules()
    x = W.match_inputs(with_batch(W.WORKLOADS[3], 2), 128, DEV, win_len=[128, 100])
    check_match(x, "LLaMA-3.1-8B + 3.2-1B, batch 2, windows 128/100")


def test_uniform_attention_all_ties():
    # zero queries: every row is uniform, every head has the same scores, every
    # TopK set is the first K tokens, every ratio is 1 and every head maps to 0
    _, W, _, _ = lib_modules()
    x = W.match_inputs(W.WORKLOADS[1], 150, DEV)
    x["l_q"].zero_()
    x["s_q"].zero_()
    hm = check_match(x, "uniform attention")
    assert not hm.any()


def test_identical_models_map_to_themselves():
    _, W, _, _ = lib_modules()
    x = W.match_inputs(W.WORKLOADS[1], 128, DEV)
    # the small model is a copy of the large one: S(i, i) = 1
    x["s_q"], x["s_k"] = x["l_q"].clone(), x["l_k"].clone()
    hm = check_match(x, "identical models")
    top = oracle_match(x)[2][0]
    nl = hm.shape[1]
    for i in range(nl):
        assert np.array_equal(top[nl + hm[0, i]], top[i])


def test_repeat_calls_are_identical():
    _, W, prepare_match, _ = lib_modules()
    x = W.match_inputs(W.WORKLOADS[2], 200, DEV)
    mc = prepare_match(x)
    mc.run()
    torch.cuda.synchronize()
    first = (mc.head_map.clone(), mc.scores.clone(), mc.top_bits.clone())
    for _ in range(3):
        mc.run()
    torch.cuda.synchronize()
    assert torch.equal(first[0], mc.head_map) and torch.equal(first[1], mc.scores)
    assert torch.equal(first[2], mc.top_bits)


def test_matched_map_drives_an_early_stopped_step():
    """Prefill matching over the small model's first 20 layers, then the
    decode step with that map: the GPU map equals the oracle's, and the step
    run with the oracle's map matches the oracle's step."""
    import parity as P
    from paper_2508_02751_amd.pipeline import prepare_step

    _, W, _, _ = lib_modules()
    w = W.WORKLOADS[7]
    win = W.match_inputs(w, 200, DEV)
    hm = check_match(win, "early-stopped small model, window 200")
    assert hm.max() < w.small.layers * w.small.q_heads
    x = W.make_step_inputs(w, DEV)
    x["head_map"] = torch.from_numpy(hm[0].copy()).to(DEV)  # the oracle's map (equal to the GPU's)
    ps = prepare_step(x)
    ps.run()
    torch.cuda.synchronize()
    ref = P.oracle_step(x, P.O.NORM_REMAINING)
    P.compare_step(ps.buf, ref, x, torch.bfloat16, "matched map, early stop")
