"""Wiring of one decode step's tensors to the C ABI (marshalling only).

`prepare_step` turns the dict produced by workloads.make_step_inputs (or any
dict with the same keys) into BatchSpec/ModelSpec objects, allocates the
caller-owned intermediates and the workspace, and builds the C step
descriptor; `run` enqueues smallkv_step on the current stream.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import torch

from . import smallkv as S


MATCH_MIN, MATCH_MAX = 100, 200  # prompt tokens the matching uses ("Method Details")


def match_window(prompt_len: int) -> Optional[int]:
    """Window of the prefill matching for a prompt: None (delay the matching
    until the context reaches MATCH_MIN tokens) below MATCH_MIN, else the
    first min(prompt_len, MATCH_MAX) tokens (a longer prompt is truncated)."""
    if prompt_len < MATCH_MIN:
        return None
    return min(prompt_len, MATCH_MAX)


def prepare_match(x: dict, scores: bool = True, top_bits: bool = True) -> S.MatchCall:
    """smallkv_match over the window operands produced by workloads.match_inputs."""
    return S.prepare_match(x["win_len"], x["top_k"], x["l_q"], x["l_k"],
                           softmax_scale(x["l_q"].shape[-1]), x["s_q"], x["s_k"],
                           softmax_scale(x["s_q"].shape[-1]), scores, top_bits)


def softmax_scale(head_dim: int) -> float:
    return float(torch.tensor(1.0 / math.sqrt(head_dim), dtype=torch.float32))


@dataclasses.dataclass
class PreparedStep:
    batch: S.BatchSpec
    small: S.ModelSpec
    large: S.ModelSpec
    head_map: torch.Tensor
    mode: int
    buf: S.StepBuffers
    desc: S.Step
    inputs: dict

    def run(self, stream=None):
        S.smallkv_step(self.desc, self.buf.ws, stream)

    def with_query(self, s_q: torch.Tensor, l_q: torch.Tensor, seq_len=None, k_crit=None,
                   k_marg=None, k_recent=None):
        """Point the descriptor at new queries/lengths (same shapes; for multi-step runs)."""
        self.small.q.copy_(s_q)
        self.large.q.copy_(l_q)
        if seq_len is not None:
            self.batch.seq_len.copy_(seq_len)
            self.batch.k_crit.copy_(k_crit)
            self.batch.k_marg.copy_(k_marg)
        if k_recent is not None:
            self.batch.k_recent.copy_(k_recent)


def prepare_step(x: dict, mode: int = S.NORM_REMAINING,
                 k_slot: Optional[torch.Tensor] = None,
                 v_slot: Optional[torch.Tensor] = None,
                 l_k: Optional[torch.Tensor] = None,
                 l_v: Optional[torch.Tensor] = None,
                 select: Optional[int] = None) -> PreparedStep:
    """`select` defaults to x["select"] when present, else per-head selection."""
    if select is None:
        select = x.get("select", S.SELECT_HEAD)
    s_q, s_k, s_v = x["s_q"], x["s_k"], x["s_v"]
    l_q = x["l_q"]
    l_k = x["l_k"] if l_k is None else l_k
    l_v = x["l_v"] if l_v is None else l_v
    n_cap = x["n_cap"] if "n_cap" in x else s_k.shape[3]
    kr = x.get("k_recent")
    batch = S.BatchSpec(x["seq_len"].contiguous(), x["k_crit"].contiguous(),
                        x["k_marg"].contiguous(), n_cap, int(x["kc_cap"]), int(x["km_cap"]),
                        kr.contiguous() if kr is not None else None)
    small = S.ModelSpec(s_q.contiguous(), s_k, s_v, torch.empty_like(s_q),
                        softmax_scale(s_q.shape[-1]), held=x.get("s_held"),
                        row_pos=x.get("s_row_pos"))
    large = S.ModelSpec(l_q.contiguous(), l_k, l_v, torch.empty_like(l_q),
                        softmax_scale(l_q.shape[-1]), k_slot, v_slot)
    hm = x["head_map"].contiguous()
    ws_bytes = S.smallkv_workspace_size(batch, small, large, hm, select)
    buf = S.alloc_step_buffers(batch, s_q, l_q, ws_bytes, select, l_k.shape[2])
    buf.small_out = small.out
    buf.large_out = large.out
    # accumulated scores: the running state, zero before the first step
    acc = (torch.zeros((batch.seq_len.numel(), buf.logits.shape[1], n_cap), dtype=torch.float32,
                       device=s_q.device) if select == S.SELECT_ACCUM else None)
    buf.acc_score = acc
    desc = S.make_step(batch, small, large, hm, mode, buf.logits, buf.row_max, buf.row_sum,
                       buf.crit_idx, buf.marg_idx, buf.marg_prob, buf.mass, select, acc)
    return PreparedStep(batch, small, large, hm, mode, buf, desc, x)
