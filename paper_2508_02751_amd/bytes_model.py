"""Byte accounting of one decode step (algorithmic, i.e. compulsory, bytes).

KV-cache size, Appendix A.1 Eq. 7: M_kv = 2 * L * N_kv * D_kv * S * B * C_b
(factor 2 for K and V).

Per decode step the method must move, at minimum:
  stage 1  the small model's K and V rows of every cached token (once), its
           queries and outputs, and the fp32 logits it emits (one per small
           head and token: the attention row that stage 2 ranks);
  stage 2  the logits of each row once, plus its index lists, marginal
           probabilities and masses;
  stage 3  per (sequence, layer, kv head) the union over the query heads that
           share the kv head of the K rows of their critical tokens and of
           the V rows of their critical and marginal tokens, plus queries and
           outputs.
Index lists read by stage 3 (4 bytes per entry) are reported separately as
metadata and are not counted in its roofline numerator.
"""
from __future__ import annotations

import dataclasses

import torch


def kv_cache_bytes(layers: int, kv_heads: int, head_dim: int, seq: int, batch: int,
                   bytes_per_value: float) -> float:
    """Eq. 7: total bytes of a K+V cache."""
    return 2 * layers * kv_heads * head_dim * seq * batch * bytes_per_value


@dataclasses.dataclass
class StepBytes:
    small_kv: int        # stage 1: K and V rows read
    small_qo: int        # stage 1: queries read and outputs written
    logits: int          # stage 1 write = stage 2 read (fp32 rows)
    part_out: int        # stage 2: index lists, marginal probabilities, masses written
    large_k_union: int   # stage 3: distinct K rows (critical union per kv head)
    large_v_union: int   # stage 3: distinct V rows (critical+marginal union per kv head)
    large_k_perhead: int # stage 3 if every query head read its own rows (no sharing)
    large_v_perhead: int
    large_qo: int        # stage 3: queries read and outputs written
    index_meta: int      # stage 3: index lists and probabilities read

    @property
    def stage1(self) -> int:
        return self.small_kv + self.small_qo + self.logits

    @property
    def stage2(self) -> int:
        return self.logits + self.part_out

    @property
    def stage3(self) -> int:
        return self.large_k_union + self.large_v_union + self.large_qo

    @property
    def step_compulsory(self) -> int:
        """Small K/V once + large union rows + queries and outputs of both models."""
        return self.small_kv + self.small_qo + self.large_k_union + self.large_v_union + self.large_qo


def step_bytes(x: dict, crit_idx: torch.Tensor, marg_idx: torch.Tensor, km_cap: int) -> StepBytes:
    """Count the bytes of one step from its inputs and the partition it produced
    (all sequences and large layers at once: one membership bitmap per
    (sequence, layer, kv head) over its tokens)."""
    s_q, s_k = x["s_q"], x["s_k"]
    l_q = x["l_q"]
    esz = s_k.element_size()
    B, l, hqs, ds = s_q.shape
    hks = s_k.shape[2]
    _, L, hq, d = l_q.shape
    hk = x["l_k"].shape[2] if "l_k" in x else hq
    g = hq // hk
    n_cap = x["n_cap"] if "n_cap" in x else s_k.shape[3]
    seq = x["seq_len"].to(torch.int64)
    # the small model reads (and scores) only the rows it holds
    s_tok = int(x["s_held"].to(torch.int64).sum()) if x.get("s_held") is not None else int(seq.sum())
    small_kv = 2 * l * hks * ds * esz * s_tok
    small_qo = 2 * B * l * hqs * ds * esz
    logits = 4 * l * hqs * s_tok
    part_out = B * l * hqs * (crit_idx.shape[-1] * 4 + km_cap * 8 + 8)
    large_qo = 2 * B * L * hq * d * esz
    dev = crit_idx.device
    rowb = d * esz
    if x.get("select", 0) == 1:  # lists per (large layer, kv head): the union is the list
        rows = torch.arange(L * hk, device=dev)[:, None].expand(L * hk, g).reshape(-1)
    else:  # each query head's lists are its small head's
        rows = x["head_map"].to(torch.int64).to(dev)
    cs = crit_idx.to(dev)[:, rows].view(B, L, hk, -1)           # [B][L][hk][g*kc]
    n_c = int((cs >= 0).sum())
    bm = torch.zeros((B, L, hk, n_cap + 1), dtype=torch.bool, device=dev)
    bm.scatter_(3, torch.where(cs >= 0, cs, n_cap).to(torch.int64), True)
    del cs
    k_union = int(bm[..., :n_cap].sum()) * rowb
    n_m = 0
    if km_cap:
        ms = marg_idx[..., :km_cap].to(dev)[:, rows].view(B, L, hk, -1)
        n_m = int((ms >= 0).sum())
        bm.scatter_(3, torch.where(ms >= 0, ms, n_cap).to(torch.int64), True)
        del ms
    v_union = int(bm[..., :n_cap].sum()) * rowb
    k_per = n_c * rowb
    v_per = (n_c + n_m) * rowb
    meta = (n_c + 2 * n_m) * 4
    return StepBytes(small_kv, small_qo, logits, part_out, k_union, v_union, k_per, v_per,
                     large_qo, meta)
