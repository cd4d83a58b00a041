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
    """Count the bytes of one step from its inputs and the partition it produced."""
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
    hm = x["head_map"].to(torch.int64).to(dev).view(L, hk, g)
    rowb = d * esz
    k_union = v_union = k_per = v_per = meta = 0
    group = x.get("select", 0) == 1  # lists per (large layer, kv head): the union is the list
    for b in range(B):
        c = crit_idx[b].to(torch.int64)          # [nsh][kc] (group selection: [L*hk][kc])
        m = marg_idx[b, :, :km_cap].to(torch.int64) if km_cap else None
        for li in range(L):
            js = hm[li]                          # [hk][g]
            if group:
                js = (li * hk + torch.arange(hk, device=dev))[:, None].expand(hk, g)
            cs = c[js.reshape(-1)].view(hk, -1)  # [hk][g*kc]
            bm = torch.zeros((hk, n_cap + 1), dtype=torch.bool, device=dev)
            bm.scatter_(1, torch.where(cs >= 0, cs, n_cap), True)
            nk = int(bm[:, :n_cap].sum())
            k_per += int((cs >= 0).sum()) * rowb
            if m is not None:
                ms = m[js.reshape(-1)].view(hk, -1)
                bm.scatter_(1, torch.where(ms >= 0, ms, n_cap), True)
                v_per += (int((cs >= 0).sum()) + int((ms >= 0).sum())) * rowb
                meta += (int((cs >= 0).sum()) + 2 * int((ms >= 0).sum())) * 4
            else:
                v_per += int((cs >= 0).sum()) * rowb
                meta += int((cs >= 0).sum()) * 4
            nv = int(bm[:, :n_cap].sum())
            k_union += nk * rowb
            v_union += nv * rowb
    return StepBytes(small_kv, small_qo, logits, part_out, k_union, v_union, k_per, v_per,
                     large_qo, meta)
