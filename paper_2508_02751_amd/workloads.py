"""Seeded synthetic decode-step workloads.

This module only draws inputs: it holds none of the method's arithmetic, and
both the GPU path and the CPU oracle consume the tensors it produces (the
oracle through a host copy of the same bytes).

Recipe (shapes of the model pairs the paper evaluates: Qwen2-0.5B/7B,
LLaMA-3.2-1B/3.1-8B, Qwen2-0.5B/72B; the efficiency experiment itself uses
synthetic padded prompts):
  * one latent z_t ~ N(0, I_64) per token and sequence, shared by both models
    and every layer; in the drifting workload positions at and after the
    prompt continue z_{t+1} = 0.9 z_t + 0.44 xi;
  * per (model, layer, kv head g) a projection W_g in R^{64 x d}, iid N(0,1);
    keys k_t = (z_t W_g + 0.1 eps) / sqrt(d); query heads use their kv head's
    W with the latent of the current (last) token: q = (z_q W_g + 0.1 eps)/sqrt(d);
  * tokens 0..3 are attention sinks: their keys are multiplied by 8 in both
    models; optionally a seeded set of "heavy hitter" positions gets keys x4;
  * values V ~ N(0, 1); everything is rounded to the storage dtype (RNE);
  * the large-to-small head map f(layer, head) is iid uniform over the small
    model's l*Hq_s heads (with an early-stopped small model, over the heads
    of the layers it runs);
  * budgets: a fixed count per sequence, or floor(N_b * pct / 100) of the
    sequence's current length N_b; workloads with recent tokens split the
    budget critical : recent : marginal = 2 : 1 : 2, as in the paper's
    experimental setup (its 20% example: 10%, 5%, 10%).

Small model's own KV eviction (slm_keep = p): each (sequence, small layer,
kv head) holds floor(N_b * p / 100) of its tokens: the sinks, the most
recent 10% of the sequence, and a seeded uniform sample of the rest, in
ascending position; its K/V rows are gathered into a compact store and
row_pos maps rows to positions.

Prefill matching window (match_inputs): the first w_cap prompt tokens of
the same latents; keys as above with the cache's projections W_g and their
own noise; query head h of kv head g projects with W_g + 0.5 E_h (E_h iid
N(0,1), so that heads of one group differ) plus 0.1 noise, over sqrt(d);
TopK budget 10% of the window (at least 1), the critical share of the
step workloads.

Seeds: base 1000 + workload id; each named tensor has its own generator
seeded from (base, tag) through crc32, so any tensor can be regenerated alone.
"""
from __future__ import annotations

import dataclasses
import zlib
from typing import Optional

import torch


@dataclasses.dataclass(frozen=True)
class ModelShape:
    layers: int
    q_heads: int
    kv_heads: int
    head_dim: int

    @property
    def group(self) -> int:
        return self.q_heads // self.kv_heads


@dataclasses.dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    batch: int
    n_ctx: int                    # context length N (max prompt length for the ragged one)
    dtype: str                    # "f32" or "bf16"
    small: ModelShape
    large: ModelShape
    crit: tuple                   # ("abs", k) or ("pct", p)
    marg: tuple
    recent: tuple = ("abs", 0)    # recent tokens kept whatever their score
    sinks: int = 4
    sink_gain: float = 8.0
    heavy_frac: float = 0.0       # fraction of positions that are heavy hitters
    heavy_gain: float = 4.0
    ragged_min: int = 0           # >0: prompt length per sequence ~ U[ragged_min, n_ctx]
    steps: int = 1                # consecutive decode steps (drifting latent)
    compact_large: bool = False   # large KV held only for retained tokens
    slm_keep: int = 0             # >0: the small model's own cache keeps this % of tokens
    select: int = 0               # 1: the query heads of a large kv head share one selection

    @property
    def n_cap(self) -> int:
        # after decode step t a sequence holds its prompt (at most n_ctx
        # tokens) and t + 1 decoded tokens
        return self.n_ctx + (self.steps if self.steps > 1 else 0)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def budget(self, spec, n: int) -> int:
        kind, v = spec
        return int(v) if kind == "abs" else (n * int(v)) // 100


QWEN2_0_5B = ModelShape(24, 14, 2, 64)
QWEN2_7B = ModelShape(28, 28, 4, 128)
QWEN2_72B = ModelShape(80, 64, 8, 128)
LLAMA32_1B = ModelShape(16, 32, 8, 64)
LLAMA3_8B = ModelShape(32, 32, 8, 128)

WORKLOADS = {
    1: Workload(1, "tiny-1layer-n512-f32", 1, 512, "f32",
                ModelShape(1, 14, 2, 64), ModelShape(1, 28, 4, 128),
                ("abs", 64), ("abs", 128)),
    2: Workload(2, "qwen2-7b+0.5b-n8192-b1-bf16", 1, 8192, "bf16",
                QWEN2_0_5B, QWEN2_7B, ("pct", 10), ("pct", 20)),
    3: Workload(3, "llama3-8b+3.2-1b-n32768-b16-bf16", 16, 32768, "bf16",
                LLAMA32_1B, LLAMA3_8B, ("pct", 5), ("pct", 15), heavy_frac=0.05),
    4: Workload(4, "qwen2-7b+0.5b-ragged1024-4096-b64-256steps-bf16", 64, 4096, "bf16",
                QWEN2_0_5B, QWEN2_7B, ("pct", 20), ("pct", 30), ragged_min=1024, steps=256),
    5: Workload(5, "qwen2-72b+0.5b-n65536-b2-bf16-compact", 2, 65536, "bf16",
                QWEN2_0_5B, QWEN2_72B, ("pct", 2), ("pct", 8), compact_large=True),
    6: Workload(6, "qwen2-7b+0.5b-n8192-b1-bf16-c10r5m10", 1, 8192, "bf16",
                QWEN2_0_5B, QWEN2_7B, ("pct", 10), ("pct", 10), recent=("pct", 5)),
    # the small model stopped after its first 20 of 24 layers (the stop with
    # no accuracy loss in the paper's early-stop table): only those layers
    # run, so only their KV exists and the head map ranges over their heads
    7: Workload(7, "qwen2-7b+0.5b@20of24-n8192-b1-bf16", 1, 8192, "bf16",
                dataclasses.replace(QWEN2_0_5B, layers=20), QWEN2_7B, ("pct", 10), ("pct", 20)),
    # the small model's own cache compressed to 40% of the tokens (the
    # paper's best small-model budget with the large model at 20%)
    8: Workload(8, "qwen2-7b+0.5b-slm40-n8192-b1-bf16", 1, 8192, "bf16",
                QWEN2_0_5B, QWEN2_7B, ("pct", 10), ("pct", 20), slm_keep=40),
    # the Qwen2 step with one selection per large kv head (summed selection)
    9: Workload(9, "qwen2-7b+0.5b-n8192-b1-bf16-groupsel", 1, 8192, "bf16",
                QWEN2_0_5B, QWEN2_7B, ("pct", 10), ("pct", 20), select=1),
    # the Qwen2 step ranked by H2O-style accumulated scores (running state)
    10: Workload(10, "qwen2-7b+0.5b-n8192-b1-bf16-accum", 1, 8192, "bf16",
                 QWEN2_0_5B, QWEN2_7B, ("pct", 10), ("pct", 20), select=2),
}

LATENT = 64


def _gen(base: int, tag: str, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((base * 1_000_003 + zlib.crc32(tag.encode())) % (2 ** 63))
    return g


def _randn(shape, base, tag, device):
    return torch.randn(shape, generator=_gen(base, tag, device), device=device,
                       dtype=torch.float32)


def prompt_lengths(w: Workload, device="cpu") -> torch.Tensor:
    """Per-sequence prompt length P_b (N for fixed-length workloads)."""
    if w.ragged_min <= 0:
        return torch.full((w.batch,), w.n_ctx, dtype=torch.int32)
    base = 1000 + w.wid
    g = _gen(base, "prompt_len", "cpu")
    return torch.randint(w.ragged_min, w.n_ctx + 1, (w.batch,), generator=g,
                         dtype=torch.int64).to(torch.int32)


def latents(w: Workload, device) -> torch.Tensor:
    """z [B][n_cap][64], fp32."""
    base = 1000 + w.wid
    z = _randn((w.batch, w.n_cap, LATENT), base, "latent", device)
    if w.steps > 1:
        P = prompt_lengths(w).to(device)
        xi = _randn((w.batch, w.n_cap, LATENT), base, "drift", device)
        for t in range(int(P.min()), w.n_cap):
            drift = (t >= P)[:, None]
            z[:, t] = torch.where(drift, 0.9 * z[:, t - 1] + 0.44 * xi[:, t], z[:, t])
    return z


def heavy_positions(w: Workload, device) -> Optional[torch.Tensor]:
    """Bool mask [B][n_cap] of heavy-hitter positions, drawn from [sinks, N)."""
    if w.heavy_frac <= 0:
        return None
    base = 1000 + w.wid
    count = int(w.heavy_frac * w.n_ctx)
    mask = torch.zeros((w.batch, w.n_cap), dtype=torch.bool)
    for b in range(w.batch):
        g = _gen(base, f"heavy/{b}", "cpu")
        pos = torch.randperm(w.n_ctx - w.sinks, generator=g)[:count] + w.sinks
        mask[b, pos] = True
    return mask.to(device)


def seq_lens(w: Workload, step: int = 0) -> torch.Tensor:
    """Current length N_b (the cache includes the current token)."""
    P = prompt_lengths(w)
    if w.steps > 1:
        return (P + step + 1).to(torch.int32)
    return P.clone()


def budgets(w: Workload, step: int = 0):
    n = seq_lens(w, step)
    kc = torch.tensor([w.budget(w.crit, int(x)) for x in n], dtype=torch.int32)
    km = torch.tensor([w.budget(w.marg, int(x)) for x in n], dtype=torch.int32)
    return n, kc, km


def recent_budget(w: Workload, step: int = 0):
    """Recent tokens per sequence [B] int32, or None for workloads without them."""
    if w.recent == ("abs", 0):
        return None
    return torch.tensor([w.budget(w.recent, int(x)) for x in seq_lens(w, step)], dtype=torch.int32)


def caps(w: Workload):
    """Widths of the index buffers: the largest budget any step can ask for."""
    n_max = w.n_cap
    return (max(1, w.budget(w.crit, n_max) + w.budget(w.recent, n_max)),
            max(1, w.budget(w.marg, n_max)))


def head_map(w: Workload, device) -> torch.Tensor:
    base = 1000 + w.wid
    g = _gen(base, "head_map", "cpu")
    hm = torch.randint(0, w.small.layers * w.small.q_heads,
                       (w.large.layers * w.large.q_heads,), generator=g, dtype=torch.int64)
    return hm.to(torch.int32).to(device)


def kv_layer(w: Workload, which: str, layer: int, z: torch.Tensor,
             heavy: Optional[torch.Tensor], device):
    """Keys and values of one layer: ([B][Hkv][n_cap][d], same) in the storage dtype."""
    m = w.small if which == "small" else w.large
    base = 1000 + w.wid
    d = m.head_dim
    W = _randn((m.kv_heads, LATENT, d), base, f"{which}/W/{layer}", device)
    k = torch.einsum("bnz,hzd->bhnd", z, W)
    k += 0.1 * _randn(k.shape, base, f"{which}/keps/{layer}", device)
    k /= d ** 0.5
    gain = torch.ones((w.batch, w.n_cap), device=device)
    gain[:, : w.sinks] = w.sink_gain
    if heavy is not None:
        gain = torch.where(heavy, torch.full_like(gain, w.heavy_gain), gain)
    k *= gain[:, None, :, None]
    v = _randn(k.shape, base, f"{which}/v/{layer}", device)
    return k.to(w.torch_dtype), v.to(w.torch_dtype)


def q_layer(w: Workload, which: str, layer: int, z: torch.Tensor, step: int, device):
    """Queries of one layer [B][Hq][d] from the current token's latent."""
    m = w.small if which == "small" else w.large
    base = 1000 + w.wid
    d = m.head_dim
    W = _randn((m.kv_heads, LATENT, d), base, f"{which}/W/{layer}", device)
    n = seq_lens(w, step).to(torch.int64).to(z.device)
    zq = z[torch.arange(w.batch, device=z.device), n - 1]          # [B][64]
    Wq = W.repeat_interleave(m.group, dim=0)                        # [Hq][64][d]
    q = torch.einsum("bz,hzd->bhd", zq, Wq)
    q += 0.1 * _randn(q.shape, base, f"{which}/qeps/{layer}/{step}", device)
    q /= d ** 0.5
    return q.to(w.torch_dtype)


def step_queries(w: Workload, z: torch.Tensor, step: int, device):
    """Queries of both models for one decode step: (s_q [B][l][Hqs][ds], l_q [B][L][Hq][d])."""
    s_q = torch.stack([q_layer(w, "small", i, z, step, device) for i in range(w.small.layers)], 1)
    l_q = torch.stack([q_layer(w, "large", i, z, step, device) for i in range(w.large.layers)], 1)
    return s_q, l_q


def make_step_inputs(w: Workload, device, step: int = 0, *, z=None, large=True):
    """All inputs of one decode step as torch tensors on `device`.

    Returns a dict with s_q [B][l][Hqs][ds], s_k/s_v [B][l][Hks][n_cap][ds],
    l_q [B][L][Hq][d], l_k/l_v [B][L][Hk][n_cap][d] (omitted when large=False),
    seq_len/k_crit/k_marg [B] int32, head_map [L*Hq] int32, kc_cap, km_cap.
    """
    if z is None:
        z = latents(w, device)
    heavy = heavy_positions(w, device)
    B, n_cap = w.batch, w.n_cap
    s, L = w.small, w.large
    out = {}
    out["s_q"] = torch.stack([q_layer(w, "small", i, z, step, device) for i in range(s.layers)], 1)
    s_k = torch.empty((B, s.layers, s.kv_heads, n_cap, s.head_dim), dtype=w.torch_dtype, device=device)
    s_v = torch.empty_like(s_k)
    for i in range(s.layers):
        k, v = kv_layer(w, "small", i, z, heavy, device)
        s_k[:, i], s_v[:, i] = k, v
    out["s_k"], out["s_v"] = s_k, s_v
    out["l_q"] = torch.stack([q_layer(w, "large", i, z, step, device) for i in range(L.layers)], 1)
    if large:
        l_k = torch.empty((B, L.layers, L.kv_heads, n_cap, L.head_dim), dtype=w.torch_dtype, device=device)
        l_v = torch.empty_like(l_k)
        for i in range(L.layers):
            k, v = kv_layer(w, "large", i, z, heavy, device)
            l_k[:, i], l_v[:, i] = k, v
        out["l_k"], out["l_v"] = l_k, l_v
    n, kc, km = budgets(w, step)
    out["seq_len"], out["k_crit"], out["k_marg"] = n.to(device), kc.to(device), km.to(device)
    if w.slm_keep:
        evict_small_cache(w, out, n, device)
    if w.select:
        out["select"] = w.select
    kr = recent_budget(w, step)
    if kr is not None:
        out["k_recent"] = kr.to(device)
    out["head_map"] = head_map(w, device)
    out["kc_cap"], out["km_cap"] = caps(w)
    return out


def match_inputs(w: Workload, w_cap: int, device, win_len=None, top_pct: int = 10):
    """Prefill operands of both models over the first w_cap prompt tokens.

    Returns l_q [B][L][Hq][w_cap][d], l_k [B][L][Hk][w_cap][d], s_q, s_k (same
    for the small model), win_len [B] int32 (w_cap when not given) and top_k
    [B] int32 = max(1, win_len * top_pct // 100).
    """
    z = latents(w, device)[:, :w_cap]
    heavy = heavy_positions(w, device)
    base = 1000 + w.wid
    gain = torch.ones((w.batch, w_cap), device=device)
    gain[:, : w.sinks] = w.sink_gain
    if heavy is not None:
        gain = torch.where(heavy[:, :w_cap], torch.full_like(gain, w.heavy_gain), gain)
    out = {}
    for which, m, pre in (("large", w.large, "l"), ("small", w.small, "s")):
        d = m.head_dim
        qs, ks = [], []
        for layer in range(m.layers):
            W = _randn((m.kv_heads, LATENT, d), base, f"{which}/W/{layer}", device)
            k = torch.einsum("bnz,hzd->bhnd", z, W)
            k += 0.1 * _randn(k.shape, base, f"prefill/{which}/keps/{layer}", device)
            k /= d ** 0.5
            k *= gain[:, None, :, None]
            E = _randn((m.q_heads, LATENT, d), base, f"prefill/{which}/E/{layer}", device)
            Wq = W.repeat_interleave(m.group, dim=0) + 0.5 * E
            q = torch.einsum("bnz,hzd->bhnd", z, Wq)
            q += 0.1 * _randn(q.shape, base, f"prefill/{which}/qeps/{layer}", device)
            q /= d ** 0.5
            qs.append(q.to(w.torch_dtype))
            ks.append(k.to(w.torch_dtype))
        out[f"{pre}_q"] = torch.stack(qs, 1).contiguous()
        out[f"{pre}_k"] = torch.stack(ks, 1).contiguous()
    if win_len is None:
        win_len = [w_cap] * w.batch
    win = torch.tensor(win_len, dtype=torch.int32)
    out["win_len"] = win.to(device)
    out["top_k"] = torch.clamp(win * top_pct // 100, min=1).to(torch.int32).to(device)
    return out


def evict_small_cache(w: Workload, x: dict, n: torch.Tensor, device):
    """Replace x's small K/V by a compact store of the rows the small model
    keeps (see the module recipe); adds s_held [B], s_row_pos
    [B][l][Hkv][n_rows] and n_cap."""
    base = 1000 + w.wid
    B, l, hk = w.batch, w.small.layers, w.small.kv_heads
    held = [max(w.sinks + 2, int(n[b]) * w.slm_keep // 100) for b in range(B)]
    rows = max(held)
    pos = torch.full((B, l, hk, rows), -1, dtype=torch.int32)
    for b in range(B):
        nb = int(n[b])
        recent = max(1, nb // 10)
        fixed = torch.cat([torch.arange(w.sinks), torch.arange(nb - recent, nb)])
        middle = torch.arange(w.sinks, nb - recent)
        extra = held[b] - fixed.numel()
        g = _gen(base, f"slm_keep/{b}", "cpu")
        for la in range(l):
            for h in range(hk):
                pick = middle[torch.randperm(middle.numel(), generator=g)[:extra]]
                keep = torch.sort(torch.cat([fixed, pick])).values
                pos[b, la, h, : keep.numel()] = keep.to(torch.int32)
    pos = pos.to(device)
    idx = pos.clamp(min=0).to(torch.int64)[..., None].expand(-1, -1, -1, -1, w.small.head_dim)
    x["s_k"] = torch.gather(x["s_k"], 3, idx).contiguous()
    x["s_v"] = torch.gather(x["s_v"], 3, idx).contiguous()
    x["s_held"] = torch.tensor(held, dtype=torch.int32, device=device)
    x["s_row_pos"] = pos.contiguous()
    x["n_cap"] = w.n_cap
