"""Pins of the byte model against the paper's printed KV-cache figures."""
import os

import pytest

from paper_2508_02751_amd.bytes_model import kv_cache_bytes

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "kv_cache_ratios.txt")


def rows():
    for line in open(GOLDEN):
        line = line.strip()
        if line and not line.startswith("#"):
            p = line.split()
            yield p[0], tuple(map(int, p[1:4])), tuple(map(int, p[4:7])), float(p[7]), int(p[8])


@pytest.mark.parametrize("pair,small,large,printed,dec", list(rows()))
def test_kv_ratio_matches_printed_table(pair, small, large, printed, dec):
    r = kv_cache_bytes(*large, 4096, 2, 2) / kv_cache_bytes(*small, 4096, 2, 2)
    assert round(r, dec) == printed


def test_slm_share_of_saved_kv():
    """Appendix A.1: with Qwen2-7B assisting Qwen2-72B at a 20% budget, the small
    model's KV is about 21.9% of the KV saved on the large model."""
    big = kv_cache_bytes(80, 8, 128, 1000, 1, 2)
    small = kv_cache_bytes(28, 4, 128, 1000, 1, 2)
    assert round(100 * small / (0.8 * big), 1) == 21.9


def test_effective_slm_kv_with_compression_and_early_stop():
    """Appendix A.3: (1/4.67) x 40% (SLM compression) x 20/24 (early stop) ~ 7.14%."""
    big = kv_cache_bytes(28, 4, 128, 1000, 1, 2)
    small = kv_cache_bytes(24, 2, 64, 1000, 1, 2)
    assert round(100 * small / big * 0.4 * 20 / 24, 2) == 7.14


def test_union_bytes_against_python_sets():
    """Stage 3's bytes: per (sequence, layer, kv head) the union of its query
    heads' critical tokens (K rows) and of their critical and marginal tokens
    (V rows), counted here with Python sets on random lists."""
    import numpy as np
    import torch

    from paper_2508_02751_amd.bytes_model import step_bytes
    rng = np.random.default_rng(7)
    B, l, hqs, hks, ds, L, hq, hk, d, n, kc, km = 3, 2, 4, 2, 64, 3, 8, 2, 128, 50, 6, 9
    nsh = l * hqs

    def lists(k):
        out = np.full((B, nsh, k), -1, np.int32)
        for b in range(B):
            for j in range(nsh):
                c = rng.integers(0, k + 1)
                out[b, j, :c] = np.sort(rng.choice(n, c, replace=False))
        return out

    crit, marg = lists(kc), lists(km)
    hm = rng.integers(0, nsh, L * hq).astype(np.int32)
    x = {"s_q": torch.zeros((B, l, hqs, ds), dtype=torch.bfloat16),
         "s_k": torch.zeros((B, l, hks, n, ds), dtype=torch.bfloat16),
         "l_q": torch.zeros((B, L, hq, d), dtype=torch.bfloat16),
         "l_k": torch.zeros((B, L, hk, 1, d), dtype=torch.bfloat16),
         "seq_len": torch.full((B,), n, dtype=torch.int32), "head_map": torch.from_numpy(hm),
         "n_cap": n}
    sb = step_bytes(x, torch.from_numpy(crit), torch.from_numpy(marg), km)
    ku = vu = kp = vp = 0
    g = hq // hk
    for b in range(B):
        for li in range(L):
            for kv in range(hk):
                js = hm[li * hq + kv * g: li * hq + (kv + 1) * g]
                cset = set().union(*[set(crit[b, j][crit[b, j] >= 0]) for j in js])
                mset = set().union(*[set(marg[b, j][marg[b, j] >= 0]) for j in js])
                ku += len(cset)
                vu += len(cset | mset)
                kp += sum(int((crit[b, j] >= 0).sum()) for j in js)
                vp += sum(int((crit[b, j] >= 0).sum() + (marg[b, j] >= 0).sum()) for j in js)
    assert sb.large_k_union == ku * d * 2 and sb.large_v_union == vu * d * 2
    assert sb.large_k_perhead == kp * d * 2 and sb.large_v_perhead == vp * d * 2
