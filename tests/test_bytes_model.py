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
