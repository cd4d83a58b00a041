"""Pins of the prefill-matching oracle (Eqs. 1-3) against facts that do not
come from the oracle itself: closed forms, fp64 brute force, set algebra on
tiny inputs, and symmetries of the head map.  CPU only."""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O

RNG = np.random.default_rng(2508)


# ------------------------------------------------------------------ exp --

def test_exp_within_one_ulp_on_its_range():
    x = np.concatenate([np.linspace(-80.0, 0.0, 400_001, dtype=np.float32),
                        -RNG.exponential(3.0, 100_000).astype(np.float32),
                        np.float32([-0.0, -1e-30, -1e-7, -0.3465736, -0.3465737, -79.99999])])
    x = x[x >= -80.0]
    y = O.exp32(x)
    ref = np.exp(x.astype(np.float64))
    ulp = np.spacing(ref.astype(np.float32)).astype(np.float64)
    err = np.abs(y.astype(np.float64) - ref) / ulp
    assert err.max() <= 1.0, f"max error {err.max():.2f} ulp at x={x[err.argmax()]}"


def test_exp_special_values_and_monotone():
    assert O.exp32(np.float32([0.0]))[0] == np.float32(1.0)
    assert O.exp32(np.float32([-0.0]))[0] == np.float32(1.0)
    assert O.exp32(np.float32([-80.00001, -1e4, np.nan, -np.inf])).tolist() == [0.0] * 4
    x = np.sort(RNG.uniform(-80, 0, 200_000).astype(np.float32))
    y = O.exp32(x)
    assert np.all(np.diff(y) >= 0), "not monotone"


# ------------------------------------------------------------- Eq. 1 --

def causal_column_sums_fp64(Q, K, scale):
    s = (Q.astype(np.float64) @ K.astype(np.float64).T) * scale
    w = s.shape[0]
    s[np.triu(np.ones((w, w), bool), 1)] = -np.inf
    p = np.exp(s - s.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    return p.sum(0)


@pytest.mark.parametrize("w", [1, 2, 17, 64, 200, 256])
def test_scores_uniform_attention_closed_form(w):
    # all logits 0: row u spreads 1/(u+1) over tokens 0..u, so
    # F_v = sum_{u=v}^{w-1} 1/(u+1) = H_w - H_v
    Q = np.zeros((w, 8), np.float32)
    K = RNG.standard_normal((w, 8)).astype(np.float32)
    F = O.match_scores(Q, K, 0.125)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, w + 1))])
    exact = H[w] - H[:w]
    np.testing.assert_allclose(F, exact, rtol=2e-5)
    assert np.all(np.diff(F) < 0), "uniform attention must favour earlier tokens"


@pytest.mark.parametrize("w,d", [(3, 4), (16, 8), (40, 64), (129, 128)])
def test_scores_match_fp64_brute_force(w, d):
    Q = RNG.standard_normal((w, d)).astype(np.float32)
    K = RNG.standard_normal((w, d)).astype(np.float32)
    K[:2] *= 6.0  # sink-like keys
    scale = 1.0 / math.sqrt(d)
    F = O.match_scores(Q, K, scale)
    ref = causal_column_sums_fp64(Q, K, scale)
    np.testing.assert_allclose(F, ref, rtol=1e-5, atol=1e-6 * w)


def test_scores_are_column_sums_of_stochastic_rows():
    for w in (1, 5, 100):
        Q = RNG.standard_normal((w, 16)).astype(np.float32)
        K = RNG.standard_normal((w, 16)).astype(np.float32)
        F = O.match_scores(Q, K, 0.25)
        assert abs(float(F.astype(np.float64).sum()) - w) <= 1e-5 * w
        assert F[-1] > 0 and np.all(F > 0)
    # one token: its only row puts all mass on itself
    assert O.match_scores(np.ones((1, 4), np.float32), np.ones((1, 4), np.float32), 1.0)[0] == 1.0


def test_scores_last_token_is_its_own_row_only():
    # F_{w-1} receives mass only from row w-1 (causal mask)
    w, d = 30, 16
    Q = RNG.standard_normal((w, d)).astype(np.float32)
    K = RNG.standard_normal((w, d)).astype(np.float32)
    F = O.match_scores(Q, K, 0.25)
    s = (Q[-1].astype(np.float64) @ K.astype(np.float64).T) * 0.25
    p = np.exp(s - s.max())
    assert abs(F[-1] - p[-1] / p.sum()) <= 1e-6


# ------------------------------------------------------------- Eq. 2 --

@pytest.mark.parametrize("w,k", [(1, 1), (10, 3), (64, 64), (200, 20), (256, 1)])
def test_topk_against_sorted_order(w, k):
    F = np.round(RNG.standard_normal(w) * 3).astype(np.float32)  # many ties
    got = O.topk_set(F, k)
    order = sorted(range(w), key=lambda v: (-float(F[v]), v))
    want = np.zeros(w, bool)
    want[order[:k]] = True
    assert np.array_equal(got, want)


def test_jaccard_is_set_algebra():
    for _ in range(200):
        w = int(RNG.integers(1, 80))
        a = RNG.random(w) < RNG.random()
        b = RNG.random(w) < RNG.random()
        A = {i for i in range(w) if a[i]}
        B = {i for i in range(w) if b[i]}
        assert O.jaccard(a, b) == (len(A & B), len(A | B))


# ------------------------------------------------------------- Eq. 3 --

def tiny_pair(B=1, w_cap=24, L=2, hq=4, hk=2, d=16, l=3, hqs=2, hks=1, ds=8, seed=0):
    r = np.random.default_rng(seed)
    f = lambda *s: r.standard_normal(s).astype(np.float32)
    return dict(l_q=f(B, L, hq, w_cap, d), l_k=f(B, L, hk, w_cap, d), l_scale=1 / math.sqrt(d),
                s_q=f(B, l, hqs, w_cap, ds), s_k=f(B, l, hks, w_cap, ds), s_scale=1 / math.sqrt(ds))


def brute_force_map(top, nl, ns):
    hm = []
    for i in range(nl):
        Ti = set(np.flatnonzero(top[i]).tolist())
        sims = []
        for j in range(ns):
            Tj = set(np.flatnonzero(top[nl + j]).tolist())
            sims.append(Fraction(len(Ti & Tj), len(Ti | Tj)))
        best = max(sims)
        hm.append(sims.index(best))  # first (lowest) j reaching the maximum
    return np.array(hm, np.int32)


@pytest.mark.parametrize("seed", range(4))
def test_map_is_argmax_of_exact_jaccard(seed):
    x = tiny_pair(B=2, seed=seed)
    win = np.array([24, 13], np.int32)
    k = np.array([5, 4], np.int32)
    hm, scores, top = O.match(win_len=win, top_k=k, **x)
    nl, ns = 2 * 4, 3 * 2
    for b in range(2):
        w = int(win[b])
        # the TopK sets are the TopK of the reported scores ...
        for h in range(nl + ns):
            order = sorted(range(w), key=lambda v: (-float(scores[b, h, v]), v))
            assert set(np.flatnonzero(top[b, h]).tolist()) == set(order[: k[b]])
            assert not top[b, h, w:].any() and not scores[b, h, w:].any()
        # ... and the map is the argmax over exact ratios, lowest j on ties
        assert np.array_equal(hm[b], brute_force_map(top[b, :, :w], nl, ns))
        # the scores are Eq. 1 for each head's own operands
        F = causal_column_sums_fp64(x["l_q"][b, 1, 3, :w], x["l_k"][b, 1, 1, :w], x["l_scale"])
        np.testing.assert_allclose(scores[b, 4 + 3, :w], F, rtol=1e-5, atol=1e-6 * w)


def test_identical_models_map_each_head_to_itself():
    x = tiny_pair(L=3, hq=2, hk=1, d=8, l=3, hqs=2, hks=1, ds=8, seed=11)
    x["s_q"], x["s_k"], x["s_scale"] = x["l_q"].copy(), x["l_k"].copy(), x["l_scale"]
    hm, scores, top = O.match(win_len=[24], top_k=[6], **x)
    nl = 6
    assert np.array_equal(scores[0, :nl], scores[0, nl:])
    for i in range(nl):
        j = int(hm[0, i])
        assert j <= i and np.array_equal(top[0, nl + j], top[0, i])
    distinct = len({top[0, i].tobytes() for i in range(nl)}) == nl
    if distinct:
        assert np.array_equal(hm[0], np.arange(nl))


def test_map_follows_a_relabelling_of_small_layers():
    x = tiny_pair(l=4, seed=5)
    hm, _, top = O.match(win_len=[24], top_k=[5], **x)
    perm = np.array([2, 0, 3, 1])  # new layer i is old layer perm[i]
    y = dict(x)
    y["s_q"], y["s_k"] = x["s_q"][:, perm].copy(), x["s_k"][:, perm].copy()
    hm2, _, _ = O.match(win_len=[24], top_k=[5], **y)
    hqs = 2
    inv = np.argsort(perm)
    old_to_new = lambda j: inv[j // hqs] * hqs + j % hqs
    nl, ns = 8, 8
    for i in range(nl):
        sims = brute_force_map_sims(top[0], nl, ns, i)
        if sims.count(max(sims)) == 1:  # unique maximum: the relabelled map follows it
            assert hm2[0, i] == old_to_new(int(hm[0, i]))


def brute_force_map_sims(top, nl, ns, i):
    Ti = set(np.flatnonzero(top[i]).tolist())
    out = []
    for j in range(ns):
        Tj = set(np.flatnonzero(top[nl + j]).tolist())
        out.append(Fraction(len(Ti & Tj), len(Ti | Tj)))
    return out


def test_budget_and_window_clamps():
    x = tiny_pair(seed=3)
    # K >= window: every TopK set is the whole window, every ratio 1, map 0
    hm, _, top = O.match(win_len=[24], top_k=[99], **x)
    assert top[0].all() and not hm.any()
    # K = 0 reads as 1; a window beyond w_cap reads as w_cap
    hm1, s1, t1 = O.match(win_len=[500], top_k=[0], **x)
    hm2, s2, t2 = O.match(win_len=[24], top_k=[1], **x)
    assert np.array_equal(hm1, hm2) and np.array_equal(s1, s2) and np.array_equal(t1, t2)
    assert t1[0].sum(1).tolist() == [1] * t1.shape[1]


# ------------------------------------------------------ window policy --

def test_match_window_policy():
    from paper_2508_02751_amd.pipeline import MATCH_MAX, MATCH_MIN, match_window
    assert (MATCH_MIN, MATCH_MAX) == (100, 200)  # "Method Details": 100 to 200 tokens
    assert match_window(99) is None              # too short: matching is delayed
    assert match_window(100) == 100 and match_window(173) == 173
    assert match_window(200) == 200 and match_window(8192) == 200  # truncated
