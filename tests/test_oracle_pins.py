"""Pins of the CPU oracle against facts fixed outside the oracle itself.

Each test checks one oracle function against something it does not compute
the same way: exact rational arithmetic with IEEE-754 binary32 rounding,
O(N^2) rank counting, exhaustive enumeration of subsets, a textbook numpy
attention in float64, closed forms of the compensated row in special cases,
and invariants the method states (three disjoint token classes with the
budgeted sizes, Top(P-K) following TopK in one order, full attention when
every token is critical).
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O

SCALE128 = float(np.float32(1.0 / math.sqrt(128.0)))


# ------------------------------------------------------------ helpers --

def round_binary32(x: Fraction) -> Fraction:
    """Round a rational to the nearest IEEE-754 binary32 value, ties to even."""
    if x == 0:
        return Fraction(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    q = Fraction(2) ** max(e - 23, -149)
    m = a / q
    n = m.numerator // m.denominator
    rem = m - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    r = n * q
    assert r < Fraction(2) ** 128, "overflow not expected in these tests"
    return sign * r


def textbook_attention(q, K, V, scale):
    """softmax(scale * q K^T) V in float64 (independent of the oracle)."""
    s = scale * (K.astype(np.float64) @ q.astype(np.float64))
    p = np.exp(s - s.max())
    p /= p.sum()
    return p @ V.astype(np.float64), p


def rank_bruteforce(logits):
    """rank_t = #{v : s_v > s_t or (s_v == s_t and v < t)}  (O(N^2))."""
    s = [float(x) for x in logits]
    n = len(s)
    return [sum(1 for v in range(n) if s[v] > s[t] or (s[v] == s[t] and v < t))
            for t in range(n)]


def small_row(rng, n, d, ties=False, scale=0.125):
    q = rng.standard_normal(d).astype(np.float32)
    K = rng.standard_normal((n, d)).astype(np.float32)
    if ties:  # duplicated key rows force equal logits
        for t in range(0, n, 3):
            K[t] = K[(t * 7 + 1) % n]
    V = rng.standard_normal((n, d)).astype(np.float32)
    return q, K, V


# --------------------------------------------------------------- keys --

@pytest.mark.parametrize("seed", range(20))
def test_logit_is_sequential_binary32_fma_chain(seed):
    """The key equals a sequential FMA chain evaluated in exact rationals
    with binary32 rounding after every step, then one rounded multiply."""
    rng = np.random.default_rng(seed)
    d = int(rng.integers(1, 24))
    q = (rng.standard_normal(d) * 10.0 ** rng.integers(-3, 3)).astype(np.float32)
    k = (rng.standard_normal(d) * 10.0 ** rng.integers(-3, 3)).astype(np.float32)
    scale = np.float32(rng.uniform(0.01, 1.0))
    a = Fraction(0)
    for c in range(d):
        a = round_binary32(Fraction(float(q[c])) * Fraction(float(k[c])) + a)
    want = float(round_binary32(a * Fraction(float(scale))))
    got = O.logit(q, k, float(scale))
    assert got == np.float32(want)


def test_logit_order_is_observable():
    """Summation order matters in fp32, so the chain order is part of the key:
    [1e8, 1, -1e8] summed left to right loses the 1."""
    q = np.array([1.0, 1.0, 1.0], np.float32)
    k = np.array([1e8, 1.0, -1e8], np.float32)
    assert O.logit(q, k, 1.0) == np.float32(0.0)
    k2 = np.array([1e8, -1e8, 1.0], np.float32)
    assert O.logit(q, k2, 1.0) == np.float32(1.0)


def test_logit_exact_on_bf16_grid():
    """bf16 inputs whose partial sums stay exact in fp32 give the exact dot
    product times the scale (a closed form)."""
    rng = np.random.default_rng(5)
    for _ in range(50):
        q = rng.integers(-64, 65, 64).astype(np.float32) / 8
        k = rng.integers(-64, 65, 64).astype(np.float32) / 16
        exact = sum(Fraction(float(a)) * Fraction(float(b)) for a, b in zip(q, k))
        assert O.logit(q, k, 0.125) == np.float32(float(exact * Fraction(1, 8)))


def test_logit_unit_vector_and_zero():
    k = np.arange(1, 65, dtype=np.float32) * 0.37
    for c in (0, 17, 63):
        q = np.zeros(64, np.float32)
        q[c] = 1.0
        assert O.logit(q, k, 0.125) == np.float32(k[c] * np.float32(0.125))
    # -0 canonicalises to +0
    s = O.logit(np.array([-1.0], np.float32), np.array([0.0], np.float32), 1.0)
    assert s == 0.0 and math.copysign(1.0, s) == 1.0


def test_key_is_order_preserving():
    rng = np.random.default_rng(1)
    vals = np.concatenate([
        rng.standard_normal(500).astype(np.float32) * 10.0 ** rng.integers(-40, 38, 500),
        np.array([0.0, -0.0, 1e-45, -1e-45, 3.4e38, -3.4e38, 1.0, -1.0], np.float32)])
    vals = vals[np.isfinite(vals)].astype(np.float32)
    keys = np.array([O.key(float(v)) for v in vals], np.uint64)
    for i in range(len(vals)):
        for j in range(0, len(vals), 7):
            assert (keys[i] > keys[j]) == (vals[i] > vals[j])
            assert (keys[i] == keys[j]) == (vals[i] == vals[j])
    assert O.key(0.0) == O.key(-0.0)


# ------------------------------------------------------------ stage 1 --

@pytest.mark.parametrize("n,d", [(1, 64), (7, 64), (300, 64), (129, 128)])
def test_small_head_is_textbook_attention(n, d):
    rng = np.random.default_rng(n * 31 + d)
    q, K, V = small_row(rng, n, d)
    scale = float(np.float32(1 / math.sqrt(d)))
    logits, m, Z, Ohat = O.small_head(q, K, V, scale)
    Oref, pref = textbook_attention(q, K, V, scale)
    np.testing.assert_allclose(Ohat, Oref, rtol=1e-6, atol=1e-6)
    p = np.exp(logits.astype(np.float64) - m) / Z
    assert abs(p.sum() - 1.0) < 1e-12
    np.testing.assert_allclose(p, pref, rtol=1e-5, atol=1e-9)
    assert m == logits.max()


# ------------------------------------------------------------ stage 2 --

@pytest.mark.parametrize("seed", range(40))
def test_partition_matches_bruteforce_ranks(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 33))
    q, K, V = small_row(rng, n, 64, ties=bool(seed % 2))
    if seed % 4 == 3:  # coarse values: many exact ties, mixed signs, zeros
        q = np.round(q * 2) / 2
        K = np.round(K * 2) / 2
    logits, m, Z, _ = O.small_head(q, K, V, 0.125)
    kc = int(rng.integers(1, n + 3))
    km = int(rng.integers(0, n + 3))
    crit, marg, mp, mass = O.partition(logits, kc, km, m, Z, kc_cap=n + 2, km_cap=n + 2)
    rank = rank_bruteforce(logits)
    nc = min(kc, n)
    nm = min(km, n - nc)
    want_c = sorted(t for t in range(n) if rank[t] < nc)
    want_m = sorted(t for t in range(n) if nc <= rank[t] < nc + nm)
    assert list(crit[:nc]) == want_c and all(crit[nc:] == -1)
    assert list(marg[:nm]) == want_m and all(marg[nm:] == -1)
    p = np.exp(logits.astype(np.float64) - m) / Z
    np.testing.assert_allclose(mp[:nm], p[want_m], rtol=1e-13, atol=0)
    assert all(mp[nm:] == 0)
    np.testing.assert_allclose(mass, [p[want_c].sum(), p[want_m].sum()], rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("seed", range(12))
def test_partition_is_max_sum_lowest_index_subset(seed):
    """Exhaustive: among all subsets of size k, C is the one with the largest
    exact logit sum and, among equal sums, the lexicographically smallest
    ascending index tuple; C u M is the same for size k + |M|."""
    rng = np.random.default_rng(300 + seed)
    n = int(rng.integers(2, 11))
    q, K, V = small_row(rng, n, 64, ties=True)
    if seed % 3 == 0:
        q = np.round(q)
        K = np.round(K)
    logits, m, Z, _ = O.small_head(q, K, V, 0.125)
    exact = [Fraction(float(x)) for x in logits]
    kc = int(rng.integers(1, n + 1))
    km = int(rng.integers(0, n - kc + 1))
    crit, marg, _, _ = O.partition(logits, kc, km, m, Z)

    def best(k):
        return min(itertools.combinations(range(n), k),
                   key=lambda S: (-sum(exact[t] for t in S), S))

    assert tuple(crit) == best(kc)
    assert tuple(sorted(list(crit) + list(marg))) == best(kc + km)


@pytest.mark.parametrize("n,kc,km", [(5, 9, 4), (5, 5, 3), (5, 3, 9), (1, 1, 0), (1, 4, 4), (8, 2, 0)])
def test_partition_budget_clamping(n, kc, km):
    rng = np.random.default_rng(n + kc + km)
    q, K, V = small_row(rng, n, 64)
    logits, m, Z, _ = O.small_head(q, K, V, 0.125)
    crit, marg, mp, mass = O.partition(logits, kc, km, m, Z, kc_cap=10, km_cap=10)
    nc, nm = min(kc, n), min(km, n - min(kc, n))
    assert (crit >= 0).sum() == nc and (marg >= 0).sum() == nm
    assert set(crit[:nc]).isdisjoint(set(marg[:nm]))
    if nc + nm == n:
        assert abs(mass.sum() - 1.0) < 1e-12
    with pytest.raises(O.OracleError):
        O.partition(logits, 0, km, m, Z, kc_cap=10, km_cap=10)


def test_partition_class_order_invariant():
    """Every critical key >= every marginal key >= every evicted key."""
    rng = np.random.default_rng(9)
    q, K, V = small_row(rng, 4096, 64, ties=True)
    logits, m, Z, _ = O.small_head(q, K, V, 0.125)
    crit, marg, _, _ = O.partition(logits, 400, 900, m, Z)
    ev = np.setdiff1d(np.arange(4096), np.concatenate([crit, marg]))
    assert len(crit) == 400 and len(marg) == 900 and len(ev) == 4096 - 1300
    assert np.all(np.diff(crit) > 0) and np.all(np.diff(marg) > 0)
    assert logits[crit].min() >= logits[marg].max() >= logits[ev].max()
    # ties across a boundary go to the lower index
    for a, b in ((crit, marg), (marg, ev)):
        t = logits[a].min()
        if t in logits[b]:
            assert a[logits[a] == t].max() < b[logits[b] == t].min()


# ------------------------------------------------- stage 2, recent tokens --
# Experimental setup: the budget is split 2 : 1 : 2 between critical, recent
# and marginal tokens; recent tokens are kept whatever their score.

@pytest.mark.parametrize("seed", range(40))
def test_partition_recent_window_matches_bruteforce(seed):
    """The last r tokens are critical; the older ones are ranked alone (O(N^2)
    counting over the older prefix) for the critical and marginal budgets."""
    rng = np.random.default_rng(500 + seed)
    n = int(rng.integers(1, 33))
    q, K, V = small_row(rng, n, 64, ties=bool(seed % 2))
    if seed % 4 == 3:
        q = np.round(q * 2) / 2
        K = np.round(K * 2) / 2
    logits, m, Z, _ = O.small_head(q, K, V, 0.125)
    kc = int(rng.integers(1, n + 3))
    km = int(rng.integers(0, n + 3))
    kr = int(rng.integers(0, n + 3))
    crit, marg, mp, mass = O.partition(logits, kc, km, m, Z, kc_cap=2 * n + 4, km_cap=n + 2,
                                       k_recent=kr)
    r = min(kr, n)
    older = n - r
    rank = rank_bruteforce(logits[:older])
    ntop = min(kc, older)
    nm = min(km, older - ntop)
    want_c = sorted([t for t in range(older) if rank[t] < ntop] + list(range(older, n)))
    want_m = sorted(t for t in range(older) if ntop <= rank[t] < ntop + nm)
    nc = ntop + r
    assert list(crit[:nc]) == want_c and all(crit[nc:] == -1)
    assert list(marg[:nm]) == want_m and all(marg[nm:] == -1)
    p = np.exp(logits.astype(np.float64) - m) / Z
    np.testing.assert_allclose(mp[:nm], p[want_m], rtol=1e-13, atol=0)
    np.testing.assert_allclose(mass, [p[want_c].sum(), p[want_m].sum()], rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("seed", range(8))
def test_partition_recent_top_is_max_sum_subset_of_older(seed):
    """Exhaustive: C minus the recent tokens is the size-k subset of the older
    tokens with the largest exact logit sum (lowest indices among equal sums)."""
    rng = np.random.default_rng(600 + seed)
    n = int(rng.integers(3, 11))
    q, K, V = small_row(rng, n, 64, ties=True)
    logits, m, Z, _ = O.small_head(q, K, V, 0.125)
    exact = [Fraction(float(x)) for x in logits]
    kr = int(rng.integers(1, n - 1))
    older = n - kr
    kc = int(rng.integers(1, older + 1))
    km = int(rng.integers(0, older - kc + 1))
    crit, marg, _, _ = O.partition(logits, kc, km, m, Z, kc_cap=kc + kr, k_recent=kr)

    def best(k):
        return min(itertools.combinations(range(older), k),
                   key=lambda S: (-sum(exact[t] for t in S), S))

    assert tuple(crit[:kc]) == best(kc) and tuple(crit[kc:]) == tuple(range(older, n))
    assert tuple(sorted(list(crit[:kc]) + list(marg))) == best(kc + km)


def test_partition_recent_window_special_cases():
    rng = np.random.default_rng(42)
    q, K, V = small_row(rng, 50, 64, ties=True)
    logits, m, Z, _ = O.small_head(q, K, V, 0.125)
    # no recent tokens: the plain partition
    for a, b in zip(O.partition(logits, 7, 11, m, Z), O.partition(logits, 7, 11, m, Z, k_recent=0)):
        np.testing.assert_array_equal(a, b)
    # the whole sequence recent: everything critical, nothing marginal
    crit, marg, mp, mass = O.partition(logits, 7, 11, m, Z, kc_cap=50, km_cap=11, k_recent=60)
    assert list(crit) == list(range(50)) and all(marg == -1)
    np.testing.assert_allclose(mass, [1.0, 0.0], rtol=1e-12, atol=0)
    # the budgets do not fit in the caps: rejected
    with pytest.raises(O.OracleError):
        O.partition(logits, 7, 11, m, Z, kc_cap=7 + 4, km_cap=11, k_recent=5)
    with pytest.raises(O.OracleError):
        O.partition(logits, 7, 11, m, Z, kc_cap=20, km_cap=11, k_recent=-1)


# ------------------------------------------------------------ stage 3 --

def _hybrid_setup(seed, n, d=64):
    """'Identical models': the large head sees the same q, K and scale as the
    small head, so its exact attention is the small model's."""
    rng = np.random.default_rng(seed)
    q, K, V = small_row(rng, n, d, ties=False)
    scale = float(np.float32(1 / math.sqrt(d)))
    logits, m, Z, _ = O.small_head(q, K, V, scale)
    Vl = rng.standard_normal((n, d)).astype(np.float32)  # the large model's V
    return q, K, Vl, scale, logits, m, Z


@pytest.mark.parametrize("mode", O.MODES)
def test_hybrid_all_critical_is_full_attention(mode):
    q, K, V, scale, logits, m, Z = _hybrid_setup(1, 200, 128)
    crit, marg, mp, mass = O.partition(logits, 200, 50, m, Z, kc_cap=200, km_cap=50)
    out = O.hybrid_head(q, K, V, crit, marg, mp, mass, scale, mode)
    ref, _ = textbook_attention(q, K, V, scale)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("mode", [O.NORM_REMAINING, O.NORM_SLM_CRIT, O.NORM_RETAINED, O.NORM_MARG_FILL])
@pytest.mark.parametrize("kc", [1, 17, 150])
def test_hybrid_identical_models_no_eviction_is_full_attention(mode, kc):
    n = 160
    q, K, V, scale, logits, m, Z = _hybrid_setup(2 + kc, n)
    crit, marg, mp, mass = O.partition(logits, kc, n - kc, m, Z)
    out = O.hybrid_head(q, K, V, crit, marg, mp, mass, scale, mode)
    ref, _ = textbook_attention(q, K, V, scale)
    np.testing.assert_allclose(out, ref, rtol=2e-6, atol=2e-6)


def test_hybrid_literal_sum_overweights_marginal():
    """O_c + O_m taken literally carries weight 1 + S'_M, so it misses full
    attention even with nothing evicted (why it is not the default)."""
    n = 160
    q, K, V, scale, logits, m, Z = _hybrid_setup(7, n)
    crit, marg, mp, mass = O.partition(logits, 10, n - 10, m, Z)
    ones = np.ones_like(V)
    w = O.hybrid_head(q, K, ones, crit, marg, mp, mass, scale, O.NORM_NONE)
    np.testing.assert_allclose(w, 1.0 + mass[1], rtol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_hybrid_identical_models_with_eviction(seed):
    """Eq. 6 with the small model exact: A on C, A' on M, 0 elsewhere.
    SLM_CRIT reproduces it; RETAINED is softmax restricted to C u M."""
    n = 240
    q, K, V, scale, logits, m, Z = _hybrid_setup(20 + seed, n)
    crit, marg, mp, mass = O.partition(logits, 30, 70, m, Z)
    _, p = textbook_attention(q, K, V, scale)
    keep = np.concatenate([crit, marg])
    eq6 = p[keep] @ V[keep].astype(np.float64)
    out = O.hybrid_head(q, K, V, crit, marg, mp, mass, scale, O.NORM_SLM_CRIT)
    np.testing.assert_allclose(out, eq6, rtol=2e-6, atol=2e-6)
    out = O.hybrid_head(q, K, V, crit, marg, mp, mass, scale, O.NORM_RETAINED)
    np.testing.assert_allclose(out, eq6 / p[keep].sum(), rtol=2e-6, atol=2e-6)


@pytest.mark.parametrize("mode,weight", [
    (O.NORM_REMAINING, lambda sc, sm: 1.0), (O.NORM_NONE, lambda sc, sm: 1.0 + sm),
    (O.NORM_SLM_CRIT, lambda sc, sm: sc + sm), (O.NORM_RETAINED, lambda sc, sm: 1.0),
    (O.NORM_MARG_FILL, lambda sc, sm: 1.0)])
def test_hybrid_weight_sum(mode, weight):
    n = 300
    rng = np.random.default_rng(77)
    q, K, _ = small_row(rng, n, 128)
    qs, Ks, Vs = small_row(rng, n, 64)
    logits, m, Z, _ = O.small_head(qs, Ks, Vs, 0.125)
    crit, marg, mp, mass = O.partition(logits, 40, 90, m, Z)
    out = O.hybrid_head(q, K, np.ones((n, 128), np.float32), crit, marg, mp, mass, SCALE128, mode)
    np.testing.assert_allclose(out, weight(mass[0], mass[1]), rtol=1e-12)


def test_hybrid_single_critical_is_its_value_row():
    n = 50
    rng = np.random.default_rng(3)
    q, K, V = small_row(rng, n, 128)
    logits, m, Z, _ = O.small_head(*small_row(rng, n, 64), 0.125)
    crit, marg, mp, mass = O.partition(logits, 1, 0, m, Z, km_cap=0)
    for mode in (O.NORM_REMAINING, O.NORM_NONE, O.NORM_RETAINED):
        out = O.hybrid_head(q, K, V, crit, marg, mp, mass, SCALE128, mode)
        np.testing.assert_allclose(out, V[crit[0]].astype(np.float64), rtol=0, atol=0)


def test_hybrid_uses_large_values_and_slots():
    """Rows reached through slot maps give the same output as identity rows;
    changing a V row outside C u M changes nothing, inside it does."""
    n, d = 120, 128
    rng = np.random.default_rng(4)
    q, K, V = small_row(rng, n, d)
    logits, m, Z, _ = O.small_head(*small_row(rng, n, 64), 0.125)
    crit, marg, mp, mass = O.partition(logits, 12, 30, m, Z)
    base = O.hybrid_head(q, K, V, crit, marg, mp, mass, SCALE128)
    perm = rng.permutation(n).astype(np.int32)
    Kp = np.empty_like(K)
    Vp = np.empty_like(V)
    Kp[perm] = K
    Vp[perm] = V
    out = O.hybrid_head(q, Kp, Vp, crit, marg, mp, mass, SCALE128, k_slot=perm, v_slot=perm)
    np.testing.assert_allclose(out, base, rtol=1e-13, atol=1e-13)
    ev = np.setdiff1d(np.arange(n), np.concatenate([crit, marg]))[0]
    V2 = V.copy()
    V2[ev] += 100
    np.testing.assert_array_equal(O.hybrid_head(q, K, V2, crit, marg, mp, mass, SCALE128), base)
    V3 = V.copy()
    V3[marg[0]] += 100
    assert np.abs(O.hybrid_head(q, K, V3, crit, marg, mp, mass, SCALE128) - base).max() > 1e-3
    # a token the store does not hold is an error
    vs = perm.copy()
    vs[marg[0]] = -1
    with pytest.raises(O.OracleError):
        O.hybrid_head(q, Kp, Vp, crit, marg, mp, mass, SCALE128, k_slot=perm, v_slot=vs)


# ----------------------------------------------------------- whole step --

def test_step_composes_the_three_stages():
    """orc_step over the tensor layout equals the per-head functions applied
    one by one, and with every token critical both models' outputs are
    textbook full attention."""
    rng = np.random.default_rng(11)
    B, ncap, l, hqs, hks, ds = 2, 40, 2, 4, 2, 64
    L, hq, hk, d = 3, 6, 3, 128
    sq = rng.standard_normal((B, l, hqs, ds)).astype(np.float32)
    sk = rng.standard_normal((B, l, hks, ncap, ds)).astype(np.float32)
    sv = rng.standard_normal((B, l, hks, ncap, ds)).astype(np.float32)
    lq = rng.standard_normal((B, L, hq, d)).astype(np.float32)
    lk = rng.standard_normal((B, L, hk, ncap, d)).astype(np.float32)
    lv = rng.standard_normal((B, L, hk, ncap, d)).astype(np.float32)
    seq = np.array([40, 23], np.int32)
    hm = rng.integers(0, l * hqs, L * hq).astype(np.int32)
    for kc, km, kr in ((np.array([5, 3]), np.array([9, 30]), None),
                       (np.array([5, 3]), np.array([9, 12]), np.array([4, 30])),
                       (np.array([40, 40]), np.array([0, 0]), None)):
        r = O.step(seq_len=seq, k_crit=kc, k_marg=km, kc_cap=40, km_cap=30, head_map=hm,
                   mode=O.NORM_REMAINING, s_q=sq, s_k=sk, s_v=sv, s_scale=0.125,
                   l_q=lq, l_k=lk, l_v=lv, l_scale=SCALE128, k_recent=kr)
        for b in range(B):
            n = seq[b]
            for j in range(l * hqs):
                lay, h = divmod(j, hqs)
                g = h // (hqs // hks)
                lg, m, Z, Os = O.small_head(sq[b, lay, h], sk[b, lay, g, :n], sv[b, lay, g, :n], 0.125)
                np.testing.assert_array_equal(r["logits"][b, j, :n], lg)
                np.testing.assert_array_equal(r["small_out"][b, lay, h], Os)
                c, mg, mp, ms = O.partition(lg, int(kc[b]), int(km[b]), m, Z, kc_cap=40, km_cap=30,
                                            k_recent=0 if kr is None else int(kr[b]))
                np.testing.assert_array_equal(r["crit"][b, j], c)
                np.testing.assert_array_equal(r["marg"][b, j], mg)
                np.testing.assert_array_equal(r["mass"][b, j], ms)
            for lay in range(L):
                for h in range(hq):
                    j = hm[lay * hq + h]
                    g = h // (hq // hk)
                    o = O.hybrid_head(lq[b, lay, h], lk[b, lay, g], lv[b, lay, g], r["crit"][b, j],
                                      r["marg"][b, j], r["marg_prob"][b, j], r["mass"][b, j], SCALE128)
                    np.testing.assert_array_equal(r["large_out"][b, lay, h], o)
                    if kc[0] == 40:
                        ref, _ = textbook_attention(lq[b, lay, h], lk[b, lay, g, :n], lv[b, lay, g, :n], SCALE128)
                        np.testing.assert_allclose(r["large_out"][b, lay, h], ref, rtol=1e-10, atol=1e-12)


# ---------------------------------------- small model's own KV eviction --

def _evicted_small_store(rng, sk, sv, held, ncap_rows):
    """Each (sequence, layer, kv head) keeps `held[b]` ascending positions
    (tokens 0 and the last one always among them); returns the compact store
    and its row -> position map."""
    B, l, hks, ncap, ds = sk.shape
    pos = np.full((B, l, hks, ncap_rows), -1, np.int32)
    ck = np.zeros((B, l, hks, ncap_rows, ds), np.float32)
    cv = np.zeros_like(ck)
    for b in range(B):
        for la in range(l):
            for g in range(hks):
                n = held[b][1]
                keep = np.sort(np.concatenate([[0, n - 1], rng.choice(np.arange(1, n - 1), held[b][0] - 2,
                                                                     replace=False)]))
                pos[b, la, g, :keep.size] = keep
                ck[b, la, g, :keep.size] = sk[b, la, g, keep]
                cv[b, la, g, :keep.size] = sv[b, la, g, keep]
    return ck, cv, pos


def test_step_with_all_rows_held_is_the_plain_step():
    rng = np.random.default_rng(21)
    B, ncap, l, hqs, hks, ds, L, hq, hk, d = 2, 48, 2, 4, 2, 64, 2, 4, 2, 128
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    sq, sk, sv = f(B, l, hqs, ds), f(B, l, hks, ncap, ds), f(B, l, hks, ncap, ds)
    lq, lk, lv = f(B, L, hq, d), f(B, L, hk, ncap, d), f(B, L, hk, ncap, d)
    seq = np.array([48, 30], np.int32)
    kc, km = np.array([6, 4], np.int32), np.array([10, 7], np.int32)
    hm = rng.integers(0, l * hqs, L * hq).astype(np.int32)
    common = dict(seq_len=seq, k_crit=kc, k_marg=km, kc_cap=8, km_cap=12, head_map=hm,
                  mode=O.NORM_REMAINING, s_q=sq, s_v=None, s_scale=0.125, l_q=lq, l_k=lk, l_v=lv,
                  l_scale=SCALE128)
    plain = O.step(**{**common, "s_k": sk, "s_v": sv})
    pos = np.broadcast_to(np.arange(ncap, dtype=np.int32), (B, l, hks, ncap)).copy()
    held = O.step(**{**common, "s_k": sk, "s_v": sv}, s_held=seq, s_row_pos=pos, n_cap=ncap)
    for k in ("crit", "marg", "marg_prob", "mass", "small_out", "large_out", "row_max", "row_sum"):
        np.testing.assert_array_equal(plain[k], held[k], err_msg=k)


@pytest.mark.parametrize("recent", [False, True])
def test_step_with_evicted_small_cache_brute_force(recent):
    """The lists are the top of the held tokens only, ranked by the small
    model's logit over its held rows (fp64 numpy), named by position; a token
    the small model dropped is never critical or marginal."""
    rng = np.random.default_rng(22 + recent)
    B, ncap, l, hqs, hks, ds, L, hq, hk, d = 2, 64, 2, 4, 2, 64, 1, 4, 2, 128
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    sq, sk, sv = f(B, l, hqs, ds), f(B, l, hks, ncap, ds), f(B, l, hks, ncap, ds)
    lq, lk, lv = f(B, L, hq, d), f(B, L, hk, ncap, d), f(B, L, hk, ncap, d)
    seq = np.array([64, 41], np.int32)
    held = np.array([26, 17], np.int32)  # about 40% of each sequence
    ck, cv, pos = _evicted_small_store(rng, sk, sv, [(26, 64), (17, 41)], 32)
    kc, km = np.array([5, 3], np.int32), np.array([8, 6], np.int32)
    kr = np.array([3, 2], np.int32) if recent else None
    hm = rng.integers(0, l * hqs, L * hq).astype(np.int32)
    r = O.step(seq_len=seq, k_crit=kc, k_marg=km, kc_cap=8, km_cap=8, head_map=hm,
               mode=O.NORM_REMAINING, s_q=sq, s_k=ck, s_v=cv, s_scale=0.125, l_q=lq, l_k=lk,
               l_v=lv, l_scale=SCALE128, k_recent=kr, s_held=held, s_row_pos=pos, n_cap=ncap)
    for b in range(B):
        nh = int(held[b])
        rr = 0 if kr is None else int(kr[b])
        for j in range(l * hqs):
            la, h = divmod(j, hqs)
            g = h // (hqs // hks)
            p = pos[b, la, g, :nh]
            s = (ck[b, la, g, :nh].astype(np.float64) @ sq[b, la, h].astype(np.float64)) * 0.125
            older = nh - rr
            order = sorted(range(older), key=lambda t: (-s[t], t))
            ntop = min(int(kc[b]), older)
            crit = sorted(set(p[order[:ntop]].tolist()) | set(p[older:].tolist()))
            marg = sorted(p[order[ntop:ntop + min(int(km[b]), older - ntop)]].tolist())
            got_c = r["crit"][b, j][r["crit"][b, j] >= 0].tolist()
            got_m = r["marg"][b, j][r["marg"][b, j] >= 0].tolist()
            assert got_c == crit and got_m == marg
            assert set(got_c + got_m) <= set(p.tolist())
            # the small model's softmax runs over its held rows only
            e = np.exp(s - s.max())
            np.testing.assert_allclose(r["row_sum"][b, j], e.sum(), rtol=1e-5)  # fp32 logits


def test_step_rejects_a_bad_position_map():
    rng = np.random.default_rng(23)
    B, ncap, l, hqs, hks, ds, L, hq, hk, d = 1, 32, 1, 2, 1, 64, 1, 2, 1, 128
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    args = dict(seq_len=np.array([32], np.int32), k_crit=np.array([3], np.int32),
                k_marg=np.array([4], np.int32), kc_cap=4, km_cap=4,
                head_map=np.zeros(2, np.int32), mode=O.NORM_REMAINING, s_q=f(1, 1, 2, 64),
                s_k=f(1, 1, 1, 16, 64), s_v=f(1, 1, 1, 16, 64), s_scale=0.125,
                l_q=f(1, 1, 2, 128), l_k=f(1, 1, 1, 32, 128), l_v=f(1, 1, 1, 32, 128),
                l_scale=SCALE128, s_held=np.array([10], np.int32), n_cap=32)
    good = np.arange(0, 32, 2, dtype=np.int32).reshape(1, 1, 1, 16)
    O.step(**args, s_row_pos=good)
    for bad in (good[..., ::-1].copy(), good + 20):  # descending; beyond the sequence
        with pytest.raises(O.OracleError):
            O.step(**args, s_row_pos=bad)


# ------------------------------------------------- group selection (GQA) --

def test_zq_closed_form_and_error_bound():
    # equal logits: every term is exactly 2^40, so Zq = n exactly
    for n in (1, 7, 4096, 65536):
        assert O.zq(np.full(n, 0.37, np.float32), 0.37) == np.float32(n)
    rng = np.random.default_rng(31)
    for n, sc in ((100, 1.0), (8192, 3.0), (65536, 0.5)):
        s = (rng.standard_normal(n) * sc).astype(np.float32)
        s[:4] += 8 * sc  # sink-like
        m = np.float32(s.max())
        z = float(O.zq(s, m))
        ref = float(np.exp(s.astype(np.float64) - float(m)).sum())
        # truncation (< 2^-40 per term), exp (1 ulp) and the final rounding
        assert abs(z - ref) <= n * 2.0 ** -40 + 3e-7 * ref, (n, z, ref)


def _group_case(rng, B=1, n=96, l=2, hqs=4, hks=2, ds=16, L=2, hq=8, hk=2, d=128, separated=True,
                head_map=None):
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    sq, sk, sv = f(B, l, hqs, ds), f(B, l, hks, n, ds), f(B, l, hks, n, ds)
    if separated:
        # logits of every small head are distinct and at least 0.02 apart:
        # q = e_0, k_t[0] = a permutation of an arithmetic sequence
        sq[:] = 0.0
        sq[..., 0] = np.sqrt(ds)
        for b in range(B):
            for la in range(l):
                for g in range(hks):
                    sk[b, la, g, :, 0] = rng.permutation(np.arange(n) * 0.02 - 1.0)
                    sk[b, la, g, :, 1:] = 0.0
    lq, lk, lv = f(B, L, hq, d), f(B, L, hk, n, d), f(B, L, hk, n, d)
    hm = rng.integers(0, l * hqs, L * hq).astype(np.int32) if head_map is None else head_map
    return dict(seq_len=np.full(B, n, np.int32), s_q=sq, s_k=sk, s_v=sv, s_scale=1 / np.sqrt(ds),
                l_q=lq, l_k=lk, l_v=lv, l_scale=SCALE128, head_map=hm)


def _run(x, kc, km, select, kr=None, mode=O.NORM_REMAINING):
    B = x["seq_len"].size
    return O.step(**x, k_crit=np.full(B, kc, np.int32), k_marg=np.full(B, km, np.int32),
                  kc_cap=kc + (kr or 0), km_cap=km, mode=mode, select=select,
                  k_recent=None if kr is None else np.full(B, kr, np.int32))


def test_group_selection_of_one_head_groups_is_per_head_selection():
    rng = np.random.default_rng(32)
    x = _group_case(rng, L=2, hq=4, hk=4)  # every kv head serves one query head
    for kr in (None, 5):
        head = _run(x, 9, 14, O.SELECT_HEAD, kr)
        grp = _run(x, 9, 14, O.SELECT_GROUP, kr)
        hm = x["head_map"]
        for i in range(8):
            j = hm[i]
            np.testing.assert_array_equal(grp["crit"][0, i], head["crit"][0, j])
            np.testing.assert_array_equal(grp["marg"][0, i], head["marg"][0, j])
            np.testing.assert_allclose(grp["marg_prob"][0, i], head["marg_prob"][0, j], rtol=1e-12)
            np.testing.assert_allclose(grp["mass"][0, i], head["mass"][0, j], rtol=1e-12)
        np.testing.assert_allclose(grp["large_out"], head["large_out"], rtol=1e-12, atol=1e-15)


def test_group_whose_heads_share_a_small_head_selects_like_it():
    rng = np.random.default_rng(33)
    hm = np.repeat(rng.integers(0, 8, 4), 4).astype(np.int32)  # 4 groups of 4 query heads
    x = _group_case(rng, L=2, hq=8, hk=2, head_map=hm)
    head = _run(x, 7, 11, O.SELECT_HEAD)
    grp = _run(x, 7, 11, O.SELECT_GROUP)
    for gi in range(4):
        j = hm[4 * gi]
        np.testing.assert_array_equal(grp["crit"][0, gi], head["crit"][0, j])
        np.testing.assert_array_equal(grp["marg"][0, gi], head["marg"][0, j])


@pytest.mark.parametrize("seed", range(3))
def test_group_selection_is_the_top_of_the_exact_sum(seed):
    """The group's C and M are a top-|C| and next-|M| of the fp64 sum of the
    heads' probabilities, up to fp32 rounding; weights are each head's own."""
    rng = np.random.default_rng(40 + seed)
    x = _group_case(rng, n=150, separated=False)
    kc, km = 12, 20
    r = _run(x, kc, km, O.SELECT_GROUP)
    L, hq, hk = 2, 8, 2
    gq = hq // hk
    logits = r["logits"][0].astype(np.float64)
    p = np.exp(logits - logits.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    for li in range(L):
        for g in range(hk):
            js = x["head_map"][li * hq + g * gq: li * hq + (g + 1) * gq]
            F = p[js].sum(0)
            c = r["crit"][0, li * hk + g]
            m = r["marg"][0, li * hk + g]
            assert c.size == kc and m.size == km and not set(c) & set(m)
            rest = np.setdiff1d(np.arange(150), np.concatenate([c, m]))
            tol = 1e-5 * F.max()
            assert F[c].min() >= F[np.concatenate([m, rest])].max() - tol
            assert F[m].min() >= F[rest].max() - tol
            for h in range(gq):
                i = li * hq + g * gq + h
                np.testing.assert_allclose(r["marg_prob"][0, i], p[js[h], m], rtol=1e-12)
                np.testing.assert_allclose(r["mass"][0, i], [p[js[h], c].sum(), p[js[h], m].sum()],
                                           rtol=1e-12)


def test_group_selection_with_everything_critical_is_full_attention():
    rng = np.random.default_rng(34)
    x = _group_case(rng, n=60, separated=False)
    r = _run(x, 60, 0, O.SELECT_GROUP)
    lq, lk, lv = x["l_q"], x["l_k"], x["l_v"]
    for li in range(2):
        for h in range(8):
            g = h // 4
            s = (lk[0, li, g].astype(np.float64) @ lq[0, li, h].astype(np.float64)) * SCALE128
            w = np.exp(s - s.max())
            w /= w.sum()
            np.testing.assert_allclose(r["large_out"][0, li, h], w @ lv[0, li, g].astype(np.float64),
                                       rtol=1e-9, atol=1e-12)


# ------------------------------------------- accumulated scores (H2O-style) --

def _acc_run(x, kc, km, acc, kr=None):
    B = x["seq_len"].size
    return O.step(**x, k_crit=np.full(B, kc, np.int32), k_marg=np.full(B, km, np.int32),
                  kc_cap=kc + (kr or 0), km_cap=km, mode=O.NORM_REMAINING,
                  select=O.SELECT_ACCUM, acc=acc,
                  k_recent=None if kr is None else np.full(B, kr, np.int32))


def test_accumulated_first_step_is_per_head_selection():
    rng = np.random.default_rng(51)
    x = _group_case(rng, n=96)
    nsh = 2 * 4
    for kr in (None, 6):
        acc = np.zeros((1, nsh, 96), np.float32)
        r = _acc_run(x, 9, 14, acc, kr)
        head = _run(x, 9, 14, O.SELECT_HEAD, kr)
        for k in ("crit", "marg", "marg_prob", "mass", "large_out"):
            np.testing.assert_allclose(r[k], head[k], rtol=1e-12, atol=1e-15, err_msg=k)
        # the state holds this step's probabilities
        lg = r["logits"][0].astype(np.float64)
        p = np.exp(lg - lg.max(1, keepdims=True))
        p /= p.sum(1, keepdims=True)
        np.testing.assert_allclose(acc[0], p, rtol=1e-6, atol=1e-12)


def test_accumulated_identical_steps_sum_up():
    rng = np.random.default_rng(52)
    x = _group_case(rng, n=64)
    acc = np.zeros((1, 8, 64), np.float32)
    for _ in range(5):
        r = _acc_run(x, 5, 8, acc)
    lg = r["logits"][0].astype(np.float64)
    p = np.exp(lg - lg.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    np.testing.assert_allclose(acc[0], 5 * p, rtol=5e-6, atol=1e-12)
    head = _run(x, 5, 8, O.SELECT_HEAD)
    np.testing.assert_array_equal(r["crit"], head["crit"])


def test_accumulated_keeps_an_earlier_heavy_hitter():
    """Step 1 attends token 7 strongly; step 2 prefers token 20 slightly.  The
    accumulated score keeps 7 critical (K = 1); the current step alone picks 20."""
    n, ds = 32, 16
    sk = np.zeros((1, 1, 1, n, ds), np.float32)
    sk[0, 0, 0, :, 0] = np.linspace(-1, 1, n)
    sk[0, 0, 0, 7, 1] = 4.0
    sk[0, 0, 0, 20, 2] = 4.0
    sv = np.ones_like(sk)
    base = dict(seq_len=np.array([n], np.int32), s_k=sk, s_v=sv, s_scale=1.0,
                l_q=np.ones((1, 1, 1, 128), np.float32), l_k=np.ones((1, 1, 1, n, 128), np.float32),
                l_v=np.ones((1, 1, 1, n, 128), np.float32), l_scale=SCALE128,
                head_map=np.zeros(1, np.int32))
    q1 = np.zeros((1, 1, 1, ds), np.float32)
    q1[..., 1] = 3.0                    # step 1: token 7 dominates
    q2 = np.zeros((1, 1, 1, ds), np.float32)
    q2[..., 1], q2[..., 2] = 1.0, 1.2   # step 2: token 20 slightly ahead of 7
    acc = np.zeros((1, 1, n), np.float32)
    _acc_run({**base, "s_q": q1}, 1, 0, acc)
    r2 = _acc_run({**base, "s_q": q2}, 1, 0, acc)
    head2 = _run({**base, "s_q": q2}, 1, 0, O.SELECT_HEAD)
    assert r2["crit"][0, 0].tolist() == [7] and head2["crit"][0, 0].tolist() == [20]


def test_accumulated_over_growing_steps_is_the_top_of_the_running_sum():
    rng = np.random.default_rng(53)
    ncap, l, hqs, hks, ds = 80, 1, 4, 2, 16
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    sk, sv = f(1, l, hks, ncap, ds), f(1, l, hks, ncap, ds)
    lk, lv = f(1, 1, 2, ncap, 128), f(1, 1, 2, ncap, 128)
    acc = np.zeros((1, l * hqs, ncap), np.float32)
    run64 = np.zeros((l * hqs, ncap))
    for step, n in enumerate((60, 61, 62, 63)):
        x = dict(seq_len=np.array([n], np.int32), s_q=f(1, l, hqs, ds), s_k=sk, s_v=sv,
                 s_scale=0.25, l_q=f(1, 1, 4, 128), l_k=lk, l_v=lv, l_scale=SCALE128,
                 head_map=np.arange(4, dtype=np.int32))
        r = _acc_run(x, 6, 9, acc)
        lg = r["logits"][0][:, :n].astype(np.float64)
        p = np.exp(lg - lg.max(1, keepdims=True))
        run64[:, :n] += p / p.sum(1, keepdims=True)
        for j in range(l * hqs):
            c, m = r["crit"][0, j], r["marg"][0, j]
            rest = np.setdiff1d(np.arange(n), np.concatenate([c, m]))
            tol = 1e-5 * run64[j].max()
            assert run64[j, c].min() >= run64[j, np.concatenate([m, rest])].max() - tol
            assert run64[j, m].min() >= run64[j, rest].max() - tol


# ----------------------------------------------------- store maintenance --

def _store_case(rng, select=O.SELECT_HEAD, B=2, n=70, L=2, hq=8, hk=2):
    x = _group_case(rng, B=B, n=n, L=L, hq=hq, hk=hk, separated=False)
    r = _run(x, 6, 10, select)
    return x, r


@pytest.mark.parametrize("select", [O.SELECT_HEAD, O.SELECT_GROUP])
def test_store_serves_stage3_like_the_full_cache(select):
    rng = np.random.default_rng(61 + select)
    x, r = _store_case(rng, select)
    B, L, hq, hk = 2, 2, 8, 2
    nk, nv, ks, vs, cnt = O.store_update(seq_len=x["seq_len"], head_map=x["head_map"],
                                         crit=r["crit"], marg=r["marg"], full_k=x["l_k"],
                                         full_v=x["l_v"], rows=70, n_small_heads=8, select=select)
    for b in range(B):
        for li in range(L):
            for h in range(hq):
                g = h // (hq // hk)
                row = (li * hk + g) if select == O.SELECT_GROUP else x["head_map"][li * hq + h]
                prow = li * hq + h if select == O.SELECT_GROUP else row
                args = (x["l_q"][b, li, h], None, None, r["crit"][b, row], r["marg"][b, row],
                        r["marg_prob"][b, prow], r["mass"][b, prow], SCALE128)
                full = O.hybrid_head(x["l_q"][b, li, h], x["l_k"][b, li, g], x["l_v"][b, li, g],
                                     *args[3:])
                store = O.hybrid_head(x["l_q"][b, li, h], nk[b, li, g], nv[b, li, g], *args[3:],
                                      k_slot=ks[b, li, g], v_slot=vs[b, li, g])
                np.testing.assert_array_equal(store, full)


def test_store_rows_are_the_ascending_unions():
    rng = np.random.default_rng(63)
    x, r = _store_case(rng)
    nk, nv, ks, vs, cnt = O.store_update(seq_len=x["seq_len"], head_map=x["head_map"],
                                         crit=r["crit"], marg=r["marg"], full_k=x["l_k"],
                                         full_v=x["l_v"], rows=70, n_small_heads=8)
    hq, hk = 8, 2
    for b in range(2):
        n = int(x["seq_len"][b])
        for li in range(2):
            for g in range(hk):
                js = x["head_map"][li * hq + g * 4: li * hq + (g + 1) * 4]
                UK = sorted(set().union(*[set(r["crit"][b, j][r["crit"][b, j] >= 0].tolist())
                                          for j in js]))
                UV = sorted(set(UK).union(*[set(r["marg"][b, j][r["marg"][b, j] >= 0].tolist())
                                            for j in js]))
                assert cnt[b, li, g].tolist() == [len(UK), len(UV)]
                assert [int(np.flatnonzero(ks[b, li, g, :n] == i)[0]) for i in range(len(UK))] == UK
                assert [int(np.flatnonzero(vs[b, li, g, :n] == i)[0]) for i in range(len(UV))] == UV
                assert (ks[b, li, g, :n] >= 0).sum() == len(UK)
                np.testing.assert_array_equal(nk[b, li, g, :len(UK)], x["l_k"][b, li, g, UK])
                np.testing.assert_array_equal(nv[b, li, g, :len(UV)], x["l_v"][b, li, g, UV])


def test_store_copies_held_rows_from_the_old_store():
    rng = np.random.default_rng(64)
    x, r = _store_case(rng)
    common = dict(seq_len=x["seq_len"], head_map=x["head_map"], full_k=x["l_k"], full_v=x["l_v"],
                  rows=70, n_small_heads=8)
    ok, ov, oks, ovs, _ = O.store_update(**common, crit=r["crit"], marg=r["marg"])
    ok, ov = ok + 1000.0, ov - 1000.0  # an old store distinguishable from the full one
    x2 = dict(x)
    x2["s_q"] = rng.standard_normal(x["s_q"].shape).astype(np.float32)
    r2 = _run(x2, 6, 10, O.SELECT_HEAD)
    nk, nv, ks, vs, cnt = O.store_update(**common, crit=r2["crit"], marg=r2["marg"], old_k=ok,
                                         old_v=ov, old_k_slot=oks, old_v_slot=ovs)
    for b in range(2):
        n = int(x["seq_len"][b])
        for li in range(2):
            for g in range(2):
                for t in range(n):
                    if ks[b, li, g, t] >= 0:
                        held = oks[b, li, g, t] >= 0
                        want = ok[b, li, g, oks[b, li, g, t]] if held else x["l_k"][b, li, g, t]
                        np.testing.assert_array_equal(nk[b, li, g, ks[b, li, g, t]], want)
                    if vs[b, li, g, t] >= 0:
                        held = ovs[b, li, g, t] >= 0
                        want = ov[b, li, g, ovs[b, li, g, t]] if held else x["l_v"][b, li, g, t]
                        np.testing.assert_array_equal(nv[b, li, g, vs[b, li, g, t]], want)


def test_store_drops_rows_past_its_capacity():
    rng = np.random.default_rng(65)
    x, r = _store_case(rng)
    nk, nv, ks, vs, cnt = O.store_update(seq_len=x["seq_len"], head_map=x["head_map"],
                                         crit=r["crit"], marg=r["marg"], full_k=x["l_k"],
                                         full_v=x["l_v"], rows=5, n_small_heads=8)
    assert (cnt[..., 1] > 5).any()
    assert ks.max() < 5 and vs.max() < 5
    for b in range(2):
        for li in range(2):
            for g in range(2):
                assert (vs[b, li, g] >= 0).sum() == min(5, cnt[b, li, g, 1])
