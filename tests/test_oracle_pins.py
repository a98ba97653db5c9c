"""Pins of the float64 oracle against what the paper and the mathematics fix.

None of these retypes the oracle's own formulas: each compares it with a
closed form worked by hand (tests/golden/hand_worked.json), a library routine
(torch's scaled_dot_product_attention in float64), an invariant the paper
states, or an exact identity (attention-sag restoration, full budget).
Brute-force enumeration on tiny inputs is in test_oracle_bruteforce.py.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import selkv_oracle as O

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_worked.json")))


def frac(s):
    return float(Fraction(s))


def rng(seed):
    return np.random.default_rng(seed)


def sdpa64(q, k, v, mask=None, causal=False, scale=None):
    """torch's reference attention in float64 on the CPU."""
    t = lambda x: torch.as_tensor(np.asarray(x, dtype=np.float64))
    m = None if mask is None else t(mask)
    return torch.nn.functional.scaled_dot_product_attention(
        t(q), t(k), t(v), attn_mask=m, is_causal=causal, scale=scale).numpy()


# ---------------------------------------------------------------- budget
def test_budget_floor_cases():
    for n, rho, m, ms in GOLD["budget_cases"]["cases"]:
        got = O.budget(n, rho, 16)
        assert got[0] == m and got[2] == ms, (n, rho, got)
    assert O.budget(100, 1.0, 16) == (100, 16, 84)
    with pytest.raises(ValueError):
        O.budget(3, 0.25, 16)          # floor(0.75) = 0 keeps nothing
    with pytest.raises(ValueError):
        O.budget(10, 0.0, 16)


# ---------------------------------------------------------------- scoring
def test_window_attention_equals_library_causal_attention():
    """Sec. 3.1: the window rows are the last W rows of ordinary causal
    attention.  With V = identity, torch's SDPA output *is* the attention
    matrix, so its last W rows must equal the oracle's A (scale 1/sqrt d)."""
    r = rng(1)
    n, d, W = 37, 16, 9
    Q = r.standard_normal((n, d))
    K = r.standard_normal((n, d))
    ref = sdpa64(Q[None], K[None], np.eye(n)[None], causal=True)[0][n - W:]
    got = O.window_attention(Q[n - W:], K, 1.0 / math.sqrt(d))
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-15)


def test_zero_query_closed_form_hand_case():
    case = GOLD["zero_query_case"]
    n, W = case["n"], case["window"]
    a = O.cumulative_attention(np.zeros((1, W, 3)), np.ones((n, 3)), 0.125)
    np.testing.assert_allclose(a, [frac(x) for x in case["expected"]], rtol=0, atol=1e-15)


@pytest.mark.parametrize("n,W,G", [(40, 8, 3), (17, 17, 1), (64, 1, 2)])
def test_zero_query_closed_form(n, W, G):
    """q = 0: row i (position p_i = n-W+i) is uniform over keys 0..p_i, so
    a_j = sum_{i: p_i >= j} 1/(p_i + 1), whatever the keys are."""
    r = rng(n)
    K = r.standard_normal((n, 8)) * 3
    a = O.cumulative_attention(np.zeros((G, W, 8)), K, 0.3)
    expect = np.array([sum(1.0 / (p + 1) for p in range(n - W, n) if p >= j) for j in range(n)])
    np.testing.assert_allclose(a, expect, rtol=1e-13)


def test_attention_mass_equals_window_length():
    """Every window row is a softmax, so sum_j a_j = W after the G-mean."""
    r = rng(2)
    for G in (1, 4):
        a = O.cumulative_attention(r.standard_normal((G, 12, 16)) * 2, r.standard_normal((50, 16)), 0.25)
        assert abs(a.sum() - 12) < 1e-12
        assert (a > 0).all()


def test_group_average_not_sum():
    """Sec. 3.3 averages the G query heads' scores: G identical heads must
    give exactly the single-head a (a sum would give G times it)."""
    r = rng(3)
    q = r.standard_normal((1, 6, 8))
    K = r.standard_normal((30, 8))
    a1 = O.cumulative_attention(q, K, 0.35)
    a4 = O.cumulative_attention(np.repeat(q, 4, axis=0), K, 0.35)
    np.testing.assert_allclose(a4, a1, rtol=1e-14)


def test_scale_enters_the_logits():
    """Two keys seen by one query with q.k = 0 and q.k = x: the attention
    ratio is exp(scale * x) (the window pass is ordinary softmax attention)."""
    q = np.array([[[1.0, 0.0]]])
    K = np.array([[0.0, 1.0], [2.0, 0.0]])
    a = O.cumulative_attention(q, K, 0.7)
    assert abs(a[1] / a[0] - math.exp(0.7 * 2.0)) < 1e-12


def test_contribution_uses_value_norm():
    """Eq. 1: c_j = a_j * ||v_j||_2; (3, 4) has norm 5, (0, 0) norm 0."""
    v = np.array([[3.0, 4.0], [0.0, 0.0], [1.0, 0.0]])
    vn = O.value_norms(v)
    np.testing.assert_array_equal(vn, [5.0, 0.0, 1.0])
    np.testing.assert_allclose(O.contribution(np.array([0.5, 2.0, 0.25]), vn), [2.5, 0.0, 0.25])


def test_pool_hand_case():
    case = GOLD["pool_case"]
    s = O.pool(np.array(case["c"], dtype=float), len(case["c"]), case["kernel"])
    np.testing.assert_allclose(s, [frac(x) for x in case["expected"]], atol=1e-15)


def test_pool_closed_forms():
    """Sec. 3.2 pooling: a delta spreads 1/K over K neighbours; a constant
    stays constant inside and loses the padded share at the edges; K = 1 is
    the identity."""
    n = 20
    delta = np.zeros(n)
    delta[9] = 1.0
    s = O.pool(delta, n, 5)
    np.testing.assert_allclose(s, [0.2 if 7 <= j <= 11 else 0.0 for j in range(n)])
    const = O.pool(np.full(n, 3.0), n, 5)
    np.testing.assert_allclose(const[2:-2], 3.0)
    np.testing.assert_allclose(const[[0, 1, -2, -1]], [3 * 3 / 5, 3 * 4 / 5, 3 * 4 / 5, 3 * 3 / 5])
    c = rng(4).random(n)
    np.testing.assert_array_equal(O.pool(c, n, 1), c)
    # only the first n_cand values are pooled: the value after the range is never read
    c2 = np.concatenate([np.ones(5), [1e9]])
    np.testing.assert_allclose(O.pool(c2, 5, 3), [2 / 3, 1, 1, 1, 2 / 3])


# ---------------------------------------------------------------- selection
def test_selection_invariants_and_ties():
    """Eq. 2: |S| = m, the recent window is always kept, S and E partition
    the positions, and equal scores go to the lower position."""
    n, m, mr = 30, 10, 4
    s = np.zeros(n - mr)
    s[[3, 7, 20]] = 5.0            # three clear winners, the rest tie at 0
    kept, ev = O.select(s, n, m, mr)
    assert len(kept) == m and len(ev) == n - m
    assert set(range(n - mr, n)) <= set(kept)
    assert sorted(set(kept) | set(ev)) == list(range(n)) and not set(kept) & set(ev)
    assert list(kept) == sorted(kept) and list(ev) == sorted(ev)
    assert list(kept[: m - mr]) == [0, 1, 2, 3, 7, 20]


def test_selection_budget_below_recent_window():
    n, m, mr = 40, 10, 10       # rho = 0.25 of 40 with m_r = 16 > m
    kept, ev = O.select(np.arange(n - mr, dtype=float), n, m, mr)
    np.testing.assert_array_equal(kept, np.arange(30, 40))


# ---------------------------------------------------------------- routing
def test_route_bucket_rules():
    """Eq. 3 reading: target = kept token of the same bucket with the most
    window attention; lowest position on ties; -1 for a bucket with no kept
    token; a kept token absorbs at most B-1 evicted tokens."""
    B = 4
    kept = np.array([1, 2, 5, 6, 13])
    ev = np.array([0, 3, 4, 7, 8, 9, 10, 11, 12, 14, 15])
    a = np.zeros(16)
    a[[1, 2]] = [0.5, 0.5]          # tie -> slot 0 (position 1)
    a[[5, 6]] = [0.1, 0.9]          # -> slot 3 (position 6)
    a[13] = 0.2                      # only candidate in bucket 3
    t = O.route_bucket(a, kept, ev, B)
    np.testing.assert_array_equal(t, [0, 0, 3, 3, -1, -1, -1, -1, 4, 4, 4])
    counts = np.bincount(t[t >= 0], minlength=len(kept))
    assert counts.max() <= B - 1


def test_route_full_cosine_picks_most_similar():
    v = np.array([[1.0, 0.0], [0.0, 1.0], [0.0, 2.0], [0.9, 0.1], [-1.0, -1.0], [0.0, 0.0]])
    kept = np.array([0, 1, 2])
    ev = np.array([3, 4, 5])
    t, best = O.route_full_cosine(v, kept, ev)
    # row 3 -> slot 0; row 4 is anti-aligned with everything, best is cos=-1/sqrt2 at slot 0
    # (ties between slots 0, 1, 2 -> lowest); zero vector -> all sims 0 -> slot 0
    np.testing.assert_array_equal(t, [0, 0, 0])
    assert abs(best[0] - 0.9 / math.hypot(0.9, 0.1)) < 1e-15
    assert abs(best[1] + 1 / math.sqrt(2)) < 1e-15 and best[2] == 0.0
    t2, _ = O.route_full_cosine(v, np.array([0, 1, 2]), np.array([5]))
    assert t2[0] == 0


# ---------------------------------------------------------------- gate / merge / ratio
@pytest.mark.parametrize("case", GOLD["gate_cases"])
def test_gate_hand_cases(case):
    v = np.array([case["u"], case["v"]], dtype=float)
    g = O.gate(v, np.array([1]), np.array([0]), np.array([0]), "cosine",
               case["threshold"], case["temperature"])
    assert abs(g[0] - frac(case["expected"])) <= case["tol"]


def test_gate_modes_and_edges():
    v = np.array([[1.0, 0.0], [-1.0, 0.0], [0.0, 0.0], [5.0, 0.0]])
    kept = np.array([0])
    ev = np.array([1, 2, 3])
    t = np.array([0, 0, -1])
    np.testing.assert_array_equal(O.gate(v, kept, ev, t, "drop"), [0, 0, 0])
    np.testing.assert_array_equal(O.gate(v, kept, ev, t, "merge_all"), [1, 1, 0])
    # anti-parallel -> 0, zero vector -> 0, unrouted -> 0
    np.testing.assert_array_equal(O.gate(v, kept, ev, t, "cosine"), [0, 0, 0])
    # parallel (different length) -> 1; clip keeps g <= 1 with tau < 0
    g = O.gate(v, kept, np.array([3]), np.array([0]), "cosine", -0.5, 0.25)
    assert g[0] == 1.0


def test_merge_and_ratio_hand_case():
    c = GOLD["merge_case"]
    v = np.array([c["v_kept"], c["v_evicted"]], dtype=float)
    k = np.array([[7.0, 8.0], [9.0, 10.0]])
    a = np.array([c["a_kept"], c["a_evicted"]], dtype=float)
    kept, ev, t = np.array([0]), np.array([1]), np.array([0])
    g = O.gate(v, kept, ev, t)
    assert abs(g[0] - frac(c["expected_gate"])) < c["tol"]
    kk, vv, w = O.merge(k, v, a, kept, ev, t, g)
    np.testing.assert_array_equal(kk, [[7.0, 8.0]])        # keys are gathered, not merged
    np.testing.assert_allclose(vv[0], [frac(x) for x in c["expected_value"]], atol=c["tol"])
    for alpha in (0.5, 1.0):
        b = O.ratio_bias(a, kept, ev, t, g, alpha)
        assert abs(b[0] - alpha * math.log(frac(c["expected_ratio"]))) < 1e-14


def _random_stage_inputs(seed, n=64, d=8, B=8, m=20):
    r = rng(seed)
    v = r.standard_normal((n, d))
    v[5] = v[3] * 2.5                       # a parallel pair
    k = r.standard_normal((n, d))
    a = r.random(n) + 0.01
    kept = np.sort(r.choice(n, m, replace=False))
    ev = np.setdiff1d(np.arange(n), kept)
    return k, v, a, kept, ev, B


def test_drop_gate_reduces_to_eviction():
    """Sec. 3.5: with g = 0 everywhere, Eq. 5 is pure drop; Eq. 6 gives R = 1."""
    k, v, a, kept, ev, B = _random_stage_inputs(5)
    t = O.route_bucket(a, kept, ev, B)
    g = O.gate(v, kept, ev, t, "drop")
    kk, vv, _ = O.merge(k, v, a, kept, ev, t, g)
    np.testing.assert_allclose(vv, v[kept], rtol=1e-15, atol=1e-15)
    np.testing.assert_array_equal(kk, k[kept])
    np.testing.assert_array_equal(O.ratio_bias(a, kept, ev, t, g, 0.5), 0.0)


def test_merge_all_is_attention_weighted_average():
    """Sec. 3.5: with g = 1, Eq. 5 is the plain a-weighted mean of each
    kept token and the evicted tokens routed to it."""
    k, v, a, kept, ev, B = _random_stage_inputs(6)
    t = O.route_bucket(a, kept, ev, B)
    g = O.gate(v, kept, ev, t, "merge_all")
    _, vv, _ = O.merge(k, v, a, kept, ev, t, g)
    for slot, i in enumerate(kept):
        members = [i] + [int(ev[e]) for e in range(len(ev)) if t[e] == slot]
        expect = np.average(v[members], axis=0, weights=a[members])
        np.testing.assert_allclose(vv[slot], expect, rtol=1e-13, atol=1e-14)


def test_merged_value_in_convex_hull_and_ratio_invariants():
    """Eq. 5 is a convex combination (weights a_i, g_j a_j >= 0); Eq. 6 gives
    R >= 1, R = 1 exactly where nothing was absorbed, and mass conservation
    sum_i a_i R_i = sum_S a_i + sum_E g_j a_j (Sec. 3.6: R is bounded by the
    redistributed attention mass)."""
    k, v, a, kept, ev, B = _random_stage_inputs(7)
    t = O.route_bucket(a, kept, ev, B)
    g = O.gate(v, kept, ev, t)
    _, vv, _ = O.merge(k, v, a, kept, ev, t, g)
    bias = O.ratio_bias(a, kept, ev, t, g, 1.0)
    R = np.exp(bias)
    for slot, i in enumerate(kept):
        members = [i] + [int(ev[e]) for e in range(len(ev)) if t[e] == slot and g[e] > 0]
        lo, hi = v[members].min(axis=0), v[members].max(axis=0)
        assert (vv[slot] >= lo - 1e-12).all() and (vv[slot] <= hi + 1e-12).all()
        absorbed = any(t[e] == slot and g[e] * a[ev[e]] > 0 for e in range(len(ev)))
        assert (R[slot] > 1.0) == absorbed
        if not absorbed:
            assert bias[slot] == 0.0
    assert (R >= 1.0).all()
    lhs = (a[kept] * R).sum()
    rhs = a[kept].sum() + sum(g[e] * a[ev[e]] for e in range(len(ev)) if t[e] >= 0)
    assert abs(lhs - rhs) < 1e-12 * rhs
    assert (g >= 0).all() and (g <= 1).all()


def test_routing_merge_ratio_invariant_to_scaling_a():
    """Every use of a after scoring is a ratio or an argmax, so the G-mean vs
    G-sum reading of Sec. 3.3 cannot change routing, merge or bias."""
    k, v, a, kept, ev, B = _random_stage_inputs(8)
    t1 = O.route_bucket(a, kept, ev, B)
    t4 = O.route_bucket(4.0 * a, kept, ev, B)
    np.testing.assert_array_equal(t1, t4)
    g = O.gate(v, kept, ev, t1)
    _, v1, _ = O.merge(k, v, a, kept, ev, t1, g)
    _, v4, _ = O.merge(k, v, 4.0 * a, kept, ev, t1, g)
    np.testing.assert_allclose(v1, v4, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(O.ratio_bias(a, kept, ev, t1, g, 0.5),
                               O.ratio_bias(4.0 * a, kept, ev, t1, g, 0.5), atol=1e-14)


# ---------------------------------------------------------------- decode
def test_decode_equals_library_attention_with_additive_bias():
    """Decode is softmax(scale q.k + bias) v; torch's SDPA adds a float mask
    to the scaled logits, so it is the same operation."""
    r = rng(9)
    Hkv, G, m, d = 3, 2, 11, 8
    q = r.standard_normal((Hkv * G, d))
    kc, vc = r.standard_normal((Hkv, m, d)), r.standard_normal((Hkv, m, d))
    bias = r.random((Hkv, m)) * 2
    got = O.decode(q, kc, vc, bias, G, 0.3)
    for h in range(Hkv * G):
        ref = sdpa64(q[h][None, None], kc[h // G][None], vc[h // G][None], mask=bias[h // G][None, None], scale=0.3)
        np.testing.assert_allclose(got[h], ref[0, 0], rtol=1e-13, atol=1e-14)
    got0 = O.decode(q, kc, vc, None, G, 0.3)
    ref0 = sdpa64(q.reshape(Hkv, G, d), kc, vc, scale=0.3).reshape(Hkv * G, d)
    np.testing.assert_allclose(got0, ref0, rtol=1e-13, atol=1e-14)


def test_decode_steps_equals_library_attention_per_step():
    """The many-step decode is, step by step, softmax(scale q.k + bias) v
    (torch SDPA in float64 with the bias as a float mask)."""
    r = rng(10)
    T, Hkv, G, m, d = 5, 2, 3, 13, 8
    qs = r.standard_normal((T, Hkv * G, d))
    kc, vc = r.standard_normal((Hkv, m, d)), r.standard_normal((Hkv, m, d))
    bias = r.random((Hkv, m)) * 3
    got = O.decode_steps(qs, kc, vc, bias, G, 0.7)
    for t in range(T):
        for h in range(Hkv * G):
            ref = sdpa64(qs[t, h][None, None], kc[h // G][None], vc[h // G][None], mask=bias[h // G][None, None],
                         scale=0.7)
            np.testing.assert_allclose(got[t, h], ref[0, 0], rtol=1e-13, atol=1e-14)
    got0 = O.decode_steps(qs, kc, vc, None, G, 0.7)
    ref0 = sdpa64(qs.reshape(T, Hkv, G, d).transpose(1, 0, 2, 3).reshape(Hkv, T * G, d), kc, vc, scale=0.7)
    np.testing.assert_allclose(got0, ref0.reshape(Hkv, T, G, d).transpose(1, 0, 2, 3).reshape(T, Hkv * G, d),
                               rtol=1e-13, atol=1e-14)


# ---------------------------------------------------------------- whole-pipeline identities
def test_full_budget_is_identity():
    """rho = 1: S = all positions, E is empty, K~ = K, V~ = V, R = 1, and the
    biased decode equals full-cache attention (spec check (a))."""
    r = rng(10)
    n, d, G, W = 48, 16, 2, 8
    k, v = r.standard_normal((n, d)), r.standard_normal((n, d))
    qw = r.standard_normal((G, W, d))
    out = O.compress_head(k, v, qw, budget_ratio=1.0, window=W)
    np.testing.assert_array_equal(out["kept"], np.arange(n))
    assert out["evicted"].size == 0
    np.testing.assert_array_equal(out["k_out"], k)
    np.testing.assert_allclose(out["v_out"], v, rtol=1e-15, atol=1e-15)
    np.testing.assert_array_equal(out["bias"], 0.0)
    q = r.standard_normal((G, d))
    dec = O.decode(q, out["k_out"][None], out["v_out"][None], out["bias"][None], G, 1 / math.sqrt(d))
    ref = sdpa64(q[None], k[None], v[None])[0]
    np.testing.assert_allclose(dec, ref, rtol=1e-13, atol=1e-14)


def _sag_case(seed, d=8, B=32, W=8):
    """A cache whose first three buckets each hold one prototype (k, v)
    repeated B times; the last bucket is B distinct tokens that the recent
    window (m_r = B) keeps.  All copies precede the window, so every copy of
    a prototype has the same window attention."""
    r = rng(seed)
    protos_k = r.standard_normal((3, d))
    protos_v = r.standard_normal((3, d))
    k = np.concatenate([np.repeat(protos_k, B, axis=0), r.standard_normal((B, d))])
    v = np.concatenate([np.repeat(protos_v, B, axis=0), r.standard_normal((B, d))])
    qw = r.standard_normal((2, W, d))
    return k, v, qw


@pytest.mark.parametrize("seed", [11, 12, 13])
def test_attention_sag_restored_exactly_with_alpha_one(seed):
    """Sec. 1 / Sec. 3.6: a cache entry standing for r identical tokens is
    under-attended by a factor r.  Evict 20 copies (rho = 108/128); each is
    routed to an identical kept copy with g = 1 and equal a, so R counts the
    copies and with alpha = 1 the biased decode over the compressed cache
    equals full-cache attention exactly (spec check (c)).  With the
    paper's alpha = 0.5 it does not."""
    k, v, qw = _sag_case(seed)
    n, d, G = k.shape[0], k.shape[1], 2
    out = O.compress_head(k, v, qw, budget_ratio=108 / 128, recent=32, bucket=32, alpha=1.0, window=8)
    assert len(out["evicted"]) == 20
    assert (out["target"] >= 0).all()
    np.testing.assert_allclose(out["gate"], 1.0, atol=1e-15)
    r = rng(seed + 100)
    q = r.standard_normal((G, d)) * 2
    sc = 1 / math.sqrt(d)
    full = sdpa64(q[None], k[None], v[None], scale=sc)[0]
    comp = O.decode(q, out["k_out"][None], out["v_out"][None], out["bias"][None], G, sc)
    np.testing.assert_allclose(comp, full, rtol=1e-12, atol=1e-13)
    half = O.compress_head(k, v, qw, budget_ratio=108 / 128, recent=32, bucket=32, alpha=0.5, window=8)
    comp_half = O.decode(q, half["k_out"][None], half["v_out"][None], half["bias"][None], G, sc)
    assert np.abs(comp_half - full).max() > 1e-6
    # without any compensation the cache is the plain eviction result
    nob = O.decode(q, out["k_out"][None], out["v_out"][None], None, G, sc)
    assert np.abs(nob - full).max() > 1e-6


# ------------------------------------------------------------------ GQA union mode (Sec. 3.3, Sec. 3.6)
def test_union_selection_hand_worked():
    """Sec. 3.3 union selection on a hand-worked case: the trim keeps the top
    mean scores among tokens some head picked, never a token no head picked."""
    c = GOLD["union_selection"]
    n, mr = c["n"], c["recent"]
    m, mr2, ms = O.budget(n, c["budget_ratio"], mr)
    kept, ev = O.select_union(np.array(c["scores"], dtype=np.float32), n, m, mr2)
    assert kept.tolist() == c["kept"] and ev.tolist() == c["evicted"]


def test_union_selection_reduces_to_per_head_cases():
    rng = np.random.default_rng(11)
    n, m, mr = 64, 24, 4
    s = rng.random((1, n - mr)).astype(np.float32)
    # a single KV head: the union is that head's own selection
    assert [x.tolist() for x in O.select_union(s, n, m, mr)] == [x.tolist() for x in O.select(s[0].astype(np.float64), n, m, mr)]
    # identical heads: every head picks the same set
    s3 = np.repeat(s, 3, axis=0)
    assert [x.tolist() for x in O.select_union(s3, n, m, mr)] == [x.tolist() for x in O.select(s[0].astype(np.float64), n, m, mr)]
    # heads picking disjoint sets that together are exactly m_s long stay whole
    s2 = np.zeros((2, n - mr), dtype=np.float32)
    ms = m - mr
    s2[0, : ms // 2] = 1.0
    s2[1, ms // 2: ms] = 1.0
    kept, _ = O.select_union(s2, n, m, mr)
    assert kept[:ms].tolist() == list(range(ms))


def test_union_selection_properties_random():
    """Shared set of exactly m; every kept candidate was picked by some head;
    no dropped union member has a larger mean (or an equal mean at a lower
    position) than a kept one."""
    rng = np.random.default_rng(5)
    for trial in range(20):
        H = int(rng.integers(2, 6))
        n = int(rng.integers(20, 120))
        mr = int(rng.integers(0, 6))
        rho = float(rng.uniform(0.1, 0.9))
        m, mr2, ms = O.budget(n, rho, mr)
        s = rng.integers(0, 6, size=(H, n - mr2)).astype(np.float32) / 4.0   # many exact ties
        kept, ev = O.select_union(s, n, m, mr2)
        assert kept.shape[0] == m and np.array_equal(np.sort(np.concatenate([kept, ev])), np.arange(n))
        picked = np.zeros(n - mr2, dtype=bool)
        for h in range(H):
            kh, _ = O.select(s[h].astype(np.float64), n, m, mr2)
            picked[kh[kh < n - mr2]] = True
        cand = kept[kept < n - mr2]
        assert picked[cand].all()
        mean = s.astype(np.float64).mean(axis=0)
        dropped = np.flatnonzero(picked & ~np.isin(np.arange(n - mr2), cand))
        for j in dropped:
            for i in cand:
                assert (mean[i], -i) > (mean[j], -j)


def test_union_ratio_bias_hand_worked():
    """Sec. 3.6 GQA rule: the bias is alpha * ln of the mean of the heads'
    ratios, not the mean of their per-head biases."""
    c = GOLD["union_ratio_bias"]
    got = O.ratio_bias_union(np.array(c["a"]), np.array(c["kept"]), np.array(c["evicted"]),
                             np.array(c["targets"]), np.array(c["gates"]), c["alpha"])
    want = [c["alpha"] * math.log(r) for r in c["mean_R"]]
    assert np.allclose(got, want, rtol=0, atol=1e-15)
    per_head = [O.ratio_bias(np.array(c["a"][h]), np.array(c["kept"]), np.array(c["evicted"]),
                             np.array(c["targets"][h]), np.array(c["gates"][h]), c["alpha"]) for h in range(2)]
    assert not np.allclose(got, np.mean(per_head, axis=0))


def test_union_ratio_bias_single_head_is_per_head():
    rng = np.random.default_rng(3)
    n = 40
    a = rng.random(n) + 0.1
    kept = np.sort(rng.choice(n, 10, replace=False))
    ev = np.setdiff1d(np.arange(n), kept)
    tg = rng.integers(-1, 10, size=ev.shape[0])
    g = rng.random(ev.shape[0])
    one = O.ratio_bias_union(a[None], kept, ev, tg[None], g[None], 0.5)
    assert np.allclose(one, O.ratio_bias(a, kept, ev, tg, g, 0.5), rtol=1e-14, atol=1e-15)


def test_compress_union_reduces_to_per_head_cases():
    """The union-mode driver against the cases the per-head pipeline fixes:
    one KV head is exactly compress_head (a union of one set, R averaged over
    one head); KV heads with identical keys, values and queries pick the same
    set, route alike and share one R, so every head equals compress_head."""
    r = rng(21)
    n, d, G, W = 96, 8, 2, 8
    k = r.standard_normal((1, n, d)) / 3
    v = r.standard_normal((1, n, d))
    q = r.standard_normal((G, W, d)) / 3
    for route in ("bucket", "full_cosine"):
        one = O.compress_union(k, v, q, group=G, window=W, bucket=8, budget_ratio=0.3, route_mode=route)
        ref = O.compress_head(k[0], v[0], q, window=W, bucket=8, budget_ratio=0.3, route_mode=route)
        for key in ("kept", "evicted", "target"):
            np.testing.assert_array_equal(one[key][0], ref[key], err_msg=key)
        for key in ("gate", "v_out", "bias", "score", "attn"):
            np.testing.assert_allclose(one[key][0], ref[key], rtol=1e-13, atol=1e-15, err_msg=key)
        three = O.compress_union(np.repeat(k, 3, 0), np.repeat(v, 3, 0), np.tile(q, (3, 1, 1)), group=G, window=W,
                                 bucket=8, budget_ratio=0.3, route_mode=route)
        for h in range(3):
            np.testing.assert_array_equal(three["kept"][h], ref["kept"])
            np.testing.assert_array_equal(three["target"][h], ref["target"])
            np.testing.assert_allclose(three["bias"][h], ref["bias"], rtol=1e-13, atol=1e-15)
            np.testing.assert_allclose(three["v_out"][h], ref["v_out"], rtol=1e-13, atol=1e-15)


# ------------------------------------------------------------------ RoPE repositioning (Eq. 7)
def test_rope_reposition_hand_worked():
    c = GOLD["rope_reposition"]
    got = O.reposition_keys(np.array([[0.0] * 4] * 2 + [c["k"]]), np.array([0, 1, c["p_old"]]), c["theta"])
    assert np.allclose(got[2], c["expected"], rtol=0, atol=1e-14)
    assert np.allclose(got[:2], 0.0)


def test_rope_properties():
    rng = np.random.default_rng(9)
    d, r = 64, 12
    x = rng.standard_normal((r, d))
    pos = rng.integers(0, 100000, size=r).astype(np.float64)
    for theta in (10000.0, 500000.0):
        y = O.rope(x, pos, theta)
        assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-12)   # rotations
        assert np.allclose(O.rope(y, -pos, theta), x, atol=1e-9)                              # inverse
        # relative position: <rope(q, a), rope(k, b)> depends on a - b only
        q, k = rng.standard_normal((1, d)), rng.standard_normal((1, d))
        l1 = float((O.rope(q, np.array([900.0]), theta) @ O.rope(k, np.array([400.0]), theta).T)[0, 0])
        l2 = float((O.rope(q, np.array([510.0]), theta) @ O.rope(k, np.array([10.0]), theta).T)[0, 0])
        assert abs(l1 - l2) < 1e-9
    # repositioning a key already at its slot changes nothing
    ks = rng.standard_normal((5, d))
    assert np.allclose(O.reposition_keys(ks, np.arange(5), 10000.0), ks, atol=1e-12)


# ------------------------------------------------------------------ alternative readings (modes)
def test_nearest_fallback_hand_worked():
    c = GOLD["nearest_fallback"]
    a, kept, ev = np.array(c["a"]), np.array(c["kept"]), np.array(c["evicted"])
    assert O.route_bucket(a, kept, ev, c["bucket"]).tolist() == c["target_bucket"]
    assert O.route_bucket_nearest(a, kept, ev, c["bucket"]).tolist() == c["target_nearest"]


def test_nearest_fallback_tie_goes_low():
    # evicted 5 sits 2 from kept 3 and 2 from kept 7: the lower position wins
    a = np.ones(12)
    kept, ev = np.array([3, 7]), np.array([0, 1, 2, 4, 5, 6, 8, 9, 10, 11])
    t = O.route_bucket_nearest(a, kept, ev, 1)      # bucket 1: every evicted bucket is empty
    assert t[ev.tolist().index(5)] == 0 and t[ev.tolist().index(6)] == 1 and t[ev.tolist().index(4)] == 0


def test_merge_keys_closed_form():
    """merge_keys applies Eq. 5's weights to keys: two tokens, one absorbed."""
    k = np.array([[1.0, 0.0], [0.0, 2.0]])
    v = np.array([[3.0, 1.0], [1.0, 1.0]])
    a = np.array([0.75, 0.25])
    kept, ev, tg, g = np.array([0]), np.array([1]), np.array([0]), np.array([0.5])
    k_out, v_out, w = O.merge(k, v, a, kept, ev, tg, g, merge_keys=True)
    # weights: a0 = 0.75, g1 a1 = 0.125, denominator 0.875
    assert np.allclose(k_out[0], [0.75 / 0.875, 0.25 / 0.875]) and np.allclose(v_out[0], [2.375 / 0.875, 1.0])
    k_plain, v_plain, _ = O.merge(k, v, a, kept, ev, tg, g)
    assert np.array_equal(k_plain[0], k[0]) and np.allclose(v_plain, v_out)
    # nothing absorbed: keys stay the kept keys either way
    k_none, _, _ = O.merge(k, v, a, kept, ev, np.array([-1]), g, merge_keys=True)
    assert np.array_equal(k_none[0], k[0])


def test_coattention_routing_hand_worked():
    c = GOLD["coattention_routing"]
    A, kept, ev = np.array(c["A"]), np.array(c["kept"]), np.array(c["evicted"])
    assert O.route_bucket(A.sum(axis=0), kept, ev, c["bucket"]).tolist() == c["target_bucket"]
    assert O.route_coattention(A, kept, ev, c["bucket"]).tolist() == c["target_coattn"]


def test_coattention_routing_reduces_to_eq3_with_one_window_row():
    """With one window row (G = W = 1) the co-attention of j and i is
    A[j] * A[i] with A[j] > 0, so its argmax over the bucket is the argmax of
    a = A: exactly the routing of Eq. 3."""
    rng = np.random.default_rng(5)
    for trial in range(20):
        n, d, B = int(rng.integers(8, 120)), 16, int(rng.integers(1, 9))
        k, q = rng.standard_normal((n, d)), rng.standard_normal((1, 1, d))
        m = int(rng.integers(1, n))
        kept = np.sort(rng.choice(n, m, replace=False))
        ev = np.setdiff1d(np.arange(n), kept)
        A = O.window_attention_group(q, k, 1.0 / 4)
        a = O.cumulative_attention(q, k, 1.0 / 4)
        assert np.array_equal(O.route_coattention(A, kept, ev, B), O.route_bucket(a, kept, ev, B))


def test_coattention_routing_properties():
    """Empty buckets route nowhere, identical candidate columns tie to the
    lower slot, and the routing ignores the order and a common scale of the
    window rows."""
    rng = np.random.default_rng(9)
    n, B = 40, 8
    A = rng.random((6, n))
    A /= A.sum(axis=1, keepdims=True)
    kept = np.array([1, 3, 17, 20, 21, 39])
    ev = np.setdiff1d(np.arange(n), kept)
    t = O.route_coattention(A, kept, ev, B)
    empty = (ev // B == 1) | (ev // B == 3)          # buckets 8..15 and 24..31 keep nothing
    assert (t[empty] == -1).all() and (t[~empty] >= 0).all()
    for e, j in enumerate(ev):
        if t[e] >= 0:
            assert kept[t[e]] // B == j // B
    assert np.array_equal(O.route_coattention(A[::-1] * 3.0, kept, ev, B), t)
    A2 = A.copy()
    A2[:, 3] = A2[:, 1]                               # kept positions 1 and 3 get identical columns
    t2 = O.route_coattention(A2, kept, ev, B)
    assert (t2[ev < 8] == 0).all()


def test_window_attention_group_equals_library_attention_per_head():
    """The stacked window attention of G query heads: G causal SDPA calls
    (V = identity) give head h's matrix, whose last W rows are rows
    h*W .. h*W + W - 1 of the stack."""
    r = rng(21)
    n, d, W, G = 29, 8, 5, 3
    Q = r.standard_normal((G, n, d))
    K = r.standard_normal((n, d))
    ref = sdpa64(Q, np.repeat(K[None], G, 0), np.repeat(np.eye(n)[None], G, 0), causal=True)[:, n - W:]
    got = O.window_attention_group(Q[:, n - W:], K, 1.0 / math.sqrt(d))
    assert got.shape == (G * W, n)
    np.testing.assert_allclose(got, ref.reshape(G * W, n), rtol=1e-13, atol=1e-15)


def test_coattention_is_linear_in_the_evicted_column():
    """Hand case: the co-attention weighs the window rows by A[r, j] itself
    (not its square).  A_j = (.4, .2), kept i1 = (.1, .35), i2 = (.2, .1):
    .04 + .07 = .11 beats .08 + .02 = .10, so i1; with squared weights
    (.16, .04) it would be .030 against .036, i2."""
    A = np.array([[0.4, 0.1, 0.2, 0.3], [0.2, 0.35, 0.1, 0.35]])
    t = O.route_coattention(A, np.array([1, 2]), np.array([0, 3]), 4)
    assert t[0] == 0
