"""Brute force on tiny inputs (n <= 16) against the float64 oracle.

The reference here is written as explicit scalar loops with math.exp and
exact Fraction sums: attention row by row, pooling by neighbour loop,
selection by enumerating every candidate subset (maximum score sum, then the
lexicographically smallest subset, which is the paper's top-k with the
lower position winning ties), routing / full-cosine routing by exhaustive
search, the gate, Eq. 5 and Eq. 6 and the decode softmax by loops.  Each
step is checked stage-wise (fed the oracle's own input for that step), so a
floating-point near-tie upstream cannot mask a mistake downstream.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import selkv_oracle as O


def bf_attention_mass(qg, k, scale):
    G, W, d = len(qg), len(qg[0]), len(k[0])
    n = len(k)
    a = [0.0] * n
    for g in range(G):
        for i in range(W):
            p = n - W + i
            logits = []
            for j in range(p + 1):
                logits.append(scale * sum(qg[g][i][t] * k[j][t] for t in range(d)))
            mx = max(logits)
            es = [math.exp(x - mx) for x in logits]
            tot = math.fsum(es)
            for j in range(p + 1):
                a[j] += es[j] / tot / G
    return a


def bf_pool(c, n_cand, K):
    out = []
    for j in range(n_cand):
        acc = 0.0
        for t in range(-(K // 2), K // 2 + 1):
            if 0 <= j + t < n_cand:
                acc += c[j + t]
        out.append(acc / K)
    return out


def bf_select(s, n, m, mr):
    ms = m - mr
    best, best_sum = None, None
    for comb in itertools.combinations(range(n - mr), ms):     # lexicographic order
        tot = sum((Fraction(s[j]) for j in comb), Fraction(0))
        if best is None or tot > best_sum:
            best, best_sum = comb, tot
    kept = list(best) + list(range(n - mr, n))
    evicted = [j for j in range(n) if j not in kept]
    return kept, evicted


def bf_route_bucket(a, kept, evicted, B):
    target = []
    for j in evicted:
        best = -1
        for slot, i in enumerate(kept):
            if i // B != j // B:
                continue
            if best == -1 or a[i] > a[kept[best]] or (a[i] == a[kept[best]] and i < kept[best]):
                best = slot
        target.append(best)
    return target


def bf_cos(u, v):
    dot = sum(x * y for x, y in zip(u, v))
    nu = math.sqrt(sum(x * x for x in u))
    nv = math.sqrt(sum(x * x for x in v))
    return 0.0 if nu == 0 or nv == 0 else dot / (nu * nv)


def bf_route_cos(v, kept, evicted):
    target = []
    for j in evicted:
        best, bs = 0, None
        for slot, i in enumerate(kept):
            c = bf_cos(v[j], v[i])
            if bs is None or c > bs:
                best, bs = slot, c
        target.append(best)
    return target


def bf_gate(v, kept, evicted, target, mode, tau, T):
    g = []
    for e, j in enumerate(evicted):
        t = target[e]
        if t < 0:
            g.append(0.0)
        elif mode == "drop":
            g.append(0.0)
        elif mode == "merge_all":
            g.append(1.0)
        else:
            g.append(min(1.0, max(0.0, (bf_cos(v[j], v[kept[t]]) - tau) / T)))
    return g


def bf_merge_ratio(v, a, kept, evicted, target, g, alpha):
    d = len(v[0])
    vout, bias = [], []
    for slot, i in enumerate(kept):
        num = [a[i] * v[i][t] for t in range(d)]
        den = a[i]
        for e, j in enumerate(evicted):
            if target[e] == slot:
                for t in range(d):
                    num[t] += g[e] * a[j] * v[j][t]
                den += g[e] * a[j]
        vout.append([x / den for x in num])
        bias.append(alpha * math.log(den / a[i]))
    return vout, bias


def bf_decode(q, kc, vc, bias, G, scale):
    out = []
    for h in range(len(q)):
        kv = h // G
        logits = [scale * sum(x * y for x, y in zip(q[h], kc[kv][i])) + (bias[kv][i] if bias is not None else 0.0)
                  for i in range(len(kc[kv]))]
        mx = max(logits)
        w = [math.exp(x - mx) for x in logits]
        tot = math.fsum(w)
        out.append([sum(w[i] * vc[kv][i][t] for i in range(len(w))) / tot for t in range(len(q[h]))])
    return out


def _case(seed, n, d, G, W, dup):
    r = np.random.default_rng(seed)
    k = r.standard_normal((n, d))
    v = r.standard_normal((n, d))
    centres = r.standard_normal((2, d))
    v[::3] = centres[0] + 0.1 * r.standard_normal((len(v[::3]), d))   # some similar values
    for j in range(1, n):
        if r.random() < dup:          # exact copies -> exact ties in a and cos = 1
            src = r.integers(0, j)
            k[j], v[j] = k[src], v[src]
    qg = r.standard_normal((G, W, d))
    return k, v, qg


@settings(max_examples=40, deadline=None)
@given(seed=st.integers(0, 10_000), n=st.integers(4, 14), d=st.sampled_from([2, 3, 5]),
       G=st.integers(1, 3), wfrac=st.floats(0.1, 1.0), rho=st.floats(0.2, 1.0),
       K=st.sampled_from([1, 3, 5]), recent=st.integers(0, 4), B=st.sampled_from([2, 4, 32]),
       mode=st.sampled_from(["cosine", "drop", "merge_all"]), route=st.sampled_from(["bucket", "full_cosine"]),
       tau=st.sampled_from([0.0, 0.3]), T=st.sampled_from([1.0, 0.5]), dup=st.sampled_from([0.0, 0.3]))
def test_pipeline_against_brute_force(seed, n, d, G, wfrac, rho, K, recent, B, mode, route, tau, T, dup):
    W = max(1, int(wfrac * n))
    if math.floor(rho * n) < 1:
        return
    k, v, qg = _case(seed, n, d, G, W, dup)
    scale = 0.7
    out = O.compress_head(k, v, qg, window=W, pool_kernel=K, recent=recent, bucket=B, budget_ratio=rho,
                          alpha=0.5, scale=scale, gate_mode=mode, gate_threshold=tau, gate_temperature=T,
                          route_mode=route)
    m, mr = out["m"], out["mr"]
    assert (m, mr) == (math.floor(rho * n), min(recent, math.floor(rho * n)))

    a = bf_attention_mass(qg.tolist(), k.tolist(), scale)
    np.testing.assert_allclose(out["attn"], a, rtol=1e-12, atol=1e-15)
    c = [a_ * math.sqrt(sum(x * x for x in row)) for a_, row in zip(out["attn"], v.tolist())]
    np.testing.assert_allclose(out["contribution"], c, rtol=1e-13, atol=1e-16)
    s = bf_pool(list(out["contribution"][: n - mr]), n - mr, K)
    np.testing.assert_allclose(out["score"], s, rtol=1e-13, atol=1e-16)

    kept, evicted = bf_select(list(out["score"]), n, m, mr)           # stage-wise: oracle's scores
    assert list(out["kept"]) == kept and list(out["evicted"]) == evicted

    if route == "bucket":
        target = bf_route_bucket(list(out["attn"]), kept, evicted, B)
    else:
        target = bf_route_cos(v.tolist(), kept, evicted)
    assert list(out["target"]) == target

    g = bf_gate(v.tolist(), kept, evicted, target, mode, tau, T)
    np.testing.assert_allclose(out["gate"], g, rtol=0, atol=1e-14)

    vout, bias = bf_merge_ratio(v.tolist(), list(out["attn"]), kept, evicted, target, list(out["gate"]), 0.5)
    np.testing.assert_allclose(out["v_out"], np.array(vout).reshape(out["v_out"].shape), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(out["bias"], bias, rtol=1e-12, atol=1e-14)
    np.testing.assert_array_equal(out["k_out"], k[kept])

    q = np.random.default_rng(seed + 1).standard_normal((G, d))
    dec = O.decode(q, out["k_out"][None], out["v_out"][None], out["bias"][None], G, scale)
    ref = bf_decode(q.tolist(), [out["k_out"].tolist()], [out["v_out"].tolist()], [list(out["bias"])], G, scale)
    np.testing.assert_allclose(dec, ref, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("n,ms", [(10, 3), (12, 5), (16, 4)])
def test_selection_enumeration_with_forced_ties(n, ms):
    """Integer scores with many ties: subset enumeration (max sum, then the
    lexicographically smallest subset) equals the oracle's top-k."""
    r = np.random.default_rng(n * 7 + ms)
    for _ in range(20):
        s = r.integers(0, 3, size=n - 2).astype(float)
        kept, ev = O.select(s, n, ms + 2, 2)
        bk, be = bf_select(list(s), n, ms + 2, 2)
        assert list(kept) == bk and list(ev) == be
