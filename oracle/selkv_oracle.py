"""Float64 CPU oracle of SelKV's one-shot KV-cache compression and biased decode.

TEST INFRASTRUCTURE ONLY.  This module is the reference the GPU library is
checked against.  Only the test-suite, the smoke check and the benchmark's
CPU-baseline leg may import it.  The library never does, and the two share
no code, headers, constants or helpers.

Paper: "SelKV: Selective KV Cache Merging with Per-Token Merge-or-Drop and
Attention Compensation" (arXiv 2607.16213).  Every function below follows one
step of Sec. 3 (Method) and Algorithm 1, in the paper's order and notation.
Arithmetic is float64 numpy.  Inputs are the storage-rounded tensors (bf16 or
fp32) that the GPU receives, upcast exactly to float64.

Readings taken where the paper is silent or garbled:
  * window pass: scale 1/sqrt(d), causal; window row i is position n-W+i and
    sees keys j <= n-W+i (Sec. 3.1, two-pass prefill);
  * GQA: query head h belongs to KV head floor(h/G); the G per-head
    cumulative attentions are averaged (Sec. 3.3, union-selection paragraph);
    that mean a is used for scoring, routing, merging and the ratio;
  * pooling (Sec. 3.2): centred moving average of width K over the candidate
    range [0, n-m_r), zero outside it, divisor always K;
  * selection (Eq. 2) is per KV head, exactly m entries; ties go to the lower
    position; m_r' = min(m_r, m);
  * routing (Eq. 3): the kept token of j's bucket with the largest window
    attention a_i, lowest position on ties, -1 (drop) for an empty bucket;
  * gate (Sec. 3.5): g = clip((sim - tau)/T, 0, 1); (tau, T) = (0, 1) is the
    paper's max(sim, 0); sim = 0 when a norm is 0; cosine against the
    pre-merge target value;
  * keys are not merged, only gathered (Eq. 5 defines only values);
  * bias (Eq. 6): natural log, alpha * ln R_i added after the softmax scale,
    per KV head (the per-head rule of Sec. 3.6);
  * GQA union mode (Sec. 3.3 union-selection paragraph, Sec. 3.6 GQA rule):
    each KV head's top-m_s set by its own scores, the union over the KV
    heads of one cache, trimmed to m_s by the mean score across KV heads
    (ties to the lower position); since every head contributes m_s tokens
    the union never falls short, so the shared kept set has exactly m
    entries.  The mean is the float64 arithmetic mean of the heads' scores.
    R is averaged across KV heads and alpha * ln(mean R) is shared by them;
  * RoPE repositioning (Sec. 3.7, Eq. 7; off by default):
    the rotate-half convention (dimension j pairs with j + d/2, frequency
    theta^(-2j/d)), retained key i moves from its position p_old = i to
    p_new = its slot in the compressed cache (0 .. m-1, contiguous);
  * alternative readings, as modes: route_bucket_nearest sends the evicted
    tokens of a bucket that keeps nothing to the nearest kept position
    instead of dropping them; merge(..., merge_keys=True) averages keys with
    the value weights of Eq. 5; route_coattention reads Eq. 3's A_{h,j,i} as
    the co-attention sum_r A[r, j] A[r, i] over the window rows of the G
    query heads (a sum, not a mean: the argmax does not depend on it).
"""
from __future__ import annotations

import math

import numpy as np

# Hyper-parameter defaults of App. F (Implementation Details) and Sec. 4.1.
DEFAULTS = dict(window=32, pool_kernel=5, recent=16, bucket=32, alpha=0.5,
                budget_ratio=0.25, gate_threshold=0.0, gate_temperature=1.0,
                gate_mode="cosine", route_mode="bucket")


# --------------------------------------------------------------------------
# Sec. 3.1: budget
# --------------------------------------------------------------------------
def budget(n: int, budget_ratio: float, recent: int = 16):
    """Target cache length m = floor(rho * n); the last m_r tokens are always
    kept and the remaining m_s = m - m_r slots are chosen by score (Sec. 3.1).

    The product rho*n is an IEEE double and is floored.  When m < m_r only m
    recent tokens fit, so m_r' = min(m_r, m).  Returns (m, m_r', m_s).
    """
    if not (0.0 < budget_ratio <= 1.0):
        raise ValueError("budget ratio must lie in (0, 1]")
    m = int(math.floor(float(budget_ratio) * float(n)))
    if m < 1:
        raise ValueError("budget keeps no token")
    mr = min(int(recent), m)
    return m, mr, m - mr


# --------------------------------------------------------------------------
# Sec. 3.1 (two-pass prefill) and Sec. 3.2 (importance scoring, Eq. 1)
# --------------------------------------------------------------------------
def window_attention(q_win: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """Attention of the last W query positions over the cached keys.

    This is the eager re-pass of Sec. 3.1: q_win [W, d] holds the queries of
    positions n-W .. n-1, k [n, d] the cached keys.  Row i sees keys
    j <= n-W+i (causal).  Returns A [W, n], each row a softmax.
    """
    q_win = np.asarray(q_win, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    W, n = q_win.shape[0], k.shape[0]
    logits = scale * (q_win @ k.T)
    row_pos = n - W + np.arange(W)
    visible = np.arange(n)[None, :] <= row_pos[:, None]
    logits = np.where(visible, logits, -np.inf)
    logits = logits - logits.max(axis=1, keepdims=True)
    e = np.exp(logits)
    return e / e.sum(axis=1, keepdims=True)


def cumulative_attention(q_win_group: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """a_j = sum over window rows of A[i, j] (Eq. 5's a), for one KV head.

    q_win_group [G, W, d] holds the window queries of the G query heads that
    share this KV head; their cumulative attentions are averaged, as Sec. 3.3
    prescribes for GQA scores.  Returns a [n].
    """
    G = q_win_group.shape[0]
    total = np.zeros(k.shape[0], dtype=np.float64)
    for g in range(G):
        total += window_attention(q_win_group[g], k, scale).sum(axis=0)
    return total / G


def value_norms(v: np.ndarray) -> np.ndarray:
    """||v_j||_2 for every cached value row (the factor in Eq. 1)."""
    v = np.asarray(v, dtype=np.float64)
    return np.sqrt((v * v).sum(axis=1))


def contribution(a: np.ndarray, vnorm: np.ndarray) -> np.ndarray:
    """Eq. 1: c_j = (sum_i A_ij) * ||v_j||_2 = a_j * ||v_j||_2."""
    return a * vnorm


def pool(c: np.ndarray, n_cand: int, kernel: int) -> np.ndarray:
    """Average-pool smoothing of Sec. 3.2 over the candidate range [0, n_cand).

    s_j = (1/K) * sum_{t=-K//2..K//2} c_{j+t}, where terms outside the
    candidate range count as zero (divisor stays K).  Returns s [n_cand].
    """
    if kernel < 1 or kernel % 2 == 0:
        raise ValueError("pooling kernel must be odd and positive")
    half = kernel // 2
    s = np.zeros(n_cand, dtype=np.float64)
    for j in range(n_cand):
        lo, hi = max(0, j - half), min(n_cand, j + half + 1)
        s[j] = c[lo:hi].sum() / kernel
    return s


# --------------------------------------------------------------------------
# Sec. 3.3: per-head selection (Eq. 2)
# --------------------------------------------------------------------------
def select(s: np.ndarray, n: int, m: int, mr: int):
    """Eq. 2: keep the m_s candidates with the largest smoothed score plus the
    last m_r positions; evict the rest.

    s holds the scores of the candidates 0 .. n-m_r-1.  Equal scores go to the
    lower position.  Returns (kept [m], evicted [n-m]) as ascending int64
    position arrays.
    """
    n_cand = n - mr
    ms = m - mr
    assert s.shape[0] == n_cand
    assert not np.isnan(s).any(), "NaN scores are outside the contract"
    positions = np.arange(n_cand)
    # primary key: larger score first; secondary: lower position first
    order = np.lexsort((positions, -s))
    chosen = np.sort(order[:ms])
    kept = np.concatenate([chosen, np.arange(n_cand, n)]).astype(np.int64)
    is_kept = np.zeros(n, dtype=bool)
    is_kept[kept] = True
    evicted = np.flatnonzero(~is_kept).astype(np.int64)
    return kept, evicted


def union_mean_score(s_heads: np.ndarray) -> np.ndarray:
    """Mean aggregate score across the KV heads of one cache, the trimming
    key of Sec. 3.3's union selection: the float64 arithmetic mean over the
    heads of each candidate's score."""
    return np.asarray(s_heads, dtype=np.float64).mean(axis=0)


def select_union(s_heads: np.ndarray, n: int, m: int, mr: int):
    """Union selection for GQA models (Sec. 3.3): every KV head picks its own
    top-m_s candidates (Eq. 2 on its scores); a candidate is kept when any
    KV head picks it; if that union holds more than m_s candidates, only the
    m_s with the largest mean score across KV heads stay (equal means: the
    lower position).  The last m_r positions are kept as in Eq. 2.  One kept
    set is shared by all KV heads.

    s_heads [H_kv, n - m_r] are the per-KV-head scores.  Returns (kept [m],
    evicted [n - m]) ascending int64 positions.
    """
    s_heads = np.asarray(s_heads)
    H, n_cand = s_heads.shape
    assert n_cand == n - mr
    ms = m - mr
    union = np.zeros(n_cand, dtype=bool)
    for h in range(H):
        kept_h, _ = select(np.asarray(s_heads[h], dtype=np.float64), n, m, mr)
        union[kept_h[kept_h < n_cand]] = True
    cand = np.flatnonzero(union)
    assert cand.shape[0] >= ms, "each head contributes m_s candidates"
    if cand.shape[0] > ms:
        mean = union_mean_score(s_heads)
        order = np.lexsort((cand, -mean[cand]))      # larger mean first, then lower position
        cand = np.sort(cand[order[:ms]])
    kept = np.concatenate([cand, np.arange(n_cand, n)]).astype(np.int64)
    is_kept = np.zeros(n, dtype=bool)
    is_kept[kept] = True
    return kept, np.flatnonzero(~is_kept).astype(np.int64)


# --------------------------------------------------------------------------
# Sec. 3.4: merge-target routing (Eq. 3)
# --------------------------------------------------------------------------
def route_bucket(a: np.ndarray, kept: np.ndarray, evicted: np.ndarray, bucket: int) -> np.ndarray:
    """Eq. 3 (bucket-attention routing): each evicted token goes to the kept
    token of its own positional bucket floor(j/B) that the observation window
    attended most (largest a_i); the lowest position wins ties.  A bucket
    with no kept token routes its evicted tokens nowhere (-1).

    Returns target [n-m]: the kept *slot* (index into `kept`) or -1.
    """
    best_slot = {}
    for slot, i in enumerate(kept):
        b = int(i) // bucket
        cur = best_slot.get(b)
        # kept is ascending, so a strict '>' keeps the lowest position on ties
        if cur is None or a[i] > a[kept[cur]]:
            best_slot[b] = slot
    target = np.full(evicted.shape[0], -1, dtype=np.int64)
    for e, j in enumerate(evicted):
        target[e] = best_slot.get(int(j) // bucket, -1)
    return target


def route_bucket_nearest(a: np.ndarray, kept: np.ndarray, evicted: np.ndarray, bucket: int) -> np.ndarray:
    """Alternative reading of Eq. 3 for a bucket that keeps no token (the
    paper is silent): instead of being dropped, each of its evicted tokens
    goes to the kept token nearest to it by position (the lower position
    when two are equally near).  Buckets that keep a token route as Eq. 3.
    """
    target = route_bucket(a, kept, evicted, bucket)
    for e, j in enumerate(evicted):
        if target[e] >= 0:
            continue
        dist = np.abs(kept.astype(np.int64) - int(j))
        target[e] = int(np.flatnonzero(dist == dist.min())[0])     # kept is ascending: lowest position
    return target


def window_attention_group(q_win_group: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """The window attention of the G query heads of one KV head stacked
    row-wise: A [G*W, n], row h*W + i = query head h at window row i."""
    return np.concatenate([window_attention(q_win_group[g], k, scale) for g in range(q_win_group.shape[0])])


def route_coattention(A: np.ndarray, kept: np.ndarray, evicted: np.ndarray, bucket: int) -> np.ndarray:
    """Alternative reading of Eq. 3 (its A_{h,j,i} taken as how much the
    window attends to j and i together): the co-attention of evicted j and
    kept i is sum over window rows r of A[r, j] * A[r, i], over the rows of
    all G query heads of the KV head (A from window_attention_group).  Each
    evicted token goes to the kept token of its own bucket with the largest
    co-attention, lowest position on ties; a bucket with no kept token
    routes nowhere (-1), as in Eq. 3.

    Returns target [n-m]: kept slots or -1.
    """
    A = np.asarray(A, dtype=np.float64)
    slots = {}
    for slot, i in enumerate(kept):
        slots.setdefault(int(i) // bucket, []).append(slot)
    target = np.full(evicted.shape[0], -1, dtype=np.int64)
    for e, j in enumerate(evicted):
        cand = slots.get(int(j) // bucket)
        if not cand:
            continue
        co = A[:, kept[cand]].T @ A[:, int(j)]
        target[e] = cand[int(np.argmax(co))]        # first maximum: candidates ascend, lowest position
    return target


def cosine(u: np.ndarray, v: np.ndarray) -> float:
    """Eq. 4: cosine similarity of two value vectors; 0 if either is zero."""
    nu = math.sqrt(float(np.dot(u, u)))
    nv = math.sqrt(float(np.dot(v, v)))
    if nu == 0.0 or nv == 0.0:
        return 0.0
    return float(np.dot(u, v)) / (nu * nv)


def route_full_cosine(v: np.ndarray, kept: np.ndarray, evicted: np.ndarray):
    """Full cosine routing, the all-pairs alternative that Eq. 3 replaces
    (Sec. 3.4, last sentence): each evicted token goes to the kept token whose
    value vector is most cosine-similar to its own; lowest slot on ties.

    Returns (target [n-m] kept slots, best cosine [n-m]).
    """
    v = np.asarray(v, dtype=np.float64)
    norms = value_norms(v)
    vk, nk = v[kept], norms[kept]
    target = np.zeros(evicted.shape[0], dtype=np.int64)
    best = np.zeros(evicted.shape[0], dtype=np.float64)
    for e, j in enumerate(evicted):
        dots = vk @ v[j]
        denom = nk * norms[j]
        sims = np.where(denom > 0, dots / np.where(denom > 0, denom, 1.0), 0.0)
        slot = int(np.argmax(sims))          # first maximum = lowest slot
        target[e] = slot
        best[e] = sims[slot]
    return target, best


# --------------------------------------------------------------------------
# Sec. 3.5: soft cosine gate (Eq. 4) and gated merge (Eq. 5)
# --------------------------------------------------------------------------
def gate(v: np.ndarray, kept: np.ndarray, evicted: np.ndarray, target: np.ndarray,
         mode: str = "cosine", threshold: float = 0.0, temperature: float = 1.0) -> np.ndarray:
    """Soft cosine gate of Sec. 3.5.

    cosine: g_j = clip((sim_j - tau)/T, 0, 1) with sim_j the cosine (Eq. 4)
            between v_j and its pre-merge target value; (tau, T) = (0, 1) is
            the paper's g = max(sim, 0).
    drop:      g_j = 0  (eviction only, the ablation of Sec. 4.3)
    merge_all: g_j = 1  (merging without the gate, Sec. 4.3)
    Unrouted tokens (target -1) get g = 0.
    """
    v = np.asarray(v, dtype=np.float64)
    g = np.zeros(evicted.shape[0], dtype=np.float64)
    for e, j in enumerate(evicted):
        t = int(target[e])
        if t < 0:
            continue
        if mode == "drop":
            g[e] = 0.0
        elif mode == "merge_all":
            g[e] = 1.0
        elif mode == "cosine":
            sim = cosine(v[j], v[kept[t]])
            g[e] = min(1.0, max(0.0, (sim - threshold) / temperature))
        else:
            raise ValueError(mode)
    return g


def merge(k: np.ndarray, v: np.ndarray, a: np.ndarray, kept: np.ndarray,
          evicted: np.ndarray, target: np.ndarray, g: np.ndarray, merge_keys: bool = False):
    """Eq. 5: the merged value of kept token i is

        v~_i = (a_i v_i + sum_{pi(j)=i} g_j a_j v_j) / (a_i + sum_{pi(j)=i} g_j a_j)

    with a the window-cumulative attention.  Keys are gathered unchanged
    (Eq. 5 defines only values); merge_keys=True is the alternative reading
    that applies the same weights to the keys.
    Returns (K~ [m, d], V~ [m, d], w [m]) where w_i is the denominator.
    """
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    a_kept = a[kept]
    assert (a_kept > 1e-30).all(), "a kept token with no window attention is outside the contract"
    num = a_kept[:, None] * v[kept]
    knum = a_kept[:, None] * k[kept]
    den = a_kept.copy()
    for e, j in enumerate(evicted):
        t = int(target[e])
        if t < 0:
            continue
        num[t] += g[e] * a[j] * v[j]
        knum[t] += g[e] * a[j] * k[j]
        den[t] += g[e] * a[j]
    k_out = knum / den[:, None] if merge_keys else k[kept].copy()
    return k_out, num / den[:, None], den


# --------------------------------------------------------------------------
# Sec. 3.6: attention-ratio compensation (Eq. 6)
# --------------------------------------------------------------------------
def ratio_bias(a: np.ndarray, kept: np.ndarray, evicted: np.ndarray, target: np.ndarray,
               g: np.ndarray, alpha: float) -> np.ndarray:
    """Eq. 6: R_i = (a_i + sum_{j->i} g_j a_j) / a_i; the decode logit bias is
    alpha * ln R_i (natural log).  Returns bias [m]."""
    absorbed = np.zeros(kept.shape[0], dtype=np.float64)
    for e, j in enumerate(evicted):
        t = int(target[e])
        if t >= 0:
            absorbed[t] += g[e] * a[j]
    a_kept = a[kept]
    R = (a_kept + absorbed) / a_kept
    return alpha * np.log(R)


def ratio_bias_union(a_heads: np.ndarray, kept: np.ndarray, evicted: np.ndarray, targets: np.ndarray,
                     gates: np.ndarray, alpha: float) -> np.ndarray:
    """Sec. 3.6, GQA rule: with one kept set shared by the KV heads, each
    head's ratio R_{h,i} of Eq. 6 is averaged across the KV heads and
    alpha * ln(mean_h R_{h,i}) is the bias of every head.

    a_heads [H, n]; targets, gates [H, n - m] (each head routes its own
    evicted tokens).  Returns bias [m], shared by the heads.
    """
    H = a_heads.shape[0]
    R = np.zeros((H, kept.shape[0]), dtype=np.float64)
    for h in range(H):
        a = np.asarray(a_heads[h], dtype=np.float64)
        absorbed = np.zeros(kept.shape[0], dtype=np.float64)
        for e, j in enumerate(evicted):
            t = int(targets[h][e])
            if t >= 0:
                absorbed[t] += gates[h][e] * a[j]
        a_kept = a[kept]
        R[h] = (a_kept + absorbed) / a_kept
    return alpha * np.log(R.mean(axis=0))


# --------------------------------------------------------------------------
# RoPE repositioning (Eq. 7)
# --------------------------------------------------------------------------
def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary position embedding of rows x [r, d] at positions pos [r]
    (negative positions rotate backwards, so rope(x, -p) is RoPE^-1 at p).
    Dimension j < d/2 pairs with j + d/2 and turns by pos * theta^(-2j/d)."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    inv_freq = float(theta) ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[:, :half], x[:, half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=1)


def reposition_keys(k_kept: np.ndarray, kept: np.ndarray, theta: float) -> np.ndarray:
    """Eq. 7: k~_i = RoPE(RoPE^-1(k_i, p_old), p_new) with p_old the original
    position of kept token i and p_new its contiguous slot in the compressed
    cache.  k_kept [m, d] rows in slot order; kept [m] original positions."""
    p_old = np.asarray(kept, dtype=np.float64)
    p_new = np.arange(kept.shape[0], dtype=np.float64)
    return rope(rope(k_kept, -p_old, theta), p_new, theta)


# --------------------------------------------------------------------------
# Decode with the compressed cache (Sec. 3.1 last paragraph; Algorithm 1)
# --------------------------------------------------------------------------
def decode(q: np.ndarray, kc: np.ndarray, vc: np.ndarray, bias, group: int,
           scale: float) -> np.ndarray:
    """Single-token attention over the compressed cache with the additive
    bias of Sec. 3.6 in the logits.

    q [H_q, d]; kc, vc [H_kv, m, d]; bias [H_kv, m] or None; query head h
    reads KV head floor(h/G).  Returns o [H_q, d].
    """
    q = np.asarray(q, dtype=np.float64)
    kc = np.asarray(kc, dtype=np.float64)
    vc = np.asarray(vc, dtype=np.float64)
    Hq, d = q.shape
    out = np.zeros((Hq, d), dtype=np.float64)
    for h in range(Hq):
        kv = h // group
        logits = scale * (kc[kv] @ q[h])
        if bias is not None:
            logits = logits + np.asarray(bias[kv], dtype=np.float64)
        logits = logits - logits.max()
        p = np.exp(logits)
        p /= p.sum()
        out[h] = p @ vc[kv]
    return out


# --------------------------------------------------------------------------
# Algorithm 1, steps 1-6, for one (sequence, KV head)
# --------------------------------------------------------------------------
def compress_head(k, v, q_win_group, *, window=None, pool_kernel=5, recent=16, bucket=32,
                  budget_ratio=0.25, alpha=0.5, scale=None, gate_mode="cosine",
                  gate_threshold=0.0, gate_temperature=1.0, route_mode="bucket"):
    """Run scoring, selection, routing, gating, merging and the ratio bias for
    one KV head.  k, v [n, d]; q_win_group [G, W, d].  Returns a dict of every
    intermediate and output (float64 / int64)."""
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    q_win_group = np.asarray(q_win_group, dtype=np.float64)
    n, d = k.shape
    W = q_win_group.shape[1]
    if window is not None:
        assert window == W
    if not (1 <= W <= n):
        raise ValueError("window must lie in [1, n]")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    m, mr, ms = budget(n, budget_ratio, recent)
    a = cumulative_attention(q_win_group, k, scale)          # step 1
    vn = value_norms(v)
    c = contribution(a, vn)
    s = pool(c[: n - mr], n - mr, pool_kernel)
    kept, evicted = select(s, n, m, mr)                      # step 2
    if route_mode == "bucket":                               # step 3
        target = route_bucket(a, kept, evicted, bucket)
    elif route_mode == "full_cosine":
        target, _ = route_full_cosine(v, kept, evicted)
    elif route_mode == "bucket_nearest":
        target = route_bucket_nearest(a, kept, evicted, bucket)
    elif route_mode == "coattn":
        target = route_coattention(window_attention_group(q_win_group, k, scale), kept, evicted, bucket)
    else:
        raise ValueError(route_mode)
    g = gate(v, kept, evicted, target, gate_mode, gate_threshold, gate_temperature)  # step 4
    k_out, v_out, w = merge(k, v, a, kept, evicted, target, g)                      # step 5
    bias = ratio_bias(a, kept, evicted, target, g, alpha)                           # step 6
    return dict(m=m, mr=mr, ms=ms, attn=a, vnorm=vn, contribution=c, score=s,
                kept=kept, evicted=evicted, target=target, gate=g,
                k_out=k_out, v_out=v_out, weight=w, bias=bias)


def compress_union(k_heads, v_heads, q_heads, *, group: int, window=None, pool_kernel=5, recent=16, bucket=32,
                   budget_ratio=0.25, alpha=0.5, scale=None, gate_mode="cosine", gate_threshold=0.0,
                   gate_temperature=1.0, route_mode="bucket"):
    """GQA union mode for the KV heads of one cache (Sec. 3.3 union
    paragraph, Sec. 3.6 GQA rule): every head is scored as in Algorithm 1
    step 1, one kept set is chosen by select_union, then each head routes,
    gates and merges its own evicted tokens into the shared set, and the
    bias alpha * ln(mean over heads of R) is shared by the heads.
    k_heads, v_heads [H, n, d]; q_heads [H*G, W, d].  Returns per-head
    stacked arrays (kept / evicted / bias shared, repeated per head)."""
    k_heads = np.asarray(k_heads, dtype=np.float64)
    v_heads = np.asarray(v_heads, dtype=np.float64)
    q_heads = np.asarray(q_heads, dtype=np.float64)
    H, n, d = k_heads.shape
    W = q_heads.shape[1]
    if window is not None:
        assert window == W
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    m, mr, ms = budget(n, budget_ratio, recent)
    a, vn, s = [], [], []
    for h in range(H):
        ah = cumulative_attention(q_heads[h * group:(h + 1) * group], k_heads[h], scale)
        vh = value_norms(v_heads[h])
        a.append(ah)
        vn.append(vh)
        s.append(pool(contribution(ah, vh)[: n - mr], n - mr, pool_kernel))
    kept, evicted = select_union(np.stack(s), n, m, mr)
    targets, gates, k_out, v_out = [], [], [], []
    for h in range(H):
        if route_mode == "bucket":
            tg = route_bucket(a[h], kept, evicted, bucket)
        elif route_mode == "full_cosine":
            tg, _ = route_full_cosine(v_heads[h], kept, evicted)
        else:
            raise ValueError(route_mode)
        g = gate(v_heads[h], kept, evicted, tg, gate_mode, gate_threshold, gate_temperature)
        ko, vo, _ = merge(k_heads[h], v_heads[h], a[h], kept, evicted, tg, g)
        targets.append(tg)
        gates.append(g)
        k_out.append(ko)
        v_out.append(vo)
    bias = ratio_bias_union(np.stack(a), kept, evicted, np.stack(targets), np.stack(gates), alpha)
    return dict(m=m, mr=mr, ms=ms, attn=np.stack(a), vnorm=np.stack(vn), score=np.stack(s),
                kept=np.stack([kept] * H), evicted=np.stack([evicted] * H), target=np.stack(targets),
                gate=np.stack(gates), k_out=np.stack(k_out), v_out=np.stack(v_out), bias=np.stack([bias] * H))


def compress(K, V, Qwin, *, group: int, **kw):
    """Batched driver: K, V [B, H_kv, n, d]; Qwin [B, H_kv*G, W, d].
    Returns a dict of per-(b, kv-head) stacked outputs."""
    K = np.asarray(K)
    B, Hkv = K.shape[:2]
    per = [[compress_head(K[b, h], V[b, h], Qwin[b, h * group:(h + 1) * group], **kw)
            for h in range(Hkv)] for b in range(B)]
    out = {}
    for key in per[0][0]:
        if key in ("m", "mr", "ms"):
            out[key] = per[0][0][key]
        else:
            out[key] = np.stack([np.stack([per[b][h][key] for h in range(Hkv)]) for b in range(B)])
    return out


def decode_steps(qs: np.ndarray, kc: np.ndarray, vc: np.ndarray, bias, group: int,
                 scale: float) -> np.ndarray:
    """decode() for many independent query steps against one compressed
    cache: qs [T, H_q, d] -> o [T, H_q, d].  Per KV head the T*G query rows
    form one matrix, so each step's logits are the same q . k products with
    the bias added, softmax over the m entries, and the weighted sum of
    values."""
    qs = np.asarray(qs, dtype=np.float64)
    kc = np.asarray(kc, dtype=np.float64)
    vc = np.asarray(vc, dtype=np.float64)
    T, Hq, d = qs.shape
    out = np.zeros((T, Hq, d), dtype=np.float64)
    for kv in range(kc.shape[0]):
        rows = qs[:, kv * group:(kv + 1) * group, :].reshape(T * group, d)
        logits = scale * (rows @ kc[kv].T)
        if bias is not None:
            logits = logits + np.asarray(bias[kv], dtype=np.float64)[None, :]
        logits = logits - logits.max(axis=1, keepdims=True)
        p = np.exp(logits)
        p /= p.sum(axis=1, keepdims=True)
        out[:, kv * group:(kv + 1) * group, :] = (p @ vc[kv]).reshape(T, group, d)
    return out


def decode_batched(q, kc, vc, bias, group: int, scale: float):
    """decode() over a leading batch dimension: q [B, H_q, d], kc/vc [B, H_kv, m, d]."""
    return np.stack([decode(q[b], kc[b], vc[b], None if bias is None else bias[b], group, scale)
                     for b in range(q.shape[0])])
