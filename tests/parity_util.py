"""Helpers shared by the GPU parity tests: run stages of the HIP path and the
float64 oracle on the same stored inputs and compare them."""
import math

import numpy as np
import torch

from oracle import selkv_oracle as O

TOL = {"fp32": 1e-4, "bf16": 2e-2}      # merged values, decode outputs, bias/alpha
SCORE_RTOL = 1e-4                       # score / attn / vnorm: fp32 arithmetic on exact inputs
GATE_ATOL = 1e-5                        # gates: fp32 arithmetic on exact inputs, in every storage dtype
NEAR_TIE = 1e-6                         # relative score gap within which two choices count as tied

# Near-tie counts of the parity tests, printed in pytest's terminal summary
# and written to parity_record.json (conftest.py).
RECORDS = []


def record(test, case, **counts):
    RECORDS.append(dict(test=test, case=str(case), **counts))


GATE = {0: "cosine", 1: "drop", 2: "merge_all"}


def make_params(S, w_or_case, **kw):
    base = dict(batch=w_or_case["batch"], n_heads_kv=w_or_case["H"], group=w_or_case["G"],
                head_dim=w_or_case["d"], seq_len=w_or_case["n"], window=w_or_case["W"],
                kv_dtype=w_or_case["dtype"])
    base.update(kw)
    return S.params(**base)


def case_from_workload(w, **over):
    return dict(batch=w.batch, H=w.n_heads_kv, G=w.group, d=w.head_dim, n=w.seq_len, W=w.window,
                dtype=w.dtype, **over)


def layers_batch(w, n_layers, device):
    """All layers' caches of a workload back to back as one batch [L*B, H, n, d]
    (and window queries [L*B, H_q, W, d]), the bench's launch layout."""
    from paper_2607_16213_amd import synth
    L = n_layers
    t0 = synth.make_layer(w, 0, device)
    K = torch.empty((L,) + tuple(t0["K"].shape), dtype=t0["K"].dtype, device=device)
    V = torch.empty_like(K)
    Q = torch.empty((L,) + tuple(t0["Qwin"].shape), dtype=t0["Qwin"].dtype, device=device)
    for layer in range(L):
        t = t0 if layer == 0 else synth.make_layer(w, layer, device)
        K[layer], V[layer], Q[layer] = t["K"], t["V"], t["Qwin"]
    return K.flatten(0, 1), V.flatten(0, 1), Q.flatten(0, 1)


def gpu_head(comp, b, h):
    """One (batch, head) slice of the GPU outputs as float64 / int numpy."""
    return dict(attn=np64(comp.attn[b, h]), score=np64(comp.score[b, h]), kept=comp.kept[b, h].cpu().numpy(),
                evicted=comp.evicted[b, h].cpu().numpy(), target=comp.target[b, h].cpu().numpy(),
                gate=np64(comp.gate[b, h]), v_out=np64(comp.V_out[b, h]), bias=np64(comp.bias[b, h]),
                K_out=np64(comp.K_out[b, h]))


def np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().double().cpu().numpy()


def dtype_name(t: torch.Tensor) -> str:
    return "bf16" if t.dtype == torch.bfloat16 else "fp32"


def assert_close_elem(got, ref, rtol, what):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    rms = np.sqrt(np.mean(ref ** 2)) if ref.size else 0.0
    err = np.abs(got - ref)
    bad = err > rtol * (np.abs(ref) + rms) + 1e-30
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} outside rtol {rtol}; max err {err.max():.3e} (rms {rms:.3e})"


def assert_close_rows(got, ref, tol, what):
    """Per-row relative L2 <= tol and elementwise |d| <= tol*(|ref| + rms_row)."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if got.size == 0:
        return
    rms = np.sqrt(np.mean(ref ** 2, axis=-1, keepdims=True))
    err = np.abs(got - ref)
    bad = err > tol * (np.abs(ref) + rms)
    assert not bad.any(), f"{what}: {bad.sum()} elements outside tol {tol}; max err {err.max():.3e}"
    rel = np.linalg.norm(got - ref, axis=-1) / np.maximum(np.linalg.norm(ref, axis=-1), 1e-300)
    assert (rel <= tol).all(), f"{what}: row rel-L2 {rel.max():.3e} > {tol}"


def oracle_kw(p, gate_mode=None):
    gm = {0: "cosine", 1: "drop", 2: "merge_all"}[p.gate_mode] if gate_mode is None else gate_mode
    return dict(pool_kernel=p.pool_kernel, recent=p.recent, bucket=p.bucket, budget_ratio=p.budget_ratio,
                alpha=float(np.float32(p.alpha)), scale=(float(np.float32(p.scale)) if p.scale > 0
                                                         else 1.0 / math.sqrt(p.head_dim)),
                gate_mode=gm, gate_threshold=float(np.float32(p.gate_threshold)),
                gate_temperature=float(np.float32(p.gate_temperature)), route_mode="bucket")


def oracle_scale(p):
    return float(np.float32(p.scale)) if p.scale > 0 else 1.0 / math.sqrt(p.head_dim)


def oracle_head_score(K64, V64, Q64, p):
    """Oracle attn, vnorm, contribution score for one KV head (float64)."""
    n = K64.shape[0]
    m, mr, ms = O.budget(n, p.budget_ratio, p.recent)
    a = O.cumulative_attention(Q64, K64, oracle_scale(p))
    vn = O.value_norms(V64)
    s = O.pool(O.contribution(a, vn)[: n - mr], n - mr, p.pool_kernel)
    return a, vn, s


def oracle_chain(K64, V64, Q64, p, gate_mode):
    """The oracle's steps for one head, chaining fp32-rounded values between
    steps exactly as they are handed to the GPU stage calls."""
    n = K64.shape[0]
    m, mr, ms = O.budget(n, p.budget_ratio, p.recent)
    a, vn, s = oracle_head_score(K64, V64, Q64, p)
    s32 = s.astype(np.float32).astype(np.float64)
    kept, ev = O.select(s32, n, m, mr)
    a32 = a.astype(np.float32).astype(np.float64)
    target = O.route_bucket(a32, kept, ev, p.bucket)
    g = O.gate(V64, kept, ev, target, gate_mode, float(np.float32(p.gate_threshold)),
               float(np.float32(p.gate_temperature)))
    k_out, v_out, _ = O.merge(K64, V64, a32, kept, ev, target, g)
    g32 = g.astype(np.float32).astype(np.float64)
    bias = O.ratio_bias(a32, kept, ev, target, g32, float(np.float32(p.alpha)))
    return dict(a=a, vn=vn, s=s, s32=s32, a32=a32, kept=kept, ev=ev, target=target, g=g, g32=g32,
                k_out=k_out, v_out=v_out, bias=bias, m=m, mr=mr, ms=ms)


def gpu_inputs_to_np(K, V, Qwin):
    return np64(K), np64(V), np64(Qwin)


def selection_differences(kept_gpu, s_ref, n, m, mr, err=0.0):
    """Positions kept by exactly one of the GPU and the oracle's top-m_s of
    s_ref, split by the oracle score's relative distance to the selection
    threshold T (the m_s-th largest score): near_tie within NEAR_TIE |T|;
    out_of_band beyond it but within 4 * err |T| (err: the measured relative
    score error); wrong beyond both.  Returns the three position counts
    (a swap moves two positions)."""
    ms = m - mr
    kept_gpu = np.asarray(kept_gpu)
    assert (kept_gpu[ms:] == np.arange(n - mr, n)).all(), "recent window not kept"
    assert (np.diff(kept_gpu) > 0).all(), "kept not ascending"
    if ms == 0:
        return 0, 0, 0
    ref_kept, _ = O.select(s_ref, n, m, mr)
    diff = set(kept_gpu[:ms].tolist()) ^ set(ref_kept[:ms].tolist())
    T = np.sort(s_ref)[::-1][ms - 1]
    near = oob = wrong = 0
    for j in diff:
        gap = abs(s_ref[j] - T)
        if gap <= NEAR_TIE * abs(T):
            near += 1
        elif gap <= 4 * err * abs(T):
            oob += 1
        else:
            wrong += 1
    return near, oob, wrong


def check_selection_near_ties(kept_gpu, s_ref, n, m, mr, err=0.0, allow_out_of_band=False):
    """The GPU kept set must equal the oracle's top-m_s except for swaps
    between candidates whose oracle scores lie within NEAR_TIE (relative) of
    the selection threshold.  Returns (near-tie swaps, out-of-band swaps);
    the latter (within 4 x the measured score error but beyond NEAR_TIE) are
    accepted only when allow_out_of_band is set.  Counts are positions."""
    near, oob, wrong = selection_differences(kept_gpu, s_ref, n, m, mr, err)
    assert wrong == 0, f"{wrong} kept positions differ from the oracle beyond the near-tie band"
    assert allow_out_of_band or oob == 0, f"{oob} kept positions differ beyond {NEAR_TIE} relative"
    return near, oob


def compare_end_to_end(gpu, ref, K_head, n, B, tol, alpha, allow_out_of_band=False, route_key=None,
                       local=True, selection=None, keys_merged=False, check_bias=True, dirty_out=None):
    """Whole-pipeline comparison of one KV head.

    gpu: numpy arrays attn, score, kept, evicted, target, gate, v_out, bias and
    the raw K_out rows; ref: the oracle's dict for that head (compress_head,
    or one head of compress_union).  Positions, not slots, are compared so a
    near-tie swap cannot shift the rest.  Selection swaps are allowed only
    between candidates within NEAR_TIE of the selection threshold (or as
    `selection` decides: a callable returning (near, out_of_band) that
    raises on anything else); routing differences only between candidate
    targets whose routing scores route_key(j, i) (default: the window
    attention a_i) lie within NEAR_TIE.  With local routes (every target in
    the token's bucket) the buckets touched by either are left out of the
    value comparisons; with non-local routes (full cosine) a head whose kept
    set differs is left out of them, and a routing near-tie leaves out its
    token and its two candidate slots.  keys_merged: K_out rows are compared
    like V_out rows (the merged-keys reading) instead of as a gather.
    check_bias=False leaves the bias out (a bias shared by several heads is
    compared once their near-ties are known); dirty_out, a set, receives
    the buckets left out (local routes).  Returns the counts."""
    rel_a = np.abs(gpu["attn"] - ref["attn"]) / np.maximum(np.abs(ref["attn"]), 1e-30)
    rel_s = np.abs(gpu["score"] - ref["score"]) / np.maximum(np.abs(ref["score"]), 1e-30)
    err = float(max(rel_a.max(initial=0), rel_s.max(initial=0)))
    m, mr = ref["m"], ref["mr"]
    if selection is None:
        swaps, oob = check_selection_near_ties(gpu["kept"], ref["score"], n, m, mr, err, allow_out_of_band)
    else:
        swaps, oob = selection(gpu["kept"], err)
    if route_key is None:
        route_key = lambda j, i: ref["attn"][i]
    kg, kr = gpu["kept"], ref["kept"]
    differ = set(kg.tolist()) ^ set(kr.tolist())
    if not keys_merged:      # gathered keys are exact for every GPU slot
        assert np.array_equal(gpu["K_out"], K_head[kg]), "K_out is not the gather of K at kept_idx"
    counts = dict(selection_swaps=swaps, out_of_band=oob, score_rel_err=err)
    if differ and not local:
        counts.update(route_ties=0, values_skipped=1)
        return counts
    dirty_b = {j // B for j in differ}          # local routes: buckets left out
    dirty_pos, dirty_ev = set(), set()          # non-local routes: kept positions and tokens left out
    ev_g = {int(j): e for e, j in enumerate(gpu["evicted"])}
    ev_r = {int(j): e for e, j in enumerate(ref["evicted"])}
    route_ties = 0
    for j, er in ev_r.items():
        if j // B in dirty_b or j not in ev_g:
            continue
        eg = ev_g[j]
        tg = -1 if gpu["target"][eg] < 0 else int(kg[gpu["target"][eg]])
        tr = -1 if ref["target"][er] < 0 else int(kr[ref["target"][er]])
        if tg == tr:
            continue
        assert tg >= 0 and tr >= 0, f"routing differs at {j}: {tg} vs {tr}"
        k1, k2 = route_key(j, tg), route_key(j, tr)
        assert abs(k1 - k2) <= NEAR_TIE * max(abs(k1), abs(k2)), f"routing differs at {j}: {k1!r} vs {k2!r}"
        route_ties += 1
        if local:
            dirty_b.add(j // B)
        else:
            dirty_pos |= {tg, tr}
            dirty_ev.add(j)
    nb = (n + B - 1) // B
    if local:
        assert len(dirty_b) <= max(2, nb // 100), f"{len(dirty_b)} of {nb} buckets touched by near-ties"
    skip_pos = lambda pos: (pos // B in dirty_b) if local else (pos in dirty_pos)
    slot_r = {int(p): s for s, p in enumerate(kr)}
    for s, pos in enumerate(kg):
        pos = int(pos)
        if skip_pos(pos):
            continue
        sr = slot_r[pos]
        assert_close_rows(gpu["v_out"][s][None], ref["v_out"][sr][None], tol, f"V_out at {pos}")
        if keys_merged:
            assert_close_rows(gpu["K_out"][s][None], ref["k_out"][sr][None], tol, f"K_out at {pos}")
        if check_bias:
            assert abs(gpu["bias"][s] - ref["bias"][sr]) <= abs(alpha) * tol, f"bias at {pos}"
    for j, er in ev_r.items():
        if (j // B in dirty_b) if local else (j in dirty_ev):
            continue
        assert abs(gpu["gate"][ev_g[j]] - ref["gate"][er]) <= GATE_ATOL, f"gate at {j}"
    counts.update(route_ties=route_ties, dirty_buckets=len(dirty_b) if local else len(dirty_pos))
    if dirty_out is not None:
        dirty_out |= dirty_b | {pos // B for pos in dirty_pos}
    return counts


def union_selection_check(kept_gpu, s_heads, n, m, mr):
    """Union selection (Sec. 3.3) of the GPU against the oracle's on the
    float64 per-head scores s_heads [H, n - m_r]: every position kept by
    exactly one of them must be a near-tie, either of the trim (its mean
    score within NEAR_TIE of the m_s-th largest mean among the union
    members) or of some head's own top-m_s (its score within NEAR_TIE of that
    head's threshold, so union membership itself may flip).  Returns
    (near-tie positions, 0)."""
    ms = m - mr
    kept_gpu = np.asarray(kept_gpu)
    assert (kept_gpu[ms:] == np.arange(n - mr, n)).all(), "recent window not kept"
    assert (np.diff(kept_gpu) > 0).all(), "kept not ascending"
    ref_kept, _ = O.select_union(s_heads, n, m, mr)
    diff = set(kept_gpu[:ms].tolist()) ^ set(ref_kept[:ms].tolist())
    if not diff:
        return 0, 0
    H = s_heads.shape[0]
    thr = [np.sort(s_heads[h])[::-1][ms - 1] for h in range(H)]
    union = np.zeros(n - mr, dtype=bool)
    for h in range(H):
        kh, _ = O.select(np.asarray(s_heads[h], np.float64), n, m, mr)
        union[kh[kh < n - mr]] = True
    mean = O.union_mean_score(s_heads)
    cand = np.flatnonzero(union)
    T = np.sort(mean[cand])[::-1][ms - 1] if cand.shape[0] > ms else -np.inf
    band = NEAR_TIE
    for j in diff:
        trim_tie = np.isfinite(T) and abs(mean[j] - T) <= band * abs(T)
        head_tie = any(abs(s_heads[h][j] - thr[h]) <= band * abs(thr[h]) for h in range(H))
        assert trim_tie or head_tie, f"union selection differs at {j}: mean {mean[j]!r} vs trim threshold {T!r}"
    return len(diff), 0
