"""Helpers shared by the GPU parity tests: run stages of the HIP path and the
float64 oracle on the same stored inputs and compare them."""
import math

import numpy as np
import torch

from oracle import selkv_oracle as O

TOL = {"fp32": 1e-4, "bf16": 2e-2}      # merged values, decode outputs, gate, bias/alpha
SCORE_RTOL = 1e-4                       # score / attn / vnorm: fp32 arithmetic on exact inputs


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


def gpu_inputs_to_np(K, V, Qwin):
    return np64(K), np64(V), np64(Qwin)


def check_selection_near_ties(kept_gpu, s_ref, n, m, mr, eps):
    """The GPU kept set must equal the oracle's top-m_s except for swaps
    between candidates whose oracle scores lie within eps (relative) of the
    selection threshold.  Returns the number of such near-tie swaps."""
    ms = m - mr
    kept_gpu = np.asarray(kept_gpu)
    assert (kept_gpu[ms:] == np.arange(n - mr, n)).all(), "recent window not kept"
    assert (np.diff(kept_gpu) > 0).all(), "kept not ascending"
    if ms == 0:
        return 0
    ref_kept, _ = O.select(s_ref, n, m, mr)
    a, b = set(kept_gpu[:ms].tolist()), set(ref_kept[:ms].tolist())
    if a == b:
        return 0
    order = np.sort(s_ref)[::-1]
    T = order[ms - 1]
    band = eps * max(abs(T), 1e-300)
    for j in a ^ b:
        assert abs(s_ref[j] - T) <= band, f"selection differs at {j}: score {s_ref[j]!r} vs threshold {T!r}"
    return len(a - b)


def compare_end_to_end(gpu, ref, K_head, n, B, tol, alpha):
    """Whole-pipeline comparison of one KV head.

    gpu: numpy arrays attn, score, kept, evicted, target, gate, v_out, bias and
    the raw K_out rows; ref: the oracle's compress_head() dict.  Positions,
    not slots, are compared so a near-tie swap cannot shift the rest.
    Selection swaps are allowed only between candidates within eps of the
    selection threshold, routing differences only between candidate targets
    whose window attention lies within eps; buckets touched by either are
    counted and left out of the value comparisons.  Returns the counts."""
    rel_a = np.abs(gpu["attn"] - ref["attn"]) / np.maximum(np.abs(ref["attn"]), 1e-30)
    rel_s = np.abs(gpu["score"] - ref["score"]) / np.maximum(np.abs(ref["score"]), 1e-30)
    eps = max(1e-6, 4 * float(max(rel_a.max(initial=0), rel_s.max(initial=0))))
    m, mr = ref["m"], ref["mr"]
    swaps = check_selection_near_ties(gpu["kept"], ref["score"], n, m, mr, eps)
    dirty = set()
    for j in set(gpu["kept"].tolist()) ^ set(ref["kept"].tolist()):
        dirty.add(j // B)
    kg, kr = gpu["kept"], ref["kept"]
    ev_g = {int(j): e for e, j in enumerate(gpu["evicted"])}
    ev_r = {int(j): e for e, j in enumerate(ref["evicted"])}
    route_ties = 0
    for j, er in ev_r.items():
        if j // B in dirty or j not in ev_g:
            continue
        eg = ev_g[j]
        tg = -1 if gpu["target"][eg] < 0 else int(kg[gpu["target"][eg]])
        tr = -1 if ref["target"][er] < 0 else int(kr[ref["target"][er]])
        if tg == tr:
            continue
        assert tg >= 0 and tr >= 0, f"routing differs at {j}: {tg} vs {tr}"
        a1, a2 = ref["attn"][tg], ref["attn"][tr]
        assert abs(a1 - a2) <= eps * max(a1, a2), f"routing differs at {j}: a {a1!r} vs {a2!r}"
        route_ties += 1
        dirty.add(j // B)
    nb = (n + B - 1) // B
    assert len(dirty) <= max(2, nb // 100), f"{len(dirty)} of {nb} buckets touched by near-ties"
    # gathered keys are exact for every GPU slot
    assert np.array_equal(gpu["K_out"], K_head[kg]), "K_out is not the gather of K at kept_idx"
    slot_r = {int(p): s for s, p in enumerate(kr)}
    for s, pos in enumerate(kg):
        pos = int(pos)
        if pos // B in dirty:
            continue
        sr = slot_r[pos]
        assert_close_rows(gpu["v_out"][s][None], ref["v_out"][sr][None], tol, f"V_out at {pos}")
        assert abs(gpu["bias"][s] - ref["bias"][sr]) <= abs(alpha) * tol, f"bias at {pos}"
    for j, er in ev_r.items():
        if j // B in dirty:
            continue
        assert abs(gpu["gate"][ev_g[j]] - ref["gate"][er]) <= tol, f"gate at {j}"
    return dict(selection_swaps=swaps, route_ties=route_ties, dirty_buckets=len(dirty), eps=eps)
