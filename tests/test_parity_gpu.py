"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
the same seeded, storage-rounded inputs.

Stage-wise checks feed every GPU call the oracle's own inputs for that step
(so a selection near-tie cannot cascade); end-to-end checks run the whole
GPU pipeline and allow only selection swaps between near-tied scores.
Bars: indices and gathered keys bit-exact, except near-ties within 1e-6
relative (counted, shown in the session's terminal summary); score / attn /
vnorm within 1e-4 relative (fp32 arithmetic on exact inputs); gates within
1e-5 absolute in every dtype (fp32 arithmetic on exact inputs); merged values
and decode outputs within 1e-4 (fp32 storage) or 2e-2 (bf16 storage); bias
within alpha * that tolerance.
"""
import math

import numpy as np
import pytest
import torch

from oracle import selkv_oracle as O
from paper_2607_16213_amd import synth
from tests.parity_util import (GATE, GATE_ATOL, NEAR_TIE, SCORE_RTOL, TOL, assert_close_elem, assert_close_rows,
                               case_from_workload, compare_end_to_end, dtype_name, gpu_head, layers_batch,
                               make_params, np64, oracle_chain, oracle_head_score, oracle_scale, record,
                               union_selection_check)

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_16213_amd import selkv
    return selkv


def to_dev(x, dtype):
    return torch.as_tensor(np.ascontiguousarray(x)).to(dtype).to(DEV).contiguous()


def random_mode_cases(kind, count):
    """`count` randomly drawn cases for one of the alternative modes: shapes,
    budget, bucket and gate parameters vary; the mode fields fit the kind."""
    out = []
    for i in range(count):
        rng = np.random.default_rng({"readings": 101, "fullcos": 202, "union": 303, "coattn": 404}[kind] * 1000 + i)
        n = int(rng.integers(60, 900))
        case = dict(batch=int(rng.integers(1, 3)), H=int(rng.integers(2 if kind == "union" else 1, 5)),
                    G=int(rng.choice([1, 2, 3, 4, 8])), d=int(rng.choice([64, 128])), n=n,
                    W=int(rng.integers(1, min(48, n) + 1)), dtype=str(rng.choice(["fp32", "bf16"])),
                    budget_ratio=float(rng.uniform(max(2.0 / n, 0.03), 0.8)), gate_mode=int(rng.integers(0, 3)),
                    gate_threshold=float(rng.choice([0.0, 0.3])), gate_temperature=float(rng.choice([0.5, 1.0])))
        if kind == "readings":
            case.update(route_mode=str(rng.choice(["bucket_nearest", "bucket"])), bucket=int(rng.choice([2, 4, 8, 32])))
            case["merge_keys"] = 1 if case["route_mode"] == "bucket" else int(rng.integers(0, 2))
            if case["route_mode"] == "bucket_nearest":   # small buckets, low budget: empty buckets occur
                case.update(bucket=int(rng.choice([2, 4])), budget_ratio=float(rng.uniform(max(2.0 / n, 0.03), 0.12)))
        elif kind == "union":
            case.update(bucket=int(rng.choice([4, 16, 32, 64])))
        elif kind == "coattn":
            case.update(bucket=int(rng.choice([8, 16, 20, 32, 64])))
        out.append(case)
    return out


def run_stagewise(S, p, K, V, Qwin, heads=None):
    """All five calls checked stage by stage; returns the oracle chains."""
    B, H, n, d = K.shape
    tol = TOL[dtype_name(K)]
    m, mr, ms = S.budget(p)
    comp = S.Compressor(p, DEV)
    # ---- score (raw inputs)
    S.score(p, K, V, Qwin, comp.score, comp.attn, comp.vnorm, comp.ws_score)
    torch.cuda.synchronize()
    K64, V64, Q64 = np64(K), np64(V), np64(Qwin)
    G = p.group
    heads = heads or [(b, h) for b in range(B) for h in range(H)]
    chains = {}
    for (b, h) in heads:
        ch = oracle_chain(K64[b, h], V64[b, h], Q64[b, h * G:(h + 1) * G], p, GATE[p.gate_mode])
        chains[(b, h)] = ch
        assert_close_elem(np64(comp.attn[b, h]), ch["a"], SCORE_RTOL, f"attn[{b},{h}]")
        assert_close_elem(np64(comp.vnorm[b, h]), ch["vn"], SCORE_RTOL, f"vnorm[{b},{h}]")
        assert_close_elem(np64(comp.score[b, h]), ch["s"], SCORE_RTOL, f"score[{b},{h}]")
    # ---- select, fed the oracle's fp32 scores (heads not sampled keep GPU scores)
    s_in = comp.score.clone()
    for (b, h), ch in chains.items():
        s_in[b, h] = torch.as_tensor(ch["s32"], dtype=torch.float32)
    S.select(p, s_in, comp.kept, comp.evicted)
    torch.cuda.synchronize()
    for (b, h), ch in chains.items():
        np.testing.assert_array_equal(comp.kept[b, h].cpu().numpy(), ch["kept"], err_msg=f"kept[{b},{h}]")
        np.testing.assert_array_equal(comp.evicted[b, h].cpu().numpy(), ch["ev"], err_msg=f"evicted[{b},{h}]")
    # ---- merge, fed oracle attn / vnorm / kept / evicted
    a_in, vn_in = comp.attn.clone(), comp.vnorm.clone()
    kept_in, ev_in = comp.kept.clone(), comp.evicted.clone()
    for (b, h), ch in chains.items():
        a_in[b, h] = torch.as_tensor(ch["a32"], dtype=torch.float32)
        vn_in[b, h] = torch.as_tensor(ch["vn"], dtype=torch.float32)
        kept_in[b, h] = torch.as_tensor(ch["kept"], dtype=torch.int32)
        ev_in[b, h] = torch.as_tensor(ch["ev"], dtype=torch.int32)
    S.merge(p, K, V, a_in, vn_in, kept_in, ev_in, comp.K_out, comp.V_out, comp.target, comp.gate, comp.ws_merge)
    torch.cuda.synchronize()
    for (b, h), ch in chains.items():
        np.testing.assert_array_equal(comp.target[b, h].cpu().numpy(), ch["target"], err_msg=f"target[{b},{h}]")
        assert np.abs(np64(comp.gate[b, h]) - ch["g"]).max(initial=0) <= GATE_ATOL, f"gate[{b},{h}]"
        assert torch.equal(comp.K_out[b, h].cpu(), K[b, h].cpu()[torch.as_tensor(ch["kept"])]), f"K_out[{b},{h}]"
        assert_close_rows(np64(comp.V_out[b, h]), ch["v_out"], tol, f"V_out[{b},{h}]")
    # ---- bias, fed oracle target / gate
    t_in, g_in = comp.target.clone(), comp.gate.clone()
    for (b, h), ch in chains.items():
        t_in[b, h] = torch.as_tensor(ch["target"], dtype=torch.int32)
        g_in[b, h] = torch.as_tensor(ch["g32"], dtype=torch.float32)
    S.bias(p, a_in, kept_in, ev_in, t_in, g_in, comp.bias, comp.ws_merge)
    torch.cuda.synchronize()
    alpha = float(np.float32(p.alpha))
    for (b, h), ch in chains.items():
        err = np.abs(np64(comp.bias[b, h]) - ch["bias"]).max(initial=0)
        assert err <= max(abs(alpha), 1e-30) * tol, f"bias[{b},{h}] err {err:.3e}"
        unabsorbed = np.setdiff1d(np.arange(m), ch["target"][ch["g32"] * ch["a32"][ch["ev"]] > 0])
        assert (comp.bias[b, h].cpu().numpy()[unabsorbed] == 0).all(), "bias must be exactly 0 where R = 1"
    return comp, chains


def run_decode_check(S, p, chains, K, steps=3, seed=0):
    """Decode over the oracle's compressed caches (values rounded to storage)."""
    B, H = p.batch, p.n_heads_kv
    G, d, dt = p.group, p.head_dim, K.dtype
    tol = TOL[dtype_name(K)]
    m = next(iter(chains.values()))["m"]
    kc = torch.zeros((B, H, m, d), dtype=dt)
    vc = torch.zeros((B, H, m, d), dtype=dt)
    bias = torch.zeros((B, H, m), dtype=torch.float32)
    for (b, h), ch in chains.items():
        kc[b, h] = torch.as_tensor(ch["k_out"]).to(dt)
        vc[b, h] = torch.as_tensor(ch["v_out"]).to(dt)
        bias[b, h] = torch.as_tensor(ch["bias"]).to(torch.float32)
    kc_d, vc_d, bias_d = kc.to(DEV), vc.to(DEV), bias.to(DEV)
    dec = S.Decoder(p, m, DEV)
    g = torch.Generator().manual_seed(1234 + seed)
    for step in range(steps):
        q = torch.randn((B, H * G, d), generator=g).to(dt)
        out = dec.run(q.to(DEV), kc_d, vc_d, bias_d).cpu().double().numpy()
        ref = O.decode_batched(np64(q), np64(kc), np64(vc), np64(bias), G, oracle_scale(p))
        for (b, h) in chains:
            assert_close_rows(out[b, h * G:(h + 1) * G], ref[b, h * G:(h + 1) * G], tol, f"decode step {step}")


# ------------------------------------------------------------------ workloads at full size
def test_tiny_workload_stagewise_and_decode(S):
    w = synth.WORKLOADS["tiny"]
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w))
    _, chains = run_stagewise(S, p, t["K"], t["V"], t["Qwin"])
    run_decode_check(S, p, chains, t["K"], steps=w.decode_steps)


def test_llama_layer_stagewise_and_decode(S):
    w = synth.WORKLOADS["llama_layer"]
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w))
    _, chains = run_stagewise(S, p, t["K"], t["V"], t["Qwin"])
    run_decode_check(S, p, chains, t["K"], steps=4)


@pytest.mark.parametrize("name", ["tiny", "llama_layer"])
def test_end_to_end_with_near_tie_accounting(S, name):
    """The full GPU pipeline on raw inputs.  Selection may differ from the
    oracle only by swaps between candidates within eps of the threshold;
    for every head whose kept set matches, all outputs are checked."""
    w = synth.WORKLOADS[name]
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w))
    comp = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
    torch.cuda.synchronize()
    K64, V64, Q64 = np64(t["K"]), np64(t["V"]), np64(t["Qwin"])
    tol = TOL[w.dtype]
    for b in range(w.batch):
        for h in range(w.n_heads_kv):
            ch = O.compress_head(K64[b, h], V64[b, h], Q64[b, h * w.group:(h + 1) * w.group],
                                 window=w.window, budget_ratio=p.budget_ratio)
            assert_close_elem(np64(comp.attn[b, h]), ch["attn"], SCORE_RTOL, "attn")
            assert_close_elem(np64(comp.score[b, h]), ch["score"], SCORE_RTOL, "score")
            counts = compare_end_to_end(gpu_head(comp, b, h), ch, K64[b, h], w.seq_len, p.bucket, tol,
                                        float(np.float32(p.alpha)))
            record("end_to_end", f"{name} b{b} h{h}", **counts)


# ------------------------------------------------------------------ edge cases, ragged shapes, modes
EDGE = [
    dict(batch=1, H=2, G=2, d=64, n=1000, W=32, dtype="fp32"),                 # ragged n
    dict(batch=2, H=1, G=3, d=128, n=77, W=20, dtype="bf16"),                  # odd G, tiny n
    dict(batch=1, H=2, G=1, d=128, n=17, W=17, dtype="fp32"),                  # W = n
    dict(batch=1, H=1, G=4, d=64, n=300, W=32, dtype="bf16", budget_ratio=1.0),   # identity
    dict(batch=1, H=2, G=2, d=128, n=200, W=8, dtype="fp32", budget_ratio=0.05),  # m < m_r
    dict(batch=1, H=1, G=2, d=64, n=513, W=32, dtype="bf16", gate_mode=1),     # drop
    dict(batch=1, H=1, G=2, d=64, n=513, W=32, dtype="bf16", gate_mode=2),     # merge all
    dict(batch=1, H=2, G=2, d=128, n=400, W=16, dtype="fp32", bucket=4, budget_ratio=0.1),  # empty buckets
    dict(batch=1, H=1, G=2, d=64, n=333, W=32, dtype="fp32", pool_kernel=1, recent=0, bucket=64),
    dict(batch=1, H=1, G=2, d=64, n=333, W=32, dtype="bf16", pool_kernel=7, bucket=1),
    dict(batch=1, H=1, G=8, d=128, n=640, W=64, dtype="bf16"),                 # 512 window rows: row groups
    dict(batch=1, H=1, G=5, d=128, n=256, W=40, dtype="fp32"),                 # fp32 row groups
    dict(batch=1, H=2, G=2, d=64, n=400, W=32, dtype="bf16", gate_threshold=0.3, gate_temperature=0.25, alpha=1.0),
    dict(batch=1, H=2, G=2, d=64, n=128, W=16, dtype="fp32", budget_ratio=1 / 128),  # m = 1: the recent slot only
    dict(batch=1, H=1, G=4, d=128, n=300, W=24, dtype="bf16", scale=0.05),     # explicit softmax scale
    dict(batch=2, H=1, G=2, d=64, n=40, W=8, dtype="bf16", bucket=64),         # n shorter than one bucket
]


MAX_SHAPES = [
    # the most window rows a KV head may have (G * W = 4096): eight row groups per key chunk
    (dict(batch=1, H=1, G=8, d=64, n=1024, W=512, dtype="bf16"), None),
    # the most heads a call may take (batch * H = 65535, the grid's y limit); three heads sampled
    (dict(batch=65535, H=1, G=1, d=64, n=48, W=8, dtype="fp32"), [(0, 0), (32767, 0), (65534, 0)]),
    # a long sequence: 2^20 tokens in one head (the ABI takes up to 2^28), 262144 kept
    (dict(batch=1, H=1, G=2, d=64, n=1 << 20, W=32, dtype="bf16"), None),
]


@pytest.mark.parametrize("case,heads", MAX_SHAPES, ids=["max_window_rows", "max_heads", "long_sequence"])
def test_maximum_shapes_stagewise(S, case, heads):
    """The largest shapes the ABI accepts along its two capped axes, and a
    sequence of 2^20 tokens, every stage checked against the oracle (on
    sampled heads for the head cap), plus one decode step."""
    t = synth.random_case(case["n"] * 3 + case["G"], batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"], device=DEV)
    p = make_params(S, case)
    _, chains = run_stagewise(S, p, t["K"], t["V"], t["Qwin"], heads=heads)
    run_decode_check(S, p, chains, t["K"], steps=1, seed=7)


@pytest.mark.parametrize("case", EDGE, ids=[f"edge{i}" for i in range(len(EDGE))])
def test_edge_cases_stagewise(S, case):
    case = dict(case)
    kw = {k: case.pop(k) for k in list(case) if k not in ("batch", "H", "G", "d", "n", "W", "dtype")}
    t = synth.random_case(case["n"] + case["d"], batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"], device=DEV)
    K, V = t["K"], t["V"]
    if case["n"] > 50:   # a few zero value rows: norm 0 -> sim 0
        V[:, :, 5].zero_()
        V[:, :, 40].zero_()
    p = make_params(S, case, **kw)
    _, chains = run_stagewise(S, p, K, V, t["Qwin"])
    run_decode_check(S, p, chains, K, steps=2)


# ------------------------------------------------------------------ determinism, bias semantics
def test_bitwise_determinism_and_zero_bias(S):
    w = synth.WORKLOADS["llama_layer"].replace(seq_len=4096)
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w))
    c1 = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"]).outputs()
    c2 = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"]).outputs()
    torch.cuda.synchronize()
    for k in c1:
        assert torch.equal(c1[k], c2[k]), k
    m = c1["K_out"].shape[2]
    dec = S.Decoder(p, m, DEV)
    q = synth.make_decode_queries(w, 0, 2, DEV)[0]
    o_null = dec.run(q, c1["K_out"], c1["V_out"], None).clone()
    o_zero = dec.run(q, c1["K_out"], c1["V_out"], torch.zeros_like(c1["bias"])).clone()
    o_b1 = dec.run(q, c1["K_out"], c1["V_out"], c1["bias"]).clone()
    o_b2 = dec.run(q, c1["K_out"], c1["V_out"], c1["bias"]).clone()
    torch.cuda.synchronize()
    assert torch.equal(o_null, o_zero)
    assert torch.equal(o_b1, o_b2)
    assert not torch.equal(o_b1, o_null)


def test_full_budget_identity_on_gpu(S):
    """rho = 1: kept = all, K~ = K and V~ = V bitwise, bias = 0, and decode
    equals full-cache decode bitwise (same kernel, same cache)."""
    w = synth.WORKLOADS["llama_layer"].replace(seq_len=1024)
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w), budget_ratio=1.0)
    c = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
    torch.cuda.synchronize()
    assert torch.equal(c.kept.cpu(), torch.arange(1024, dtype=torch.int32).expand(1, 8, 1024))
    assert torch.equal(c.K_out, t["K"]) and torch.equal(c.V_out, t["V"])
    assert (c.bias == 0).all()
    q = synth.make_decode_queries(w, 0, 1, DEV)[0]
    dec = S.Decoder(p, 1024, DEV)
    a = dec.run(q, c.K_out, c.V_out, c.bias).clone()
    b = dec.run(q, t["K"], t["V"], None).clone()
    assert torch.equal(a, b)
    ref = O.decode_batched(np64(q), np64(t["K"]), np64(t["V"]), None, 4, 1 / math.sqrt(128))
    assert_close_rows(a.cpu().double().numpy(), ref, TOL["bf16"], "decode")


def test_full_cache_decode_100k(S):
    """The comparison decode of the long-context point: the whole 102400-entry
    cache, no bias, sampled heads against the oracle."""
    w = synth.WORKLOADS["ctx100k"]
    t = synth.make_layer(w, 5, DEV)
    p = S.params(batch=1, n_heads_kv=8, group=4, head_dim=128, kv_dtype="bf16")
    dec = S.Decoder(p, w.seq_len, DEV)
    q = synth.make_decode_queries(w, 5, 2, DEV)
    for st in range(2):
        out = dec.run(q[st], t["K"], t["V"], None).cpu().double().numpy()[0]
        for h in (0, 7):
            ref = O.decode(np64(q[st][0, 4 * h:4 * h + 4]), np64(t["K"][0, h])[None], np64(t["V"][0, h])[None],
                           None, 4, 1 / math.sqrt(128))
            assert_close_rows(out[4 * h:4 * h + 4], ref, TOL["bf16"], "full decode")


def test_abi_errors_with_device_memory(S):
    w = synth.WORKLOADS["tiny"]
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w))
    c = S.Compressor(p, DEV)
    small = torch.empty(16, dtype=torch.uint8, device=DEV)
    with pytest.raises(S.SelkvError) as e:
        S.score(p, t["K"], t["V"], t["Qwin"], c.score, c.attn, c.vnorm, small)
    assert e.value.status == 5
    raw = torch.empty(t["K"].numel() * 4 + 16, dtype=torch.uint8, device=DEV)
    import ctypes
    st = S.lib.selkv_score(ctypes.byref(p), ctypes.c_void_p(raw.data_ptr() + 4), ctypes.c_void_p(t["V"].data_ptr()),
                           ctypes.c_void_p(t["Qwin"].data_ptr()), ctypes.c_void_p(c.score.data_ptr()),
                           ctypes.c_void_p(c.attn.data_ptr()), ctypes.c_void_p(c.vnorm.data_ptr()),
                           ctypes.c_void_p(c.ws_score.data_ptr()), c.ws_score.numel(), None)
    assert st == 4
    torch.cuda.synchronize()


def test_decode_hip_graph_replays_match_eager(S):
    """Decode captured in a HIP graph: every replay (with eager work and
    synchronisation in between) equals the eager result bitwise; no state
    carries over in the workspace between graph and eager launches."""
    w = synth.WORKLOADS["llama_layer"].replace(seq_len=4096)
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w))
    c = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
    dec = S.Decoder(S.params(batch=1, n_heads_kv=8, group=4, head_dim=128, kv_dtype="bf16"), c.m, DEV)
    qs = synth.make_decode_queries(w, 0, 4, DEV)
    outs = torch.zeros((4,) + tuple(dec.out.shape), dtype=torch.float32, device=DEV)
    for i in range(4):
        dec.run(qs[i], c.K_out, c.V_out, c.bias, out=outs[i])
    torch.cuda.synchronize()
    ref = outs.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dec.run(qs[0], c.K_out, c.V_out, c.bias)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(4):
            dec.run(qs[i], c.K_out, c.V_out, c.bias, out=outs[i])
    for rep in range(3):
        outs.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(outs, ref), f"replay {rep}"
        dec.run(qs[1], c.K_out, c.V_out, None)       # eager work between replays
        torch.cuda.synchronize()


# ------------------------------------------------------------------ full-cosine routing (all-pairs variant)
def oracle_fullcos(K64, V64, a32, vn, kept, ev, p, gate_mode):
    target, best = O.route_full_cosine(V64, kept, ev)
    g = O.gate(V64, kept, ev, target, gate_mode, float(np.float32(p.gate_threshold)),
               float(np.float32(p.gate_temperature)))
    _, v_out, _ = O.merge(K64, V64, a32, kept, ev, target, g)
    return target, best, g, v_out


FULLCOS = [
    dict(batch=1, H=2, G=2, d=64, n=512, W=32, dtype="fp32"),
    dict(batch=1, H=2, G=4, d=128, n=1000, W=32, dtype="bf16"),
    dict(batch=2, H=1, G=3, d=64, n=300, W=16, dtype="bf16", gate_mode=2),
    dict(batch=1, H=1, G=2, d=128, n=200, W=8, dtype="fp32", gate_mode=1),
    dict(batch=1, H=2, G=2, d=64, n=700, W=32, dtype="bf16", gate_threshold=0.2, gate_temperature=0.5,
         budget_ratio=0.1),
    dict(batch=1, H=1, G=2, d=64, n=300, W=32, dtype="bf16", budget_ratio=1.0),       # nothing evicted
    dict(batch=1, H=1, G=2, d=64, n=100, W=8, dtype="fp32", budget_ratio=0.05),       # m < 16: one partial tile
    dict(batch=1, H=1, G=2, d=64, n=20000, W=32, dtype="bf16", budget_ratio=0.9),     # m > 16384 cursor slots
    # the kept range split into runs of 9 tiles (odd: each run's extra trip reads the next run's first tile,
    # the last run's reads the repeated last kept row), merged in slot order
    dict(batch=1, H=2, G=2, d=128, n=4400, W=32, dtype="bf16", budget_ratio=0.5),
    dict(batch=2, H=1, G=4, d=64, n=9000, W=32, dtype="bf16", budget_ratio=0.3, gate_mode=2),
]
FULLCOS += random_mode_cases("fullcos", 8)
# larger random cases: at least 1024 kept rows, so the match splits the kept range into runs
FULLCOS += [dict(c, n=int(3000 + 1700 * i), budget_ratio=0.35 + 0.1 * i, dtype="bf16")
            for i, c in enumerate(random_mode_cases("fullcos", 12)[8:])]


@pytest.mark.parametrize("case", FULLCOS, ids=[f"fullcos{i}" for i in range(len(FULLCOS))])
def test_full_cosine_routing_stagewise(S, case):
    """a9: the all-pairs cosine routing on MFMA, the stable grouping by
    target and the segmented merge / bias, each fed the oracle's inputs.
    Target slots must match except where the two best cosines lie within
    1e-6 of each other relative (fp32 accumulation over d <= 128 terms of
    unit-scale products); such rows are counted and their two candidate
    slots left out of the value checks."""
    case = dict(case)
    kw = {k: case.pop(k) for k in list(case) if k not in ("batch", "H", "G", "d", "n", "W", "dtype")}
    t = synth.random_case(case["n"] * 7 + 1, batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"],
                          clusters=8, device=DEV)
    K, V, Q = t["K"], t["V"], t["Qwin"]
    V[:, :, 7].zero_()
    p = make_params(S, case, route_mode="full_cosine", **kw)
    tol = TOL[case["dtype"]]
    B, H, n, d = K.shape
    m, mr, ms = S.budget(p)
    comp = S.Compressor(p, DEV)
    S.score(p, K, V, Q, comp.score, comp.attn, comp.vnorm, comp.ws_score)
    torch.cuda.synchronize()
    K64, V64, Q64 = np64(K), np64(V), np64(Q)
    chains = {}
    a_in, vn_in = comp.attn.clone(), comp.vnorm.clone()
    for b in range(B):
        for h in range(H):
            ch = oracle_chain(K64[b, h], V64[b, h], Q64[b, h * p.group:(h + 1) * p.group], p, GATE[p.gate_mode])
            chains[(b, h)] = ch
            comp.kept[b, h] = torch.as_tensor(ch["kept"], dtype=torch.int32)
            comp.evicted[b, h] = torch.as_tensor(ch["ev"], dtype=torch.int32)
            a_in[b, h] = torch.as_tensor(ch["a32"], dtype=torch.float32)
            vn_in[b, h] = torch.as_tensor(ch["vn"], dtype=torch.float32)
    S.merge(p, K, V, a_in, vn_in, comp.kept, comp.evicted, comp.K_out, comp.V_out, comp.target, comp.gate,
            comp.ws_merge)
    torch.cuda.synchronize()
    ties = 0
    for (b, h), ch in chains.items():
        target, best, g, v_out = oracle_fullcos(K64[b, h], V64[b, h], ch["a32"], ch["vn"], ch["kept"], ch["ev"], p,
                                                GATE[p.gate_mode])
        tg = comp.target[b, h].cpu().numpy()
        skip = set()
        vk = V64[b, h][ch["kept"]]
        nk = np.linalg.norm(vk, axis=1)
        for e in np.flatnonzero(tg != target):
            vj = V64[b, h][ch["ev"][e]]
            nj = np.linalg.norm(vj)
            cos = lambda s: 0.0 if nk[s] == 0 or nj == 0 else float(vk[s] @ vj) / (nk[s] * nj)
            c1, c2 = cos(tg[e]), cos(target[e])
            assert abs(c1 - c2) <= NEAR_TIE * max(abs(c1), abs(c2)), \
                f"routing differs at evicted {e}: {tg[e]} vs {target[e]} (cosines {c1!r}, {c2!r})"
            skip |= {int(tg[e]), int(target[e])}
            ties += 1
        keep_e = np.array([int(target[e]) not in skip for e in range(len(target))], dtype=bool)
        assert np.abs(np64(comp.gate[b, h])[keep_e] - g[keep_e]).max(initial=0) <= GATE_ATOL
        assert torch.equal(comp.K_out[b, h].cpu(), K[b, h].cpu()[torch.as_tensor(ch["kept"])])
        rows = np.array([s not in skip for s in range(m)], dtype=bool)
        assert_close_rows(np64(comp.V_out[b, h])[rows], v_out[rows], tol, "V_out")
        # bias through the same grouping, fed the oracle's targets and gates
        g32 = g.astype(np.float32).astype(np.float64)
        comp.target[b, h] = torch.as_tensor(target, dtype=torch.int32)
        comp.gate[b, h] = torch.as_tensor(g32, dtype=torch.float32)
        chains[(b, h)]["fc_bias"] = O.ratio_bias(ch["a32"], ch["kept"], ch["ev"], target, g32,
                                                 float(np.float32(p.alpha)))
    S.bias(p, a_in, comp.kept, comp.evicted, comp.target, comp.gate, comp.bias, comp.ws_merge)
    torch.cuda.synchronize()
    for (b, h), ch in chains.items():
        err = np.abs(np64(comp.bias[b, h]) - ch["fc_bias"]).max(initial=0)
        assert err <= max(abs(float(np.float32(p.alpha))), 1e-30) * tol, f"bias err {err:.3e}"
    record("full_cosine_routing_stagewise", case, route_ties=ties)


def test_full_cosine_deterministic_and_grouped_in_order(S):
    w = synth.WORKLOADS["llama_layer"].replace(seq_len=2048, n_heads_kv=4)
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w), route_mode="full_cosine")
    outs = []
    for _ in range(2):
        c = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in c.outputs().items()})
    for k in outs[0]:
        assert torch.equal(outs[0][k], outs[1][k]), k
    tg = outs[0]["target"].cpu().numpy()
    assert ((tg >= 0) & (tg < outs[0]["kept"].shape[2])).all()


# ------------------------------------------------------------------ GQA union mode (Sec. 3.3, Sec. 3.6)
UNION = [
    dict(batch=1, H=2, G=2, d=64, n=512, W=32, dtype="fp32"),
    dict(batch=2, H=4, G=2, d=128, n=700, W=16, dtype="bf16"),
    dict(batch=1, H=8, G=4, d=128, n=2048, W=32, dtype="bf16"),
    dict(batch=1, H=3, G=1, d=64, n=300, W=8, dtype="fp32", budget_ratio=0.05),        # m < m_r: recent only
    dict(batch=1, H=2, G=2, d=64, n=400, W=32, dtype="bf16", route_mode="full_cosine"),
    dict(batch=1, H=4, G=2, d=64, n=256, W=32, dtype="fp32", budget_ratio=1.0),         # nothing evicted
]
UNION += random_mode_cases("union", 8)


@pytest.mark.parametrize("case", UNION, ids=[f"union{i}" for i in range(len(UNION))])
def test_gqa_union_select_merge_bias(S, case):
    """Union selection fed the oracle's fp32 scores must match the oracle's
    (float64 trim mean) except for near-ties of the trim or of a head's own
    top-m_s (within 1e-6 relative, counted).  On the GPU's kept set, merge
    (bucket or full-cosine routing, per head) and the head-averaged bias are
    then checked per head against the oracle."""
    case = dict(case)
    kw = {k: case.pop(k) for k in list(case) if k not in ("batch", "H", "G", "d", "n", "W", "dtype")}
    t = synth.random_case(case["n"] * 3 + case["H"], batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"], device=DEV)
    K, V, Q = t["K"], t["V"], t["Qwin"]
    p = make_params(S, case, select_mode="union", **kw)
    tol = TOL[case["dtype"]]
    B, H, n, d = K.shape
    m, mr, ms = S.budget(p)
    comp = S.Compressor(p, DEV)
    S.score(p, K, V, Q, comp.score, comp.attn, comp.vnorm, comp.ws_score)
    torch.cuda.synchronize()
    K64, V64, Q64 = np64(K), np64(V), np64(Q)
    s_in, a_in, vn_in = comp.score.clone(), comp.attn.clone(), comp.vnorm.clone()
    heads = {}
    for b in range(B):
        for h in range(H):
            a, vn, sc = oracle_head_score(K64[b, h], V64[b, h], Q64[b, h * p.group:(h + 1) * p.group], p)
            heads[(b, h)] = dict(a32=a.astype(np.float32).astype(np.float64), vn=vn,
                                 s32=sc.astype(np.float32))
            s_in[b, h] = torch.as_tensor(heads[(b, h)]["s32"])
            a_in[b, h] = torch.as_tensor(heads[(b, h)]["a32"], dtype=torch.float32)
            vn_in[b, h] = torch.as_tensor(vn, dtype=torch.float32)
    S.select(p, s_in, comp.kept, comp.evicted, comp.ws_select)
    torch.cuda.synchronize()
    gate_mode = GATE[p.gate_mode]
    alpha = float(np.float32(p.alpha))
    t_in, g_in = comp.target.clone(), comp.gate.clone()
    want = {}
    ties = 0
    for b in range(B):
        kept = comp.kept[b, 0].cpu().numpy()
        ev = comp.evicted[b, 0].cpu().numpy()
        s_heads = np.stack([heads[(b, h)]["s32"] for h in range(H)]).astype(np.float64)
        near, _ = union_selection_check(kept, s_heads, n, m, mr)
        ties += near
        for h in range(H):
            np.testing.assert_array_equal(comp.kept[b, h].cpu().numpy(), kept, err_msg=f"shared kept[{b},{h}]")
            np.testing.assert_array_equal(comp.evicted[b, h].cpu().numpy(), ev, err_msg=f"shared evicted[{b},{h}]")
        tgs, gs = [], []
        for h in range(H):
            hd = heads[(b, h)]
            if p.route_mode == 1:
                tg, _ = O.route_full_cosine(V64[b, h], kept, ev)
            else:
                tg = O.route_bucket(hd["a32"], kept, ev, p.bucket)
            g = O.gate(V64[b, h], kept, ev, tg, gate_mode, float(np.float32(p.gate_threshold)),
                       float(np.float32(p.gate_temperature)))
            g32 = g.astype(np.float32).astype(np.float64)
            _, v_out, _ = O.merge(K64[b, h], V64[b, h], hd["a32"], kept, ev, tg, g)
            want[(b, h)] = dict(target=tg, g=g, v_out=v_out, kept=kept, ev=ev)
            tgs.append(tg)
            gs.append(g32)
            t_in[b, h] = torch.as_tensor(tg, dtype=torch.int32)
            g_in[b, h] = torch.as_tensor(g32, dtype=torch.float32)
        want[b] = O.ratio_bias_union(np.stack([heads[(b, h)]["a32"] for h in range(H)]), kept, ev,
                                     np.stack(tgs), np.stack(gs), alpha)
    # merge with the shared set, per head
    S.merge(p, K, V, a_in, vn_in, comp.kept, comp.evicted, comp.K_out, comp.V_out, comp.target, comp.gate,
            comp.ws_merge)
    torch.cuda.synchronize()
    route_ties = 0
    for b in range(B):
        for h in range(H):
            r = want[(b, h)]
            tg = comp.target[b, h].cpu().numpy()
            skip = set()
            if p.route_mode == 1:      # all-pairs cosine: near-tied best cosines may pick either slot
                vk = V64[b, h][r["kept"]]
                nk = np.linalg.norm(vk, axis=1)
                for e in np.flatnonzero(tg != r["target"]):
                    vj = V64[b, h][r["ev"][e]]
                    nj = np.linalg.norm(vj)
                    cos = lambda s: 0.0 if nk[s] == 0 or nj == 0 else float(vk[s] @ vj) / (nk[s] * nj)
                    c1, c2 = cos(tg[e]), cos(r["target"][e])
                    assert abs(c1 - c2) <= NEAR_TIE * max(abs(c1), abs(c2)), f"routing differs at evicted {e}"
                    skip |= {int(tg[e]), int(r["target"][e])}
                    route_ties += 1
            else:
                np.testing.assert_array_equal(tg, r["target"], err_msg=f"target[{b},{h}]")
            keep_e = np.array([int(x) not in skip for x in r["target"]], dtype=bool)
            assert np.abs(np64(comp.gate[b, h])[keep_e] - r["g"][keep_e]).max(initial=0) <= GATE_ATOL
            assert torch.equal(comp.K_out[b, h].cpu(), K[b, h].cpu()[torch.as_tensor(r["kept"])])
            rows = np.array([s not in skip for s in range(m)], dtype=bool)
            assert_close_rows(np64(comp.V_out[b, h])[rows], r["v_out"][rows], tol, f"V_out[{b},{h}]")
    # bias fed the oracle's targets and gates
    S.bias(p, a_in, comp.kept, comp.evicted, t_in, g_in, comp.bias, comp.ws_merge)
    torch.cuda.synchronize()
    for b in range(B):
        for h in range(H):
            err = np.abs(np64(comp.bias[b, h]) - want[b]).max(initial=0)
            assert err <= max(abs(alpha), 1e-30) * tol, f"bias[{b},{h}] err {err:.3e}"
        assert all(torch.equal(comp.bias[b, 0], comp.bias[b, h]) for h in range(H))
    record("gqa_union_stagewise", case, selection_swaps=ties, route_ties=route_ties)


def union_oracle_compare(S, p, comp, K64, V64, Q64, b, tol):
    """The GPU's union-mode outputs of cache b against compress_union, head
    by head (near-ties of the union selection and of routing counted)."""
    H, G, n = p.n_heads_kv, p.group, p.seq_len
    m, mr, ms = S.budget(p)
    route = "full_cosine" if p.route_mode == 1 else "bucket"
    ref = O.compress_union(K64[b], V64[b], Q64[b], group=G, window=p.window, budget_ratio=p.budget_ratio,
                           bucket=p.bucket, alpha=float(np.float32(p.alpha)), gate_mode=GATE[p.gate_mode],
                           gate_threshold=float(np.float32(p.gate_threshold)),
                           gate_temperature=float(np.float32(p.gate_temperature)), route_mode=route)
    sel = lambda kept, err: union_selection_check(kept, ref["score"], n, m, mr)
    totals = {}
    dirty, skipped = set(), False
    for h in range(H):
        ref_h = {k: (v[h] if isinstance(v, np.ndarray) else v) for k, v in ref.items()}
        vk = None
        if route == "full_cosine":
            vk = V64[b, h]
            nrm = np.linalg.norm(vk, axis=1)
            key = lambda j, i: 0.0 if nrm[i] == 0 or nrm[j] == 0 else float(vk[i] @ vk[j]) / (nrm[i] * nrm[j])
        else:
            key = lambda j, i, a=ref_h["attn"]: a[i]
        c = compare_end_to_end(gpu_head(comp, b, h), ref_h, K64[b, h], n, p.bucket, tol, float(np.float32(p.alpha)),
                               route_key=key, local=route != "full_cosine", selection=sel, check_bias=False,
                               dirty_out=dirty)
        skipped |= bool(c.get("values_skipped"))
        for k, v in c.items():
            totals[k] = max(totals.get(k, 0), v) if k == "score_rel_err" else totals.get(k, 0) + v
    # the shared bias: every head's ratio enters it, so a near-tie of any head leaves its buckets out
    gk, rk = comp.kept[b, 0].cpu().numpy(), ref["kept"][0]
    if not skipped and np.array_equal(gk, rk):
        alpha = float(np.float32(p.alpha))
        keep = np.array([int(x) // p.bucket not in dirty for x in gk], dtype=bool)
        err = np.abs(np64(comp.bias[b, 0])[keep] - ref["bias"][0][keep]).max(initial=0)
        assert err <= abs(alpha) * tol, f"shared bias err {err:.3e}"
    elif not skipped:
        slot_r = {int(x): s for s, x in enumerate(rk)}
        for s, x in enumerate(gk):
            if int(x) // p.bucket in dirty or int(x) not in slot_r:
                continue
            assert abs(float(comp.bias[b, 0, s]) - ref["bias"][0][slot_r[int(x)]]) <= abs(float(p.alpha)) * tol
    return totals


@pytest.mark.parametrize("case", UNION, ids=[f"union{i}" for i in range(len(UNION))])
def test_gqa_union_end_to_end(S, case):
    """The whole union-mode pipeline (fused merge + bias) on the GPU's own
    scores against the oracle's union mode: the shared kept set but for
    near-ties of the trim or of a head's own top-m_s, per-head targets,
    gates and merged values, and the head-averaged bias."""
    case = dict(case)
    kw = {k: case.pop(k) for k in list(case) if k not in ("batch", "H", "G", "d", "n", "W", "dtype")}
    t = synth.random_case(case["n"] * 5 + case["H"], batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"], device=DEV)
    p = make_params(S, case, select_mode="union", **kw)
    comp = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
    torch.cuda.synchronize()
    K64, V64, Q64 = np64(t["K"]), np64(t["V"]), np64(t["Qwin"])
    for b in range(case["batch"]):
        counts = union_oracle_compare(S, p, comp, K64, V64, Q64, b, TOL[case["dtype"]])
        record("gqa_union_end_to_end", f"{case} {kw} b{b}", **counts)


def test_gqa_union_end_to_end_llama_layer(S):
    """The whole union-mode compression of a Llama-shaped layer on the GPU
    against the oracle's union mode (float64 scores, float64 trim mean):
    one kept set of m entries shared by the eight KV heads, equal to the
    oracle's but for near-ties (counted); per-head targets, gates, merged
    values and the head-averaged bias to their bars."""
    w = synth.WORKLOADS["llama_layer"]
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w), select_mode="union")
    comp = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
    torch.cuda.synchronize()
    m, mr, ms = S.budget(p)
    kept = comp.kept[0].cpu().numpy()
    assert (kept == kept[0]).all(), "all KV heads share one kept set"
    assert all(torch.equal(comp.bias[0, 0], comp.bias[0, h]) for h in range(p.n_heads_kv))
    counts = union_oracle_compare(S, p, comp, np64(t["K"]), np64(t["V"]), np64(t["Qwin"]), 0, TOL[w.dtype])
    record("gqa_union_end_to_end", "llama_layer", **counts)


def test_gqa_union_full_size(S):
    """Union-mode compression at the bench's layer size (one ctx100k layer:
    8 KV heads x 102400 tokens, 25600 kept) on the GPU against the oracle's
    union mode: the shared kept set equal to the oracle's but for near-ties
    of the float64 trim mean (counted), then every head's targets, gates,
    merged values and the head-averaged bias to their bars."""
    w = synth.WORKLOADS["ctx100k"]
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w), select_mode="union")
    comp = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
    torch.cuda.synchronize()
    kept = comp.kept[0].cpu().numpy()
    assert (kept == kept[0]).all(), "all KV heads share one kept set"
    counts = union_oracle_compare(S, p, comp, np64(t["K"]), np64(t["V"]), np64(t["Qwin"]), 0, TOL[w.dtype])
    record("gqa_union_full_size", "ctx100k layer 0", **counts)


# ------------------------------------------------------------------ RoPE repositioning (Eq. 7)
ROPE = [
    dict(batch=1, H=2, d=64, n=512, dtype="fp32", theta=10000.0),
    dict(batch=2, H=2, d=128, n=3000, dtype="bf16", theta=500000.0),
    dict(batch=1, H=1, d=128, n=20000, dtype="fp32", theta=10000.0),       # angles up to 1.5e4 rad
    dict(batch=1, H=2, d=64, n=700, dtype="bf16", theta=10000.0, budget_ratio=1.0),
    # the benchmark's size: a 102400-token layer (25600 kept keys per head), Llama-3 theta
    dict(batch=1, H=8, d=128, n=102400, dtype="bf16", theta=500000.0),
    dict(batch=1, H=2, d=128, n=102400, dtype="fp32", theta=500000.0),     # angles up to 1e5 rad
]


@pytest.mark.parametrize("case", ROPE, ids=[f"rope{i}" for i in range(len(ROPE))])
def test_rope_reposition(S, case):
    """Eq. 7 on the GPU against the oracle's two rotations, for kept sets
    spread over the whole sequence; rows already at their slot stay bit for
    bit (a full budget keeps every key where it was)."""
    B, H, d, n = case["batch"], case["H"], case["d"], case["n"]
    dt = torch.bfloat16 if case["dtype"] == "bf16" else torch.float32
    p = S.params(batch=B, n_heads_kv=H, group=1, head_dim=d, seq_len=n, window=8, kv_dtype=case["dtype"],
                 budget_ratio=case.get("budget_ratio", 0.25))
    m, mr, ms = S.budget(p)
    g = torch.Generator().manual_seed(n + d)
    K = torch.randn((B, H, n, d), generator=g).to(dt)
    kept = torch.empty((B, H, m), dtype=torch.int32)
    for b in range(B):
        for h in range(H):
            kept[b, h] = torch.sort(torch.randperm(n, generator=g)[:m]).values.to(torch.int32)
    K_out = torch.gather(K, 2, kept.long()[..., None].expand(B, H, m, d)).contiguous()
    kd, Kd = kept.to(DEV), K_out.to(DEV)
    S.rope_reposition(p, kd, Kd, case["theta"])
    torch.cuda.synchronize()
    got = Kd.cpu()
    tol = TOL[case["dtype"]]
    for b in range(B):
        for h in range(H):
            ks = kept[b, h].numpy()
            want = O.reposition_keys(K_out[b, h].double().numpy(), ks, case["theta"])
            assert_close_rows(got[b, h].double().numpy(), want, tol, f"K~[{b},{h}]")
            same = ks == np.arange(m)
            assert torch.equal(got[b, h][torch.as_tensor(same)], K_out[b, h][torch.as_tensor(same)])
    if case.get("budget_ratio") == 1.0:
        assert torch.equal(got, K_out)


# ------------------------------------------------------------------ generation loop with appended tokens
@pytest.mark.parametrize("name", ["tiny", "llama_layer", "ctx100k"])
def test_decode_with_appended_tokens(S, name):
    """The decode loop after compression: each step appends the new token's
    key and value (bias 0) to the compressed cache and attends over all of
    it.  Checked against the oracle's decode over the compressed cache plus
    the appended rows, at every step."""
    w = synth.WORKLOADS[name]
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w))
    B, H, G, d = p.batch, p.n_heads_kv, p.group, p.head_dim
    heads = [(0, 0)] if name == "tiny" else [(0, 0), (0, 5)]
    # the compressed cache comes from the oracle (its outputs rounded to storage)
    K64, V64, Q64 = np64(t["K"]), np64(t["V"]), np64(t["Qwin"])
    m = S.budget(p)[0]
    steps = 12
    cap = m + steps
    dt = t["K"].dtype
    Kh = torch.zeros((B, H, cap, d), dtype=dt)
    Vh = torch.zeros_like(Kh)
    bh = torch.full((B, H, cap), 7.0, dtype=torch.float32)      # overwritten where appended
    bh[:, :, :m] = 0.0
    for (b, h) in heads:
        ch = oracle_chain(K64[b, h], V64[b, h], Q64[b, h * G:(h + 1) * G], p, GATE[p.gate_mode])
        Kh[b, h, :m] = torch.as_tensor(ch["k_out"]).to(dt)
        Vh[b, h, :m] = torch.as_tensor(ch["v_out"]).to(dt)
        bh[b, h, :m] = torch.as_tensor(ch["bias"]).to(torch.float32)
    Kc, Vc, bias = Kh.to(DEV), Vh.to(DEV), bh.to(DEV)
    ws = S.workspace(p, S.CALL_DECODE, DEV, cap)
    out = torch.empty((B, H * G, d), dtype=torch.float32, device=DEV)
    g = torch.Generator().manual_seed(77)
    tol = TOL[dtype_name(t["K"])]
    for step in range(steps):
        q = torch.randn((B, H * G, d), generator=g).to(dt)
        kn = torch.randn((B, H, d), generator=g).to(dt)
        vn = torch.randn((B, H, d), generator=g).to(dt)
        S.decode_append(p, q.to(DEV), kn.to(DEV), vn.to(DEV), Kc, Vc, bias, m + step, out, ws)
        torch.cuda.synchronize()
        L = m + step + 1
        assert torch.equal(Kc[:, :, m + step].cpu(), kn) and torch.equal(Vc[:, :, m + step].cpu(), vn)
        assert (bias[:, :, m + step] == 0).all()
        Kh[:, :, m + step], Vh[:, :, m + step], bh[:, :, m + step] = kn, vn, 0.0
        ref = O.decode_batched(np64(q), np64(Kh[:, :, :L]), np64(Vh[:, :, :L]), np64(bh[:, :, :L]), G,
                               oracle_scale(p))
        got = out.cpu().double().numpy()
        for (b, h) in heads:
            assert_close_rows(got[b, h * G:(h + 1) * G], ref[b, h * G:(h + 1) * G], tol, f"append step {step}")
    assert torch.equal(bias.cpu(), bh)


def test_decode_append_from_empty_cache_without_bias(S):
    """Generation from an empty cache with no bias array (fp32, d 64, G 1):
    the first step attends over the new token alone (output = its value),
    every later step over all tokens appended so far."""
    p = S.params(batch=2, n_heads_kv=3, group=1, head_dim=64, seq_len=64, window=8, kv_dtype="fp32")
    B, H, G, d = 2, 3, 1, 64
    steps = 40
    Kc = torch.zeros((B, H, steps, d), dtype=torch.float32, device=DEV)
    Vc = torch.zeros_like(Kc)
    ws = S.workspace(p, S.CALL_DECODE, DEV, steps)
    out = torch.empty((B, H * G, d), dtype=torch.float32, device=DEV)
    g = torch.Generator().manual_seed(5)
    Kh, Vh = torch.zeros((B, H, steps, d)), torch.zeros((B, H, steps, d))
    for step in range(steps):
        q = torch.randn((B, H * G, d), generator=g)
        kn, vn = torch.randn((B, H, d), generator=g), torch.randn((B, H, d), generator=g)
        S.decode_append(p, q.to(DEV), kn.to(DEV), vn.to(DEV), Kc, Vc, None, step, out, ws)
        torch.cuda.synchronize()
        Kh[:, :, step], Vh[:, :, step] = kn, vn
        got = out.cpu().double().numpy()
        if step == 0:
            np.testing.assert_allclose(got, vn.double().numpy().reshape(B, H * G, d), rtol=1e-6, atol=1e-6)
        ref = O.decode_batched(np64(q), np64(Kh[:, :, :step + 1]), np64(Vh[:, :, :step + 1]), None, G,
                               1.0 / math.sqrt(d))
        assert_close_rows(got, ref, TOL["fp32"], f"append step {step}")
    assert torch.equal(Kc.cpu(), Kh) and torch.equal(Vc.cpu(), Vh)


# ------------------------------------------------------------------ alternative readings as modes
READINGS = [
    # many empty buckets: bucket 4 at a 10% budget leaves most buckets without a kept token
    dict(batch=1, H=2, G=2, d=64, n=600, W=16, dtype="fp32", route_mode="bucket_nearest", bucket=4,
         budget_ratio=0.1),
    dict(batch=2, H=1, G=4, d=128, n=1000, W=32, dtype="bf16", route_mode="bucket_nearest", bucket=4,
         budget_ratio=0.1),
    dict(batch=1, H=2, G=2, d=128, n=777, W=16, dtype="fp32", route_mode="bucket_nearest", bucket=8,
         budget_ratio=0.05, gate_mode=2, merge_keys=1),
    dict(batch=1, H=1, G=2, d=64, n=300, W=8, dtype="bf16", route_mode="bucket_nearest", bucket=2,
         budget_ratio=0.02, gate_mode=1),
    dict(batch=1, H=1, G=2, d=64, n=200, W=8, dtype="fp32", route_mode="bucket_nearest", budget_ratio=1.0),
    dict(batch=1, H=2, G=2, d=64, n=513, W=16, dtype="fp32", merge_keys=1),                # bucket routing
    dict(batch=1, H=2, G=4, d=128, n=1000, W=32, dtype="bf16", merge_keys=1, gate_mode=2),
    dict(batch=1, H=2, G=2, d=128, n=640, W=16, dtype="bf16", route_mode="bucket_nearest", bucket=4,
         budget_ratio=0.1, merge_keys=1),
]
READINGS += random_mode_cases("readings", 8)


@pytest.mark.parametrize("case", READINGS, ids=[f"reading{i}" for i in range(len(READINGS))])
def test_alternative_readings_stagewise(S, case):
    """Nearest-kept fallback for empty buckets and key merging, each fed the
    oracle's fp32 attention, norms and kept / evicted lists: targets are
    integers decided on identical fp32 inputs (bit-exact), gates, merged
    values and merged keys within the storage tolerance, gathered keys
    bit-exact where keys are not merged, and the bias through the grouping by
    target slot fed the oracle's targets and gates."""
    case = dict(case)
    kw = {k: case.pop(k) for k in list(case) if k not in ("batch", "H", "G", "d", "n", "W", "dtype")}
    t = synth.random_case(case["n"] * 11 + 3, batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"],
                          clusters=6, device=DEV)
    K, V, Q = t["K"], t["V"], t["Qwin"]
    p = make_params(S, case, **kw)
    nearest = p.route_mode == S.ROUTE_BUCKET_NEAREST
    mk = bool(p.merge_keys)
    tol = TOL[case["dtype"]]
    B, H, n, d = K.shape
    m, mr, ms = S.budget(p)
    comp = S.Compressor(p, DEV)
    S.score(p, K, V, Q, comp.score, comp.attn, comp.vnorm, comp.ws_score)
    torch.cuda.synchronize()
    K64, V64, Q64 = np64(K), np64(V), np64(Q)
    refs = {}
    a_in, vn_in = comp.attn.clone(), comp.vnorm.clone()
    tau, temp = float(np.float32(p.gate_threshold)), float(np.float32(p.gate_temperature))
    fallbacks = 0
    for b in range(B):
        for h in range(H):
            ch = oracle_chain(K64[b, h], V64[b, h], Q64[b, h * p.group:(h + 1) * p.group], p, GATE[p.gate_mode])
            comp.kept[b, h] = torch.as_tensor(ch["kept"], dtype=torch.int32)
            comp.evicted[b, h] = torch.as_tensor(ch["ev"], dtype=torch.int32)
            a_in[b, h] = torch.as_tensor(ch["a32"], dtype=torch.float32)
            vn_in[b, h] = torch.as_tensor(ch["vn"], dtype=torch.float32)
            if nearest:
                target = O.route_bucket_nearest(ch["a32"], ch["kept"], ch["ev"], p.bucket)
                fallbacks += int((ch["target"] < 0).sum())
            else:
                target = ch["target"]
            g = O.gate(V64[b, h], ch["kept"], ch["ev"], target, GATE[p.gate_mode], tau, temp)
            k_out, v_out, _ = O.merge(K64[b, h], V64[b, h], ch["a32"], ch["kept"], ch["ev"], target, g,
                                      merge_keys=mk)
            g32 = g.astype(np.float32).astype(np.float64)
            bias = O.ratio_bias(ch["a32"], ch["kept"], ch["ev"], target, g32, float(np.float32(p.alpha)))
            refs[(b, h)] = dict(kept=ch["kept"], target=target, g=g, g32=g32, k_out=k_out, v_out=v_out, bias=bias)
    if nearest and n > m:
        assert fallbacks > 0, "the case must leave some bucket without a kept token"
    S.merge(p, K, V, a_in, vn_in, comp.kept, comp.evicted, comp.K_out, comp.V_out, comp.target, comp.gate,
            comp.ws_merge)
    torch.cuda.synchronize()
    for (b, h), r in refs.items():
        np.testing.assert_array_equal(comp.target[b, h].cpu().numpy(), r["target"], err_msg=f"target[{b},{h}]")
        assert np.abs(np64(comp.gate[b, h]) - r["g"]).max(initial=0) <= GATE_ATOL, f"gate[{b},{h}]"
        assert_close_rows(np64(comp.V_out[b, h]), r["v_out"], tol, f"V_out[{b},{h}]")
        if mk:
            assert_close_rows(np64(comp.K_out[b, h]), r["k_out"], tol, f"K_out[{b},{h}]")
            untouched = np.setdiff1d(np.arange(m), r["target"][r["target"] >= 0])    # nothing routed there
            got = comp.K_out[b, h].cpu()[torch.as_tensor(untouched, dtype=torch.long)]
            assert torch.equal(got, K[b, h].cpu()[torch.as_tensor(r["kept"][untouched])]), "unmerged keys gathered"
        else:
            assert torch.equal(comp.K_out[b, h].cpu(), K[b, h].cpu()[torch.as_tensor(r["kept"])]), f"K_out[{b},{h}]"
        comp.target[b, h] = torch.as_tensor(r["target"], dtype=torch.int32)
        comp.gate[b, h] = torch.as_tensor(r["g32"], dtype=torch.float32)
    S.bias(p, a_in, comp.kept, comp.evicted, comp.target, comp.gate, comp.bias, comp.ws_merge)
    torch.cuda.synchronize()
    for (b, h), r in refs.items():
        err = np.abs(np64(comp.bias[b, h]) - r["bias"]).max(initial=0)
        assert err <= max(abs(float(np.float32(p.alpha))), 1e-30) * tol, f"bias[{b},{h}] err {err:.3e}"
    record("alternative_readings_stagewise", case, nearest_fallbacks=fallbacks)


def test_nearest_fallback_end_to_end_llama_layer(S):
    """The whole pipeline with the nearest-kept fallback on one Llama-shaped
    layer (bucket 8 at a 10% budget): every evicted token gets a kept target
    (no -1), buckets that keep a token route exactly as the plain bucket
    routing on the same call's outputs, and the run is bitwise repeatable."""
    w = synth.WORKLOADS["llama_layer"].replace(seq_len=4096, n_heads_kv=4)
    t = synth.make_layer(w, 0, DEV)
    p_near = make_params(S, case_from_workload(w), route_mode="bucket_nearest", bucket=8, budget_ratio=0.1)
    p_plain = make_params(S, case_from_workload(w), bucket=8, budget_ratio=0.1)
    outs = []
    for p in (p_near, p_near, p_plain):
        c = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in c.outputs().items()})
    for k in outs[0]:
        assert torch.equal(outs[0][k], outs[1][k]), k
    near, plain = outs[0], outs[2]
    assert torch.equal(near["kept"], plain["kept"])
    tn, tp = near["target"].cpu().numpy(), plain["target"].cpu().numpy()
    m = near["kept"].shape[2]
    assert ((tn >= 0) & (tn < m)).all()
    routed = tp >= 0
    assert (~routed).any(), "a 10% budget with bucket 8 must leave empty buckets"
    np.testing.assert_array_equal(tn[routed], tp[routed])


# ------------------------------------------------------------------ co-attention routing (alternative reading of Eq. 3)
COATTN = [
    dict(batch=1, H=2, G=2, d=64, n=500, W=16, dtype="fp32"),
    dict(batch=2, H=1, G=4, d=128, n=1000, W=32, dtype="bf16"),                      # shared-tile row statistics
    dict(batch=1, H=2, G=4, d=128, n=700, W=16, dtype="bf16", bucket=64, budget_ratio=0.1),
    dict(batch=1, H=1, G=3, d=64, n=333, W=8, dtype="bf16", bucket=20, gate_mode=2, merge_keys=1),
    dict(batch=1, H=1, G=8, d=64, n=600, W=32, dtype="bf16", bucket=8),              # 256 rows: general passes
    dict(batch=1, H=2, G=2, d=128, n=400, W=8, dtype="fp32", bucket=16, budget_ratio=0.05, gate_mode=1),
    dict(batch=1, H=1, G=2, d=64, n=200, W=8, dtype="fp32", budget_ratio=1.0),       # nothing evicted
]
COATTN += random_mode_cases("coattn", 8)


@pytest.mark.parametrize("case", COATTN, ids=[f"coattn{i}" for i in range(len(COATTN))])
def test_coattn_routing_stagewise(S, case):
    """Co-attention routing fed the oracle's kept / evicted lists: every
    target equals the oracle's argmax of sum_r A[r, j] A[r, i] (float64 A)
    except where the two candidates' co-attentions lie within 1e-6 of each
    other relative (NEAR_TIE, counted).  Merge and bias with route_mode COATTN are then
    fed the oracle's targets: gates, merged values (and keys), gathered keys
    and the bias as for the bucket routing."""
    case = dict(case)
    kw = {k: case.pop(k) for k in list(case) if k not in ("batch", "H", "G", "d", "n", "W", "dtype")}
    t = synth.random_case(case["n"] * 13 + 5, batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"],
                          clusters=6, device=DEV)
    K, V, Q = t["K"], t["V"], t["Qwin"]
    p = make_params(S, case, route_mode="coattn", **kw)
    mk = bool(p.merge_keys)
    tol = TOL[case["dtype"]]
    B, H, n, d = K.shape
    G = p.group
    m, mr, ms = S.budget(p)
    comp = S.Compressor(p, DEV)
    S.score(p, K, V, Q, comp.score, comp.attn, comp.vnorm, comp.ws_score)
    torch.cuda.synchronize()
    K64, V64, Q64 = np64(K), np64(V), np64(Q)
    a_in, vn_in = comp.attn.clone(), comp.vnorm.clone()
    refs = {}
    for b in range(B):
        for h in range(H):
            ch = oracle_chain(K64[b, h], V64[b, h], Q64[b, h * G:(h + 1) * G], p, GATE[p.gate_mode])
            comp.kept[b, h] = torch.as_tensor(ch["kept"], dtype=torch.int32)
            comp.evicted[b, h] = torch.as_tensor(ch["ev"], dtype=torch.int32)
            a_in[b, h] = torch.as_tensor(ch["a32"], dtype=torch.float32)
            vn_in[b, h] = torch.as_tensor(ch["vn"], dtype=torch.float32)
            A = O.window_attention_group(Q64[b, h * G:(h + 1) * G], K64[b, h], oracle_scale(p))
            refs[(b, h)] = dict(ch=ch, A=A, target=O.route_coattention(A, ch["kept"], ch["ev"], p.bucket))
    comp.target.fill_(-7)
    S.route_coattn(p, K, Q, comp.kept, comp.evicted, comp.target, comp.ws_route)
    torch.cuda.synchronize()
    ties = 0
    for (b, h), r in refs.items():
        ch, A, tg_ref = r["ch"], r["A"], r["target"]
        tg = comp.target[b, h].cpu().numpy()
        np.testing.assert_array_equal(tg < 0, tg_ref < 0, err_msg="empty buckets")
        for e in np.flatnonzero(tg != tg_ref):
            j = ch["ev"][e]
            co = lambda s: float(A[:, ch["kept"][s]] @ A[:, j])
            c_gpu, c_ref = co(tg[e]), co(tg_ref[e])
            assert ch["kept"][tg[e]] // p.bucket == j // p.bucket, "target outside the bucket"
            assert abs(c_gpu - c_ref) <= NEAR_TIE * abs(c_ref), f"routing differs at evicted {e}: {c_gpu!r} {c_ref!r}"
            ties += 1
    # merge / bias fed the oracle's targets
    for (b, h), r in refs.items():
        ch, tg = r["ch"], r["target"]
        comp.target[b, h] = torch.as_tensor(tg, dtype=torch.int32)
        g = O.gate(V64[b, h], ch["kept"], ch["ev"], tg, GATE[p.gate_mode], float(np.float32(p.gate_threshold)),
                   float(np.float32(p.gate_temperature)))
        r["g"] = g
        r["g32"] = g.astype(np.float32).astype(np.float64)
        r["k_out"], r["v_out"], _ = O.merge(K64[b, h], V64[b, h], ch["a32"], ch["kept"], ch["ev"], tg, g,
                                            merge_keys=mk)
        r["bias"] = O.ratio_bias(ch["a32"], ch["kept"], ch["ev"], tg, r["g32"], float(np.float32(p.alpha)))
    t_in = comp.target.clone()
    S.merge(p, K, V, a_in, vn_in, comp.kept, comp.evicted, comp.K_out, comp.V_out, comp.target, comp.gate,
            comp.ws_merge)
    torch.cuda.synchronize()
    assert torch.equal(comp.target, t_in), "merge must not write the given targets"
    for (b, h), r in refs.items():
        ch = r["ch"]
        assert np.abs(np64(comp.gate[b, h]) - r["g"]).max(initial=0) <= GATE_ATOL, f"gate[{b},{h}]"
        assert_close_rows(np64(comp.V_out[b, h]), r["v_out"], tol, f"V_out[{b},{h}]")
        if mk:
            assert_close_rows(np64(comp.K_out[b, h]), r["k_out"], tol, f"K_out[{b},{h}]")
        else:
            assert torch.equal(comp.K_out[b, h].cpu(), K[b, h].cpu()[torch.as_tensor(ch["kept"])]), f"K_out[{b},{h}]"
        untouched = np.setdiff1d(np.arange(m), r["target"][r["target"] >= 0])
        sel = torch.as_tensor(untouched, dtype=torch.long)
        assert torch.equal(comp.V_out[b, h].cpu()[sel], V[b, h].cpu()[torch.as_tensor(ch["kept"][untouched])])
        comp.gate[b, h] = torch.as_tensor(r["g32"], dtype=torch.float32)
    S.bias(p, a_in, comp.kept, comp.evicted, comp.target, comp.gate, comp.bias, comp.ws_merge)
    torch.cuda.synchronize()
    for (b, h), r in refs.items():
        err = np.abs(np64(comp.bias[b, h]) - r["bias"]).max(initial=0)
        assert err <= max(abs(float(np.float32(p.alpha))), 1e-30) * tol, f"bias[{b},{h}] err {err:.3e}"
    record("coattn_routing_stagewise", case, route_ties=ties)


def test_coattn_end_to_end_llama_layer(S):
    """The whole pipeline with co-attention routing on a Llama-shaped layer:
    every target lies in its token's bucket, -1 exactly for the buckets that
    keep nothing, at least one bucket routes differently from Eq. 3, the run
    is bitwise repeatable, and every head matches the oracle's co-attention
    pipeline end to end (near-ties of selection and routing counted)."""
    w = synth.WORKLOADS["llama_layer"].replace(seq_len=4096, n_heads_kv=4)
    t = synth.make_layer(w, 0, DEV)
    p_co = make_params(S, case_from_workload(w), route_mode="coattn")
    p_eq3 = make_params(S, case_from_workload(w))
    outs = []
    for p in (p_co, p_co, p_eq3):
        c = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in c.outputs().items()})
    for k in outs[0]:
        assert torch.equal(outs[0][k], outs[1][k]), k
    co, eq3 = outs[0], outs[2]
    assert torch.equal(co["kept"], eq3["kept"])
    kept, ev = co["kept"].cpu().numpy(), co["evicted"].cpu().numpy()
    tc, te = co["target"].cpu().numpy(), eq3["target"].cpu().numpy()
    np.testing.assert_array_equal(tc < 0, te < 0)
    Bk = p_co.bucket
    for b in range(kept.shape[0]):
        for h in range(kept.shape[1]):
            ok = tc[b, h] >= 0
            assert (kept[b, h][tc[b, h][ok]] // Bk == ev[b, h][ok] // Bk).all()
    assert (tc != te).any(), "co-attention should route some token differently from Eq. 3"
    # the whole co-attention pipeline against the oracle's, head by head
    K64, V64, Q64 = np64(t["K"]), np64(t["V"]), np64(t["Qwin"])
    G = p_co.group
    for h in range(p_co.n_heads_kv):
        ch = O.compress_head(K64[0, h], V64[0, h], Q64[0, h * G:(h + 1) * G], window=w.window, route_mode="coattn")
        A = O.window_attention_group(Q64[0, h * G:(h + 1) * G], K64[0, h], oracle_scale(p_co))
        gpu = {k: (np64(v[0, h]) if v.is_floating_point() else v[0, h].cpu().numpy()) for k, v in co.items()}
        gpu = dict(attn=gpu["attn"], score=gpu["score"], kept=gpu["kept"], evicted=gpu["evicted"],
                   target=gpu["target"], gate=gpu["gate"], v_out=gpu["V_out"], bias=gpu["bias"], K_out=gpu["K_out"])
        counts = compare_end_to_end(gpu, ch, K64[0, h], w.seq_len, Bk, TOL[w.dtype], float(np.float32(p_co.alpha)),
                                    route_key=lambda j, i, A=A: float(A[:, i] @ A[:, j]))
        record("coattn_end_to_end", f"llama_layer n=4096 h{h}", **counts)


# ------------------------------------------------------------------ alternative modes end to end
def _oracle_mode_compare(S, p, comp, case, K64, V64, Q64, tag):
    """Every (sequence, KV head) of the GPU's whole pipeline in p's mode
    against compress_head in the same mode (keys merged with the Eq. 5
    weights when p.merge_keys is set), near-ties counted."""
    route = {S.ROUTE_BUCKET: "bucket", S.ROUTE_FULL_COSINE: "full_cosine", S.ROUTE_BUCKET_NEAREST: "bucket_nearest",
             S.ROUTE_COATTN: "coattn"}[p.route_mode]
    G, Bk = case["G"], p.bucket
    tol, alpha = TOL[case["dtype"]], float(np.float32(p.alpha))
    for b in range(case["batch"]):
        for h in range(case["H"]):
            ch = O.compress_head(K64[b, h], V64[b, h], Q64[b, h * G:(h + 1) * G], window=case["W"],
                                 budget_ratio=p.budget_ratio, bucket=Bk, gate_mode=GATE[p.gate_mode],
                                 gate_threshold=float(np.float32(p.gate_threshold)),
                                 gate_temperature=float(np.float32(p.gate_temperature)), route_mode=route)
            if p.merge_keys:
                ch["k_out"], _, _ = O.merge(K64[b, h], V64[b, h], ch["attn"], ch["kept"], ch["evicted"],
                                            ch["target"], ch["gate"], merge_keys=True)
            key = None
            if route == "coattn":
                A = O.window_attention_group(Q64[b, h * G:(h + 1) * G], K64[b, h], oracle_scale(p))
                key = lambda j, i, A=A: float(A[:, i] @ A[:, j])
            counts = compare_end_to_end(gpu_head(comp, b, h), ch, K64[b, h], case["n"], Bk, tol, alpha, route_key=key,
                                        local=route in ("bucket", "coattn"), keys_merged=bool(p.merge_keys))
            record(tag, f"{case} b{b} h{h}", **counts)


@pytest.mark.parametrize("mode", [dict(route_mode="bucket_nearest"), dict(merge_keys=1)],
                         ids=["bucket_nearest", "merge_keys"])
def test_alternative_modes_full_size(S, mode):
    """The nearest-kept fallback and the merged-keys reading at the bench's
    layer size (one ctx100k layer, 8 KV heads x 102400 tokens): the whole
    GPU pipeline, then KV heads 0 and 1 against the oracle's pipeline in the
    same mode (near-ties of selection and routing counted)."""
    w = synth.WORKLOADS["ctx100k"]
    t = synth.make_layer(w, 0, DEV)
    p = make_params(S, case_from_workload(w), **mode)
    comp = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
    torch.cuda.synchronize()
    case = dict(batch=1, H=2, G=w.group, d=w.head_dim, n=w.seq_len, W=w.window, dtype=w.dtype)
    _oracle_mode_compare(S, p, comp, case, np64(t["K"][:, :2]), np64(t["V"][:, :2]), np64(t["Qwin"][:, :2 * w.group]),
                         "alternative_modes_full_size_" + ("bucket_nearest" if "route_mode" in mode else "merge_keys"))


@pytest.mark.parametrize("case", READINGS + [dict(c, route_mode="coattn") for c in COATTN],
                         ids=[f"reading{i}" for i in range(len(READINGS))] + [f"coattn{i}" for i in range(len(COATTN))])
def test_alternative_modes_end_to_end(S, case):
    """The nearest-kept fallback, merged keys and co-attention routing run
    as whole GPU pipelines (score, select, [route,] fused merge + bias) on
    the GPU's own intermediate results, against the oracle's pipeline in the
    same mode."""
    case = dict(case)
    kw = {k: case.pop(k) for k in list(case) if k not in ("batch", "H", "G", "d", "n", "W", "dtype")}
    t = synth.random_case(case["n"] * 17 + 9, batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"],
                          clusters=6, device=DEV)
    p = make_params(S, case, **kw)
    comp = S.Compressor(p, DEV).run(t["K"], t["V"], t["Qwin"])
    torch.cuda.synchronize()
    _oracle_mode_compare(S, p, comp, dict(case, **kw), np64(t["K"]), np64(t["V"]), np64(t["Qwin"]),
                         "alternative_modes_end_to_end")


# ------------------------------------------------------------------ fused merge + bias (steps 3 - 6 in one pass)
FUSED = [
    dict(batch=1, H=2, G=4, d=128, n=2000, W=32, dtype="bf16"),
    dict(batch=2, H=2, G=2, d=64, n=777, W=16, dtype="fp32", gate_mode=2),
    dict(batch=1, H=2, G=2, d=128, n=640, W=16, dtype="bf16", route_mode="bucket_nearest", bucket=4,
         budget_ratio=0.1),
    dict(batch=1, H=2, G=2, d=64, n=513, W=16, dtype="fp32", route_mode="bucket_nearest", bucket=2,
         budget_ratio=0.02, merge_keys=1),
    dict(batch=1, H=2, G=4, d=128, n=1000, W=32, dtype="bf16", merge_keys=1),
    dict(batch=1, H=2, G=4, d=128, n=1500, W=32, dtype="bf16", route_mode="coattn"),
    dict(batch=1, H=2, G=2, d=64, n=700, W=16, dtype="fp32", route_mode="coattn", bucket=64),
    dict(batch=1, H=2, G=4, d=128, n=1200, W=32, dtype="bf16", route_mode="full_cosine"),
    dict(batch=2, H=4, G=2, d=128, n=900, W=32, dtype="bf16", select_mode="union"),
    dict(batch=1, H=4, G=2, d=64, n=600, W=16, dtype="fp32", select_mode="union", route_mode="full_cosine"),
    dict(batch=1, H=2, G=2, d=64, n=100, W=8, dtype="fp32", budget_ratio=1.0),         # nothing evicted
]


@pytest.mark.parametrize("case", FUSED, ids=[f"fused{i}" for i in range(len(FUSED))])
def test_merge_bias_fused_equals_merge_then_bias(S, case):
    """selkv_merge_bias gives bit for bit what selkv_merge followed by
    selkv_bias gives, in every routing, gate, key and selection mode: the
    bias kernels sum a slot's absorbed mass in the merge kernels' order.
    The fused outputs are then checked against the oracle's whole pipeline
    in the same mode (near-ties of selection and routing counted)."""
    case = dict(case)
    kw = {k: case.pop(k) for k in list(case) if k not in ("batch", "H", "G", "d", "n", "W", "dtype")}
    t = synth.random_case(case["n"] * 7 + 5, batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"],
                          clusters=6, device=DEV)
    p = make_params(S, case, **kw)
    print(f"fused case {case} {kw}", flush=True)
    comp = S.Compressor(p, DEV)
    comp.run(t["K"], t["V"], t["Qwin"], fused=False)
    torch.cuda.synchronize()
    sep = {k: v.clone() for k, v in comp.outputs().items()}
    for v in (comp.K_out, comp.V_out, comp.gate, comp.bias):
        v.fill_(float("nan"))
    comp.target.fill_(-7)
    comp.run(t["K"], t["V"], t["Qwin"], fused=True)
    torch.cuda.synchronize()
    fused = comp.outputs()
    for k in ("kept", "evicted", "target", "gate", "K_out", "V_out", "bias"):
        a, b = sep[k], fused[k]
        assert torch.equal(a.view(torch.int32) if a.is_floating_point() and a.element_size() == 4 else a,
                           b.view(torch.int32) if b.is_floating_point() and b.element_size() == 4 else b), k
    # and the fused outputs against the oracle's whole pipeline in the same mode
    K64, V64, Q64 = np64(t["K"]), np64(t["V"]), np64(t["Qwin"])
    alpha = float(np.float32(p.alpha))
    tol = TOL[case["dtype"]]
    G, B = case["G"], p.bucket
    if kw.get("select_mode") == "union":
        for b in range(case["batch"]):
            record("fused_vs_oracle", f"{case} {kw} b{b}", **union_oracle_compare(S, p, comp, K64, V64, Q64, b, tol))
        return
    route = {S.ROUTE_BUCKET: "bucket", S.ROUTE_FULL_COSINE: "full_cosine", S.ROUTE_BUCKET_NEAREST: "bucket_nearest",
             S.ROUTE_COATTN: "coattn"}[p.route_mode]
    for b in range(case["batch"]):
        for h in range(case["H"]):
            ch = O.compress_head(K64[b, h], V64[b, h], Q64[b, h * G:(h + 1) * G], window=case["W"],
                                 budget_ratio=p.budget_ratio, bucket=B, gate_mode=GATE[p.gate_mode], route_mode=route)
            if p.merge_keys:    # the merged-keys reading: keys take the Eq. 5 weights
                ch["k_out"], _, _ = O.merge(K64[b, h], V64[b, h], ch["attn"], ch["kept"], ch["evicted"],
                                            ch["target"], ch["gate"], merge_keys=True)
            if route == "coattn":
                A = O.window_attention_group(Q64[b, h * G:(h + 1) * G], K64[b, h], oracle_scale(p))
                key = lambda j, i, A=A: float(A[:, i] @ A[:, j])
            elif route == "full_cosine":
                vv = V64[b, h]
                nrm = np.linalg.norm(vv, axis=1)
                key = lambda j, i, vv=vv, nrm=nrm: (0.0 if nrm[i] == 0 or nrm[j] == 0
                                                    else float(vv[i] @ vv[j]) / (nrm[i] * nrm[j]))
            else:
                key = None
            counts = compare_end_to_end(gpu_head(comp, b, h), ch, K64[b, h], case["n"], B, tol, alpha,
                                        route_key=key, local=route in ("bucket", "coattn"),
                                        keys_merged=bool(p.merge_keys))
            record("fused_vs_oracle", f"{case} {kw} b{b} h{h}", **counts)


# ------------------------------------------------------------------ workspaces need no initialisation
DIRTY = FUSED + [
    dict(batch=1, H=2, G=2, d=64, n=300, W=16, dtype="bf16", route_mode="full_cosine", budget_ratio=1.0),
    dict(batch=1, H=2, G=2, d=64, n=300, W=16, dtype="fp32", select_mode="union", budget_ratio=1.0),
]


@pytest.mark.parametrize("case", DIRTY, ids=[f"dirty{i}" for i in range(len(DIRTY))])
def test_compression_workspaces_need_no_zero_fill(S, case):
    """The score, select, route and merge workspaces are scratch the library
    writes before it reads: filled with seeded random bytes instead of zeros,
    every output of the compression (fused and merge-then-bias) is bit for bit
    the same, in every routing, selection and key mode and with nothing
    evicted (rho = 1, where the full-cosine grouping writes no offsets)."""
    case = dict(case)
    kw = {k: case.pop(k) for k in list(case) if k not in ("batch", "H", "G", "d", "n", "W", "dtype")}
    t = synth.random_case(case["n"] * 11 + 3, batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"],
                          clusters=6, device=DEV)
    p = make_params(S, case, **kw)
    print(f"dirty workspace case {case} {kw}", flush=True)
    gen = torch.Generator(device="cpu").manual_seed(case["n"])
    for fused in (True, False):
        comp = S.Compressor(p, DEV)
        comp.run(t["K"], t["V"], t["Qwin"], fused=fused)
        torch.cuda.synchronize()
        clean = {k: v.clone() for k, v in comp.outputs().items()}
        for ws in (comp.ws_score, comp.ws_select, comp.ws_merge, comp.ws_route):
            if ws is not None:
                ws.copy_(torch.randint(0, 256, ws.shape, dtype=torch.uint8, generator=gen))
        comp.run(t["K"], t["V"], t["Qwin"], fused=fused)
        torch.cuda.synchronize()
        for k, v in comp.outputs().items():
            a, b = clean[k], v
            if a.is_floating_point():
                a, b = a.view(torch.int16 if a.element_size() == 2 else torch.int32), \
                    b.view(torch.int16 if b.element_size() == 2 else torch.int32)
            assert torch.equal(a, b), f"{k} differs after a dirty workspace (fused={fused})"


# ------------------------------------------------------------------ selection: the threshold's bin
def _select_case(rng, kind):
    """(n, m, scores [2, n - 16] fp32) for a selection whose threshold falls
    in a bin of a chosen population.  The kernel bins the offsets of the
    order-preserving keys from the head's smallest key into 4096 bins whose
    width fits the head's key range, stages the threshold's bin in LDS when it
    holds at most 12288 keys, and resolves the remaining low bits there (or in
    global passes) at most 10 bits at a time."""
    if kind in ("at_cap", "over_cap"):
        # a cluster within 8 ulps of 1.0 (one bin: the range reaches 100) holding the threshold
        inbin = 12288 if kind == "at_cap" else 12289
        hi, top = 7712, 10
        n_cand = inbin + hi + top
        clus = np.float32(1.0) + np.float32(2.0 ** -23) * rng.integers(0, 8, (2, inbin)).astype(np.float32)
        s = np.concatenate([clus, 4.0 + rng.random((2, hi)), np.full((2, top), 100.0)], axis=1)
        s = np.stack([rng.permutation(r) for r in s])
        ms = top + hi + 5000
    elif kind == "all_equal":       # zero key range: no low pass, ties decide
        n_cand, ms = 30000, 7000
        s = np.full((2, n_cand), 0.75)
    elif kind == "ties":            # five values 8 ulps apart: exact bins, many ties at the threshold
        n_cand, ms = 10000, 4000
        vals = np.float32(1.0) + np.float32(2.0 ** -20) * np.arange(5, dtype=np.float32)
        s = vals[rng.integers(0, 5, (2, n_cand))]
    elif kind == "one_low_pass":    # 20000 consecutive floats: bins of 8 keys, one 3-bit low pass
        n_cand, ms = 20000, 6000
        s = np.float32(1.0) + np.float32(2.0 ** -23) * np.stack([rng.permutation(n_cand) for _ in range(2)]).astype(np.float32)
    elif kind == "minus_inf":       # -inf marks candidates that must not be chosen (the GQA union's non-members)
        n_cand, ms = 40000, 9000
        s = np.float32(1.0) + np.float32(0.01) * rng.random((2, n_cand)).astype(np.float32)
        s[rng.random((2, n_cand)) < 0.4] = -np.inf
    elif kind == "few_finite":      # fewer finite keys than m_s: the threshold is -inf, ties by position
        n_cand, ms = 20000, 7000
        s = np.full((2, n_cand), -np.inf, dtype=np.float32)
        for r in range(2):
            s[r, rng.choice(n_cand, 3000, replace=False)] = 1.0 + rng.random(3000)
    else:                           # "mixed_sign": keys span nearly 2^32, two full low passes
        n_cand, ms = 30000, 9000
        s = np.stack([np.concatenate([-np.exp(rng.normal(0, 20, n_cand // 2)), np.exp(rng.normal(0, 20, n_cand // 2))])
                      for _ in range(2)])
        s = np.stack([rng.permutation(r) for r in s.astype(np.float32)])
    n = n_cand + 16
    return n, ms + 16, np.asarray(s, dtype=np.float32)


@pytest.mark.parametrize("kind", ["at_cap", "over_cap", "all_equal", "ties", "one_low_pass", "mixed_sign", "minus_inf",
                                  "few_finite"])
def test_select_threshold_bin_staged_or_not(S, kind):
    """Whichever way the threshold's bin is resolved (staged in LDS or by
    passes over the scores, with zero, one or two low passes, over the keys
    above -inf or over all keys), the kept and evicted lists are the
    oracle's bit for bit (equal scores: the lower position wins)."""
    rng = np.random.default_rng({"at_cap": 1, "over_cap": 2, "all_equal": 3, "ties": 4, "one_low_pass": 5,
                                 "mixed_sign": 6, "minus_inf": 7, "few_finite": 8}[kind])
    n, m, s = _select_case(rng, kind)
    p = S.params(batch=1, n_heads_kv=2, group=1, head_dim=64, seq_len=n, window=8, kv_dtype="fp32",
                 budget_ratio=(m + 0.5) / n)
    mm, mr, ms = S.budget(p)
    assert (mm, mr) == (m, 16)
    print(f"select {kind}: n={n} m={m}", flush=True)
    score = torch.as_tensor(s)[None].to(DEV).contiguous()
    kept = torch.empty((1, 2, m), dtype=torch.int32, device=DEV)
    ev = torch.empty((1, 2, n - m), dtype=torch.int32, device=DEV)
    S.select(p, score, kept, ev)
    torch.cuda.synchronize()
    for h in range(2):
        k_ref, e_ref = O.select(s[h].astype(np.float64), n, m, mr)
        assert np.array_equal(kept[0, h].cpu().numpy(), k_ref), (kind, h)
        assert np.array_equal(ev[0, h].cpu().numpy(), e_ref), (kind, h)


# ------------------------------------------------------------------ random configurations, stage by stage
def _random_config(seed):
    rng = np.random.default_rng(9000 + seed)
    d = int(rng.choice([64, 128]))
    n = int(rng.integers(40, 900))
    W = int(rng.integers(1, min(64, n) + 1))
    G = int(rng.choice([1, 2, 3, 4, 5, 8]))
    case = dict(batch=int(rng.integers(1, 3)), H=int(rng.integers(1, 4)), G=G, d=d, n=n, W=W,
                dtype=str(rng.choice(["fp32", "bf16"])))
    kw = dict(bucket=int(rng.choice([1, 3, 8, 16, 32, 48, 64])), pool_kernel=int(rng.choice([1, 3, 5, 9, 33])),
              recent=int(rng.integers(0, 33)), budget_ratio=float(rng.uniform(max(2.0 / n, 0.02), 1.0)),
              gate_mode=int(rng.integers(0, 3)), gate_threshold=float(rng.choice([0.0, 0.2, 0.5])),
              gate_temperature=float(rng.choice([0.25, 0.5, 1.0, 2.0])), alpha=float(rng.uniform(0.1, 2.0)),
              scale=float(rng.choice([0.0, 0.05, 0.2])))
    return case, kw


def _random_mid_config(seed):
    """Mid-size draws: several score chunks, select chunks and match tiles per
    head, window rows up to 512, budgets up to 60%."""
    rng = np.random.default_rng(77000 + seed)
    d = int(rng.choice([64, 128]))
    n = int(rng.integers(1000, 24000))
    W = int(rng.integers(1, 129))
    G = int(rng.choice([1, 2, 4, 8]))
    while G * W > 512:
        W //= 2
    case = dict(batch=int(rng.integers(1, 3)), H=int(rng.integers(1, 3)), G=G, d=d, n=n, W=W,
                dtype=str(rng.choice(["fp32", "bf16"])))
    kw = dict(bucket=int(rng.choice([8, 16, 32, 48, 64])), pool_kernel=int(rng.choice([1, 5, 9])),
              recent=int(rng.integers(0, 65)), budget_ratio=float(rng.uniform(0.05, 0.6)),
              gate_mode=int(rng.integers(0, 3)), gate_threshold=float(rng.choice([0.0, 0.2])),
              gate_temperature=float(rng.choice([0.5, 1.0])), alpha=float(rng.uniform(0.1, 1.0)),
              scale=float(rng.choice([0.0, 0.05])))
    return case, kw


@pytest.mark.parametrize("seed", range(64))
def test_random_configs_stagewise(S, seed):
    """Randomly drawn shapes and parameters (batch, heads, group, d, n, W,
    bucket, pooling kernel, recent window, budget, gate mode / threshold /
    temperature, alpha, softmax scale, storage dtype): every stage fed the
    oracle's inputs matches it (indices bit-exact), one decode step over the
    oracle's cache matches, and the fused merge + bias call reproduces the
    separate calls bit for bit on the GPU's own chain."""
    _random_check(S, seed, *_random_config(seed))


@pytest.mark.parametrize("seed", range(16))
def test_random_mid_size_configs_stagewise(S, seed):
    """As test_random_configs_stagewise, at 1000 - 24000 tokens per head."""
    _random_check(S, seed, *_random_mid_config(seed))


def _random_check(S, seed, case, kw):
    print(f"random config {seed}: {case} {kw}", flush=True)
    t = synth.random_case(seed * 31 + 7, batch=case["batch"], n_heads_kv=case["H"], group=case["G"],
                          head_dim=case["d"], seq_len=case["n"], window=case["W"], dtype=case["dtype"],
                          clusters=5, device=DEV)
    p = make_params(S, case, **kw)
    _, chains = run_stagewise(S, p, t["K"], t["V"], t["Qwin"])
    run_decode_check(S, p, chains, t["K"], steps=1, seed=seed)
    comp = S.Compressor(p, DEV)
    comp.run(t["K"], t["V"], t["Qwin"], fused=False)
    sep = {k: v.clone() for k, v in comp.outputs().items()}
    comp.run(t["K"], t["V"], t["Qwin"], fused=True)
    torch.cuda.synchronize()
    for k, v in comp.outputs().items():
        assert torch.equal(v, sep[k]), k


# ------------------------------------------------------------------ all-pairs routing with more than 65535 kept slots
def test_full_cosine_three_sort_passes(S):
    """70000 kept slots: the slot keys 0 .. m need 17 bits, so the grouping
    by target slot takes three 8-bit radix passes.  Sampled rows are checked
    against the float64 cosine argmax (near-ties within 1e-6 counted); then
    every slot's merged value and bias against the oracle's Eq. 5 / Eq. 6
    fed the GPU's own targets and gates, which holds only if every slot's
    list is exactly its tokens."""
    case = dict(batch=1, H=1, G=2, d=64, n=140000, W=16, dtype="bf16")
    t = synth.random_case(140001, batch=1, n_heads_kv=1, group=2, head_dim=64, seq_len=case["n"], window=16,
                          dtype="bf16", clusters=8, device=DEV)
    K, V, Q = t["K"], t["V"], t["Qwin"]
    p = make_params(S, case, budget_ratio=0.5)
    comp = S.Compressor(p, DEV).run(K, V, Q)
    pf = make_params(S, case, budget_ratio=0.5, route_mode="full_cosine")
    ws = S.workspace(pf, S.CALL_MERGE, DEV)
    K_out, V_out = torch.empty_like(comp.K_out), torch.empty_like(comp.V_out)
    target, gate = torch.empty_like(comp.target), torch.empty_like(comp.gate)
    S.merge(pf, K, V, comp.attn, comp.vnorm, comp.kept, comp.evicted, K_out, V_out, target, gate, ws)
    bias = torch.empty_like(comp.bias)
    S.bias(pf, comp.attn, comp.kept, comp.evicted, target, gate, bias, ws)
    torch.cuda.synchronize()
    m = comp.m
    assert m > 65535
    kept, ev = comp.kept[0, 0].cpu().numpy(), comp.evicted[0, 0].cpu().numpy()
    tg, g = target[0, 0].cpu().numpy(), gate[0, 0].cpu().double().numpy()
    assert ((tg >= 0) & (tg < m)).all()
    V64, K64 = np64(V[0, 0]), np64(K[0, 0])
    vk = V64[kept]
    nk = np.linalg.norm(vk, axis=1)
    rows = np.random.default_rng(3).choice(len(ev), 256, replace=False)
    ties = 0
    for r in rows:
        vj = V64[ev[r]]
        cos = (vk @ vj) / (nk * np.linalg.norm(vj))
        best = int(np.argmax(cos))
        if tg[r] != best:
            assert cos[tg[r]] >= cos[best] - NEAR_TIE * abs(cos[best]), f"row {ev[r]}"
            ties += 1
    a = comp.attn[0, 0].cpu().double().numpy()
    _, v_out, _ = O.merge(K64, V64, a, kept, ev, tg, g)
    assert_close_rows(np64(V_out[0, 0]), v_out, TOL["bf16"], "V_out")
    want = O.ratio_bias(a, kept, ev, tg, g, float(np.float32(p.alpha)))
    # fp32 sums of the same fp32 inputs: any slot holding a wrong list would be off by far more
    assert (np.abs(np64(bias[0, 0]) - want) <= 1e-5 * (1 + np.abs(want))).all()
    assert torch.equal(K_out[0, 0].cpu(), K[0, 0].cpu()[torch.as_tensor(kept)])
    record("full_cosine_three_sort_passes", "n 140000, m 70000", route_ties=ties)


# ------------------------------------------------------------------ all-pairs routing at the full ctx100k size, sampled
def test_full_cosine_full_size_sampled(S):
    """a9 at the bench's size: one ctx100k layer (8 KV heads, 76800 evicted x
    25600 kept rows each, the kept range split into runs).  The GPU's own
    attn / vnorm / kept / evicted feed the full-cosine merge call; for 512
    sampled evicted rows of two heads the float64 cosine argmax over all
    kept rows (lowest slot on ties) must be the GPU's target, except where
    the two cosines lie within 1e-6 of each other relative (counted); gates
    follow the chosen target's cosine.  Every kept slot of those heads is
    then checked: keys gathered bit for bit, merged values (Eq. 5) and
    biases (Eq. 6) against float64 on the GPU's own targets and gates."""
    w = synth.WORKLOADS["ctx100k"]
    t = synth.make_layer(w, 0, DEV)
    K, V, Q = t["K"], t["V"], t["Qwin"]
    p = make_params(S, case_from_workload(w))
    comp = S.Compressor(p, DEV).run(K, V, Q)
    pf = make_params(S, case_from_workload(w), route_mode="full_cosine")
    ws = S.workspace(pf, S.CALL_MERGE, DEV)
    K_out, V_out = torch.empty_like(comp.K_out), torch.empty_like(comp.V_out)
    target, gate = torch.empty_like(comp.target), torch.empty_like(comp.gate)
    S.merge(pf, K, V, comp.attn, comp.vnorm, comp.kept, comp.evicted, K_out, V_out, target, gate, ws)
    torch.cuda.synchronize()
    rng = np.random.default_rng(77)
    ties = 0
    for h in (0, 5):
        kept = comp.kept[0, h].cpu().numpy()
        ev = comp.evicted[0, h].cpu().numpy()
        V64 = np64(V[0, h])
        Vk = V64[kept]
        nk = np.linalg.norm(Vk, axis=1)
        rows = rng.choice(len(ev), 512, replace=False)
        vj = V64[ev[rows]]
        cos = (vj @ Vk.T) / (np.linalg.norm(vj, axis=1)[:, None] * nk[None, :])
        ref = cos.argmax(axis=1)                      # first (lowest) slot of the maximum
        got = target[0, h].cpu().numpy()[rows]
        g = gate[0, h].cpu().numpy()[rows]
        for r in range(len(rows)):
            c_ref, c_got = cos[r, ref[r]], cos[r, got[r]]
            if got[r] != ref[r]:
                assert c_got >= c_ref - NEAR_TIE * abs(c_ref), f"head {h} row {ev[rows[r]]}: {c_got!r} vs {c_ref!r}"
                ties += 1
            assert abs(g[r] - min(1.0, max(0.0, c_got))) <= GATE_ATOL, f"gate head {h} row {ev[rows[r]]}"
    # the grouping and the segmented merge at this size: every kept slot of the two heads against
    # the float64 Eq. 5 and Eq. 6 on the GPU's own targets and gates (so no near-tie can differ)
    bias = torch.empty_like(comp.bias)
    S.bias(pf, comp.attn, comp.kept, comp.evicted, target, gate, bias, S.workspace(pf, S.CALL_BIAS, DEV))
    torch.cuda.synchronize()
    alpha = float(np.float32(pf.alpha))
    for h in (0, 5):
        kept = comp.kept[0, h].cpu().numpy()
        ev = comp.evicted[0, h].cpu().numpy()
        a = np64(comp.attn[0, h])
        tg = target[0, h].cpu().numpy()
        g = np64(gate[0, h])
        _, v_ref, _ = O.merge(np64(K[0, h]), np64(V[0, h]), a, kept, ev, tg, g)
        assert torch.equal(K_out[0, h].cpu(), K[0, h].cpu()[torch.as_tensor(kept, dtype=torch.long)]), f"K_out head {h}"
        assert_close_rows(np64(V_out[0, h]), v_ref, TOL["bf16"], f"V_out head {h}")
        b_ref = O.ratio_bias(a, kept, ev, tg, g, alpha)
        err = np.abs(np64(bias[0, h]) - b_ref).max()
        assert err <= alpha * TOL["fp32"], f"bias head {h} err {err:.3e}"
        absorbed = np.unique(tg[(tg >= 0) & (g * a[ev] > 0)])
        assert (np64(bias[0, h])[np.setdiff1d(np.arange(len(kept)), absorbed)] == 0).all(), "bias 0 where R = 1"
    record("full_cosine_full_size_sampled", "ctx100k layer 0 heads 0,5 (1024 rows)", route_ties=ties)


# ------------------------------------------------------------------ co-attention routing at the full ctx100k size, sampled
def test_coattn_full_size_sampled(S):
    """The co-attention route mode at the bench's layer size (8 KV heads of
    4 query heads, 102400 tokens, W = 32).  The whole pipeline runs on the
    GPU; for 512 sampled evicted tokens of two heads the float64 argmax over
    the kept tokens of the token's bucket of sum_r A[r, j] A[r, i] (A over
    all 4 x 32 window rows, lowest position on ties) must be the GPU's
    target, except within 1e-6 relative of each other; -1 exactly where the
    bucket keeps nothing; gates follow the chosen target's value cosine.
    Every kept slot of those heads: keys gathered bit for bit, merged values
    and biases against float64 on the GPU's own targets and gates."""
    w = synth.WORKLOADS["ctx100k"]
    t = synth.make_layer(w, 0, DEV)
    K, V, Q = t["K"], t["V"], t["Qwin"]
    p = make_params(S, case_from_workload(w), route_mode="coattn")
    comp = S.Compressor(p, DEV).run(K, V, Q)
    torch.cuda.synchronize()
    G, Bk = p.group, p.bucket
    rng = np.random.default_rng(78)
    ties = unrouted = 0
    for h in (2, 7):
        kept = comp.kept[0, h].cpu().numpy()
        ev = comp.evicted[0, h].cpu().numpy()
        tg = comp.target[0, h].cpu().numpy()
        g = comp.gate[0, h].cpu().numpy()
        K64, V64 = np64(K[0, h]), np64(V[0, h])
        A = O.window_attention_group(np64(Q[0, h * G:(h + 1) * G]), K64, oracle_scale(p))
        rows = np.sort(rng.choice(len(ev), 512, replace=False))
        by_bucket = {}
        for slot, i in enumerate(kept):
            by_bucket.setdefault(int(i) // Bk, []).append(slot)
        for r in rows:
            j = int(ev[r])
            cand = by_bucket.get(j // Bk)
            if not cand:
                assert tg[r] == -1, f"head {h} evicted {j}: bucket keeps nothing, target {tg[r]}"
                assert g[r] == 0.0
                unrouted += 1
                continue
            co = A[:, kept[cand]].T @ A[:, j]
            ref = cand[int(np.argmax(co))]
            assert tg[r] in cand, f"head {h} evicted {j}: target {tg[r]} outside its bucket"
            if tg[r] != ref:
                c_got = float(A[:, kept[tg[r]]] @ A[:, j])
                assert abs(c_got - co.max()) <= NEAR_TIE * abs(co.max()), f"head {h} evicted {j}"
                ties += 1
            g_ref = O.gate(V64, kept, ev[r:r + 1], tg[r:r + 1], GATE[p.gate_mode], float(np.float32(p.gate_threshold)),
                           float(np.float32(p.gate_temperature)))[0]
            assert abs(g[r] - g_ref) <= GATE_ATOL, f"gate head {h} evicted {j}"
        # the merge per target at this size: every kept slot against the float64 Eq. 5 / Eq. 6 on
        # the GPU's own attention, targets and gates
        a = np64(comp.attn[0, h])
        ga = np64(comp.gate[0, h])
        _, v_ref, _ = O.merge(K64, V64, a, kept, ev, tg, ga)
        assert torch.equal(comp.K_out[0, h].cpu(), K[0, h].cpu()[torch.as_tensor(kept, dtype=torch.long)])
        assert_close_rows(np64(comp.V_out[0, h]), v_ref, TOL["bf16"], f"V_out head {h}")
        alpha = float(np.float32(p.alpha))
        err = np.abs(np64(comp.bias[0, h]) - O.ratio_bias(a, kept, ev, tg, ga, alpha)).max()
        assert err <= alpha * TOL["fp32"], f"bias head {h} err {err:.3e}"
    record("coattn_full_size_sampled", "ctx100k layer 0 heads 2,7 (1024 rows)", route_ties=ties, unrouted=unrouted)


# ------------------------------------------------------------------ decode over long, ragged and many-head caches
LONG_DECODE = [
    dict(B=1, H=8, G=4, d=128, L=25600, bias=True),      # the 100k point's compressed cache
    dict(B=1, H=8, G=4, d=128, L=11003, bias=True),      # ragged last chunk
    dict(B=32, H=8, G=4, d=128, L=3000, bias=True),      # 256 heads: one chunk per head
    dict(B=1, H=2, G=8, d=64, L=20000, bias=False),
    dict(B=2, H=4, G=1, d=128, L=9001, bias=True),
    dict(B=1, H=8, G=3, d=128, L=8300, bias=True),
]


@pytest.mark.parametrize("case", LONG_DECODE, ids=[f"long{i}" for i in range(len(LONG_DECODE))])
def test_decode_long_caches(S, case):
    """bf16 decode over long and ragged caches, many heads (one chunk per
    head), G = 1 .. 8, d = 64 / 128, with and without bias, a few dominant
    entries: sampled heads against the float64 oracle; bitwise the same over
    repeated calls, with a workspace first filled with garbage (no
    initialisation is needed), and over HIP graph replays."""
    B, H, G, d, L = case["B"], case["H"], case["G"], case["d"], case["L"]
    gen = torch.Generator(device=DEV)
    gen.manual_seed(L * 7 + H)
    K = (torch.randn((B, H, L, d), device=DEV, generator=gen) * 0.35).to(torch.bfloat16)
    V = torch.randn((B, H, L, d), device=DEV, generator=gen).to(torch.bfloat16)
    bias = None
    if case["bias"]:
        bias = torch.rand((B, H, L), device=DEV, generator=gen) * 0.5
        bias[:, :, ::97] += 4.0                       # a few dominant entries, spread over the chunks
    q = torch.randn((3, B, H * G, d), device=DEV, generator=gen).to(torch.bfloat16)
    p = S.params(batch=B, n_heads_kv=H, group=G, head_dim=d, kv_dtype="bf16")
    dec = S.Decoder(p, L, DEV)
    outs = torch.empty((3, B, H * G, d), dtype=torch.float32, device=DEV)
    for i in range(3):
        dec.run(q[i], K, V, bias, out=outs[i])
    torch.cuda.synchronize()
    ref = outs.clone()
    scale = 1 / math.sqrt(d)
    rng = np.random.default_rng(L)
    for b, h in {(0, 0), (B - 1, H - 1), (int(rng.integers(B)), int(rng.integers(H)))}:
        for i in (0, 2):
            want = O.decode(np64(q[i][b, h * G:(h + 1) * G]), np64(K[b, h])[None], np64(V[b, h])[None],
                            None if bias is None else np64(bias[b, h])[None], G, scale)
            assert_close_rows(np64(outs[i][b, h * G:(h + 1) * G]), want, TOL["bf16"], f"decode b{b} h{h} q{i}")
    dec.ws.fill_(0xAB)                                 # garbage in the partials
    for i in range(3):
        dec.run(q[i], K, V, bias, out=outs[i])
    torch.cuda.synchronize()
    assert torch.equal(outs, ref), "decode differs after the workspace was filled with garbage"
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dec.run(q[0], K, V, bias)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(3):
            dec.run(q[i], K, V, bias, out=outs[i])
    for rep in range(3):
        outs.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(outs, ref), f"graph replay {rep}"
        dec.run(q[1], K, V, None)                      # eager work between replays
        torch.cuda.synchronize()
