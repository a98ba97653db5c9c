"""The C ABI library on the host: it loads, exports every symbol declared in
include/selkv.h, its struct layout matches the binding, and its host-only
logic (budget, workspace sizing, argument validation) behaves as documented.
No call here reaches a kernel launch."""
import ctypes
import json
import os
import re
import subprocess
import tempfile

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "selkv.h")


@pytest.fixture(scope="module")
def S():
    from paper_2607_16213_amd import selkv
    return selkv


def declared_functions():
    text = open(HEADER).read()
    return re.findall(r"SELKV_API\s+[\w\s\*]+?\b(selkv_\w+)\s*\(", text)


def test_header_symbols_exported(S):
    names = declared_functions()
    assert len(names) >= 10
    for name in names:
        assert hasattr(S.lib, name), name
    dyn = subprocess.run(["nm", "-D", "--defined-only", S.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(line.split()[-1] for line in dyn.splitlines() if line.strip())
    missing = [n for n in names if n not in exported]
    assert not missing, missing


def test_struct_layout_matches_c(S):
    fields = [f for f, _ in S.Params._fields_]
    src = ["#include <stdio.h>", "#include <stddef.h>", '#include "selkv.h"', "int main(void){",
           'printf("{\\"size\\": %zu", sizeof(selkv_params));']
    for f in fields:
        src.append(f'printf(", \\"{f}\\": %zu", offsetof(selkv_params, {f}));')
    src.append('printf("}\\n"); return 0; }')
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "layout.c")
        open(c, "w").write("\n".join(src))
        exe = os.path.join(d, "layout")
        r = subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", f"-I{ROOT}/include", "-I/opt/rocm/include", c, "-o", exe],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        layout = json.loads(subprocess.run([exe], capture_output=True, text=True).stdout)
    assert layout["size"] == ctypes.sizeof(S.Params)
    for f in fields:
        assert layout[f] == getattr(S.Params, f).offset, f


def test_params_init_defaults(S):
    p = S.params()
    assert p.struct_size == ctypes.sizeof(S.Params)
    assert (p.window, p.pool_kernel, p.recent, p.bucket) == (32, 5, 16, 32)
    assert abs(p.alpha - 0.5) < 1e-7 and p.budget_ratio == 0.25
    assert S.lib.selkv_abi_version() == 6
    assert S.lib.selkv_status_string(0) == b"success"


def test_budget_matches_golden(S):
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "hand_worked.json")))["budget_cases"]["cases"]
    for n, rho, m, ms in gold:
        p = S.params(seq_len=n, budget_ratio=rho, window=min(32, n))
        got = S.budget(p)
        assert got[0] == m and got[2] == ms, (n, rho, got)


def test_workspace_sizes(S):
    p = S.params(seq_len=8192)
    assert S.workspace_bytes(p, S.CALL_SCORE) > 8 * 8192 * 4
    assert S.workspace_bytes(p, S.CALL_SELECT) == 0
    assert S.workspace_bytes(p, S.CALL_MERGE) >= 8 * (8192 // 32 + 1) * 4
    assert S.workspace_bytes(p, S.CALL_DECODE, 2048) > 0


def test_validation_codes(S):
    def st(p, call=S.CALL_SCORE):
        b = ctypes.c_size_t()
        return S.lib.selkv_workspace_size(ctypes.byref(p), call, 16, ctypes.byref(b))
    assert st(S.params(seq_len=100)) == 0
    assert st(S.params(seq_len=100, head_dim=96)) == 3          # EUNSUPPORTED
    assert st(S.params(seq_len=100, kv_dtype=7)) == 2           # EDTYPE
    assert st(S.params(seq_len=100, window=101)) == 1           # W > n
    assert st(S.params(seq_len=100, pool_kernel=4)) == 1        # even K
    assert st(S.params(seq_len=100, pool_kernel=1027)) == 3     # K above 1025: unsupported
    assert st(S.params(seq_len=100, budget_ratio=0.0)) == 1
    assert st(S.params(seq_len=100, budget_ratio=1.5)) == 1
    assert st(S.params(seq_len=3, window=3, budget_ratio=0.25)) == 1   # m = 0
    assert st(S.params(seq_len=100, gate_temperature=0.0)) == 1
    assert st(S.params(seq_len=100, bucket=65)) == 3
    assert st(S.params(seq_len=(1 << 28) + 1)) == 3
    assert st(S.params(seq_len=1 << 28)) == 0
    assert st(S.params(seq_len=100, group=9), S.CALL_DECODE) == 1
    p = S.params(seq_len=100)
    p.struct_size = 4
    assert st(p) == 1


@pytest.mark.skipif(torch.cuda.is_available(), reason="fake pointers are only passed where no GPU exists")
def test_call_validation_before_launch(S):
    """Invalid calls return a status before any launch (fake pointers never
    get dereferenced: a launch here would fail with EHIP instead)."""
    p = S.params(seq_len=256)
    fake = ctypes.c_void_p(0x10000)
    mis = ctypes.c_void_p(0x10002)
    null = None
    f = S.lib.selkv_score
    assert f(ctypes.byref(p), null, fake, fake, fake, fake, fake, fake, 1 << 30, None) == 1
    assert f(ctypes.byref(p), mis, fake, fake, fake, fake, fake, fake, 1 << 30, None) == 4
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, null, 0, None) == 5
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, fake, 16, None) == 5
    g = S.lib.selkv_decode_attn
    assert g(ctypes.byref(p), fake, fake, fake, null, 0, fake, fake, 1 << 30, None) == 1      # cache_len 0
    assert g(ctypes.byref(p), fake, fake, fake, ctypes.c_void_p(0x10001), 64, fake, fake, 1 << 30, None) == 4
    pf = S.params(seq_len=256, route_mode="full_cosine")
    m = S.lib.selkv_merge
    assert m(ctypes.byref(pf), fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, 16, None) == 5
    assert m(ctypes.byref(pf), fake, fake, fake, fake, fake, fake, mis, fake, fake, fake, fake, 1 << 30, None) == 4
    assert S.workspace_bytes(pf, S.CALL_MERGE) > S.workspace_bytes(S.params(seq_len=256), S.CALL_MERGE)


def test_union_mode_validation_and_workspace(S):
    b = ctypes.c_size_t()
    bad = S.params(seq_len=256, select_mode=2)
    assert S.lib.selkv_workspace_size(ctypes.byref(bad), S.CALL_SELECT, 0, ctypes.byref(b)) == 1
    per_head = S.params(seq_len=256)
    union = S.params(seq_len=256, select_mode="union")
    assert S.workspace_bytes(per_head, S.CALL_SELECT) == 0
    assert S.workspace_bytes(union, S.CALL_SELECT) >= 4 * (256 - 16) * 2
    assert S.workspace_bytes(union, S.CALL_BIAS) >= S.workspace_bytes(per_head, S.CALL_BIAS) + 4 * 8 * 64
    assert S.workspace_bytes(union, S.CALL_MERGE) == S.workspace_bytes(per_head, S.CALL_MERGE)


@pytest.mark.skipif(torch.cuda.is_available(), reason="fake pointers are only passed where no GPU exists")
def test_rope_reposition_validation(S):
    p = S.params(seq_len=256)
    fake, mis = ctypes.c_void_p(0x10000), ctypes.c_void_p(0x10004)
    f = S.lib.selkv_rope_reposition
    assert f(ctypes.byref(p), fake, fake, 1.0, None) == 1          # theta must exceed 1
    assert f(ctypes.byref(p), fake, fake, float("nan"), None) == 1
    assert f(ctypes.byref(p), None, fake, 10000.0, None) == 1
    assert f(ctypes.byref(p), fake, mis, 10000.0, None) == 4       # K_out 16-byte aligned


@pytest.mark.skipif(torch.cuda.is_available(), reason="fake pointers are only passed where no GPU exists")
def test_decode_workspace_covers_every_shorter_cache(S):
    """The decode workspace sized for a capacity serves every cache length up
    to it: the size never shrinks as the length grows (so the capacity's
    size is the largest), for head counts that split the cache into few or
    many chunks, including a capacity whose rounded chunk count is below
    that of shorter caches (2175 entries over 8 KV heads)."""
    for (B, H, G, d) in [(1, 8, 4, 128), (1, 2, 2, 64), (4, 32, 1, 128), (1, 1, 8, 128), (3, 5, 3, 64)]:
        p = S.params(batch=B, n_heads_kv=H, group=G, head_dim=d, seq_len=64)
        for cap in (1, 17, 100, 2175, 2176, 4113, 9000):
            sizes = [S.workspace_bytes(p, S.CALL_DECODE, L) for L in range(1, cap + 1)]
            assert all(a <= b for a, b in zip(sizes, sizes[1:])), (B, H, cap)


@pytest.mark.skipif(torch.cuda.is_available(), reason="fake pointers are only passed where no GPU exists")
def test_decode_append_accepts_the_capacity_workspace_at_every_length(S):
    """Every append step of a cache grown up to its capacity passes the
    workspace check with the size returned for the capacity (the call then
    fails at the launch, there being no GPU, never with EWORKSPACE)."""
    fake = ctypes.c_void_p(0x10000)
    for (H, G, cap) in [(8, 4, 2175), (8, 4, 8191 // 4 + 128), (2, 2, 700), (32, 1, 4096 + 128)]:
        p = S.params(batch=1, n_heads_kv=H, group=G, head_dim=128, seq_len=64)
        ws = S.workspace_bytes(p, S.CALL_DECODE, cap)
        for L in range(0, cap):
            st = S.lib.selkv_decode_append(ctypes.byref(p), fake, fake, fake, fake, fake, None, L, cap, fake, fake,
                                           ws, None)
            assert st != 5, (H, cap, L)


def test_decode_append_validation(S):
    p = S.params(seq_len=256)
    fake = ctypes.c_void_p(0x10000)
    f = S.lib.selkv_decode_append
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, 8, 8, fake, fake, 1 << 30, None) == 1   # full
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, -1, 8, fake, fake, 1 << 30, None) == 1
    assert f(ctypes.byref(p), fake, ctypes.c_void_p(0x10008), fake, fake, fake, fake, 3, 8, fake, fake, 1 << 30,
             None) == 4
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, 3, 8, fake, fake, 0, None) == 5


def test_alternative_readings_validation_and_workspace(S):
    """Nearest-kept fallback and key merging: the flags are checked, and both
    stay bucket-local (the workspace of the plain bucket routing)."""
    b = ctypes.c_size_t()
    for bad in (S.params(seq_len=256, route_mode=4), S.params(seq_len=256, route_mode=-1),
                S.params(seq_len=256, merge_keys=2)):
        assert S.lib.selkv_workspace_size(ctypes.byref(bad), S.CALL_MERGE, 0, ctypes.byref(b)) == 1
    plain = S.params(seq_len=256)
    near = S.params(seq_len=256, route_mode="bucket_nearest")
    full = S.params(seq_len=256, route_mode="full_cosine")
    for call in (S.CALL_MERGE, S.CALL_BIAS):
        assert S.workspace_bytes(near, call) == S.workspace_bytes(plain, call)
        assert S.workspace_bytes(full, call) > S.workspace_bytes(plain, call)
    keys = S.params(seq_len=256, merge_keys=1)
    assert S.workspace_bytes(keys, S.CALL_MERGE) == S.workspace_bytes(plain, S.CALL_MERGE)


def test_coattn_route_validation_and_workspace(S):
    """Co-attention routing: the route mode is accepted, its workspace holds
    the score pass's row statistics plus the bucket offsets, and the call
    checks its arguments before any launch."""
    p = S.params(seq_len=4096, route_mode="coattn")
    assert S.workspace_bytes(p, S.CALL_ROUTE) >= S.workspace_bytes(p, S.CALL_SCORE) - 4 * 8 * 4096
    assert S.workspace_bytes(p, S.CALL_MERGE) == S.workspace_bytes(S.params(seq_len=4096), S.CALL_MERGE)
    b = ctypes.c_size_t()
    bad = S.params(seq_len=256, route_mode=4)
    assert S.lib.selkv_workspace_size(ctypes.byref(bad), S.CALL_ROUTE, 0, ctypes.byref(b)) == 1
    assert S.lib.selkv_workspace_size(ctypes.byref(p), 7, 0, ctypes.byref(b)) == 1


@pytest.mark.skipif(torch.cuda.is_available(), reason="fake pointers are only passed where no GPU exists")
def test_coattn_route_call_validation(S):
    p = S.params(seq_len=256, route_mode="coattn")
    fake, mis = ctypes.c_void_p(0x10000), ctypes.c_void_p(0x10004)
    f = S.lib.selkv_route_coattn
    assert f(ctypes.byref(p), None, fake, fake, fake, fake, fake, 1 << 30, None) == 1
    assert f(ctypes.byref(p), fake, fake, fake, None, fake, fake, 1 << 30, None) == 1        # evicted needed
    assert f(ctypes.byref(p), fake, mis, fake, fake, fake, fake, 1 << 30, None) == 4         # Qwin 16-byte aligned
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, 64, None) == 5             # workspace too small


def test_merge_bias_workspace_is_the_bias_workspace(S):
    """The fused merge + bias call needs the merge's routing scratch plus, in
    union mode, the per-head ratios: exactly what selkv_bias needs."""
    for kw in ({}, dict(route_mode="full_cosine"), dict(route_mode="bucket_nearest"), dict(route_mode="coattn"),
               dict(select_mode="union"), dict(select_mode="union", route_mode="full_cosine")):
        p = S.params(seq_len=1000, **kw)
        assert S.workspace_bytes(p, S.CALL_MERGE_BIAS) == S.workspace_bytes(p, S.CALL_BIAS)
        assert S.workspace_bytes(p, S.CALL_MERGE_BIAS) >= S.workspace_bytes(p, S.CALL_MERGE)


@pytest.mark.skipif(torch.cuda.is_available(), reason="fake pointers are only passed where no GPU exists")
def test_merge_bias_call_validation(S):
    p = S.params(seq_len=256)
    fake, mis4, mis2 = ctypes.c_void_p(0x10000), ctypes.c_void_p(0x10004), ctypes.c_void_p(0x10002)
    f = S.lib.selkv_merge_bias
    big = 1 << 30
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, None, fake, big, None) == 1
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, mis2, fake, big, None) == 4
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, mis4, fake, fake, fake, fake, fake, big, None) == 4
    assert f(ctypes.byref(p), None, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, big, None) == 1
    assert f(ctypes.byref(p), fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, 16, None) == 5
    union = S.params(seq_len=256, select_mode="union")
    need = S.workspace_bytes(union, S.CALL_MERGE_BIAS)
    assert f(ctypes.byref(union), fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, need - 1,
             None) == 5
