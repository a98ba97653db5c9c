"""The allocation-free decode entry point (selkv_decode_attn_noalloc) against
selkv_decode_attn with a caller workspace: the same kernels, so the outputs
must agree bit for bit.  Two calls in a row on the shared per-GPU scratch,
the second with a smaller problem (fewer heads, a shorter cache), each
compared with the workspace call on the same inputs; plus the float64
oracle's decode to the bf16 bar, and the oversize rejection."""
import ctypes
import math

import numpy as np
import pytest
import torch

from oracle import selkv_oracle as O
from tests.parity_util import TOL, assert_close_rows, np64

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_16213_amd import selkv
    return selkv


def _case(S, B, H, G, d, L, seed, bias=True):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn((B, H * G, d), generator=g).to(torch.bfloat16).to(DEV)
    K = (torch.randn((B, H, L, d), generator=g) / math.sqrt(d)).to(torch.bfloat16).to(DEV)
    V = torch.randn((B, H, L, d), generator=g).to(torch.bfloat16).to(DEV)
    b = (torch.rand((B, H, L), generator=g) * 0.7).to(DEV) if bias else None
    p = S.params(batch=B, n_heads_kv=H, group=G, head_dim=d, kv_dtype="bf16")
    return p, q, K, V, b


@pytest.mark.parametrize("first,second", [
    (dict(B=1, H=8, G=4, d=128, L=25600), dict(B=1, H=4, G=4, d=128, L=3001)),
    (dict(B=4, H=32, G=1, d=128, L=4096), dict(B=1, H=2, G=8, d=64, L=777)),
])
def test_noalloc_decode_matches_workspace_decode(S, first, second):
    for i, c in enumerate((first, second)):
        p, q, K, V, b = _case(S, c["B"], c["H"], c["G"], c["d"], c["L"], seed=100 + i)
        out_ws = torch.full((c["B"], c["H"] * c["G"], c["d"]), float("nan"), device=DEV)
        out_na = torch.full_like(out_ws, float("nan"))
        dec = S.Decoder(p, c["L"], DEV)
        dec.run(q, K, V, b, out=out_ws)
        S.decode_attn_noalloc(p, q, K, V, b, out_na)
        torch.cuda.synchronize()
        assert torch.equal(out_na, out_ws), f"call {i}: noalloc differs from the workspace decode"
        ref = O.decode_batched(np64(q), np64(K), np64(V), None if b is None else np64(b), c["G"], 1 / math.sqrt(c["d"]))
        assert_close_rows(out_na.cpu().double().numpy(), ref, TOL["bf16"], f"call {i} vs oracle")


def test_noalloc_decode_rejects_shapes_beyond_the_scratch(S):
    # 8192 KV heads with G = 8, d = 128: one split each needs 8192 * 8 * 520 B = 34 MB > 16 MiB
    p = S.params(batch=8192, n_heads_kv=1, group=8, head_dim=128, kv_dtype="bf16")
    nbytes = S.workspace_bytes(p, S.CALL_DECODE, 64)
    assert nbytes > (16 << 20)
    q = torch.empty((8192, 8, 128), dtype=torch.bfloat16, device=DEV)
    K = torch.empty((8192, 1, 64, 128), dtype=torch.bfloat16, device=DEV)
    out = torch.empty((8192, 8, 128), dtype=torch.float32, device=DEV)
    st = S.lib.selkv_decode_attn_noalloc(ctypes.byref(p), ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(K.data_ptr()),
                                         ctypes.c_void_p(K.data_ptr()), None, 64, ctypes.c_void_p(out.data_ptr()),
                                         None)
    assert st == 5      # SELKV_EWORKSPACE, before any launch
