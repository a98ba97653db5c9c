"""Thin ctypes binding of libselkv.so (C ABI in include/selkv.h).

Argument marshalling only: every step runs in the HIP kernels of the
library.  Tensors are torch device tensors (PyTorch provides device memory
and the current stream); the functions check dtype, shape, device and
contiguity, then pass raw pointers.  Importing this module raises if the
built library is missing -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libselkv.so")

F32, BF16 = 0, 1
GATE_COSINE, GATE_DROP, GATE_MERGE_ALL = 0, 1, 2
ROUTE_BUCKET, ROUTE_FULL_COSINE, ROUTE_BUCKET_NEAREST, ROUTE_COATTN = 0, 1, 2, 3
SELECT_PER_HEAD, SELECT_UNION = 0, 1
ABI_VERSION = 6
CALL_SCORE, CALL_SELECT, CALL_MERGE, CALL_BIAS, CALL_DECODE, CALL_ROUTE, CALL_MERGE_BIAS = range(7)
STATUS = {0: "SELKV_OK", 1: "SELKV_EINVAL", 2: "SELKV_EDTYPE", 3: "SELKV_EUNSUPPORTED", 4: "SELKV_EALIGN",
          5: "SELKV_EWORKSPACE", 6: "SELKV_EHIP"}
GATE_MODES = {"cosine": GATE_COSINE, "drop": GATE_DROP, "merge_all": GATE_MERGE_ALL}
ROUTE_MODES = {"bucket": ROUTE_BUCKET, "full_cosine": ROUTE_FULL_COSINE, "bucket_nearest": ROUTE_BUCKET_NEAREST,
               "coattn": ROUTE_COATTN}
SELECT_MODES = {"per_head": SELECT_PER_HEAD, "union": SELECT_UNION}


class SelkvError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)}")


class Params(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_uint32),
        ("batch", ctypes.c_int32),
        ("n_heads_kv", ctypes.c_int32),
        ("group", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("seq_len", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("pool_kernel", ctypes.c_int32),
        ("recent", ctypes.c_int32),
        ("bucket", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("gate_mode", ctypes.c_int32),
        ("route_mode", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("alpha", ctypes.c_float),
        ("gate_threshold", ctypes.c_float),
        ("gate_temperature", ctypes.c_float),
        ("budget_ratio", ctypes.c_double),
        ("select_mode", ctypes.c_int32),
        ("merge_keys", ctypes.c_int32),
    ]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2607_16213_amd.build.build() first")
    lib = ctypes.CDLL(LIB_PATH)
    vp, sz, i32, fp, ip = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p
    P = ctypes.POINTER(Params)
    sigs = {
        "selkv_params_init": (None, [P]),
        "selkv_budget": (ctypes.c_int, [P, ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(i32)]),
        "selkv_workspace_size": (ctypes.c_int, [P, i32, i32, ctypes.POINTER(sz)]),
        "selkv_score": (ctypes.c_int, [P, vp, vp, vp, fp, fp, fp, vp, sz, vp]),
        "selkv_select": (ctypes.c_int, [P, fp, ip, ip, vp, sz, vp]),
        "selkv_route_coattn": (ctypes.c_int, [P, vp, vp, ip, ip, ip, vp, sz, vp]),
        "selkv_merge": (ctypes.c_int, [P, vp, vp, fp, fp, ip, ip, vp, vp, ip, fp, vp, sz, vp]),
        "selkv_bias": (ctypes.c_int, [P, fp, ip, ip, ip, fp, fp, vp, sz, vp]),
        "selkv_merge_bias": (ctypes.c_int, [P, vp, vp, fp, fp, ip, ip, vp, vp, ip, fp, fp, vp, sz, vp]),
        "selkv_decode_attn": (ctypes.c_int, [P, vp, vp, vp, fp, i32, fp, vp, sz, vp]),
        "selkv_decode_attn_noalloc": (ctypes.c_int, [P, vp, vp, vp, fp, i32, fp, vp]),
        "selkv_rope_reposition": (ctypes.c_int, [P, ip, vp, ctypes.c_double, vp]),
        "selkv_decode_append": (ctypes.c_int, [P, vp, vp, vp, vp, vp, fp, i32, i32, fp, vp, sz, vp]),
        "selkv_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "selkv_abi_version": (ctypes.c_int32, []),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


lib = _load()
if lib.selkv_abi_version() != ABI_VERSION:
    raise ImportError(f"{LIB_PATH} has ABI version {lib.selkv_abi_version()}, this binding expects {ABI_VERSION}")


def params(**kw) -> Params:
    """selkv_params with the paper's defaults, overridden by keyword."""
    p = Params()
    lib.selkv_params_init(ctypes.byref(p))
    for k, v in kw.items():
        if k == "gate_mode" and isinstance(v, str):
            v = GATE_MODES[v]
        if k == "route_mode" and isinstance(v, str):
            v = ROUTE_MODES[v]
        if k == "select_mode" and isinstance(v, str):
            v = SELECT_MODES[v]
        if k == "kv_dtype" and isinstance(v, (str, torch.dtype)):
            v = BF16 if v in ("bf16", torch.bfloat16) else F32
        if not hasattr(p, k):
            raise AttributeError(k)
        setattr(p, k, v)
    return p


def _check(status: int, where: str):
    if status != 0:
        raise SelkvError(status, where)


def budget(p: Params):
    m, mr, ms = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check(lib.selkv_budget(ctypes.byref(p), ctypes.byref(m), ctypes.byref(mr), ctypes.byref(ms)), "selkv_budget")
    return m.value, mr.value, ms.value


def workspace_bytes(p: Params, call: int, cache_len: int = 0) -> int:
    b = ctypes.c_size_t()
    _check(lib.selkv_workspace_size(ctypes.byref(p), call, cache_len, ctypes.byref(b)), "selkv_workspace_size")
    return b.value


def workspace(p: Params, call: int, device, cache_len: int = 0) -> torch.Tensor:
    """Scratch for `call` (zero-filled for tidiness; no call needs it initialised)."""
    nbytes = workspace_bytes(p, call, cache_len)
    return torch.zeros(max(nbytes, 1), dtype=torch.uint8, device=device)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, shape, dtype, name):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _nbytes(ws):
    """Size in bytes of a workspace tensor (any dtype), 0 for none."""
    if ws is None:
        return 0
    if not ws.is_cuda or not ws.is_contiguous():
        raise ValueError("workspace must be a contiguous device tensor")
    return ws.numel() * ws.element_size()


def _kvdt(p: Params):
    return torch.bfloat16 if p.kv_dtype == BF16 else torch.float32


def score(p, K, V, Qwin, score_out, attn, vnorm, ws, stream=None):
    B, H, n, d = p.batch, p.n_heads_kv, p.seq_len, p.head_dim
    m, mr, ms = budget(p)
    dt = _kvdt(p)
    _dev(K, (B, H, n, d), dt, "K"); _dev(V, (B, H, n, d), dt, "V")
    _dev(Qwin, (B, H * p.group, p.window, d), dt, "Qwin")
    _dev(score_out, (B, H, n - mr), torch.float32, "score")
    _dev(attn, (B, H, n), torch.float32, "attn"); _dev(vnorm, (B, H, n), torch.float32, "vnorm")
    _check(lib.selkv_score(ctypes.byref(p), _ptr(K), _ptr(V), _ptr(Qwin), _ptr(score_out), _ptr(attn), _ptr(vnorm),
                           _ptr(ws), _nbytes(ws), _stream(stream)), "selkv_score")


def select(p, score_in, kept, evicted, ws=None, stream=None):
    B, H, n = p.batch, p.n_heads_kv, p.seq_len
    m, mr, ms = budget(p)
    _dev(score_in, (B, H, n - mr), torch.float32, "score")
    _dev(kept, (B, H, m), torch.int32, "kept_idx")
    _dev(evicted, (B, H, n - m), torch.int32, "evicted_idx")
    _check(lib.selkv_select(ctypes.byref(p), _ptr(score_in), _ptr(kept), _ptr(evicted), _ptr(ws),
                            _nbytes(ws), _stream(stream)), "selkv_select")


def route_coattn(p, K, Qwin, kept, evicted, target, ws, stream=None):
    """Co-attention routing (route_mode COATTN): target slots for selkv_merge / selkv_bias."""
    B, H, n, d = p.batch, p.n_heads_kv, p.seq_len, p.head_dim
    m, mr, ms = budget(p)
    dt = _kvdt(p)
    _dev(K, (B, H, n, d), dt, "K"); _dev(Qwin, (B, H * p.group, p.window, d), dt, "Qwin")
    _dev(kept, (B, H, m), torch.int32, "kept_idx"); _dev(evicted, (B, H, n - m), torch.int32, "evicted_idx")
    _dev(target, (B, H, n - m), torch.int32, "target")
    _check(lib.selkv_route_coattn(ctypes.byref(p), _ptr(K), _ptr(Qwin), _ptr(kept), _ptr(evicted), _ptr(target),
                                  _ptr(ws), _nbytes(ws), _stream(stream)),
           "selkv_route_coattn")


def merge(p, K, V, attn, vnorm, kept, evicted, K_out, V_out, target, gate, ws, stream=None):
    B, H, n, d = p.batch, p.n_heads_kv, p.seq_len, p.head_dim
    m, mr, ms = budget(p)
    dt = _kvdt(p)
    _dev(K, (B, H, n, d), dt, "K"); _dev(V, (B, H, n, d), dt, "V")
    _dev(attn, (B, H, n), torch.float32, "attn"); _dev(vnorm, (B, H, n), torch.float32, "vnorm")
    _dev(kept, (B, H, m), torch.int32, "kept_idx"); _dev(evicted, (B, H, n - m), torch.int32, "evicted_idx")
    _dev(K_out, (B, H, m, d), dt, "K_out"); _dev(V_out, (B, H, m, d), dt, "V_out")
    _dev(target, (B, H, n - m), torch.int32, "target"); _dev(gate, (B, H, n - m), torch.float32, "gate")
    _check(lib.selkv_merge(ctypes.byref(p), _ptr(K), _ptr(V), _ptr(attn), _ptr(vnorm), _ptr(kept), _ptr(evicted),
                           _ptr(K_out), _ptr(V_out), _ptr(target), _ptr(gate), _ptr(ws),
                           _nbytes(ws), _stream(stream)), "selkv_merge")


def merge_bias(p, K, V, attn, vnorm, kept, evicted, K_out, V_out, target, gate, bias_out, ws, stream=None):
    """selkv_merge and selkv_bias in one pass (the bias from the merge's own sums)."""
    B, H, n, d = p.batch, p.n_heads_kv, p.seq_len, p.head_dim
    m, mr, ms = budget(p)
    dt = _kvdt(p)
    _dev(K, (B, H, n, d), dt, "K"); _dev(V, (B, H, n, d), dt, "V")
    _dev(attn, (B, H, n), torch.float32, "attn"); _dev(vnorm, (B, H, n), torch.float32, "vnorm")
    _dev(kept, (B, H, m), torch.int32, "kept_idx"); _dev(evicted, (B, H, n - m), torch.int32, "evicted_idx")
    _dev(K_out, (B, H, m, d), dt, "K_out"); _dev(V_out, (B, H, m, d), dt, "V_out")
    _dev(target, (B, H, n - m), torch.int32, "target"); _dev(gate, (B, H, n - m), torch.float32, "gate")
    _dev(bias_out, (B, H, m), torch.float32, "bias")
    _check(lib.selkv_merge_bias(ctypes.byref(p), _ptr(K), _ptr(V), _ptr(attn), _ptr(vnorm), _ptr(kept),
                                _ptr(evicted), _ptr(K_out), _ptr(V_out), _ptr(target), _ptr(gate), _ptr(bias_out),
                                _ptr(ws), _nbytes(ws), _stream(stream)), "selkv_merge_bias")


def bias(p, attn, kept, evicted, target, gate, bias_out, ws, stream=None):
    B, H, n = p.batch, p.n_heads_kv, p.seq_len
    m, mr, ms = budget(p)
    _dev(attn, (B, H, n), torch.float32, "attn")
    _dev(kept, (B, H, m), torch.int32, "kept_idx"); _dev(evicted, (B, H, n - m), torch.int32, "evicted_idx")
    _dev(target, (B, H, n - m), torch.int32, "target"); _dev(gate, (B, H, n - m), torch.float32, "gate")
    _dev(bias_out, (B, H, m), torch.float32, "bias")
    _check(lib.selkv_bias(ctypes.byref(p), _ptr(attn), _ptr(kept), _ptr(evicted), _ptr(target), _ptr(gate),
                          _ptr(bias_out), _ptr(ws), _nbytes(ws), _stream(stream)),
           "selkv_bias")


def rope_reposition(p, kept, K_out, rope_theta, stream=None):
    B, H, d = p.batch, p.n_heads_kv, p.head_dim
    m, mr, ms = budget(p)
    _dev(kept, (B, H, m), torch.int32, "kept_idx")
    _dev(K_out, (B, H, m, d), _kvdt(p), "K_out")
    _check(lib.selkv_rope_reposition(ctypes.byref(p), _ptr(kept), _ptr(K_out), float(rope_theta), _stream(stream)),
           "selkv_rope_reposition")


def decode_attn(p, q, K, V, bias_in, out, ws, stream=None):
    B, H, d = p.batch, p.n_heads_kv, p.head_dim
    L = K.shape[2]
    dt = _kvdt(p)
    _dev(q, (B, H * p.group, d), dt, "q")
    _dev(K, (B, H, L, d), dt, "K"); _dev(V, (B, H, L, d), dt, "V")
    if bias_in is not None:
        _dev(bias_in, (B, H, L), torch.float32, "bias")
    _dev(out, (B, H * p.group, d), torch.float32, "out")
    _check(lib.selkv_decode_attn(ctypes.byref(p), _ptr(q), _ptr(K), _ptr(V), _ptr(bias_in), L, _ptr(out), _ptr(ws),
                                 _nbytes(ws), _stream(stream)), "selkv_decode_attn")


def decode_attn_noalloc(p, q, K, V, bias_in, out, stream=None):
    """selkv_decode_attn with the library's fixed per-GPU scratch instead of a
    workspace (nothing is allocated; calls overlapping on one GPU race)."""
    B, H, d = p.batch, p.n_heads_kv, p.head_dim
    L = K.shape[2]
    dt = _kvdt(p)
    _dev(q, (B, H * p.group, d), dt, "q")
    _dev(K, (B, H, L, d), dt, "K"); _dev(V, (B, H, L, d), dt, "V")
    if bias_in is not None:
        _dev(bias_in, (B, H, L), torch.float32, "bias")
    _dev(out, (B, H * p.group, d), torch.float32, "out")
    _check(lib.selkv_decode_attn_noalloc(ctypes.byref(p), _ptr(q), _ptr(K), _ptr(V), _ptr(bias_in), L, _ptr(out),
                                         _stream(stream)), "selkv_decode_attn_noalloc")


def decode_append(p, q, k_new, v_new, K, V, bias_io, cache_len, out, ws, stream=None):
    """Append (k_new, v_new) at entry cache_len (bias 0 there) and attend over
    cache_len + 1 entries; K, V [B, H, capacity, d] and bias [B, H, capacity]."""
    B, H, d = p.batch, p.n_heads_kv, p.head_dim
    cap = K.shape[2]
    dt = _kvdt(p)
    _dev(q, (B, H * p.group, d), dt, "q")
    _dev(k_new, (B, H, d), dt, "k_new"); _dev(v_new, (B, H, d), dt, "v_new")
    _dev(K, (B, H, cap, d), dt, "K"); _dev(V, (B, H, cap, d), dt, "V")
    if bias_io is not None:
        _dev(bias_io, (B, H, cap), torch.float32, "bias")
    _dev(out, (B, H * p.group, d), torch.float32, "out")
    _check(lib.selkv_decode_append(ctypes.byref(p), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(K), _ptr(V),
                                   _ptr(bias_io), int(cache_len), cap, _ptr(out), _ptr(ws),
                                   _nbytes(ws), _stream(stream)), "selkv_decode_append")


class Compressor:
    """Owns the output and scratch tensors of one problem size and runs the
    compression calls (score, select, [route_coattn,] merge_bias, or merge then
    bias with fused=False) on the current stream.  Allocation happens once, in
    the constructor."""

    def __init__(self, p: Params, device):
        self.p = p
        B, H, n, d = p.batch, p.n_heads_kv, p.seq_len, p.head_dim
        self.m, self.mr, self.ms = budget(p)
        m, mr = self.m, self.mr
        dt = _kvdt(p)
        f32, i32 = torch.float32, torch.int32
        self.score = torch.empty((B, H, n - mr), dtype=f32, device=device)
        self.attn = torch.empty((B, H, n), dtype=f32, device=device)
        self.vnorm = torch.empty((B, H, n), dtype=f32, device=device)
        self.kept = torch.empty((B, H, m), dtype=i32, device=device)
        self.evicted = torch.empty((B, H, n - m), dtype=i32, device=device)
        self.K_out = torch.empty((B, H, m, d), dtype=dt, device=device)
        self.V_out = torch.empty((B, H, m, d), dtype=dt, device=device)
        self.target = torch.empty((B, H, n - m), dtype=i32, device=device)
        self.gate = torch.empty((B, H, n - m), dtype=f32, device=device)
        self.bias = torch.empty((B, H, m), dtype=f32, device=device)
        self.ws_score = workspace(p, CALL_SCORE, device)
        self.ws_select = workspace(p, CALL_SELECT, device)
        self.ws_merge = workspace(p, CALL_MERGE_BIAS, device)   # covers merge and bias alone too
        self.ws_route = workspace(p, CALL_ROUTE, device) if p.route_mode == ROUTE_COATTN else None

    def run(self, K, V, Qwin, stream=None, fused=True):
        p = self.p
        score(p, K, V, Qwin, self.score, self.attn, self.vnorm, self.ws_score, stream)
        select(p, self.score, self.kept, self.evicted, self.ws_select, stream)
        if p.route_mode == ROUTE_COATTN:
            route_coattn(p, K, Qwin, self.kept, self.evicted, self.target, self.ws_route, stream)
        if fused:
            merge_bias(p, K, V, self.attn, self.vnorm, self.kept, self.evicted, self.K_out, self.V_out, self.target,
                       self.gate, self.bias, self.ws_merge, stream)
        else:
            merge(p, K, V, self.attn, self.vnorm, self.kept, self.evicted, self.K_out, self.V_out, self.target,
                  self.gate, self.ws_merge, stream)
            bias(p, self.attn, self.kept, self.evicted, self.target, self.gate, self.bias, self.ws_merge, stream)
        return self

    def outputs(self):
        return dict(score=self.score, attn=self.attn, vnorm=self.vnorm, kept=self.kept, evicted=self.evicted,
                    K_out=self.K_out, V_out=self.V_out, target=self.target, gate=self.gate, bias=self.bias)


class Decoder:
    """Owns the split-K workspace for decode over caches of `cache_len` entries."""

    def __init__(self, p: Params, cache_len: int, device):
        self.p = p
        self.cache_len = cache_len
        self.ws = workspace(p, CALL_DECODE, device, cache_len)
        self.out = torch.empty((p.batch, p.n_heads_kv * p.group, p.head_dim), dtype=torch.float32, device=device)

    def run(self, q, K, V, bias_in=None, out=None, stream=None):
        o = self.out if out is None else out
        decode_attn(self.p, q, K, V, bias_in, o, self.ws, stream)
        return o
