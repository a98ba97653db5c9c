"""Seeded synthetic KV caches with the shapes of the paper's workloads.

This module only draws random tensors.  It holds none of SelKV's arithmetic,
and both the GPU path and the float64 reference read the very same stored
tensors that it returns.

The paper evaluates LLaMA-3.1-8B (32 query / 8 KV heads, d = 128) prompts up
to 100k tokens and an MHA model (32 / 32 heads) at 25% retention (Sec. 4.1,
Sec. 4.4).  Its data (LongBench prompts run through trained weights) is not
available, so seeded generators with those shapes stand in for it:

``scaled``  keys and window queries ~ N(0, 1)/sqrt(d) per coordinate.
``heavy``   keys ~ N(0, 1); every KV head has a unit direction u; queries are
            z + u with z ~ N(0, I); a fraction of key positions (the heavy
            hitters) gets 4*sqrt(d)*u added, raising their mean logit by ~4.
Values      a few unit-norm cluster centres per KV head plus Gaussian noise
            of per-coordinate std sigma/sqrt(d) (so the noise norm is ~sigma).
Duplicates  a fraction of positions are exact (k, v) copies of a uniformly
            chosen earlier position in the same 32-token bucket, so exact
            attention ties and unit cosines occur.

Tensors are drawn in float32 with a ``torch.Generator`` seeded from
(workload, layer, tag) and then rounded to the storage dtype (bf16 by
round-to-nearest-even).  Layouts: K, V [B, H_kv, n, d]; window queries
[B, H_q, W, d]; decode queries [steps, B, H_q, d].
"""
from __future__ import annotations

import dataclasses
import hashlib
import math

import torch

TAG_K, TAG_V, TAG_QWIN, TAG_QDEC, TAG_STRUCT = 1, 2, 3, 4, 5


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int                 # independent sequences
    layers: int
    n_heads_kv: int
    group: int                 # query heads per KV head
    head_dim: int
    seq_len: int
    window: int
    budgets: tuple             # retention ratios rho
    dtype: str                 # "fp32" | "bf16"
    key_gen: str               # "scaled" | "heavy"
    value_clusters: int
    value_noise: float         # sigma: per-coordinate noise std is sigma/sqrt(d)
    dup_fraction: float
    heavy_fraction: float
    decode_steps: int
    gate_sweep: tuple = ((0.0, 1.0),)   # (threshold tau, temperature T) pairs
    decode_cache_full: bool = False      # also time decode over the full n-entry cache

    @property
    def n_heads_q(self) -> int:
        return self.n_heads_kv * self.group

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "fp32" else torch.bfloat16

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # 1 layer, 4 query / 2 KV heads, d = 64, n = 512, W = 32, 25% budget, fp32
    "tiny": Workload("tiny", 1, 1, 2, 2, 64, 512, 32, (0.25,), "fp32", "scaled",
                     16, 0.3, 0.10, 0.0, 16),
    # one Llama-3-8B-shaped layer, bf16: 32 query / 8 KV heads, d = 128, n = 8192
    "llama_layer": Workload("llama_layer", 1, 1, 8, 4, 128, 8192, 32, (0.25,), "bf16", "heavy",
                            256, 0.5, 0.0, 0.02, 128),
    # the full 32-layer cache at 32k tokens, batch 1, bf16
    "ctx32k": Workload("ctx32k", 1, 32, 8, 4, 128, 32768, 32, (0.25,), "bf16", "scaled",
                       16, 0.3, 0.10, 0.0, 256),
    # the paper's long-context speed point: 32 layers at 102400 tokens
    "ctx100k": Workload("ctx100k", 1, 32, 8, 4, 128, 102400, 32, (0.25,), "bf16", "scaled",
                        16, 0.3, 0.10, 0.0, 512, decode_cache_full=True),
    # MHA shape, batch 4, W = 64, budget and gate sweep
    "mha_sweep": Workload("mha_sweep", 4, 1, 32, 1, 128, 16384, 64, (0.10, 0.25, 0.50), "bf16",
                          "heavy", 256, 0.5, 0.0, 0.02, 128,
                          gate_sweep=tuple((tau, T) for tau in (0.0, 0.2, 0.4) for T in (0.25, 0.5, 1.0))),
}


def seed_for(workload: str, layer: int, tag: int, extra: int = 0) -> int:
    """A 63-bit seed derived from (workload name, layer, tag, extra)."""
    h = hashlib.sha256(f"selkv|{workload}|{layer}|{tag}|{extra}".encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _normal(shape, seed, device):
    return torch.randn(shape, generator=_gen(device, seed), device=device, dtype=torch.float32)


def _unit_rows(x: torch.Tensor) -> torch.Tensor:
    return x / x.norm(dim=-1, keepdim=True)


def _duplicate_sources(n: int, frac: float, bucket: int, lead: int, seed: int, device) -> torch.Tensor:
    """For every (leading index, position) the position whose (k, v) it copies
    (itself when it is not a duplicate).  Duplicates copy a uniformly chosen
    earlier position of the same bucket; chains resolve to their first source."""
    g = _gen(device, seed)
    pos = torch.arange(n, device=device).expand(lead, n)
    offset = pos % bucket
    pick = torch.rand((lead, n), generator=g, device=device) < frac
    pick &= offset > 0
    u = torch.rand((lead, n), generator=g, device=device)
    src_off = torch.clamp((u * offset.to(torch.float32)).floor().to(torch.int64), max=bucket - 1)
    src = torch.where(pick, pos - offset + torch.minimum(src_off, offset - 1), pos)
    for _ in range(bucket):                       # resolve copy chains
        nxt = torch.gather(src, 1, src)
        if torch.equal(nxt, src):
            break
        src = nxt
    return src


def make_layer(w: Workload, layer: int = 0, device="cpu", seq_len: int | None = None):
    """K, V [B, H_kv, n, d] and window queries [B, H_q, W, d] of one layer, in
    the workload's storage dtype, on `device`."""
    n = w.seq_len if seq_len is None else seq_len
    B, Hkv, G, d, W = w.batch, w.n_heads_kv, w.group, w.head_dim, w.window
    name = w.name
    if w.key_gen == "scaled":
        K = _normal((B, Hkv, n, d), seed_for(name, layer, TAG_K), device) / math.sqrt(d)
        Qw = _normal((B, Hkv * G, W, d), seed_for(name, layer, TAG_QWIN), device) / math.sqrt(d)
    elif w.key_gen == "heavy":
        u = _unit_rows(_normal((B, Hkv, d), seed_for(name, layer, TAG_STRUCT, 1), device))
        K = _normal((B, Hkv, n, d), seed_for(name, layer, TAG_K), device)
        hit = torch.rand((B, Hkv, n), generator=_gen(device, seed_for(name, layer, TAG_STRUCT, 2)),
                         device=device) < w.heavy_fraction
        K = K + hit[..., None].to(torch.float32) * (4.0 * math.sqrt(d)) * u[:, :, None, :]
        z = _normal((B, Hkv * G, W, d), seed_for(name, layer, TAG_QWIN), device)
        Qw = z + u.repeat_interleave(G, dim=1)[:, :, None, :]
    else:
        raise ValueError(w.key_gen)

    centres = _unit_rows(_normal((B, Hkv, w.value_clusters, d), seed_for(name, layer, TAG_STRUCT, 3), device))
    assign = torch.randint(0, w.value_clusters, (B, Hkv, n),
                           generator=_gen(device, seed_for(name, layer, TAG_STRUCT, 4)), device=device)
    V = torch.gather(centres, 2, assign[..., None].expand(B, Hkv, n, d))
    V = V + _normal((B, Hkv, n, d), seed_for(name, layer, TAG_V), device) * (w.value_noise / math.sqrt(d))

    if w.dup_fraction > 0:
        src = _duplicate_sources(n, w.dup_fraction, 32, B * Hkv, seed_for(name, layer, TAG_STRUCT, 5), device)
        src = src.view(B, Hkv, n, 1).expand(B, Hkv, n, d)
        K = torch.gather(K, 2, src)
        V = torch.gather(V, 2, src)

    dt = w.torch_dtype
    return dict(K=K.to(dt).contiguous(), V=V.to(dt).contiguous(), Qwin=Qw.to(dt).contiguous())


def make_decode_queries(w: Workload, layer: int = 0, steps: int | None = None, device="cpu"):
    """Decode queries [steps, B, H_q, d] (fresh draws per step, same family as
    the window queries: N(0, 1) per coordinate, plus u for `heavy`)."""
    steps = w.decode_steps if steps is None else steps
    B, Hkv, G, d = w.batch, w.n_heads_kv, w.group, w.head_dim
    q = _normal((steps, B, Hkv * G, d), seed_for(w.name, layer, TAG_QDEC), device)
    if w.key_gen == "heavy":
        u = _unit_rows(_normal((B, Hkv, d), seed_for(w.name, layer, TAG_STRUCT, 1), device))
        q = q + u.repeat_interleave(G, dim=1)[None]
    return q.to(w.torch_dtype).contiguous()


def random_case(seed: int, *, batch=1, n_heads_kv=2, group=2, head_dim=64, seq_len=100, window=8,
                dtype="fp32", dup_fraction=0.1, clusters=4, noise=0.3, device="cpu"):
    """A small free-form case for edge-case tests: scaled keys, clustered
    values with duplicates.  Returns K, V, Qwin like make_layer."""
    w = Workload(f"case{seed}", batch, 1, n_heads_kv, group, head_dim, seq_len, window, (0.25,), dtype,
                 "scaled", clusters, noise, dup_fraction, 0.0, 1)
    return make_layer(w, 0, device)
