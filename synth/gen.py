"""Seeded synthetic Q/K/V shaped like a Llama-3.1-8B attention layer at long context.

The paper measures on real prompts through Llama 3.1-8B-Instruct (Sec. 4.1); those
weights and datasets are not available, so these generators stand in for the shape of
that workload: grouped-query attention with 32 query and 8 key/value heads, head dim
128, rotary position encoding with base 500000, and contexts up to 128K tokens.  The
structure the sparse patterns exploit (attention sinks, vertical key columns, a local
band, dispersed evidence spans) is planted explicitly so that each pattern family has
something to find.

Recipe (all draws from numpy PCG64, ``seed = 1000 * config + layer``):

* base: Q, K, V ~ N(0, 1), float32, one independent stream per head
  (``[seed, 1, h]`` for query head h, ``[seed, 2, g]`` / ``[seed, 3, g]`` for K / V of
  key/value head g), so any subset of heads can be regenerated on its own;
* local bias (before RoPE): a fixed unit vector ``c`` spread evenly over the rotary pairs
  whose frequency lies in [1e-3, 1e-1] is added as ``sqrt(lam*sqrt(d)) * c`` to every
  query and key, which after RoPE adds ``lam * mean_f cos(theta_f (i-j))`` to logit i,j;
* RoPE, rotate-half convention: pair f = dims (f, f + d/2), theta_f = 500000^(-2f/d),
  position = token index (no long-context frequency rescaling);
* planted "+k sigma" boosts (after RoPE): direction u (orthonormal set drawn from the
  structure stream ``[seed, 7]``, orthogonal to the rotary pairs of the local-band
  vector), ``sqrt(k*sqrt(d)) * u`` added to the chosen keys and to the chosen queries, so
  the logit rises by k background standard deviations;
* cast: round-to-nearest-even to bf16 (configs 2-5); config 1 stays float32.

Config 5 draws a regime per key/value group (local 0.35, sink 0.30, vertical 0.28,
diffuse 0.07) with context-scaled strengths so that the structured regimes hold about
98% of the softmax mass at 128K: local band lam = 17; sinks (4 keys) and 64 vertical
columns at k = ln(1.65 n / count) + 4; sink and vertical heads also carry the local band;
diffuse heads get no plants.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

ROPE_BASE = 500000.0

# Five workloads: a single-head fp32 case, then GQA 32/8 d=128 bf16 layers of growing length.
CONFIGS = {
    1: dict(n=2048, hq=1, hkv=1, d=64, dtype="f32", layers=1),
    2: dict(n=8192, hq=32, hkv=8, d=128, dtype="bf16", layers=1),
    3: dict(n=32768, hq=32, hkv=8, d=128, dtype="bf16", layers=1),
    4: dict(n=131072, hq=32, hkv=8, d=128, dtype="bf16", layers=1),
    5: dict(n=131072, hq=32, hkv=8, d=128, dtype="bf16", layers=32),
}

REGIMES = ("local", "sink", "vertical", "diffuse")
REGIME_P = (0.35, 0.30, 0.28, 0.07)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return the 16-bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    u = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (u >> np.uint32(16)).astype(np.uint16)


def bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 values rounded to the nearest bf16 value, still stored as float32."""
    return bits_to_f32(bf16_bits(x))


@dataclass
class GroupPlants:
    """Planted structure of one key/value head group (shared by its query heads)."""
    regime: str
    sink_k: float = 0.0          # logit boost of keys [0, sink_n), in background std units
    sink_n: int = 4
    vert_k: float = 0.0          # logit boost of the vertical key columns
    vert_cols: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))
    local_lam: float = 0.0       # peak local-band logit bias


@dataclass
class LayerSpec:
    cfg: int
    layer: int
    seed: int
    n: int
    hq: int
    hkv: int
    d: int
    dtype: str
    groups: list
    dirs: np.ndarray             # [16, d] orthonormal planted directions
    span_starts: np.ndarray      # [n_spans] evidence span starts (config 4)
    span_len: int
    span_k: float
    chunk_span: np.ndarray       # [n // 1024] span id each 1024-row query chunk follows, -1 none

    @property
    def group_size(self) -> int:
        return self.hq // self.hkv


def _plant_amp(k: float, d: int) -> float:
    return math.sqrt(k * math.sqrt(d))


def layer_spec(cfg: int, layer: int = 0, n: int | None = None) -> LayerSpec:
    """Structure of one layer: everything but the Gaussian background (cheap)."""
    c = CONFIGS[cfg]
    n = int(c["n"] if n is None else n)
    hq, hkv, d = c["hq"], c["hkv"], c["d"]
    seed = 1000 * cfg + layer
    rs = np.random.default_rng([seed, 7])
    g = rs.standard_normal((d, 16))
    # planted directions live outside the rotary pairs that carry the local-band vector, so
    # that u . R_j c = 0 for every position j (no position-dependent cross terms)
    theta = ROPE_BASE ** (-2.0 * np.arange(d // 2, dtype=np.float64) / d)
    band = np.nonzero((theta >= 1e-3) & (theta <= 1e-1))[0]
    g[band] = 0.0
    g[band + d // 2] = 0.0
    qmat, _ = np.linalg.qr(g)
    dirs = qmat.T.astype(np.float64)          # rows orthonormal
    groups = []
    for _g in range(hkv):
        if cfg == 5:
            regime = REGIMES[int(rs.choice(4, p=REGIME_P))]
        else:
            regime = "mixed"
        if regime == "mixed":
            nv = 16
            cols = np.sort(rs.choice(np.arange(4, n), size=min(nv, max(n - 4, 0)), replace=False))
            lam = 0.0 if cfg == 1 else 4.0
            groups.append(GroupPlants(regime, sink_k=4.0, vert_k=3.0, vert_cols=cols, local_lam=lam))
        elif regime == "sink":       # attention sinks plus a local band (A-shape-like head)
            k = math.log(1.65 * n / 4) + 4.0
            groups.append(GroupPlants(regime, sink_k=k, local_lam=17.0))
        elif regime == "vertical":   # vertical key columns plus a local band (vertical-slash head)
            nv = 64
            cols = np.sort(rs.choice(np.arange(4, n), size=min(nv, max(n - 4, 0)), replace=False))
            k = math.log(1.65 * n / nv) + 4.0
            groups.append(GroupPlants(regime, vert_k=k, vert_cols=cols, local_lam=17.0))
        elif regime == "local":
            groups.append(GroupPlants(regime, local_lam=17.0))
        else:
            groups.append(GroupPlants(regime))
    span_len = 512
    if cfg == 4:
        n_spans = 8
        eighth = n // n_spans
        starts = np.array([k * eighth + int(rs.integers(0, max(eighth - span_len, 1)))
                           for k in range(n_spans)], dtype=np.int64)
        nchunk = (n + 1023) // 1024
        chunk_span = np.full(nchunk, -1, dtype=np.int64)
        for ch in range(nchunk):
            elig = np.nonzero(starts < ch * 1024)[0]
            if elig.size:
                chunk_span[ch] = int(elig[int(rs.integers(0, elig.size))])
    else:
        starts = np.zeros(0, dtype=np.int64)
        chunk_span = np.full((n + 1023) // 1024, -1, dtype=np.int64)
    return LayerSpec(cfg, layer, seed, n, hq, hkv, d, c["dtype"], groups, dirs, starts,
                     span_len, 3.0, chunk_span)


_TABLES = {}


def _rope_tables(n: int, d: int, device="cpu"):
    import torch
    key = (n, d, str(device))
    if key not in _TABLES:
        half = d // 2
        theta = ROPE_BASE ** (-2.0 * np.arange(half, dtype=np.float64) / d)
        ang = np.arange(n, dtype=np.float64)[:, None] * theta[None, :]
        _TABLES.clear()
        _TABLES[key] = (torch.from_numpy(np.cos(ang).astype(np.float32)).to(device),
                        torch.from_numpy(np.sin(ang).astype(np.float32)).to(device), theta)
    return _TABLES[key]


def _local_vec(d: int, theta: np.ndarray) -> np.ndarray:
    half = d // 2
    band = np.nonzero((theta >= 1e-3) & (theta <= 1e-1))[0]
    c = np.zeros(d, dtype=np.float64)
    c[band] = 1.0
    c[band + half] = 1.0
    return (c / np.linalg.norm(c)).astype(np.float32)


def _rope(x, cos, sin):
    """Rotate-half RoPE on a [n, d] float32 torch tensor (elementwise float32 ops)."""
    import torch
    half = x.shape[1] // 2
    x1, x2 = x[:, :half], x[:, half:]
    out = torch.empty_like(x)
    out[:, :half] = x1 * cos - x2 * sin
    out[:, half:] = x2 * cos + x1 * sin
    return out


_DEV = ["cpu"]


def _vec(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(_DEV[0])


def _finish(x, dtype: str):
    """bf16 configs: round to nearest even and return the bf16 tensor; else float32."""
    import torch
    return x.to(torch.bfloat16) if dtype == "bf16" else x.contiguous()


def _normals(seed_key, n, d):
    return np.random.default_rng(seed_key).standard_normal((n, d), dtype=np.float32)


def _gen_q(spec: LayerSpec, h: int, tabs, base):
    import torch
    cos, sin, theta = tabs
    d = spec.d
    gp = spec.groups[h // spec.group_size]
    x = torch.from_numpy(base).to(_DEV[0])
    if gp.local_lam > 0:
        x += _vec(_plant_amp(gp.local_lam, d) * _local_vec(d, theta))[None, :]
    x = _rope(x, cos, sin)
    if gp.sink_k > 0:
        x += _vec(_plant_amp(gp.sink_k, d) * spec.dirs[0])[None, :]
    if gp.vert_k > 0 and gp.vert_cols.size:
        x += _vec(_plant_amp(gp.vert_k, d) * spec.dirs[1])[None, :]
    if spec.span_starts.size:
        amp = _plant_amp(spec.span_k, d)
        for ch, sid in enumerate(spec.chunk_span):
            if sid >= 0:
                x[ch * 1024:(ch + 1) * 1024] += _vec(amp * spec.dirs[2 + sid])
    return _finish(x, spec.dtype)


def _gen_k(spec: LayerSpec, g: int, tabs, base):
    cos, sin, theta = tabs
    d = spec.d
    gp = spec.groups[g]
    import torch
    x = torch.from_numpy(base).to(_DEV[0])
    if gp.local_lam > 0:
        x += _vec(_plant_amp(gp.local_lam, d) * _local_vec(d, theta))[None, :]
    x = _rope(x, cos, sin)
    if gp.sink_k > 0:
        x[:gp.sink_n] += _vec(_plant_amp(gp.sink_k, d) * spec.dirs[0])
    if gp.vert_k > 0 and gp.vert_cols.size:
        x[torch.from_numpy(gp.vert_cols).to(_DEV[0])] += _vec(_plant_amp(gp.vert_k, d) * spec.dirs[1])
    if spec.span_starts.size:
        amp = _plant_amp(spec.span_k, d)
        for sid, st in enumerate(spec.span_starts):
            x[st:st + spec.span_len] += _vec(amp * spec.dirs[2 + sid])
    return _finish(x, spec.dtype)


def _gen_v(spec: LayerSpec, g: int, base):
    import torch
    return _finish(torch.from_numpy(base).to(_DEV[0]), spec.dtype)


def make_layer_torch(cfg: int, layer: int = 0, n: int | None = None, q_heads=None, kv_heads=None,
                     threads: int | None = None, device="cpu") -> dict:
    """Like make_layer, but returns torch tensors on ``device`` (bf16 for bf16 configs):
    q [hq, n, d], k, v [hkv, n, d].  Heads not requested are zero.  The Gaussian background
    is always drawn on the host (PCG64); the elementwise float32 transforms (bias, RoPE,
    plants, rounding) are single IEEE operations, so every device gives the same bits."""
    import torch
    spec = layer_spec(cfg, layer, n)
    n, d = spec.n, spec.d
    q_heads = list(range(spec.hq)) if q_heads is None else list(q_heads)
    kv_heads = list(range(spec.hkv)) if kv_heads is None else list(kv_heads)
    _DEV[0] = device
    tabs = _rope_tables(n, d, device)
    tdt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
    q = torch.zeros((spec.hq, n, d), dtype=tdt, device=device)
    k = torch.zeros((spec.hkv, n, d), dtype=tdt, device=device)
    v = torch.zeros((spec.hkv, n, d), dtype=tdt, device=device)
    items = [(0, h) for h in q_heads] + [(1, g) for g in kv_heads] + [(2, g) for g in kv_heads]
    keys = {0: 1, 1: 2, 2: 3}
    nthreads = threads or min(16, os.cpu_count() or 1)
    # Gaussian background: one PCG64 stream per head, drawn in parallel threads
    with ThreadPoolExecutor(nthreads) as ex:
        bases = list(ex.map(lambda it: _normals([spec.seed, keys[it[0]], it[1]], n, d), items))
    for (kind, h), base in zip(items, bases):
        if kind == 0:
            q[h] = _gen_q(spec, h, tabs, base)
        elif kind == 1:
            k[h] = _gen_k(spec, h, tabs, base)
        else:
            v[h] = _gen_v(spec, h, base)
    return dict(q=q, k=k, v=v, spec=spec)


def make_layer(cfg: int, layer: int = 0, n: int | None = None, q_heads=None, kv_heads=None,
               threads: int | None = None) -> dict:
    """Generate Q [hq, n, d], K, V [hkv, n, d] as float32 numpy arrays (bf16-exact for bf16
    configs).  ``q_heads`` / ``kv_heads`` restrict generation to a subset of heads; the other
    heads are zeros.  Values of a generated head do not depend on the subset chosen."""
    t = make_layer_torch(cfg, layer, n, q_heads, kv_heads, threads)
    return dict(q=t["q"].float().numpy(), k=t["k"].float().numpy(), v=t["v"].float().numpy(),
                spec=t["spec"])
