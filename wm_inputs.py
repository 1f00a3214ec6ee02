"""Seeded synthetic KV caches shared by the tests and the benchmark.

This module only draws random numbers; it holds none of the mover's
arithmetic (no checksum, diff or codec).  Both the HIP library and the CPU
oracle consume the bytes it produces: GPU tests generate on the device and
hand a host copy to the oracle.

The paper's real cache (a warmed world-model attention cache of 1.67 GB,
420 bf16 tensors, about 75% of it rewritten per generation step; §3.1,
§3.3, §6.4) and its traces are not available, so these generators stand in
for it with the shapes and value distributions below.  A "channel" is one
(layer, K/V, head, head_dim index); the layout is [L, 2, H, T, D]
contiguous, so a 64 KiB chunk of the production cache holds 256 tokens x
128 dims of one (layer, K/V, head).
"""
from __future__ import annotations

import dataclasses

import torch

CHUNK = 65536


@dataclasses.dataclass(frozen=True)
class CacheSpec:
    name: str
    shape: tuple  # (L, 2, H, T, D)
    seed: int
    dist: str = "normal"  # "normal" (N(0,1) x per-channel scale) or "t3"
    channel_scale: bool = True  # LogNormal(0, 0.5) per channel
    outlier_frac: float = 0.0  # channels scaled x20
    outlier_seed: int = 2
    raw_frac: float = 0.0  # chunks overwritten with uniform 16-bit patterns
    raw_seed: int = 5

    @property
    def nbytes(self) -> int:
        n = 1
        for s in self.shape:
            n *= s
        return 2 * n


TINY = CacheSpec("tiny", (2, 2, 8, 512, 64), seed=0)
PRODUCTION = CacheSpec("production", (28, 2, 16, 7296, 128), seed=0,
                       outlier_frac=0.02)
FANIN = tuple(CacheSpec(f"fanin{s}", (24, 2, 8, 4096, 128), seed=100 + s)
              for s in range(8))
LONG = CacheSpec("long_context", (32, 2, 8, 32768, 128), seed=4, dist="t3",
                 channel_scale=False, raw_frac=0.10)


def _channel_scales(spec: CacheSpec, device) -> torch.Tensor:
    L, two, H, _, D = spec.shape
    n_ch = L * two * H * D
    g = torch.Generator(device=device).manual_seed(spec.seed)
    if spec.channel_scale:
        scale = torch.exp(0.5 * torch.randn(n_ch, generator=g, device=device))
    else:
        scale = torch.ones(n_ch, device=device)
    if spec.outlier_frac > 0:
        go = torch.Generator(device=device).manual_seed(spec.outlier_seed)
        k = round(spec.outlier_frac * n_ch)
        sel = torch.randperm(n_ch, generator=go, device=device)[:k]
        scale[sel] *= 20.0
    return scale.view(L, two, H, 1, D)


def _draw(shape, dist: str, g: torch.Generator, device) -> torch.Tensor:
    z = torch.randn(shape, generator=g, device=device)
    if dist == "t3":
        # Student-t with 3 degrees of freedom: z / sqrt(chi2_3 / 3)
        chi = torch.zeros(shape, device=device)
        for _ in range(3):
            chi += torch.randn(shape, generator=g, device=device) ** 2
        z = z / torch.sqrt(chi / 3.0)
    return z


def make_cache(spec: CacheSpec, device="cpu") -> torch.Tensor:
    """bf16 tensor of spec.shape, generated layer by layer from spec.seed."""
    L, two, H, T, D = spec.shape
    scale = _channel_scales(spec, device)
    g = torch.Generator(device=device).manual_seed(spec.seed + 1_000_003)
    out = torch.empty(spec.shape, dtype=torch.bfloat16, device=device)
    for l in range(L):
        z = _draw((two, H, T, D), spec.dist, g, device)
        out[l] = (z * scale[l]).to(torch.bfloat16)
    if spec.raw_frac > 0:
        flat = out.view(-1).view(torch.int16)
        n_chunks = spec.nbytes // CHUNK
        k = round(spec.raw_frac * n_chunks)
        gr = torch.Generator(device=device).manual_seed(spec.raw_seed)
        sel = torch.randperm(n_chunks, generator=gr, device=device)[:k]
        words = CHUNK // 2
        for s in torch.sort(sel).values.tolist():
            bits = torch.randint(0, 65536, (words,), generator=gr,
                                 device=device, dtype=torch.int32)
            flat[s * words:(s + 1) * words] = bits.to(torch.int16)
    return out


def chunk_scales(spec: CacheSpec, chunk_ids: torch.Tensor,
                 device="cpu") -> torch.Tensor:
    """Per-element channel scale of every element of the given chunks."""
    L, two, H, T, D = spec.shape
    scale = _channel_scales(spec, device).view(L * two * H, D)
    words = CHUNK // 2
    e = chunk_ids.to(device).view(-1, 1) * words + torch.arange(
        words, device=device).view(1, -1)
    return scale[e // (T * D), e % D]


def rewrite_chunks(state: torch.Tensor, spec: CacheSpec, chunk_ids: torch.Tensor,
                   seed: int) -> None:
    """In place: the listed 64 KiB chunks of state (ids may repeat) get fresh
    draws from the same per-channel distribution."""
    device = state.device
    flat = state.view(-1)
    words = CHUNK // 2
    ids = torch.unique(chunk_ids.to(device))
    g = torch.Generator(device=device).manual_seed(seed)
    step = 2048  # chunks per batch, bounds temporary memory
    for b in range(0, ids.numel(), step):
        part = ids[b:b + step]
        z = _draw((part.numel(), words), spec.dist, g, device)
        z = z * chunk_scales(spec, part, device)
        pos = (part.view(-1, 1) * words +
               torch.arange(words, device=device).view(1, -1)).view(-1)
        flat[pos] = z.view(-1).to(torch.bfloat16)


def regenerate(prev: torch.Tensor, spec: CacheSpec, chunk_ids: torch.Tensor,
               seed: int) -> torch.Tensor:
    """Copy of prev whose listed 64 KiB chunks hold fresh draws from the same
    per-channel distribution (the active-generation step)."""
    cur = prev.clone()
    rewrite_chunks(cur, spec, chunk_ids, seed)
    return cur


def chunk_writes(n_chunks: int, count: int, seed: int, device="cpu") -> torch.Tensor:
    """`count` chunk writes of a generating session, each to a chunk drawn
    uniformly with replacement (the occupancy model of pre-copy)."""
    g = torch.Generator(device=device).manual_seed(seed)
    return torch.randint(0, n_chunks, (count,), generator=g, device=device)


def bernoulli_chunks(n_chunks: int, p: float, seed: int,
                     device="cpu") -> torch.Tensor:
    g = torch.Generator(device=device).manual_seed(seed)
    mask = torch.rand(n_chunks, generator=g, device=device) < p
    return torch.nonzero(mask).view(-1)


def permuted_chunks(n_chunks: int, count: int, seed: int,
                    device="cpu") -> torch.Tensor:
    g = torch.Generator(device=device).manual_seed(seed)
    return torch.sort(torch.randperm(n_chunks, generator=g,
                                     device=device)[:count]).values


def tiny_step(device="cpu"):
    """Tiny cache and its step: exactly 24 of 32 chunks rewritten."""
    prev = make_cache(TINY, device)
    ids = permuted_chunks(TINY.nbytes // CHUNK, 24, seed=1, device=device)
    return prev, regenerate(prev, TINY, ids, seed=11), ids


def production_step(prev: torch.Tensor, device=None):
    """Active-generation step: each chunk regenerated iff Bernoulli(0.75)."""
    device = device or prev.device
    ids = bernoulli_chunks(PRODUCTION.nbytes // CHUNK, 0.75, seed=3,
                           device=device)
    return regenerate(prev, PRODUCTION, ids, seed=13), ids


def as_bytes(t: torch.Tensor) -> torch.Tensor:
    return t.contiguous().view(-1).view(torch.uint8)


# ---- session manifests ------------------------------------------------------
# The paper's suspend manifest has 450 leaves: the 420 movable tensors plus
# scalar control flags (§5 "Implementation").  A stand-in of the same
# structure is cut from a cache of the specs above: per layer, the K and the V
# slab split into 7 head groups (392 tensors for 28 layers), one fp32 [T]
# per-layer tensor (28), and 30 scalar control leaves of 1, 4 or 8 bytes.

N_CONTROL_LEAVES = 30


def head_groups(n_heads: int) -> tuple:
    """Split n_heads into min(7, n_heads) groups, the larger groups last
    (16 heads -> 2,2,2,2,2,3,3)."""
    g = min(7, n_heads)
    base, extra = divmod(n_heads, g)
    return tuple(base + (1 if i >= g - extra else 0) for i in range(g))


def make_manifest(spec: CacheSpec, device="cpu", cache=None) -> list:
    """Leaves of a session manifest built on `spec`'s cache: a list of
    separate contiguous tensors (bf16 head-group slabs, fp32 per-layer
    tensors, uint8/int32/int64 control scalars)."""
    if cache is None:
        cache = make_cache(spec, device)
    L, _, H, T, _ = spec.shape
    g = torch.Generator(device=cache.device).manual_seed(spec.seed + 7000)
    leaves = []
    groups = head_groups(H)
    for layer in range(L):
        for kv in range(2):
            h0 = 0
            for n in groups:
                leaves.append(cache[layer, kv, h0:h0 + n].clone())
                h0 += n
        leaves.append(torch.rand(T, generator=g, device=cache.device))
    dtypes = (torch.uint8, torch.int32, torch.int64)
    for i in range(N_CONTROL_LEAVES):
        leaves.append(torch.randint(0, 1 << 30, (1,), generator=g, device=cache.device,
                                    dtype=torch.int64).to(dtypes[i % 3]))
    return leaves


def ragged_sizes(n: int, seed: int) -> list:
    """Leaf sizes mixing the edge cases of a flat layout (0, 1, 15, 16, 17,
    64 KiB +- 1 ...) with uniform sizes up to 300 KB."""
    g = torch.Generator().manual_seed(seed)
    edge = [0, 1, 15, 16, 17, 4095, 4096, 65535, 65536, 65537, 131071, 2]
    sizes = []
    for i in range(n):
        if i % 3 == 0:
            sizes.append(edge[(i // 3) % len(edge)])
        else:
            sizes.append(int(torch.randint(1, 300_000, (1,), generator=g).item()))
    return sizes
