"""Seeded synthetic inputs for the KV-composition workloads.

This module only DRAWS inputs: shapes, token coordinates, chunk offsets and
random tensors.  It holds none of the method's arithmetic (no rotation, norm,
ranking or attention); the tests and the benchmark turn these draws into
post-rotary caches themselves.

Workloads (model geometry from the paper's experimental setup, Section 3:
36 layers, 16 query heads, 2 KV heads, head dim 128, mRoPE sections 16/24/24):

  tiny      1 layer, 4 Q / 2 KV heads, D=16, sections (2,3,3), fp32 storage,
            2 chunks of 2x4x4 tokens, chunk 2 shifted by dt=2, rho=0.25
  qwen8k    Qwen2.5-VL-3B geometry, bf16, 4 chunks of 8x16x16 tokens,
            chunk c shifted by dt=8c, rho=0.1
  long65k   the same geometry with 32 chunks (65,536 tokens); chunk c is
            shifted by dt_c = dt_{c-1} + 8 + gap_c, gap_c ~ U{0..16}, rho=0.1
  rebase_*  K only, 2048-token chunks, every chunk shifted by
            dt ~ U{0..1e5}, dh, dw ~ U{-16..16} (8k / 65k / 262k tokens)
  attn32k   the same geometry with 16 chunks (32,768 tokens), dt_c = 8c,
            rho in {0.05, 0.1, 0.2, 0.5, 1.0}

Random streams (each tensor and layer has its own counter-free seed, so any
layer can be drawn alone):
  stream 0  pre-rotary K and V ~ N(0, 1)
  stream 1  fresh-row noise z ~ N(0, 0.1^2) (K and V separately) and the
            per-token noise scale s_t ~ LogNormal(0, 1)
  stream 2  fresh queries ~ N(0, 1)
  stream 3  chunk offsets and gaps
"""
from dataclasses import dataclass, field

import numpy as np

QWEN = dict(n_layers=36, n_q_heads=16, n_kv_heads=2, head_dim=128,
            sections=(16, 24, 24), base=1.0e6, dtype="bf16")

# tensor tags inside a stream
TAG_K, TAG_V, TAG_ZK, TAG_ZV, TAG_S, TAG_Q, TAG_OFF = range(7)


@dataclass(frozen=True)
class Workload:
    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    sections: tuple
    base: float
    dtype: str                 # 'bf16' or 'f32'
    chunk_grid: tuple          # (temporal groups, height, width) per chunk
    n_chunks: int
    rho: float
    score_layer: int
    offsets: str               # offset recipe name
    seed: int = 0
    rhos: tuple = field(default=())
    chunk_lens: tuple = field(default=())   # ragged chunks: explicit token counts (overrides the grid)

    @property
    def chunk_tokens(self):
        t, h, w = self.chunk_grid
        return t * h * w

    @property
    def chunk_start(self):
        if self.chunk_lens:
            return np.concatenate([[0], np.cumsum(self.chunk_lens)]).astype(np.int64)
        return np.arange(self.n_chunks + 1, dtype=np.int64) * self.chunk_tokens

    @property
    def n_tokens(self):
        return int(self.chunk_start[-1])

    @property
    def cs1(self):
        return int(self.chunk_start[1])

    @property
    def n_candidates(self):
        return self.n_tokens - self.cs1


WORKLOADS = {
    "tiny": Workload("tiny", 1, 4, 2, 16, (2, 3, 3), 1.0e6, "f32", (2, 4, 4), 2,
                     0.25, 0, "tiny"),
    "qwen8k": Workload("qwen8k", chunk_grid=(8, 16, 16), n_chunks=4, rho=0.1,
                       score_layer=1, offsets="cumulative8", **QWEN),
    "long65k": Workload("long65k", chunk_grid=(8, 16, 16), n_chunks=32, rho=0.1,
                        score_layer=1, offsets="cumulative8_gap16", **QWEN),
    "rebase8k": Workload("rebase8k", chunk_grid=(8, 16, 16), n_chunks=4, rho=0.0,
                         score_layer=1, offsets="random_all_axes", **QWEN),
    "rebase65k": Workload("rebase65k", chunk_grid=(8, 16, 16), n_chunks=32, rho=0.0,
                          score_layer=1, offsets="random_all_axes", **QWEN),
    "rebase262k": Workload("rebase262k", chunk_grid=(8, 16, 16), n_chunks=128, rho=0.0,
                           score_layer=1, offsets="random_all_axes", **QWEN),
    "attn32k": Workload("attn32k", chunk_grid=(8, 16, 16), n_chunks=16, rho=0.1,
                        score_layer=1, offsets="cumulative8",
                        rhos=(0.05, 0.1, 0.2, 0.5, 1.0), **QWEN),
}


def _rng(seed, stream, tag, layer=0):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, tag, layer])))


def local_coords(w: Workload):
    """Local (t, h, w) of every token: raster order inside each chunk, from 0
    (a ragged chunk ends with a partial frame)."""
    _, hh, ww = w.chunk_grid
    cs = w.chunk_start
    parts = []
    for c in range(w.n_chunks):
        j = np.arange(cs[c + 1] - cs[c], dtype=np.int64)
        parts.append(np.stack([j // (hh * ww), (j // ww) % hh, j % ww], axis=-1))
    return np.concatenate(parts)


def chunk_offsets(w: Workload):
    """Per-chunk global offsets (dt, dh, dw) = p' - p, int64 [N, 3]."""
    N = w.n_chunks
    off = np.zeros((N, 3), dtype=np.int64)
    if w.offsets == "none":
        pass
    elif w.offsets == "tiny":
        off[1] = (2, 0, 0)
    elif w.offsets == "cumulative8":
        off[:, 0] = 8 * np.arange(N)
    elif w.offsets == "cumulative8_gap16":
        gaps = _rng(w.seed, 3, TAG_OFF).integers(0, 17, size=N)
        for c in range(1, N):
            off[c, 0] = off[c - 1, 0] + w.chunk_grid[0] + gaps[c]
    elif w.offsets == "random_all_axes":
        r = _rng(w.seed, 3, TAG_OFF)
        off[:, 0] = r.integers(0, 100_001, size=N)
        off[:, 1] = r.integers(-16, 17, size=N)
        off[:, 2] = r.integers(-16, 17, size=N)
    else:
        raise ValueError(w.offsets)
    return off


def draw_normal(shape, seed, stream, tag, layer=0, std=1.0):
    """N(0, std^2) draw of one tensor slice (one layer): float32 samples
    returned as float64."""
    x = _rng(seed, stream, tag, layer).standard_normal(shape, dtype=np.float32).astype(np.float64)
    return x * std if std != 1.0 else x


LAYER_TENSORS = ("k_pre", "v", "zk", "zv", "q_pre")


def draw_layer(w: Workload, layer, which=LAYER_TENSORS):
    """Random tensors of one layer, float64, pre-rotary.

    k_pre, v     [H_kv, T, D]   stored keys (before rotation) and values
    zk, zv       [H_kv, n, D]   fresh-row noise, N(0, 0.1^2)
    q_pre        [H_q, n, D]    fresh queries (before rotation)
    """
    T, n, D = w.n_tokens, w.n_candidates, w.head_dim
    spec = dict(k_pre=((w.n_kv_heads, T, D), 0, TAG_K, 1.0),
                v=((w.n_kv_heads, T, D), 0, TAG_V, 1.0),
                zk=((w.n_kv_heads, n, D), 1, TAG_ZK, 0.1),
                zv=((w.n_kv_heads, n, D), 1, TAG_ZV, 0.1),
                q_pre=((w.n_q_heads, n, D), 2, TAG_Q, 1.0))
    return {k: draw_normal(spec[k][0], w.seed, spec[k][1], spec[k][2], layer, spec[k][3]) for k in which}


def draw_token_scale(w: Workload):
    """Per-token noise scale s_t ~ LogNormal(0, 1) for the n candidates (shared by all layers)."""
    return _rng(w.seed, 1, TAG_S).lognormal(0.0, 1.0, size=w.n_candidates)


# ---------------------------------------------------------------- device draws
def torch_seed(seed, stream, tag, layer=0):
    """A 63-bit torch seed for one (stream, tensor, layer) slice."""
    return int(np.random.SeedSequence([seed, stream, tag, layer]).generate_state(2, np.uint64)[0]
               & np.uint64(0x7FFFFFFFFFFFFFFF))


def torch_normal(shape, seed, stream, tag, layer, device, dtype, std=1.0):
    """N(0, std^2) draw on a device with torch's generator (for the large workloads)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(torch_seed(seed, stream, tag, layer))
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)


def torch_token_scale(w: Workload, device):
    """s_t ~ LogNormal(0, 1) on a device, float32 [n]."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(torch_seed(w.seed, 1, TAG_S))
    return torch.randn(w.n_candidates, generator=g, device=device, dtype=torch.float32).exp_()
