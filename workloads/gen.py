"""Seeded clustered-Gaussian shallow-key indices and text-token queries.

Every array is bfloat16, carried as its raw 16-bit pattern in ``numpy.uint16``.
Values are drawn in float32 and rounded to bfloat16 with round-to-nearest-even.

Workload shapes (7B-class GQA language model, one frame = one video unit at 1 FPS):

==== ============================================================================
C1   tiny: 2 shallow layers, 4 query / 2 KV heads, d=64, 64 frames x 16 tokens,
     2 planted frames, 8 query tokens, top-k 32, 4 frames selected
C2   10-minute stream: 4 layers, 28/4 heads, d=128, 600 x 196, 8 planted,
     32 query tokens, top-k 256, 16 frames
C3   C2 with per-frame k-means compression to 32 centroids (10 iterations),
     top-k 64, 16 frames
C4   1-hour stream: 4 layers, 28/4 heads, d=128, 3600 x 196, 24 planted,
     64 query tokens, top-k 512, 32 frames
C5   16 streams, 6 layers, 16/2 heads, d=128, lengths uniform on 300..3600
     frames x 196 tokens, odd streams compressed to 32 centroids, 32 query
     tokens, top-k 256, 16 frames per stream
P4   C4's stream with the paper's own selection settings: one query token (the
     last prompt token), scores averaged over heads (one list per layer),
     top 64 per layer, pool of 32, 8 frames
==== ============================================================================

Generator: for each (frame, layer, KV head) a centroid ``z ~ N(0, I_d)`` and
tokens ``z + 0.5 * N(0, I_d)``.  A planted frame replaces ``z`` by
``||z|| * m_hat`` where ``m_hat`` is the unit mean of the bfloat16 queries of
that layer over the KV head's query-head group and all query tokens; planted
frames sit at ``floor((i + 1/2) * F / n_planted)``.  Query tokens are
``N(0, 1)``.  Each frame has its own ``SeedSequence([seed, stream, 1, frame])``
so blocks of frames can be drawn in parallel and in any order with identical
bytes.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

_PURPOSE_QUERY = 0
_PURPOSE_FRAME = 1
_PURPOSE_LENGTHS = 2


@dataclass(frozen=True)
class Config:
    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    tokens_per_frame: int
    n_q: int
    top_k: int
    n_select: int
    n_frames: int = 0                 # single-stream workloads
    n_planted: int = 0
    compress: tuple | None = None     # (n_centroids, n_iters) for every stream
    n_streams: int = 1
    frames_range: tuple | None = None  # ragged batches: inclusive (lo, hi)
    compress_odd_streams: bool = False
    planted_every: int = 150           # ragged batches: one planted frame per this many frames
    pool_mult: int = 4
    head_mode: int = 0                 # 1: the paper's head-averaged lists, one per layer
    description: str = ""

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


CONFIGS: dict[str, Config] = {
    "C1": Config("C1", 2, 4, 2, 64, 16, 8, 32, 4, n_frames=64, n_planted=2,
                 description="tiny index, 64 frames x 16 tokens"),
    "C2": Config("C2", 4, 28, 4, 128, 196, 32, 256, 16, n_frames=600, n_planted=8,
                 description="10-minute stream, 600 frames x 196 tokens"),
    "C3": Config("C3", 4, 28, 4, 128, 196, 32, 64, 16, n_frames=600, n_planted=8,
                 compress=(32, 10),
                 description="10-minute stream compressed to 600 x 32 centroids"),
    "C4": Config("C4", 4, 28, 4, 128, 196, 64, 512, 32, n_frames=3600, n_planted=24,
                 description="1-hour stream, 3600 frames x 196 tokens"),
    "C5": Config("C5", 6, 16, 2, 128, 196, 32, 256, 16, n_streams=16,
                 frames_range=(300, 3600), compress_odd_streams=True,
                 description="16 ragged streams (300..3600 frames), odd streams compressed"),
    "P4": Config("P4", 4, 28, 4, 128, 196, 1, 64, 8, n_frames=3600, n_planted=24, head_mode=1,
                 description="the paper's selection settings on the 1-hour stream: last prompt token, "
                             "head-averaged scores, top 64 per layer, pool of 32, 8 units"),
}


@dataclass(frozen=True)
class StreamSpec:
    stream: int
    n_frames: int
    n_planted: int
    compress: tuple | None = None
    planted: tuple = field(default=())


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return the bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).copy()
    if np.any((u & 0x7F800000) == 0x7F800000):
        raise ValueError("non-finite value in generated data")
    lsb = (u >> 16) & np.uint32(1)
    u += np.uint32(0x7FFF)
    u += lsb
    return (u >> 16).astype(np.uint16)


def _bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def planted_frames(n_frames: int, n_planted: int) -> tuple:
    if n_planted <= 0:
        return ()
    return tuple(int(math.floor((i + 0.5) * n_frames / n_planted)) for i in range(n_planted))


def stream_specs(cfg: Config, seed: int = 0) -> list[StreamSpec]:
    if cfg.frames_range is None:
        return [StreamSpec(0, cfg.n_frames, cfg.n_planted, cfg.compress,
                           planted_frames(cfg.n_frames, cfg.n_planted))]
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0, _PURPOSE_LENGTHS])))
    lo, hi = cfg.frames_range
    lengths = rng.integers(lo, hi + 1, size=cfg.n_streams)
    specs = []
    for s, f in enumerate(lengths):
        f = int(f)
        n_p = int(math.ceil(f / cfg.planted_every))
        comp = (32, 10) if (cfg.compress_odd_streams and s % 2 == 1) else cfg.compress
        specs.append(StreamSpec(s, f, n_p, comp, planted_frames(f, n_p)))
    return specs


def make_queries(cfg: Config, seed: int = 0, stream: int = 0) -> list[np.ndarray]:
    """Per shallow layer, the query tokens ``[H_q][n_q][d]`` as bfloat16 bits."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, _PURPOSE_QUERY])))
    out = []
    for _ in range(cfg.n_layers):
        q = rng.standard_normal((cfg.n_q_heads, cfg.n_q, cfg.head_dim), dtype=np.float32)
        out.append(bf16_bits(q))
    return out


def _planted_directions(cfg: Config, queries: list[np.ndarray]) -> np.ndarray:
    """Unit mean query direction per (layer, KV head): ``[L][H_kv][d]`` float64."""
    G = cfg.group
    dirs = np.zeros((cfg.n_layers, cfg.n_kv_heads, cfg.head_dim))
    for l, q in enumerate(queries):
        qf = _bf16_to_f64(q)
        for g in range(cfg.n_kv_heads):
            m = qf[g * G:(g + 1) * G].reshape(-1, cfg.head_dim).mean(axis=0)
            n = np.linalg.norm(m)
            dirs[l, g] = m / n if n > 0 else m
    return dirs


def _one_frame(cfg: Config, seed: int, stream: int, frame: int, planted: bool,
               dirs: np.ndarray) -> np.ndarray:
    """Keys of one frame: ``[L][H_kv][T][d]`` bfloat16 bits.

    Draw order per frame: all centroids ``[L][H_kv][d]``, then all token noise
    ``[L][H_kv][T][d]``.
    """
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, _PURPOSE_FRAME, frame])))
    L, Hk, T, d = cfg.n_layers, cfg.n_kv_heads, cfg.tokens_per_frame, cfg.head_dim
    z = rng.standard_normal((L, Hk, d), dtype=np.float32)
    noise = rng.standard_normal((L, Hk, T, d), dtype=np.float32)
    if planted:
        norms = np.linalg.norm(z.astype(np.float64), axis=2, keepdims=True)
        z = (norms * dirs).astype(np.float32)
    noise *= np.float32(0.5)
    noise += z[:, :, None, :]
    return bf16_bits(noise)


def frame_block_keys(cfg: Config, spec: StreamSpec, queries: list[np.ndarray], f0: int, f1: int,
                     seed: int = 0, threads: int | None = None) -> list[np.ndarray]:
    """Keys of frames ``[f0, f1)`` in append layout: per layer ``[H_kv][(f1-f0)*T][d]``."""
    dirs = _planted_directions(cfg, queries)
    planted = set(spec.planted)
    nthreads = threads or min(16, len(os.sched_getaffinity(0)))
    L, Hk, T, d = cfg.n_layers, cfg.n_kv_heads, cfg.tokens_per_frame, cfg.head_dim
    out = [np.empty((Hk, (f1 - f0) * T, d), dtype=np.uint16) for _ in range(L)]

    def fill(f):
        fr = _one_frame(cfg, seed, spec.stream, f, f in planted, dirs)
        i = f - f0
        for l in range(L):
            out[l][:, i * T:(i + 1) * T, :] = fr[l]

    with ThreadPoolExecutor(max(1, nthreads)) as ex:
        list(ex.map(fill, range(f0, f1)))
    return out


def make_stream(cfg: Config, spec: StreamSpec, seed: int = 0, threads: int | None = None):
    """Queries and the whole stream's keys: ``(queries, per-layer keys)``."""
    q = make_queries(cfg, seed, spec.stream)
    keys = frame_block_keys(cfg, spec, q, 0, spec.n_frames, seed, threads)
    return q, keys
