"""Workload geometry of the five benchmark/parity configurations (data only).

Shapes follow the paper's rollout geometry: 832x480 video at 16 FPS, 4x
temporal VAE compression, chunks of three latent frames, 30x52 patch grid per
latent frame (1560 tokens), a Wan2.1-1.3B-shaped DiT (hidden 1536, 12 heads
of 128, MLP 8960), four denoising levels.  Levels are the paper's: 0 clean,
K = 4 pure noise.  Node lists are oldest chunk first.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple


@dataclass
class Geometry:
    heads: int
    head_dim: int
    grid_h: int
    grid_w: int
    frames_per_chunk: int
    K: int = 4
    W: int = 6
    hidden: int = 0
    mlp: int = 0
    rope_dims: Tuple[int, int, int] = (44, 42, 42)
    theta: float = 10000.0

    @property
    def tokens_per_page(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def tokens_per_chunk(self) -> int:
        return self.tokens_per_page * self.frames_per_chunk


# Tiny oracle case: 4 chunks x 2 latent frames x 16 tokens; 2 heads of 64; K = 4.
TINY = Geometry(heads=2, head_dim=64, grid_h=4, grid_w=4, frames_per_chunk=2, K=4, W=3,
                rope_dims=(24, 20, 20))

# Wan2.1-1.3B-shaped block.
WAN = Geometry(heads=12, head_dim=128, grid_h=30, grid_w=52, frames_per_chunk=3, K=4, W=6,
               hidden=1536, mlp=8960)

# Small bf16 shape spanning several 64-key tiles, with pages (104 tokens)
# that end inside a tile and nodes whose last tile is ragged; used by the
# fast GPU parity tests.
SMALL = Geometry(heads=2, head_dim=128, grid_h=8, grid_w=13, frames_per_chunk=3, K=4, W=6,
                 hidden=256, mlp=512, rope_dims=(44, 42, 42))


# Short nodes (one 96-token latent frame per chunk, 96 queries): the
# 128-query work-group shape of the bf16 kernel, with pages that end inside
# 64-key tiles.
SHORT = Geometry(heads=2, head_dim=128, grid_h=8, grid_w=12, frames_per_chunk=1, K=4, W=6,
                 hidden=256, mlp=512)


# Narrow nodes (one 40-token latent frame per chunk, 40 queries): the
# 64-query work-group shape of the bf16 kernel with its 32-key tiles, pages
# (40 tokens) that end inside tiles and ragged last tiles.
NARROW = Geometry(heads=2, head_dim=128, grid_h=5, grid_w=8, frames_per_chunk=1, K=4, W=6,
                  hidden=256, mlp=512)


def kv_stream(nq: int, W: int = 20) -> Geometry:
    """Short-context K/V streaming shape: Wan heads (12 x 128), one latent
    frame of ``nq`` tokens per chunk, up to W + 1 = 21 pages per node."""
    grid_w = {64: 8, 128: 16}[nq]
    return Geometry(heads=12, head_dim=128, grid_h=8, grid_w=grid_w, frames_per_chunk=1, K=4, W=W,
                    hidden=1536, mlp=8960)


@dataclass
class Workload:
    name: str
    policy: str
    pack: List[Tuple[int, int]]           # nodes run in one packed forward
    resident: List[Tuple[int, int]]       # states cached before the forward
    description: str = ""


def cfg2_clean(level: int = 4) -> Workload:
    """Clean history, one node at a time: chunk 6 with clean chunks 0..5 cached."""
    return Workload("cfg2-clean", "clean", [(6, level)], [(c, 0) for c in range(6)],
                    "Wan block, clean history, one node, 6 prior chunks (28080 keys)")


def cfg3_same(level: int = 2) -> Workload:
    """Same-level history: 4 consecutive chunks at one level packed together."""
    return Workload("cfg3-same", "same", [(6 + i, level) for i in range(4)],
                    [(c, level) for c in range(6)],
                    "Wan block, same-level history, 4 nodes at one level")


def cfg4_prog(refresh: bool = False) -> Workload:
    """Progressive-history diagonal in steady state (levels in the paper's
    numbering: the oldest in-flight chunk is the least noisy)."""
    pack = [(6, 1), (7, 2), (8, 3), (9, 4)]
    resident = [(c, 0) for c in range(6)]
    if refresh:
        pack = [(6, 0), (7, 1), (8, 2), (9, 3), (10, 4)]
    return Workload("cfg4-prog" + ("+R" if refresh else ""), "prog", pack, resident,
                    "Wan block, progressive diagonal pack, 21-frame per-node window")
