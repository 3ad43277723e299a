"""3D rotary position embedding -- oracle, test infrastructure only.

The paper does not define the positional encoding of its DiT; this is the
reading used for the Wan-shaped workload.  Pinned by mathematical
properties (identity at position 0, norm preservation, relative-position
invariance of the logits) and by a hand table of single-pair rotation angles
for the 44/42/42 split (pairs 0, 1, 2 and the last of each axis); the choice
of split and theta itself is the reading, not a statement of the paper.

The head dimension d is split into three axis groups of d_t, d_h, d_w
channels (44/42/42 for d = 128).  Channels are taken in interleaved pairs
(x[2p], x[2p+1]); pair p belongs to the time axis for p < d_t/2, to the
height axis for the next d_h/2 pairs and to the width axis for the rest.
Within axis a, its i-th pair is rotated by the angle pos_a * theta**(-2 i / d_a)
-- multiplication of the complex number x[2p] + 1j * x[2p+1] by exp(1j * angle).

Token positions: a chunk holds F latent frames of grid_h x grid_w tokens,
row-major; token n of frame f of chunk c sits at time c * F + f, height
n // grid_w, width n % grid_w.
"""
from __future__ import annotations

import numpy as np


def axis_of_pairs(dims):
    """For each channel pair: (axis index, index i within the axis)."""
    out = []
    for a, da in enumerate(dims):
        for i in range(da // 2):
            out.append((a, i))
    return out


def chunk_positions(chunk: int, frames_per_chunk: int, grid_h: int, grid_w: int) -> np.ndarray:
    """[frames*grid_h*grid_w, 3] integer (t, h, w) positions of one chunk's tokens."""
    f, n = np.meshgrid(np.arange(frames_per_chunk), np.arange(grid_h * grid_w), indexing="ij")
    t = chunk * frames_per_chunk + f
    return np.stack([t.ravel(), (n // grid_w).ravel(), (n % grid_w).ravel()], axis=1)


def rope(x: np.ndarray, pos: np.ndarray, dims=(44, 42, 42), theta: float = 10000.0) -> np.ndarray:
    """Rotate x [N, H, d] at positions pos [N, 3]; returns fp64 [N, H, d]."""
    x = np.asarray(x, dtype=np.float64)
    N, H, d = x.shape
    assert sum(dims) == d and all(da % 2 == 0 for da in dims)
    z = x[..., 0::2] + 1j * x[..., 1::2]                     # [N, H, d/2]
    angle = np.empty((N, d // 2), dtype=np.float64)
    for p, (a, i) in enumerate(axis_of_pairs(dims)):
        angle[:, p] = pos[:, a] * theta ** (-2.0 * i / dims[a])
    z = z * np.exp(1j * angle)[:, None, :]
    out = np.empty_like(x)
    out[..., 0::2] = z.real
    out[..., 1::2] = z.imag
    return out
