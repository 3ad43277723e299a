"""One DiT block over a pack of nodes -- oracle, test infrastructure only.

The paper fixes only the network's role (F_theta in Eq. 1, reading the
context of each node through the visibility mask of Eq. 6).  The block form
is the Wan-shaped reading used for the workload (no trained weights exist
here to compare a real model with; the reading itself is pinned by a block
worked by hand at hidden 4, every intermediate listed, and by closed-form
special cases):

    h  = RMSNorm(x)                          eps = 1e-6, unit gain
    q, k, v = h Wq^T, h Wk^T, h Wv^T          heads of d channels
    q, k = RoPE(q), RoPE(k)                   at each token's (t, h, w) position
    o  = attention of each node over its selected states (Eq. 6)
    x' = x + o Wo^T
    y  = x' + GELU_tanh(RMSNorm(x') Wup^T) Wdown^T

Noise-level conditioning (optional): the denoiser of Eq. 1 takes the node's
level j.  With a per-level table mod[j] = (shift_a, scale_a, gate_a,
shift_m, scale_m, gate_m) the block is

    h  = RMSNorm(x) (1 + scale_a) + shift_a
    x' = x + gate_a (o Wo^T)
    y  = x' + gate_m (GELU_tanh((RMSNorm(x') (1 + scale_m) + shift_m) Wup^T) Wdown^T)

(an adaLN-style reading; the table itself, e.g. a projected timestep
embedding, is an input).  Without it the block is the form above.

Two further options of the Wan block form (readings: the paper's F_theta
takes the condition c of Eq. 1, and Wan-style blocks read it by
cross-attention; both normalise queries and keys):

    qk-norm:  q = RMSNorm(h Wq^T) g_q, k = RMSNorm(h Wk^T) g_k over the whole
              hidden width, before RoPE
    cross-attention to a condition sequence c [L, hidden] (K_c, V_c cached
    once: K_c = RMSNorm(c Wck^T) g_ck or c Wck^T, V_c = c Wcv^T, no RoPE),
    after the self-attention residual:
              x'' = x' + Attn(RMSNorm(RMSNorm(x') Wcq^T) g_cq, K_c, V_c) Wco^T
              (the inner RMSNorm of the query only when g_cq is given)
    and the MLP then reads x''.

Weights are in [out, in] layout (y = x W^T); Wqkv stacks Wq, Wk, Wv along
its output axis.  Every product here is an fp64 numpy matmul.  The K and V a
node produces become the cached representation of its state (Sec. 3.2,
"Effective context and visibility"): later nodes read them.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, Optional, Sequence, Tuple

import numpy as np

from .attention import node_attention, softmax_attention
from .rope import chunk_positions, rope

RMS_EPS = 1e-6


def rmsnorm(x: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


class BlockShape:
    def __init__(self, hidden=1536, heads=12, head_dim=128, mlp=8960,
                 frames_per_chunk=3, grid_h=30, grid_w=52, rope_dims=(44, 42, 42),
                 theta=10000.0):
        self.hidden, self.heads, self.head_dim, self.mlp = hidden, heads, head_dim, mlp
        self.frames_per_chunk, self.grid_h, self.grid_w = frames_per_chunk, grid_h, grid_w
        self.rope_dims, self.theta = tuple(rope_dims), theta

    @property
    def tokens_per_chunk(self):
        return self.frames_per_chunk * self.grid_h * self.grid_w


def modulated_norm(x: np.ndarray, mod_row: Optional[np.ndarray], which: int) -> np.ndarray:
    """RMSNorm(x), then * (1 + scale) + shift of part ``which`` (0 attention,
    1 MLP) of one level's modulation row [6][hidden]; plain without a row."""
    h = rmsnorm(x)
    if mod_row is None:
        return h
    shift = np.asarray(mod_row[3 * which], dtype=np.float64)
    scale = np.asarray(mod_row[3 * which + 1], dtype=np.float64)
    return h * (1.0 + scale) + shift


def norm_gain(x: np.ndarray, gain) -> np.ndarray:
    """RMSNorm over the last axis times a per-channel gain (qk-norm)."""
    return rmsnorm(x) * np.asarray(gain, dtype=np.float64)


def project_kv(x: np.ndarray, chunk: int, w_qkv: np.ndarray, shp: BlockShape, mod_row=None,
               g_k=None):
    """Rotated K and plain V of one node's tokens: x [Nq, hidden] -> [Nq, H, d] x 2."""
    D = shp.hidden
    h = modulated_norm(x, mod_row, 0)
    w = np.asarray(w_qkv, dtype=np.float64)
    k = h @ w[D:2 * D].T
    if g_k is not None:
        k = norm_gain(k, g_k)
    k = k.reshape(-1, shp.heads, shp.head_dim)
    v = (h @ w[2 * D:3 * D].T).reshape(-1, shp.heads, shp.head_dim)
    pos = chunk_positions(chunk, shp.frames_per_chunk, shp.grid_h, shp.grid_w)
    return rope(k, pos, shp.rope_dims, shp.theta), v


def project_q(x: np.ndarray, chunk: int, w_qkv: np.ndarray, shp: BlockShape, rows=None,
              mod_row=None, g_q=None):
    D = shp.hidden
    x = np.asarray(x, dtype=np.float64)
    pos = chunk_positions(chunk, shp.frames_per_chunk, shp.grid_h, shp.grid_w)
    if rows is not None:
        x, pos = x[rows], pos[rows]
    h = modulated_norm(x, mod_row, 0)
    q = h @ np.asarray(w_qkv, dtype=np.float64)[0:D].T
    if g_q is not None:
        q = norm_gain(q, g_q)
    return rope(q.reshape(-1, shp.heads, shp.head_dim), pos, shp.rope_dims, shp.theta)


def condition_kv(ctx: np.ndarray, w_k: np.ndarray, w_v: np.ndarray, shp: BlockShape, g_k=None):
    """Cached K and V of a condition sequence ctx [L, hidden] -> [L, H, d] x 2
    (no RoPE: the condition has no position in the video)."""
    ctx = np.asarray(ctx, dtype=np.float64)
    k = ctx @ np.asarray(w_k, dtype=np.float64).T
    if g_k is not None:
        k = norm_gain(k, g_k)
    v = ctx @ np.asarray(w_v, dtype=np.float64).T
    return k.reshape(-1, shp.heads, shp.head_dim), v.reshape(-1, shp.heads, shp.head_dim)


def cross_attention(x: np.ndarray, cross: Dict[str, np.ndarray], shp: BlockShape) -> np.ndarray:
    """Attn(RMSNorm(x) Wcq^T [RMSNorm * g_cq], K_c, V_c) Wco^T for rows x [N, hidden].

    cross: "k", "v" (the condition's [L, H, d] from condition_kv), "w_q",
    "w_o" ([hidden, hidden]) and optionally "g_q"."""
    q = rmsnorm(x) @ np.asarray(cross["w_q"], dtype=np.float64).T
    if cross.get("g_q") is not None:
        q = norm_gain(q, cross["g_q"])
    q = q.reshape(-1, shp.heads, shp.head_dim)
    k, v = np.asarray(cross["k"], dtype=np.float64), np.asarray(cross["v"], dtype=np.float64)
    scale = 1.0 / math.sqrt(shp.head_dim)
    o = np.empty_like(q)
    for h in range(shp.heads):
        o[:, h, :] = softmax_attention(q[:, h, :], k[:, h, :], v[:, h, :], scale)
    return o.reshape(q.shape[0], -1) @ np.asarray(cross["w_o"], dtype=np.float64).T


def block_forward(sel, x_of: Callable[[int], np.ndarray], weights: Dict[str, np.ndarray],
                  resident_kv: Callable[[Tuple[int, int]], Tuple[np.ndarray, np.ndarray]],
                  shp: BlockShape, rows: Optional[Sequence[int]] = None,
                  mod: Optional[np.ndarray] = None, qk_norm=None, cross=None,
                  trace: Optional[dict] = None):
    """Run one block for every node of ``sel``.

    x_of(i) gives node i's input [Nq, hidden].  resident_kv(state) gives the
    cached (rotated K, V) of a state that no pack node produces.  ``rows``
    restricts the outputs to those token rows of every node (the K/V of all
    rows are still computed, since every row reads all of them).  ``mod``
    is the optional per-level modulation table [levels][6][hidden];
    ``qk_norm`` the optional gains (g_q, g_k); ``cross`` the optional
    cross-attention (see cross_attention), one for every node or a function
    of the node (c, j) (nodes of one pack may read different conditions).
    With ``trace`` (a dict) the intermediates of each node's output rows are
    stored in it: trace[i] = {"q": rotated queries [rows, H, d], "o": the
    attention output [rows, H, d], "a": o Wo^T [rows, hidden] (before any
    gate)}.
    Returns ({i: y_i}, {i: (k_i, v_i)}).
    """
    def mod_row(j):
        return None if mod is None else np.asarray(mod[j], dtype=np.float64)

    g_q, g_k = (None, None) if qk_norm is None else qk_norm
    new_kv = {}
    for i, (c, j) in enumerate(sel.nodes):
        new_kv[i] = project_kv(x_of(i), c, weights["w_qkv"], shp, mod_row(j), g_k)
    index_of = {node: i for i, node in enumerate(sel.nodes)}

    def kv_of(state):
        if state in index_of:
            return new_kv[index_of[state]]
        return resident_kv(state)

    scale = 1.0 / math.sqrt(shp.head_dim)
    out = {}
    for i, (c, j) in enumerate(sel.nodes):
        m = mod_row(j)
        x = np.asarray(x_of(i), dtype=np.float64)
        if rows is not None:
            x = x[rows]
        q = project_q(x_of(i), c, weights["w_qkv"], shp, rows, m, g_q)
        o = node_attention(q, sel.segments(i), kv_of, scale).reshape(q.shape[0], -1)
        a = o @ np.asarray(weights["w_o"], dtype=np.float64).T
        if trace is not None:
            trace[i] = {"q": q, "o": o.reshape(q.shape), "a": a}
        x1 = x + (a if m is None else m[2] * a)
        if cross is not None:
            x1 = x1 + cross_attention(x1, cross((c, j)) if callable(cross) else cross, shp)
        u = modulated_norm(x1, m, 1) @ np.asarray(weights["w_up"], dtype=np.float64).T
        f = gelu_tanh(u) @ np.asarray(weights["w_down"], dtype=np.float64).T
        out[i] = x1 + (f if m is None else m[5] * f)
    return out, new_kv
