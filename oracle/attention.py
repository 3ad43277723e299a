"""Softmax attention of each node over its selected context -- oracle, test infrastructure only.

Eq. 6 adds a mask M(u, v) in {0, -inf} to the attention logits before the
softmax.  For node i, M is 0 exactly on the key tokens of the states its
selection table lists (history plus its own chunk) and -inf elsewhere, so
the masked softmax over all keys equals the plain softmax over the gathered
visible keys.  This module computes the latter, in fp64, one node and one
head at a time:

    s = q k^T * scale,   p = exp(s - max_row s) / sum_row exp(s - max_row s),   o = p v

Layouts (numpy): q, o are [Nq, H, d]; the K and V of one state are
[tokens, H, d] with tokens ordered frame by frame.
"""
from __future__ import annotations

from typing import Callable, Dict, Sequence, Tuple

import numpy as np


def softmax_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
                      return_probs: bool = False):
    """One head: q [Nq, d], k [Nk, d], v [Nk, dv] -> o [Nq, dv] in fp64."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    s = (q @ k.T) * scale
    s = s - s.max(axis=1, keepdims=True)
    e = np.exp(s)
    p = e / e.sum(axis=1, keepdims=True)
    o = p @ v
    return (o, p) if return_probs else o


def gather_context(segments: Sequence[Tuple[int, int]],
                   kv_of: Callable[[Tuple[int, int]], Tuple[np.ndarray, np.ndarray]]):
    """Concatenate the K and V of the selected states in selection order."""
    ks, vs = [], []
    for state in segments:
        k, v = kv_of(state)
        ks.append(np.asarray(k, dtype=np.float64))
        vs.append(np.asarray(v, dtype=np.float64))
    return np.concatenate(ks, axis=0), np.concatenate(vs, axis=0)


def node_attention(q: np.ndarray, segments, kv_of, scale: float, rows=None) -> np.ndarray:
    """Attention of one node: q [Nq, H, d] over its segments -> [Nq, H, d] fp64.

    ``rows`` restricts the computation to a subset of query rows (each row is
    independent of the others, so sampled rows are exact).
    """
    k, v = gather_context(segments, kv_of)
    q = np.asarray(q, dtype=np.float64)
    if rows is not None:
        q = q[rows]
    H = q.shape[1]
    out = np.empty((q.shape[0], H, v.shape[2]), dtype=np.float64)
    for h in range(H):
        out[:, h, :] = softmax_attention(q[:, h, :], k[:, h, :], v[:, h, :], scale)
    return out


def packed_attention(sel, q_of, kv_of, scale: float, rows=None) -> Dict[int, np.ndarray]:
    """Every node of a selection table, independently: {node index: o}."""
    return {i: node_attention(q_of(i), sel.segments(i), kv_of, scale, rows)
            for i in range(len(sel.nodes))}


def row_probabilities(q: np.ndarray, segments, kv_of, scale: float, head: int) -> np.ndarray:
    """Softmax rows of one head (debug form used by the row-sum pin)."""
    k, v = gather_context(segments, kv_of)
    _, p = softmax_attention(np.asarray(q)[:, head, :], k[:, head, :], v[:, head, :],
                             scale, return_probs=True)
    return p
