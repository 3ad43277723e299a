"""History selection (Sec. 3.2, Eq. 4-5) -- oracle, test infrastructure only.

A *node* is one denoising update: chunk ``c`` (0-based; the paper's b = c + 1)
at noise level ``j`` (0 = clean endpoint, K = initial noise), Eq. 1.

For a history window of W chunks the node reads the offsets
r in R subset of {1, ..., min(W, c)} (Eq. 4 with b - 1 = c), and from chunk c - r
the state at level phi(j, r).  The three policies of Eq. 5:

    clean  phi(j, r) = 0
    same   phi(j, r) = j
    prog   phi(j, r) = max(j - r, 0)

A fourth kind, ``table``, takes phi from a user table.  Eq. 4 lets the
policy and the offset set depend on the chunk (Phi_b, R_b,j): with
``n_chunks`` > 0 the tables are indexed [c][j][r - 1].  Each node also sees its own chunk at
its own level (the query chunk's own features, Eq. 6 text; attention inside a
chunk is bidirectional).

Canonical order of one node's segments: history offsets from the oldest chunk
(r = min(W, c)) to the newest (r = 1), then the node's own state.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

CLEAN, SAME, PROG, TABLE = 0, 1, 2, 3
KIND_NAMES = {"clean": CLEAN, "same": SAME, "prog": PROG, "table": TABLE}


class SelectionError(ValueError):
    """Invalid policy or node set (the C ABI's SC_EINVAL)."""


@dataclass
class Policy:
    kind: int
    K: int
    W: int
    phi_table: Optional[Sequence] = None  # [K+1][W] (or [n_chunks][K+1][W]), kind TABLE
    r_mask: Optional[Sequence] = None     # [K+1][W] (or [n_chunks][K+1][W]), None = dense
    n_chunks: int = 0                     # > 0: tables depend on the chunk (Phi_b of Eq. 4)

    def _entry(self, table, c: int, j: int, r: int):
        return table[c][j][r - 1] if self.n_chunks > 0 else table[j][r - 1]

    def phi(self, j: int, r: int, c: int = 0) -> int:
        """Level selected from chunk c - r for a node (c, j) (Eq. 4-5)."""
        if self.kind == CLEAN:
            return 0
        if self.kind == SAME:
            return j
        if self.kind == PROG:
            return max(j - r, 0)
        return int(self._entry(self.phi_table, c, j, r))

    def selected(self, j: int, r: int, c: int = 0) -> bool:
        """Whether offset r is in R_b,j for node (c, j) (Eq. 4)."""
        if self.r_mask is None:
            return True
        return bool(self._entry(self.r_mask, c, j, r))


def policy(name: str, K: int, W: int, **kw) -> Policy:
    return Policy(KIND_NAMES[name], K, W, **kw)


@dataclass
class Selection:
    """Canonical selection table of a pack of nodes.

    seg_off[i]..seg_off[i+1] index node i's segments; segment s is the state
    (seg_chunk[s], seg_level[s]); seg_src[s] is the index of the pack node that
    produces that state in this call, or -1 when it must already be cached.
    ``states`` lists every distinct state read by the pack, sorted by
    (chunk, level); ``vis[i][k]`` is 1 when node i reads ``states[k]``.
    """
    nodes: List[Tuple[int, int]]
    seg_off: List[int] = field(default_factory=list)
    seg_chunk: List[int] = field(default_factory=list)
    seg_level: List[int] = field(default_factory=list)
    seg_src: List[int] = field(default_factory=list)
    states: List[Tuple[int, int]] = field(default_factory=list)
    vis: List[List[int]] = field(default_factory=list)

    def segments(self, i: int) -> List[Tuple[int, int]]:
        lo, hi = self.seg_off[i], self.seg_off[i + 1]
        return list(zip(self.seg_chunk[lo:hi], self.seg_level[lo:hi]))


def _validate(pol: Policy, nodes: Sequence[Tuple[int, int]]) -> None:
    if pol.kind not in (CLEAN, SAME, PROG, TABLE):
        raise SelectionError("unknown policy kind")
    if pol.K < 1 or pol.W < 0 or pol.n_chunks < 0:
        raise SelectionError("K must be >= 1, W >= 0 and n_chunks >= 0")

    def check_shape(table, what, entries_ok):
        per_chunk = list(table) if pol.n_chunks > 0 else [table]
        if pol.n_chunks > 0 and len(per_chunk) != pol.n_chunks:
            raise SelectionError(f"{what} needs n_chunks x (K+1) x W entries")
        for t in per_chunk:
            if len(t) != pol.K + 1 or any(len(row) != pol.W for row in t):
                raise SelectionError(f"{what} must be (K+1) x W per chunk")
            if any(not entries_ok(int(v)) for row in t for v in row):
                raise SelectionError(f"{what} entries out of range")
    if pol.kind == TABLE:
        if pol.phi_table is None:
            raise SelectionError("table policy needs a phi table")
        check_shape(pol.phi_table, "phi table", lambda v: 0 <= v <= pol.K)
    if pol.r_mask is not None:
        check_shape(pol.r_mask, "r_mask", lambda v: True)
    seen = set()
    for c, j in nodes:
        if c < 0 or (pol.n_chunks > 0 and c >= pol.n_chunks) or not (0 <= j <= pol.K):
            raise SelectionError("node chunk must be in [0, n_chunks) and level in [0, K]")
        if (c, j) in seen:
            raise SelectionError("duplicate node in pack")
        seen.add((c, j))


def select(pol: Policy, nodes: Sequence[Tuple[int, int]]) -> Selection:
    """Selection table for a pack of nodes under ``pol`` (Eq. 4-5)."""
    nodes = [(int(c), int(j)) for c, j in nodes]
    _validate(pol, nodes)
    index_of = {node: i for i, node in enumerate(nodes)}
    sel = Selection(nodes=nodes)
    sel.seg_off.append(0)
    for i, (c, j) in enumerate(nodes):
        segs = []
        for r in range(min(pol.W, c), 0, -1):          # oldest history first
            if pol.selected(j, r, c):
                segs.append((c - r, pol.phi(j, r, c)))
        segs.append((c, j))                             # own chunk, own level
        for (sc, sl) in segs:
            sel.seg_chunk.append(sc)
            sel.seg_level.append(sl)
            sel.seg_src.append(index_of.get((sc, sl), -1))
        sel.seg_off.append(len(sel.seg_chunk))
    sel.states = sorted(set(zip(sel.seg_chunk, sel.seg_level)))
    pos = {s: k for k, s in enumerate(sel.states)}
    for i in range(len(nodes)):
        row = [0] * len(sel.states)
        for s in sel.segments(i):
            row[pos[s]] = 1
        sel.vis.append(row)
    return sel
