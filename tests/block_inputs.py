"""Seeded inputs of one DiT block over a pack, and the oracle's view of them.

CPU only (numpy): shared by the GPU block tests, which upload these exact
bf16 values, and by the CPU tests of the branch gates, which plant mistakes
in the oracle and check that the gates reject them.

Branch gates.  The block output is O(1) while its attention branch
a = o Wo^T is O(1e-3) at N(0, 0.02) weights, so block-level gates cannot see
the attention.  The branches are therefore compared where they are formed:
the rotated queries q and the attention output o that the block leaves in its
workspace, against the oracle's q and o of the same inputs, and the
attention branch itself as y - x of a block run with w_down = 0 and x scaled
by 2^-8 (exact in bf16), where the residual rounding of x' = x + a is small
against a.  Gate (the attention tolerances of the workload, with the
relative one that sees a dropped page): |d| <= 2e-2 max(1, |ref|) per
element, mean |d| <= 2e-3 + 2^-8 mean |ref|, and relative Frobenius error
<= 1e-2 per (node, head) -- per node for a.  The error model behind the
scaled terms: one bf16 rounding (round to nearest even, 8 significant bits)
moves a value v by at most 2^-8 |v| and by at most 2^-9 |v| on average, and
q and the cached K are stored after up to two roundings (qk-norm rounds the
raw projection, then the normalised one).  So on top of the attention
tolerances the gate allows two roundings of the values themselves.  o and a
are far below 1 (mean |ref| ~ 1e-2), where these are the plain attention
tolerances; q and K are O(1) (|q| ~ 5 at Wan shape).
"""
from __future__ import annotations

import contextlib
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

import oracle.block as oblock
from oracle.block import BlockShape, block_forward
from oracle.policy import policy as oracle_policy
from oracle.policy import select
from oracle.rope import chunk_positions, rope
from synth import (TAG_K, TAG_V, TAG_W_DOWN, TAG_W_O, TAG_W_QKV, TAG_W_UP, TAG_X, bf16_bits,
                   bf16_value, normal, normal_parallel)

BRANCH_MAX_ABS = 2e-2
BRANCH_MEAN_ABS = 2e-3
BRANCH_REL_FROB = 1e-2
X_SMALL = 2.0 ** -8      # input scale of the attention-branch case


def exact(bits: np.ndarray) -> np.ndarray:
    return bf16_value(bits).astype(np.float64)


def block_shape(geo) -> BlockShape:
    return BlockShape(geo.hidden, geo.heads, geo.head_dim, geo.mlp, geo.frames_per_chunk,
                      geo.grid_h, geo.grid_w, geo.rope_dims, geo.theta)


def weight_bits(geo, layer: int, seed: int, zero_down: bool = False) -> Dict[str, np.ndarray]:
    D, M = geo.hidden, geo.mlp
    gen = normal_parallel if D * M > 1 << 22 else normal
    w = {"w_qkv": gen((3 * D, D), (seed, TAG_W_QKV, layer), 0.02),
         "w_o": gen((D, D), (seed, TAG_W_O, layer), 0.02),
         "w_up": gen((M, D), (seed, TAG_W_UP, layer), 0.02),
         "w_down": gen((D, M), (seed, TAG_W_DOWN, layer), 0.02)}
    if zero_down:
        w["w_down"][:] = 0.0
    return {k: bf16_bits(v) for k, v in w.items()}


class BlockInputs:
    """x of every pack node, the block weights and the resident states' K/V
    (drawn unrotated; the cache rotates K on append, the oracle rotates them
    here), all as bf16 bit patterns plus their exact values."""

    def __init__(self, geo, kind: str, pack: Sequence[Tuple[int, int]],
                 resident: Sequence[Tuple[int, int]], seed: int = 0, x_scale: float = 1.0,
                 zero_down: bool = False):
        self.geo, self.kind, self.pack, self.seed = geo, kind, list(pack), seed
        self.resident = list(resident)
        big = geo.tokens_per_chunk * geo.hidden > 1 << 20
        self.gen = normal_parallel if big else normal
        self.kv_shape = (geo.tokens_per_chunk, geo.heads, geo.head_dim)
        self.res_bits, self.res_kv = {}, {}
        for st in self.resident:
            self._draw_state(st)
        xs = [self.gen((geo.tokens_per_chunk, geo.hidden), (seed, TAG_X) + tuple(st)) for st in self.pack]
        self.x_bits = bf16_bits(np.concatenate(xs) * np.float32(x_scale))
        xv = exact(self.x_bits)
        n = geo.tokens_per_chunk
        self.x = [xv[i * n:(i + 1) * n] for i in range(len(self.pack))]
        self.w_bits = weight_bits(geo, 0, seed, zero_down)
        self.w = {k: exact(v) for k, v in self.w_bits.items()}
        self.shape = block_shape(geo)

    def _draw_state(self, st):
        g = self.geo
        kb = bf16_bits(self.gen(self.kv_shape, (self.seed, TAG_K) + tuple(st)))
        vb = bf16_bits(self.gen(self.kv_shape, (self.seed, TAG_V) + tuple(st)))
        self.res_bits[st] = (kb, vb)
        pos = chunk_positions(st[0], g.frames_per_chunk, g.grid_h, g.grid_w)
        self.res_kv[st] = (rope(exact(kb), pos, g.rope_dims, g.theta), exact(vb))

    def resident_kv(self, st):
        if st not in self.res_kv:          # a state only a planted mistake reads
            self._draw_state(st)
        return self.res_kv[st]

    def selection(self):
        return select(oracle_policy(self.kind, self.geo.K, self.geo.W), self.pack)

    def oracle(self, rows=None, trace=None, sel=None, **options):
        return block_forward(sel or self.selection(), lambda i: self.x[i], self.w, self.resident_kv,
                             self.shape, rows=rows, trace=trace, **options)


# ----------------------------------------------------------- planted mistakes
class _EditedSelection:
    """A selection whose segment lists are edited (a planted mistake)."""

    def __init__(self, sel, edit):
        self.nodes, self._sel, self._edit = sel.nodes, sel, edit

    def segments(self, i):
        return self._edit(i, list(self._sel.segments(i)))


def drop_oldest_history(sel):
    return _EditedSelection(sel, lambda i, segs: segs[1:] if len(segs) > 1 else segs)


def oldest_level_off_by_one(sel, K):
    def edit(i, segs):
        if len(segs) < 2:
            return segs
        c, l = segs[0]
        return [(c, l + 1 if l < K else l - 1)] + segs[1:]
    return _EditedSelection(sel, edit)


@contextlib.contextmanager
def queries_without_rope():
    """The oracle's block with q left unrotated (keys still rotated)."""
    orig = oblock.project_q

    def unrotated(x, chunk, w_qkv, shp, rows=None, mod_row=None, g_q=None):
        x = np.asarray(x, dtype=np.float64)
        if rows is not None:
            x = x[rows]
        h = oblock.modulated_norm(x, mod_row, 0)
        q = h @ np.asarray(w_qkv, dtype=np.float64)[0:shp.hidden].T
        if g_q is not None:
            q = oblock.norm_gain(q, g_q)
        return q.reshape(-1, shp.heads, shp.head_dim)

    oblock.project_q = unrotated
    try:
        yield
    finally:
        oblock.project_q = orig


PLANTED = ("drop oldest history chunk", "oldest level off by one", "q without RoPE")


@contextlib.contextmanager
def _shared_projections():
    """project_kv memoised per (input array, chunk): the planted mistakes
    leave the pack's K/V unchanged, so the traces share one projection."""
    orig, memo = oblock.project_kv, {}

    def memoised(x, chunk, w_qkv, shp, mod_row=None, g_k=None):
        key = (id(x), chunk, id(w_qkv), id(mod_row), id(g_k))
        if key not in memo:
            memo[key] = (x, orig(x, chunk, w_qkv, shp, mod_row, g_k))
        return memo[key][1]

    oblock.project_kv = memoised
    try:
        yield
    finally:
        oblock.project_kv = orig


def traces_of(sel, x_of, weights, resident_kv, shp, K, rows, **options) -> Dict[str, dict]:
    """Oracle traces of one block ("exact", with its outputs under "y" and
    the pack's K/V under "kv") and of the block with each planted mistake,
    for the given output rows.  Arguments are block_forward's; ``options``
    its keywords (mod, qk_norm, cross)."""
    out = {}

    def run(s, tr):
        return block_forward(s, x_of, weights, resident_kv, shp, rows=rows, trace=tr, **options)

    with _shared_projections():
        out["exact"] = {}
        out["y"], out["kv"] = run(sel, out["exact"])
        for name in PLANTED:
            tr = {}
            if name == PLANTED[0]:
                run(drop_oldest_history(sel), tr)
            elif name == PLANTED[1]:
                run(oldest_level_off_by_one(sel, K), tr)
            else:
                with queries_without_rope():
                    run(sel, tr)
            out[name] = tr
    return out


def oracle_traces(inp: BlockInputs, rows, **options) -> Dict[str, dict]:
    """traces_of on a BlockInputs case."""
    return traces_of(inp.selection(), lambda i: inp.x[i], inp.w, inp.resident_kv, inp.shape, inp.geo.K,
                     rows, **options)


def planted_must_fail(traces: Dict[str, dict], keys=("o", "a")) -> Dict[str, float]:
    """Every planted mistake must fail the branch gate on o and a of every
    node that reads history (q without RoPE also on q); returns the smallest
    error/limit ratio per mistake."""
    exact_tr, worst = traces["exact"], {}
    for name in PLANTED:
        ks = keys + ("q",) if name == PLANTED[2] else keys
        ratios = [branch_ratio(traces[name][i][k], exact_tr[i][k]) for i in exact_tr for k in ks]
        worst[name] = min(ratios)
        assert worst[name] > 1.0, f"planted mistake '{name}' passes the branch gate ({worst[name]:.3g})"
    return worst


# --------------------------------------------------------------------- gates
def branch_errors(got: np.ndarray, want: np.ndarray):
    """(max |d| / max(1, |ref|), mean |d| scaled to the 2e-3 limit (see the
    module docstring), worst relative Frobenius error over the middle axis)
    of [N, H, d] arrays ([N, hidden] counts as one head)."""
    if got.ndim == 2:
        got, want = got[:, None, :], want[:, None, :]
    d = np.abs(got - want)
    rel = max(float(np.linalg.norm(got[:, h] - want[:, h]) / np.linalg.norm(want[:, h]))
              for h in range(want.shape[1]))
    mx = float((d / np.maximum(1.0, np.abs(want))).max())
    mean = float(d.mean()) * BRANCH_MEAN_ABS / (BRANCH_MEAN_ABS + 2.0 ** -8 * float(np.abs(want).mean()))
    return mx, mean, rel


def branch_ratio(got: np.ndarray, want: np.ndarray) -> float:
    """Worst error / limit over the three branch gates (<= 1 passes)."""
    mx, mean, rel = branch_errors(got, want)
    return max(mx / BRANCH_MAX_ABS, mean / BRANCH_MEAN_ABS, rel / BRANCH_REL_FROB)


def branch_gate(got: np.ndarray, want: np.ndarray, what: str) -> float:
    assert np.all(np.isfinite(got)), f"{what}: non-finite"
    r = branch_ratio(got, want)
    mx, mean, rel = branch_errors(got, want)
    assert r <= 1.0, f"{what}: max {mx:.3g} mean {mean:.3g} rel {rel:.3g} (ratio {r:.3g})"
    return r
