"""GPU parity of RoPE append, the DiT block and the sampler against the oracle.

Block outputs pass through seven bf16 roundings (normalised input, q/k/v,
attention output, residual stream, second norm, GELU output, final output).
Two of them land on the residual stream itself (x' = x + o Wo, then y), and a
bf16 rounding moves a value by half a spacing at most (2^-8 relative) and by
a quarter spacing on average (~2^-9 of the value over a binade); the others
are averaged over >= 256-term dot products.  Gates: elementwise
|gpu - oracle| <= 2e-2 * max(1, |oracle|), and
mean |gpu - oracle| <= 4e-3 * max(1, mean |oracle|) (two residual roundings
of ~2^-9 each, with margin).  The K/V the block writes into the cache use the
attention gates.
"""
import math

import numpy as np
import pytest

import paper_2609_22283_amd as sc
from oracle.block import BlockShape, block_forward, project_kv
from oracle.pipeline import sampler_step
from oracle.policy import policy as oracle_policy
from oracle.policy import select
from oracle.rope import chunk_positions, rope
from synth import (TAG_K, TAG_NOISE, TAG_V, TAG_W_DOWN, TAG_W_O, TAG_W_QKV, TAG_W_UP, TAG_X,
                   normal, normal_parallel)
from synth.configs import SHORT, SMALL, WAN, cfg4_prog

from gpu_cases import bf16_gates, from_device, sample_rows, to_device, torch_mod

pytestmark = pytest.mark.gpu


def read_pages(pool, geo, n_slots, slots, layer=0, dtype_bytes=2):
    """Pool pages of one state -> (K [tokens, H, d], V [tokens, H, d]) fp64."""
    torch = torch_mod()
    H, d, tpp = geo.heads, geo.head_dim, geo.tokens_per_page
    slot_elems = 2 * H * tpp * d
    view = pool.view(torch.bfloat16)
    ks, vs = [], []
    for s in slots:
        base = (layer * n_slots + s) * slot_elems
        page = from_device(view[base:base + slot_elems].clone())
        k = page[:H * tpp * d].reshape(H, tpp, d).transpose(1, 0, 2)
        v = page[H * tpp * d:].reshape(H, d, tpp).transpose(2, 0, 1)
        ks.append(k)
        vs.append(v)
    return np.concatenate(ks), np.concatenate(vs)


def make_rope(geo, max_frames=64):
    torch = torch_mod()
    nbytes = sc.sc_rope_table_bytes(geo.grid_h, geo.grid_w, geo.rope_dims, max_frames, geo.theta)
    table = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    return sc.sc_rope_table_build(table, geo.grid_h, geo.grid_w, geo.rope_dims, max_frames, geo.theta)


def test_append_with_rope_matches_oracle():
    torch = torch_mod()
    geo = SMALL
    n_slots = 12
    nbytes = sc.sc_cache_pool_bytes(1, geo.heads, geo.head_dim, geo.tokens_per_page,
                                    geo.frames_per_chunk, n_slots)
    pool = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
    cache = sc.sc_cache_create(pool, 1, geo.heads, geo.head_dim, geo.tokens_per_page,
                               geo.frames_per_chunk, n_slots)
    rp = make_rope(geo)
    shape = (geo.tokens_per_chunk, geo.heads, geo.head_dim)
    for st in [(0, 0), (5, 2)]:
        kd, kv = to_device(normal(shape, (1, TAG_K) + st), sc.SC_DTYPE_BF16)
        vd, vv = to_device(normal(shape, (1, TAG_V) + st), sc.SC_DTYPE_BF16)
        cache.append(0, st, kd, vd, rope=rp)
        torch.cuda.synchronize()
        k_got, v_got = read_pages(pool, geo, n_slots, cache.slots(st))
        pos = chunk_positions(st[0], geo.frames_per_chunk, geo.grid_h, geo.grid_w)
        k_want = rope(kv, pos, geo.rope_dims, geo.theta)
        assert np.array_equal(v_got, vv)                       # V moved, not changed
        err = np.abs(k_got - k_want)
        assert err.max() <= np.abs(k_want).max() * 2.0 ** -8 + 1e-6
    with pytest.raises(sc.ScError) as e:
        cache.append(0, (0, 0), kd, vd, rope=rp)
    assert e.value.code == sc.SC_EEXIST


def _weights(geo, layer, seed):
    D, M = geo.hidden, geo.mlp
    big = D * M > 1 << 22
    gen = normal_parallel if big else normal
    w = {"w_qkv": gen((3 * D, D), (seed, TAG_W_QKV, layer), 0.02),
         "w_o": gen((D, D), (seed, TAG_W_O, layer), 0.02),
         "w_up": gen((M, D), (seed, TAG_W_UP, layer), 0.02),
         "w_down": gen((D, M), (seed, TAG_W_DOWN, layer), 0.02)}
    dev, exact = {}, {}
    for k, v in w.items():
        dev[k], exact[k] = to_device(v, sc.SC_DTYPE_BF16)
    return dev, exact


def _mod_table(geo, seed):
    """Random per-level modulation [K+1][6][hidden] fp32 (gates around 1)."""
    m = np.stack([np.stack([normal((geo.hidden,), (seed, 30, j, r), 0.2) for r in range(6)])
                  for j in range(geo.K + 1)]).astype(np.float32)
    m[:, 2] += 1.0
    m[:, 5] += 1.0
    return m


class BlockCase:
    """One block over a pack.  Options: ``mod`` (host fp32 modulation table),
    ``qk`` (host fp32 qk-norm gains [2][hidden]), ``cross`` (a ConditionCase
    whose condition 0 every node reads)."""

    def __init__(self, geo, kind, pack, resident, seed=0, mod=None, qk=None, cross=None):
        torch = torch_mod()
        self.mod = mod                                   # host fp32 table or None
        self.qk, self.cross = qk, cross
        self.geo, self.kind, self.pack = geo, kind, pack
        ppc, tpp = geo.frames_per_chunk, geo.tokens_per_page
        n_slots = (len(resident) + len(pack) + 2) * ppc
        nbytes = sc.sc_cache_pool_bytes(1, geo.heads, geo.head_dim, tpp, ppc, n_slots)
        self.pool = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
        self.n_slots = n_slots
        self.cache = sc.sc_cache_create(self.pool, 1, geo.heads, geo.head_dim, tpp, ppc, n_slots)
        self.rope = make_rope(geo)
        big = geo.tokens_per_chunk * geo.hidden > 1 << 20
        gen = normal_parallel if big else normal
        shape = (geo.tokens_per_chunk, geo.heads, geo.head_dim)
        self.res_kv, keep = {}, []
        for st in resident:
            kd, kv = to_device(gen(shape, (seed, TAG_K) + st), sc.SC_DTYPE_BF16)
            vd, vv = to_device(gen(shape, (seed, TAG_V) + st), sc.SC_DTYPE_BF16)
            self.cache.append(0, st, kd, vd, rope=self.rope)
            pos = chunk_positions(st[0], ppc, geo.grid_h, geo.grid_w)
            self.res_kv[st] = (rope(kv, pos, geo.rope_dims, geo.theta), vv)
            keep += [kd, vd]
        torch.cuda.synchronize()
        del keep
        self.sel = sc.sc_selection_build(kind, geo.K, geo.W, pack)
        self.plan = sc.sc_plan_build(self.sel, self.cache)
        xs = [gen((geo.tokens_per_chunk, geo.hidden), (seed, TAG_X) + st) for st in pack]
        self.x_dev, xv = to_device(np.concatenate(xs), sc.SC_DTYPE_BF16)
        n = geo.tokens_per_chunk
        self.x = [xv[i * n:(i + 1) * n] for i in range(len(pack))]
        self.w_dev, self.w = _weights(geo, 0, seed)
        self.mod_dev = None if mod is None else torch.from_numpy(mod).cuda()
        self.qk_dev = None if qk is None else torch.from_numpy(np.ascontiguousarray(qk)).cuda()
        ca = None if cross is None else cross.cross_attn(len(pack), geo.tokens_per_chunk)
        self.bw = sc.BlockWeights(geo.hidden, geo.heads, geo.head_dim, geo.mlp, self.w_dev["w_qkv"],
                                  self.w_dev["w_o"], self.w_dev["w_up"], self.w_dev["w_down"],
                                  mod=self.mod_dev, qk_norm=self.qk_dev, cross=ca)
        T = len(pack) * n
        self.ws_bytes = sc.sc_block_workspace_bytes(self.bw, T)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device="cuda")
        self.shape = BlockShape(geo.hidden, geo.heads, geo.head_dim, geo.mlp, geo.frames_per_chunk,
                                geo.grid_h, geo.grid_w, geo.rope_dims, geo.theta)

    def run(self):
        torch = torch_mod()
        sc.sc_block_forward(self.bw, self.cache, 0, self.plan, self.x_dev, self.rope, self.ws,
                            self.ws_bytes)
        torch.cuda.synchronize()
        out = from_device(self.x_dev)
        n = self.geo.tokens_per_chunk
        return [out[i * n:(i + 1) * n] for i in range(len(self.pack))]

    def oracle(self, rows=None):
        sel = select(oracle_policy(self.kind, self.geo.K, self.geo.W), self.pack)
        qk = None if self.qk is None else tuple(self.qk.astype(np.float64))
        cross = None if self.cross is None else self.cross.oracle_dict(0)
        return block_forward(sel, lambda i: self.x[i], self.w, self.res_kv.__getitem__, self.shape,
                             rows=rows, mod=self.mod, qk_norm=qk, cross=cross)


def block_gate(got, want, what, roundings=7):
    """Block output against the fp64 oracle: |d| <= 2e-2 max(1, |ref|) per
    element and mean |d| <= 4e-3 max(1, mean |ref|), set for the plain
    block's seven bf16 roundings (two on the residual stream).  A path with
    more roundings scales both limits by sqrt(roundings / 7): independent
    rounding errors add in quadrature."""
    assert np.all(np.isfinite(got)), what
    scale = math.sqrt(roundings / 7)
    d = np.abs(got - want)
    lim = 2e-2 * scale * np.maximum(1.0, np.abs(want))
    worst = float((d / lim).max())
    assert worst <= 1.0, f"{what}: worst error/limit {worst:.3g}"
    mean_lim = 4e-3 * scale * max(1.0, float(np.abs(want).mean()))
    assert d.mean() <= mean_lim, f"{what}: mean abs {d.mean():.3g}"
    return worst, float(d.mean())


SMALL_BLOCK_PACKS = [
    ("prog", [(6, 1), (7, 2), (8, 3), (9, 4)], [(c, 0) for c in range(6)]),
    ("prog", [(6, 0), (7, 1), (8, 2), (9, 3), (10, 4)], [(c, 0) for c in range(6)]),
    ("same", [(6 + i, 3) for i in range(4)], [(c, 3) for c in range(6)]),
    ("clean", [(6, 4)], [(c, 0) for c in range(6)]),
]


@pytest.mark.parametrize("kind,pack,resident", SMALL_BLOCK_PACKS)
def test_small_block(kind, pack, resident):
    case = BlockCase(SMALL, kind, pack, resident, seed=11)
    got = case.run()
    want, new_kv = case.oracle()
    for i in range(len(pack)):
        block_gate(got[i], want[i], f"{kind} node {pack[i]}")
        k_got, v_got = read_pages(case.pool, SMALL, case.n_slots, case.cache.slots(pack[i]))
        bf16_gates(k_got, new_kv[i][0], "cached K")
        bf16_gates(v_got, new_kv[i][1], "cached V")
    with pytest.raises(sc.ScError) as e:                      # K/V of the pack already written
        case.run()
    assert e.value.code == sc.SC_EEXIST


@pytest.mark.parametrize("kind,pack,resident", SMALL_BLOCK_PACKS[:2])
def test_small_block_level_modulation(kind, pack, resident):
    """Noise-level conditioning: per-level shift/scale after both RMSNorms
    and gates on both residual branches, each node using its own level's
    row."""
    case = BlockCase(SMALL, kind, pack, resident, seed=15, mod=_mod_table(SMALL, 15))
    got = case.run()
    want, new_kv = case.oracle()
    for i in range(len(pack)):
        block_gate(got[i], want[i], f"modulated {kind} node {pack[i]}")
        k_got, v_got = read_pages(case.pool, SMALL, case.n_slots, case.cache.slots(pack[i]))
        bf16_gates(k_got, new_kv[i][0], "cached K (modulated)")
        bf16_gates(v_got, new_kv[i][1], "cached V (modulated)")


def test_short_block_prog():
    """A progressive pack of one-frame, 96-token chunks (the attention's
    128-query work-group shape inside the block)."""
    pack = [(6, 0), (7, 1), (8, 2), (9, 3), (10, 4)]
    case = BlockCase(SHORT, "prog", pack, [(c, 0) for c in range(6)], seed=13)
    got = case.run()
    want, _ = case.oracle()
    for i in range(len(pack)):
        block_gate(got[i], want[i], f"short node {pack[i]}")


def test_block_rejects_level_beyond_modulation_table():
    mod = _mod_table(SMALL, 16)[:3]                       # levels 0..2 only
    case = BlockCase(SMALL, "prog", [(6, 1), (7, 2), (8, 3)], [(c, 0) for c in range(6)], seed=16,
                     mod=mod)
    with pytest.raises(sc.ScError) as e:
        case.run()
    assert e.value.code == sc.SC_EINVAL


def test_block_rejects_oversized_pack():
    """More pack nodes than the QKV epilogue's node table holds (64) is
    refused before any launch, leaving the pack's pages unwritten."""
    import dataclasses
    geo = dataclasses.replace(SHORT, W=0)                    # each node reads only itself
    case = BlockCase(geo, "clean", [(c, 4) for c in range(65)], [], seed=14)
    with pytest.raises(sc.ScError) as e:
        case.run()
    assert e.value.code == sc.SC_EUNSUPPORTED


# Wan-shaped packs of 4, 5 and 1 nodes (T = 18720, 23400, 4680 tokens).
# The GEMMs pick their token-tile width from T, so between them these run
# every width: QKV on 192 / 256 / 192 tokens, the MLP-up GEMM on 256, and the
# out-projection and MLP-down GEMMs on 256 / 192 / 128.
WAN_BLOCK_PACKS = [
    ("prog", cfg4_prog(False).pack, cfg4_prog(False).resident),
    ("prog", cfg4_prog(True).pack, cfg4_prog(True).resident),
    ("clean", [(6, 4)], [(c, 0) for c in range(6)]),
]


@pytest.mark.parametrize("kind,pack,resident", WAN_BLOCK_PACKS, ids=["4-node", "5-node", "1-node"])
def test_wan_block_sampled_rows(kind, pack, resident):
    case = BlockCase(WAN, kind, pack, resident, seed=12)
    got = case.run()
    rows = sample_rows(WAN.tokens_per_chunk, 24, seed=3)
    want, _ = case.oracle(rows=rows)
    for i in range(len(pack)):
        block_gate(got[i][rows], want[i], f"wan {kind} node {pack[i]}")


def test_wan_width_block_1800_tokens():
    """Wan widths (hidden 1536, 12 heads, MLP 8960) over one 1800-token chunk
    (one 15 x 120 frame) with one resident state: the MLP-up GEMM runs on
    192-token tiles here (350 tiles, 2 rounds at 0.75 of a tile, against 280
    tiles in 2 full rounds at 256), as do the QKV GEMM, and the out/down GEMMs
    on 128-token tiles."""
    import dataclasses
    geo = dataclasses.replace(WAN, grid_h=15, grid_w=120, frames_per_chunk=1)
    case = BlockCase(geo, "clean", [(1, 4)], [(0, 0)], seed=17)
    got = case.run()
    rows = sample_rows(geo.tokens_per_chunk, 32, seed=5)
    want, _ = case.oracle(rows=rows)
    block_gate(got[0][rows], want[0], "wan-width 1800-token node (1, 4)")


def test_sampler_matches_oracle():
    torch = torch_mod()
    nodes = [(3, 0), (4, 1), (5, 2), (6, 3), (7, 4)]
    t = (0.0, 5 / 8, 5 / 6, 15 / 16, 1.0)
    E = 4680 * 16
    y = normal((len(nodes), E), (1, TAG_X))
    xi = normal((len(nodes), E), (1, TAG_NOISE))
    yd, yv = to_device(y, sc.SC_DTYPE_BF16)
    nd, nv = to_device(xi, sc.SC_DTYPE_BF16)
    out = torch.full_like(yd, 7.0)
    sc.sc_sampler_step(nodes, t, 4, out, yd, nd, E)
    torch.cuda.synchronize()
    got = from_device(out)
    for i, (c, j) in enumerate(nodes):
        if j == 0:
            assert np.all(got[i] == 7.0)
            continue
        want = sampler_step(yv[i], nv[i], t[j - 1])
        assert np.abs(got[i] - want).max() <= np.abs(want).max() * 2.0 ** -8 + 1e-6
