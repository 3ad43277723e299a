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
attention gates.  Without level modulation both norms are folded into the
GEMMs that follow them and their outputs are never rounded, so that block has
five roundings; the gates keep the count of seven.
"""
import math

import numpy as np
import pytest

import paper_2609_22283_amd as sc
from oracle.pipeline import sampler_step
from oracle.rope import chunk_positions, rope
from synth import TAG_K, TAG_NOISE, TAG_V, TAG_X, bf16_bits, normal
from synth.configs import SHORT, SMALL, WAN, cfg3_same, cfg4_prog

from block_inputs import X_SMALL, BlockInputs, branch_gate, exact, oracle_traces, planted_must_fail
from gpu_cases import bf16_gates, bits_to_device, from_device, sample_rows, to_device, torch_mod

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


def _mod_table(geo, seed):
    """Random per-level modulation [K+1][6][hidden] fp32 (gates around 1)."""
    m = np.stack([np.stack([normal((geo.hidden,), (seed, 30, j, r), 0.2) for r in range(6)])
                  for j in range(geo.K + 1)]).astype(np.float32)
    m[:, 2] += 1.0
    m[:, 5] += 1.0
    return m


class BlockCase:
    """One block over a pack, on the inputs of ``BlockInputs`` (the same
    bf16 values the oracle reads).  Options: ``mod`` (host fp32 modulation
    table), ``qk`` (host fp32 qk-norm gains [2][hidden]), ``cross`` (a
    ConditionCase whose condition 0 every node reads), ``x_scale`` and
    ``zero_down`` (the attention-branch case: x scaled by a power of two and
    w_down = 0)."""

    def __init__(self, geo, kind, pack, resident, seed=0, mod=None, qk=None, cross=None, x_scale=1.0,
                 zero_down=False):
        torch = torch_mod()
        self.inp = BlockInputs(geo, kind, pack, resident, seed, x_scale, zero_down)
        self.mod = mod                                   # host fp32 table or None
        self.qk, self.cross = qk, cross
        self.geo, self.kind, self.pack = geo, kind, list(pack)
        ppc, tpp = geo.frames_per_chunk, geo.tokens_per_page
        n_slots = (len(resident) + len(pack) + 2) * ppc
        nbytes = sc.sc_cache_pool_bytes(1, geo.heads, geo.head_dim, tpp, ppc, n_slots)
        self.pool = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
        self.n_slots = n_slots
        self.cache = sc.sc_cache_create(self.pool, 1, geo.heads, geo.head_dim, tpp, ppc, n_slots)
        self.rope = make_rope(geo)
        keep = []
        for st in resident:                              # K rotated by the cache on append
            kd, vd = (bits_to_device(b) for b in self.inp.res_bits[tuple(st)])
            self.cache.append(0, st, kd, vd, rope=self.rope)
            keep += [kd, vd]
        torch.cuda.synchronize()
        del keep
        self.res_kv = self.inp.res_kv
        self.sel = sc.sc_selection_build(kind, geo.K, geo.W, pack)
        self.plan = sc.sc_plan_build(self.sel, self.cache)
        self.x_dev = bits_to_device(self.inp.x_bits)
        self.x = self.inp.x
        self.w_dev = {k: bits_to_device(v) for k, v in self.inp.w_bits.items()}
        self.w = self.inp.w
        self.mod_dev = None if mod is None else torch.from_numpy(mod).cuda()
        self.qk_dev = None if qk is None else torch.from_numpy(np.ascontiguousarray(qk)).cuda()
        ca = None if cross is None else cross.cross_attn(len(pack), geo.tokens_per_chunk)
        self.bw = sc.BlockWeights(geo.hidden, geo.heads, geo.head_dim, geo.mlp, self.w_dev["w_qkv"],
                                  self.w_dev["w_o"], self.w_dev["w_up"], self.w_dev["w_down"],
                                  mod=self.mod_dev, qk_norm=self.qk_dev, cross=ca)
        self.T = len(pack) * geo.tokens_per_chunk
        self.ws_bytes = sc.sc_block_workspace_bytes(self.bw, self.T)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device="cuda")
        self.shape = self.inp.shape

    def run(self):
        torch = torch_mod()
        sc.sc_block_forward(self.bw, self.cache, 0, self.plan, self.x_dev, self.rope, self.ws,
                            self.ws_bytes)
        torch.cuda.synchronize()
        out = from_device(self.x_dev)
        n = self.geo.tokens_per_chunk
        return [out[i * n:(i + 1) * n] for i in range(len(self.pack))]

    def views(self):
        """The block's rotated q and attention output o from its workspace,
        per node, as [Nq, H, d] fp64 (after run())."""
        qo, oo = sc.sc_block_workspace_views(self.bw, self.T)
        g, n = self.geo, self.geo.tokens_per_chunk
        out = []
        for off in (qo, oo):
            t = self.ws[off:off + self.T * g.hidden * 2].view(torch_mod().bfloat16)
            a = from_device(t).reshape(len(self.pack), n, g.heads, g.head_dim)
            out.append([a[i] for i in range(len(self.pack))])
        return out

    def oracle_options(self):
        qk = None if self.qk is None else tuple(self.qk.astype(np.float64))
        cross = None if self.cross is None else self.cross.oracle_dict(0)
        return {"mod": self.mod, "qk_norm": qk, "cross": cross}

    def oracle(self, rows=None, trace=None):
        return self.inp.oracle(rows, trace, **self.oracle_options())


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


def test_small_block_extreme_rows():
    """Rows at the ends of the RMSNorms' range, which the plain block folds
    into its GEMMs as per-token factors: an all-zero input row (its factor
    is 1 / sqrt(eps) = 1000 and every projection of it is zero) and a row
    2^12 times larger than the others (exact in bf16; its normalised rows
    equal the unscaled row's), through the block and its cached K/V,
    against the oracle on the same values."""
    kind, pack, resident = SMALL_BLOCK_PACKS[0]
    case = BlockCase(SMALL, kind, pack, resident, seed=19)
    n = SMALL.tokens_per_chunk
    bits = case.inp.x_bits.copy()
    bits[3] = 0                                                # node 0, row 3
    bits[n + 5] = bf16_bits(exact(bits[n + 5]) * 4096.0)       # node 1, row 5
    xv = exact(bits)
    case.inp.x_bits = bits
    case.inp.x = case.x = [xv[i * n:(i + 1) * n] for i in range(len(pack))]
    case.x_dev = bits_to_device(bits)
    got = case.run()
    want, new_kv = case.oracle()
    assert np.abs(want[1][5]).max() > 1000.0                   # the large row stays large
    for i in range(len(pack)):
        block_gate(got[i], want[i], f"extreme rows, node {pack[i]}")
        k_got, v_got = read_pages(case.pool, SMALL, case.n_slots, case.cache.slots(pack[i]))
        bf16_gates(k_got, new_kv[i][0], "cached K (extreme rows)")
        bf16_gates(v_got, new_kv[i][1], "cached V (extreme rows)")
    k0, v0 = read_pages(case.pool, SMALL, case.n_slots, case.cache.slots(pack[0]))
    assert not np.any(k0[3]) and not np.any(v0[3])            # the zero row's K and V are zero


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


def check_branches(case, got, rows, what, options=None, small_x=False):
    """The block's branches against the oracle's trace of the same inputs:
    the rotated q and attention output o read from the workspace, and for
    the small-x case (w_down = 0) the attention branch y - x (gated by
    gate_a when modulated); the pack's K/V written into the cache.  The
    oracle with each planted mistake must fail the same gates (checked on
    the CPU, on these inputs).  Returns the worst error/limit ratio."""
    tr = oracle_traces(case.inp, rows, **(options or {}))
    planted_must_fail(tr)
    q_got, o_got = case.views()
    sel = slice(None) if rows is None else rows
    worst = 0.0
    for i, node in enumerate(case.pack):
        t = tr["exact"][i]
        worst = max(worst, branch_gate(q_got[i][sel], t["q"], f"{what} node {node}: q"))
        worst = max(worst, branch_gate(o_got[i][sel], t["o"], f"{what} node {node}: o"))
        if small_x:
            a = t["a"]
            if case.mod is not None:
                a = case.mod[node[1], 2] * a
            worst = max(worst, branch_gate(got[i][sel] - case.x[i][sel], a,
                                           f"{what} node {node}: y - x (attention branch)"))
        else:
            block_gate(got[i][sel], tr["y"][i], f"{what} node {node}: block output")
        k_got, v_got = read_pages(case.pool, case.geo, case.n_slots, case.cache.slots(node))
        worst = max(worst, branch_gate(k_got[sel], tr["kv"][i][0][sel], f"{what} node {node}: cached K"))
        worst = max(worst, branch_gate(v_got[sel], tr["kv"][i][1][sel], f"{what} node {node}: cached V"))
    return worst


@pytest.mark.parametrize("small_x", [False, True], ids=["x", "small-x"])
@pytest.mark.parametrize("kind,pack,resident", SMALL_BLOCK_PACKS, ids=["prog4", "prog5", "same", "clean"])
def test_small_block_branches(kind, pack, resident, small_x):
    """q, o, the attention branch and the cached K/V at small shapes, every
    row (Eq. 6 through the block: the in-pack pages written by the QKV
    epilogue are read by the attention in the same forward)."""
    case = BlockCase(SMALL, kind, pack, resident, seed=11, x_scale=X_SMALL if small_x else 1.0,
                     zero_down=small_x)
    got = case.run()
    check_branches(case, got, None, f"small {kind}", small_x=small_x)


@pytest.mark.parametrize("use_qk", [False, True], ids=["mod", "mod+qk-norm"])
def test_small_block_branches_modulated(use_qk):
    """The attention branch with level modulation (its gate_a) and qk-norm
    (q and k normalised over the hidden width before RoPE)."""
    from gpu_cases import gains
    qk = np.stack([gains(SMALL.hidden, (18, 45, 0)), gains(SMALL.hidden, (18, 45, 1))]) if use_qk else None
    case = BlockCase(SMALL, *SMALL_BLOCK_PACKS[1], seed=18, mod=_mod_table(SMALL, 18), qk=qk,
                     x_scale=X_SMALL, zero_down=True)
    got = case.run()
    check_branches(case, got, None, "small modulated", case.oracle_options(), small_x=True)


def test_block_error_leaves_pack_unwritten():
    """A block refused before its launches (an MLP width the GEMMs do not
    support) leaves the pack unwritten; a two-layer stack whose second layer
    is refused leaves the first layer unwritten too, and runs again once the
    weights are fixed."""
    torch = torch_mod()
    geo, (kind, pack, resident) = SMALL, SMALL_BLOCK_PACKS[0]
    case = BlockCase(geo, kind, pack, resident, seed=19)
    w = case.w_dev
    bad = sc.BlockWeights(geo.hidden, geo.heads, geo.head_dim, 320, w["w_qkv"], w["w_o"], w["w_up"],
                          w["w_down"])
    with pytest.raises(sc.ScError) as e:
        sc.sc_block_forward(bad, case.cache, 0, case.plan, case.x_dev, case.rope, case.ws, case.ws_bytes)
    assert e.value.code == sc.SC_EUNSUPPORTED
    assert not any(case.cache.contains(st, 0) for st in pack)
    # two layers: the first runs, the second is refused
    ppc, tpp = geo.frames_per_chunk, geo.tokens_per_page
    n_slots = (len(resident) + len(pack) + 2) * ppc
    pool = torch.full((sc.sc_cache_pool_bytes(2, geo.heads, geo.head_dim, tpp, ppc, n_slots),), 0xFF,
                      dtype=torch.uint8, device="cuda")
    cache = sc.sc_cache_create(pool, 2, geo.heads, geo.head_dim, tpp, ppc, n_slots)
    for layer in range(2):
        for st in resident:
            kd, vd = (bits_to_device(b) for b in case.inp.res_bits[tuple(st)])
            cache.append(layer, st, kd, vd, rope=case.rope)
    plan = sc.sc_plan_build(sc.sc_selection_build(kind, geo.K, geo.W, pack), cache)
    x = case.x_dev.clone()
    with pytest.raises(sc.ScError) as e:
        sc.sc_stack_forward([case.bw, bad], cache, plan, x, case.rope, case.ws, case.ws_bytes)
    assert e.value.code == sc.SC_EUNSUPPORTED
    assert not any(cache.contains(st, l) for st in pack for l in range(2))
    x.copy_(case.x_dev)
    sc.sc_stack_forward([case.bw, case.bw], cache, plan, x, case.rope, case.ws, case.ws_bytes)
    torch.cuda.synchronize()
    assert all(cache.contains(st, l) for st in pack for l in range(2))
    assert np.all(np.isfinite(from_device(x)))


# Wan-shaped packs: progressive diagonals of 4 and 5 nodes (T = 18720, 23400
# tokens), the same-level pack of 4 (level 2) and one clean node (4680).
# The GEMMs pick their token-tile width from T, so between them these run
# every width: QKV on 192 / 256 / 192 tokens, the MLP-up GEMM on 256, and the
# out-projection and MLP-down GEMMs on 256 / 192 / 128.
WAN_BLOCK_PACKS = [
    ("prog", cfg4_prog(False).pack, cfg4_prog(False).resident),
    ("prog", cfg4_prog(True).pack, cfg4_prog(True).resident),
    ("same", cfg3_same(2).pack, cfg3_same(2).resident),
    ("clean", [(6, 4)], [(c, 0) for c in range(6)]),
]


@pytest.mark.parametrize("kind,pack,resident", WAN_BLOCK_PACKS, ids=["4-node", "5-node", "same-4-node",
                                                                     "1-node"])
def test_wan_block_sampled_rows(kind, pack, resident):
    """Wan shape, sampled rows: block output, q, o and the cached K/V."""
    case = BlockCase(WAN, kind, pack, resident, seed=12)
    got = case.run()
    rows = sample_rows(WAN.tokens_per_chunk, 24, seed=3)
    check_branches(case, got, rows, f"wan {kind}")


def test_wan_block_attention_branch():
    """Wan shape, x of scale 2^-8 and w_down = 0: y - x is the attention
    branch o Wo^T of each node of the progressive diagonal."""
    case = BlockCase(WAN, "prog", cfg4_prog(False).pack, cfg4_prog(False).resident, seed=12,
                     x_scale=X_SMALL, zero_down=True)
    got = case.run()
    rows = sample_rows(WAN.tokens_per_chunk, 24, seed=4)
    check_branches(case, got, rows, "wan small-x", small_x=True)


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
