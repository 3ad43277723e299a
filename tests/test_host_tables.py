"""C ABI host core vs the oracle, on the CPU (no kernel launches).

Selection tables, visibility and plan tables (page slots under the
lowest-free-first allocator) must match the oracle bit for bit; error codes
must match the oracle's failures.  Also checks that the library exports every
function the headers under include/ declare.
"""
import os
import random
import re

import pytest

import paper_2609_22283_amd as sc
from oracle.plan import CacheModel, PlanError, build_plan
from oracle.policy import Policy, SelectionError, policy, select

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_header_symbols_exported():
    declared = set()
    inc = os.path.join(ROOT, "include")
    for name in sorted(os.listdir(inc)):
        if name.endswith(".h"):
            with open(os.path.join(inc, name)) as f:
                declared |= set(re.findall(r"\b(sc_[a-z_0-9]+)\s*\(", f.read()))
    assert declared == set(sc.EXPORTED_SYMBOLS)
    for name in declared:
        assert hasattr(sc.lib, name), name
    assert sc.sc_abi_version() == sc.ABI_VERSION == 7


def _random_pack(rnd, K, max_chunk=9, max_n=6):
    cand = [(c, j) for c in range(max_chunk) for j in range(K + 1)]
    return rnd.sample(cand, rnd.randint(1, min(max_n, len(cand))))


def _oracle_policy(kind, K, W, phi, mask):
    return Policy({"clean": 0, "same": 1, "prog": 2, "table": 3}[kind], K, W, phi, mask)


def test_selection_tables_bit_exact():
    rnd = random.Random(1)
    for trial in range(400):
        K, W = rnd.randint(1, 6), rnd.randint(0, 7)
        kind = rnd.choice(["clean", "same", "prog", "table"])
        phi = [[rnd.randint(0, K) for _ in range(W)] for _ in range(K + 1)] if kind == "table" else None
        mask = None
        if rnd.random() < 0.3:
            mask = [[rnd.randint(0, 1) for _ in range(W)] for _ in range(K + 1)]
        pack = _random_pack(rnd, K)
        want = select(_oracle_policy(kind, K, W, phi, mask), pack)
        got = sc.sc_selection_build(kind, K, W, pack, phi_table=phi, r_mask=mask)
        off, ch, lv, src = got.tables()
        assert off == want.seg_off and ch == want.seg_chunk
        assert lv == want.seg_level and src == want.seg_src
        states, vis = got.visibility()
        assert states == want.states and vis == want.vis


@pytest.mark.parametrize("bad", [
    dict(kind="prog", K=0, W=2, pack=[(0, 0)]),
    dict(kind="prog", K=4, W=-1, pack=[(0, 0)]),
    dict(kind="prog", K=4, W=2, pack=[(0, 5)]),
    dict(kind="prog", K=4, W=2, pack=[(-1, 1)]),
    dict(kind="prog", K=4, W=2, pack=[(1, 1), (1, 1)]),
    dict(kind="table", K=2, W=2, pack=[(1, 1)], phi=[[0, 3], [0, 0], [0, 0]]),
    dict(kind=7, K=2, W=2, pack=[(1, 1)]),
])
def test_selection_errors(bad):
    with pytest.raises(sc.ScError) as e:
        sc.sc_selection_build(bad["kind"], bad["K"], bad["W"], bad["pack"], phi_table=bad.get("phi"))
    assert e.value.code == sc.SC_EINVAL
    if isinstance(bad["kind"], str):
        with pytest.raises(SelectionError):
            select(_oracle_policy(bad["kind"], bad["K"], bad["W"], bad.get("phi"), None), bad["pack"])


def _host_cache(n_slots, ppc, tpp=16):
    # a fake device address: no kernel is launched by plan building
    return sc.sc_cache_create(0x100000, 1, 2, 128, tpp, ppc, n_slots)


def test_plan_tables_and_allocator_bit_exact():
    """Random sequences of plans and releases: page lists, slots, frames and
    error codes equal the oracle's cache model step by step."""
    rnd = random.Random(2)
    for trial in range(60):
        K, W, ppc = rnd.randint(1, 4), rnd.randint(0, 4), rnd.randint(1, 3)
        n_slots = rnd.randint(4, 60)
        cache = _host_cache(n_slots, ppc)
        model = CacheModel(n_slots=n_slots, pages_per_chunk=ppc)
        for step in range(25):
            if model.slots and rnd.random() < 0.3:
                st = rnd.choice(sorted(model.slots))
                model.release(st)
                cache.release(st)
                continue
            kind = rnd.choice(["clean", "same", "prog"])
            pack = _random_pack(rnd, K, max_chunk=7, max_n=4)
            sel_o = select(policy(kind, K, W), pack)
            sel_c = sc.sc_selection_build(kind, K, W, pack)
            try:
                want = build_plan(sel_o, model, 16)
                err = None
            except PlanError as e:
                err = e.code
            if err is not None:
                with pytest.raises(sc.ScError) as e:
                    sc.sc_plan_build(sel_c, cache)
                assert e.value.code == {"EUNAVAILABLE": sc.SC_EUNAVAILABLE,
                                        "ECAPACITY": sc.SC_ECAPACITY}[err]
                continue
            got = sc.sc_plan_build(sel_c, cache)
            off, slot, tok, frame = got.tables()
            assert off == want.page_off and slot == want.page_slot
            assert tok == want.page_tokens and frame == want.page_frame
            for st in model.slots:
                assert cache.slots(st) == model.slots[st]
            assert cache.free_slot_count() == len(model.free_slots())


def test_worked_example_through_abi():
    """Sec. 3.3, K = 3 round two, through the C ABI."""
    for kind, expect in [("same", ((0, 3), -1)), ("prog", ((0, 2), 0)), ("clean", None)]:
        cache = _host_cache(16, 1)
        sc.sc_plan_build(sc.sc_selection_build("same", 3, 0, [(0, 3)]), cache)  # (0,3) cached
        sel = sc.sc_selection_build(kind, 3, 1, [(0, 2), (1, 3)])
        off, ch, lv, src = sel.tables()
        if expect is None:
            with pytest.raises(sc.ScError) as e:
                sc.sc_plan_build(sel, cache)
            assert e.value.code == sc.SC_EUNAVAILABLE
            continue
        g = off[1]
        assert (ch[g], lv[g]) == expect[0] and src[g] == expect[1]
        sc.sc_plan_build(sel, cache)


def test_cache_errors_without_device():
    cache = _host_cache(4, 2)
    with pytest.raises(sc.ScError) as e:
        cache.release((3, 3))
    assert e.value.code == sc.SC_ENOTFOUND
    with pytest.raises(sc.ScError) as e:
        cache.slots((3, 3))
    assert e.value.code == sc.SC_ENOTFOUND
    sc.sc_plan_build(sc.sc_selection_build("prog", 4, 0, [(0, 4), (1, 4)]), cache)
    assert cache.free_slot_count() == 0
    with pytest.raises(sc.ScError) as e:
        sc.sc_plan_build(sc.sc_selection_build("prog", 4, 0, [(2, 4)]), cache)
    assert e.value.code == sc.SC_ECAPACITY
    assert cache.contains((0, 4)) and not cache.contains((0, 4), 0)
    with pytest.raises(sc.ScError) as e:
        sc.sc_cache_create(0x1000, 1, 2, 128, 12, 2, 4)         # tokens_per_page % 8 != 0
    assert e.value.code == sc.SC_EINVAL
    with pytest.raises(sc.ScError) as e:
        sc.sc_cache_create(0x1000, 1, 2, 96, 16, 2, 4)          # head_dim 96
    assert e.value.code == sc.SC_EUNSUPPORTED
    assert sc.sc_cache_pool_bytes(2, 12, 128, 1560, 3, 10) == 2 * 10 * 2 * 12 * 1560 * 128 * 2


def test_stale_plan_detected_on_cpu():
    """A plan whose slot was released must not reach a kernel: sc_attention
    fails with SC_ESTALE before launching anything."""
    cache = _host_cache(8, 1)
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(0, 0)]), cache)
    plan = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 1, [(1, 4)]), cache)
    cache.release((0, 0))
    with pytest.raises(sc.ScError) as e:
        sc.sc_attention(plan, cache, 0, 0x1000, 0x2000, 0.125)
    assert e.value.code == sc.SC_ESTALE
    plan2 = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(2, 4)]), cache)
    with pytest.raises(sc.ScError) as e:                       # reserved but never written
        sc.sc_attention(plan2, cache, 0, 0x1000, 0x2000, 0.125)
    assert e.value.code == sc.SC_EUNAVAILABLE


def test_attention_workspace_size():
    """Workspace of the bf16 attention: units (head, node, query tile) that
    fill whole rounds of the CUs' work-group slots run whole; when units are
    long (a mean of at least 2048 keys, 32 key tiles of 64) the remaining
    units are cut into S pieces, each leaving a partial (one row per query of
    the tile: 128 fp32 outputs plus max and sum).  Nodes of at most 64
    queries use 64-query tiles with 32-key tiles (1024 slots), of at most 128
    128-query tiles (512 slots), larger ones 256-query tiles (256 slots), the
    last two with 64-key tiles.  S minimises the tail's rounds plus a
    per-piece cost of two key tiles, within 1024 pieces and the shortest
    node's key tiles.  No workspace for fp32 caches or when nothing is cut."""
    row = (128 + 2) * 4
    cache = sc.sc_cache_create(0x100000, 1, 2, 128, 64, 1, 64)      # 64 queries per node
    plan = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(0, 0)]), cache)
    assert sc.sc_attention_workspace_bytes(plan, cache) == 0          # 2 key tiles: no cut
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(c, 0) for c in range(1, 40)]), cache)
    plan = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 3, [(40, 4)]), cache)
    assert sc.sc_attention_workspace_bytes(plan, cache) == 0          # 256 keys: too short to cut
    plan = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 39, [(40, 4)]), cache)
    # 2 units of 2560 keys (80 tiles of 32): S = 16 (one round of sixteenths + 16 x 2/80 overhead)
    assert sc.sc_attention_workspace_bytes(plan, cache) == 2 * 16 * 64 * row
    mid = sc.sc_cache_create(0x100000, 1, 2, 128, 128, 1, 64)       # 128 queries per node
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(c, 0) for c in range(20)]), mid)
    plan = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 20, [(20, 4)]), mid)
    # 2 units of 2688 keys (42 tiles of 64): S = 16
    assert sc.sc_attention_workspace_bytes(plan, mid) == 2 * 16 * 128 * row
    wide = sc.sc_cache_create(0x100000, 1, 2, 128, 160, 1, 64)      # 160 queries per node
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(c, 0) for c in range(13)]), wide)
    plan = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 13, [(13, 4)]), wide)
    # 2 units of 35 tiles (14 pages x 160 keys): S = 16 (the cap)
    assert sc.sc_attention_workspace_bytes(plan, wide) == 2 * 16 * 256 * row
    big = sc.sc_cache_create(0x100000, 1, 12, 128, 1560, 3, 64)
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(0, 0)]), big)
    plan = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 1, [(1, 4)]), big)
    assert sc.sc_attention_workspace_bytes(plan, big) == 0            # 228 units: one round
    f32 = sc.sc_cache_create(0x100000, 1, 2, 64, 16, 1, 8, sc.SC_DTYPE_F32)
    plan = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(0, 0)]), f32)
    assert sc.sc_attention_workspace_bytes(plan, f32) == 0


def test_empty_pack_is_a_no_op():
    """An empty pack selects nothing, plans nothing and launches nothing."""
    sel = sc.sc_selection_build("prog", 4, 6, [])
    cache = _host_cache(8, 1)
    plan = sc.sc_plan_build(sel, cache)
    assert plan.tables() == ([0], [], [], [])
    sc.sc_attention(plan, cache, 0, 0x1000, 0x2000, 0.125)
    assert sc.sc_attention_workspace_bytes(plan, cache) == 0
    assert cache.free_slot_count() == 8


def test_position_dependent_selection_bit_exact():
    """Chunk-dependent phi tables and offset masks (Eq. 4's Phi_b, R_b,j)
    through the C ABI against the oracle."""
    rnd = random.Random(2)
    for trial in range(200):
        K, W, n = rnd.randint(1, 5), rnd.randint(0, 6), rnd.randint(1, 10)
        kind = rnd.choice(["clean", "same", "prog", "table"])
        phi = ([[[rnd.randint(0, K) for _ in range(W)] for _ in range(K + 1)] for _ in range(n)]
               if kind == "table" else None)
        mask = None
        if kind != "table" or rnd.random() < 0.5:
            mask = [[[rnd.randint(0, 1) for _ in range(W)] for _ in range(K + 1)] for _ in range(n)]
        pack = _random_pack(rnd, K, max_chunk=n)
        want = select(Policy({"clean": 0, "same": 1, "prog": 2, "table": 3}[kind], K, W, phi, mask,
                             n_chunks=n), pack)
        got = sc.sc_selection_build(kind, K, W, pack, phi_table=phi, r_mask=mask, n_chunks=n)
        off, ch, lv, src = got.tables()
        assert off == want.seg_off and ch == want.seg_chunk
        assert lv == want.seg_level and src == want.seg_src
    K, W, n = 2, 2, 3
    phi = [[[0, 0] for _ in range(K + 1)] for _ in range(n)]
    with pytest.raises(sc.ScError) as e:                       # node beyond the tables
        sc.sc_selection_build("table", K, W, [(3, 1)], phi_table=phi, n_chunks=n)
    assert e.value.code == sc.SC_EINVAL
    phi[2][1][0] = 3                                           # entry > K in the last chunk's table
    with pytest.raises(sc.ScError) as e:
        sc.sc_selection_build("table", K, W, [(0, 1)], phi_table=phi, n_chunks=n)
    assert e.value.code == sc.SC_EINVAL
    with pytest.raises(sc.ScError) as e:
        sc.sc_selection_build("prog", K, W, [(0, 1)], n_chunks=-1)
    assert e.value.code == sc.SC_EINVAL


def test_condition_plan_tables_and_errors():
    """sc_plan_condition: node i reads every page of its condition state (one
    state may serve several nodes); unknown states and empty or query-less
    packs are refused."""
    cond = sc.sc_cache_create(0x100000, 2, 2, 128, 64, 2, 6)
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(0, 0), (1, 0)]), cond)  # reserve
    s0, s1 = cond.slots((0, 0)), cond.slots((1, 0))
    plan = sc.sc_plan_condition(cond, [(1, 0), (0, 0), (1, 0)], 4680)
    off, slot, tok, frame = plan.tables()
    assert off == [0, 2, 4, 6] and slot == s1 + s0 + s1
    assert tok == [64] * 6 and frame == [0, 1] * 3
    for conds, nq, code in [([(2, 0)], 8, sc.SC_ENOTFOUND), ([], 8, sc.SC_EINVAL),
                            ([(0, 0)], 0, sc.SC_EINVAL)]:
        with pytest.raises(sc.ScError) as e:
            sc.sc_plan_condition(cond, conds, nq)
        assert e.value.code == code
    # a condition reserved but never written is refused when read
    with pytest.raises(sc.ScError) as e:
        sc.sc_attention(plan, cond, 0, 0x1000, 0x2000, 0.125)
    assert e.value.code == sc.SC_EUNAVAILABLE


def test_condition_append_and_cross_block_checks_without_device():
    """Argument checks of the condition projection and of the block's
    cross-attention and qk-norm options, all taken before any launch."""
    cond = sc.sc_cache_create(0x100000, 1, 2, 128, 64, 1, 1)
    need = sc.sc_condition_workspace_bytes(cond)
    L, D = 64, 256
    assert need == 2 * L * D * 2 + L * (D // 64) * 4
    args = dict(ctx=0x1000, w_k=0x2000, w_v=0x3000, k_norm=None, ws=0x4000)
    for layer, ws_bytes, extra, code in [(1, need, {}, sc.SC_EINVAL),         # layer out of range
                                         (0, need - 1, {}, sc.SC_EINVAL),     # workspace too small
                                         (0, need, {"k_norm": 0x5004}, sc.SC_EINVAL)]:  # misaligned gain
        a = dict(args, **extra)
        with pytest.raises(sc.ScError) as e:
            sc.sc_condition_append(cond, layer, (0, 0), a["ctx"], a["w_k"], a["w_v"], a["k_norm"],
                                   a["ws"], ws_bytes)
        assert e.value.code == code
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(5, 0)]), cond)     # fills the pool
    with pytest.raises(sc.ScError) as e:
        sc.sc_condition_append(cond, 0, (0, 0), 0x1000, 0x2000, 0x3000, None, 0x4000, need)
    assert e.value.code == sc.SC_ECAPACITY

    # block with cross-attention: the condition plan must match the pack
    cache = sc.sc_cache_create(0x100000, 1, 2, 128, 64, 1, 8)
    plan = sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(0, 4), (1, 4)]), cache)
    cond2 = sc.sc_cache_create(0x200000, 1, 2, 128, 64, 1, 2)
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(0, 0)]), cond2)
    good = sc.sc_plan_condition(cond2, [(0, 0), (0, 0)], 64)
    wrong_n = sc.sc_plan_condition(cond2, [(0, 0)], 64)
    wrong_nq = sc.sc_plan_condition(cond2, [(0, 0), (0, 0)], 32)
    mism = sc.sc_cache_create(0x300000, 1, 4, 128, 64, 1, 2)                  # 4 heads
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(0, 0)]), mism)
    mism_plan = sc.sc_plan_condition(mism, [(0, 0), (0, 0)], 64)
    bw0 = sc.BlockWeights(D, 2, 128, 512, 0x1000, 0x2000, 0x3000, 0x4000)
    ws_bytes = sc.sc_block_workspace_bytes(bw0, 128)
    cases = [(sc.CrossAttn(0x1000, 0x2000, cond2, wrong_n), None, sc.SC_EINVAL),
             (sc.CrossAttn(0x1000, 0x2000, cond2, wrong_nq), None, sc.SC_EINVAL),
             (sc.CrossAttn(0x1000, 0x2000, mism, mism_plan), None, sc.SC_EINVAL),
             (sc.CrossAttn(0x1000, 0x2000, cond2, good, q_norm=0x5008), None, sc.SC_EINVAL),
             (sc.CrossAttn(0x1000, 0x2000, cond2, good), None, sc.SC_EUNAVAILABLE),  # not written
             (None, 0x5004, sc.SC_EINVAL)]                                       # misaligned gains
    for cross, qk, code in cases:
        bw = sc.BlockWeights(D, 2, 128, 512, 0x1000, 0x2000, 0x3000, 0x4000, qk_norm=qk,
                             cross=cross)
        assert sc.sc_block_workspace_bytes(bw, 128) == ws_bytes
        with pytest.raises(sc.ScError) as e:
            sc.sc_block_forward(bw, cache, 0, plan, 0x6000, None, 0x7000, ws_bytes)
        assert e.value.code == code, (cross, qk)
    assert not cache.contains((0, 4), 0)                  # nothing was written
    # condition pages shorter than one key tile (32 keys for nodes of at most
    # 64 queries, 64 keys above) have no bf16 kernel
    short = sc.sc_cache_create(0x400000, 1, 2, 128, 24, 1, 1)
    sc.sc_plan_build(sc.sc_selection_build("clean", 4, 0, [(0, 0)]), short)
    sp = sc.sc_plan_condition(short, [(0, 0), (0, 0)], 64)
    bw = sc.BlockWeights(D, 2, 128, 512, 0x1000, 0x2000, 0x3000, 0x4000,
                         cross=sc.CrossAttn(0x1000, 0x2000, short, sp))
    with pytest.raises(sc.ScError) as e:
        sc.sc_block_forward(bw, cache, 0, plan, 0x6000, None, 0x7000, ws_bytes)
    assert e.value.code == sc.SC_EUNSUPPORTED
    # the condition projection is bf16 only
    f32 = sc.sc_cache_create(0x500000, 1, 2, 128, 64, 1, 1, sc.SC_DTYPE_F32)
    with pytest.raises(sc.ScError) as e:
        sc.sc_condition_append(f32, 0, (0, 0), 0x1000, 0x2000, 0x3000, None, 0x4000, 1 << 30)
    assert e.value.code == sc.SC_EUNSUPPORTED
