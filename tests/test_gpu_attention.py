"""GPU parity of the packed paged attention against the CPU oracle.

Covers the tiny fp32 case (every node of 4 chunks x 5 levels under all three
policies, several pack shapes), small bf16 packs on each work-group shape
(256, 128 and 64 queries) whose pages (104, 96 and 40 tokens) leave ragged
tails inside key tiles, the short-context streaming shape and long windows
cut into key-range pieces, the Wan-shaped clean / same-level /
progressive packs on sampled rows, the segment probe, negative controls
(mistakes planted in the oracle must fail the gates), NaN poisoning of
unused slots, packed vs sequential, run-to-run determinism and the workspace
check.
"""
import dataclasses

import numpy as np
import pytest

import paper_2609_22283_amd as sc
from oracle.attention import node_attention
from oracle.pipeline import pipeline_rounds
from oracle.policy import policy as oracle_policy
from oracle.policy import select
from synth.configs import (NARROW, SHORT, SMALL, TINY, WAN, cfg2_clean, cfg3_same, cfg4_prog,
                           kv_stream)

from gpu_cases import (AttnCase, BF16_MAX_ABS, F32_MAX_ABS, bf16_gates, from_device, sample_rows,
                       to_device, torch_mod)

pytestmark = pytest.mark.gpu

ALL_TINY = [(c, j) for c in range(4) for j in range(TINY.K + 1)]


def _tiny_packs(kind):
    packs = [[n] for n in ALL_TINY]
    if kind == "prog":
        packs += [p for p in pipeline_rounds(4, TINY.K, refresh=True) if len(p) > 1]
    if kind == "same":
        packs += [[(c, j) for c in range(4)] for j in range(TINY.K + 1)]
    packs.append(list(ALL_TINY))           # everything resident, one pack of 20
    return packs


@pytest.mark.parametrize("kind", ["clean", "same", "prog"])
def test_tiny_fp32_every_node(kind):
    for pack in _tiny_packs(kind):
        case = AttnCase(TINY, sc.SC_DTYPE_F32, kind, pack, resident=ALL_TINY, seed=1)
        out = case.run()
        for i, node in enumerate(pack):
            want = case.oracle(i)
            err = np.abs(out[i] - want).max()
            assert err <= F32_MAX_ABS, (kind, pack, node, err)


SMALL_PACKS = [
    ("prog", [(6, 1), (7, 2), (8, 3), (9, 4)], [(c, 0) for c in range(6)]),
    ("prog", [(6, 0), (7, 1), (8, 2), (9, 3), (10, 4)], [(c, 0) for c in range(6)]),
    ("same", [(6 + i, 2) for i in range(4)], [(c, 2) for c in range(6)]),
    ("clean", [(6, 3)], [(c, 0) for c in range(6)]),
    ("clean", [(2, 4)], [(c, 0) for c in range(2)]),
    ("prog", [(0, 4)], []),
]


@pytest.mark.parametrize("kind,pack,resident", SMALL_PACKS)
def test_small_bf16_packs(kind, pack, resident):
    case = AttnCase(SMALL, sc.SC_DTYPE_BF16, kind, pack, resident, seed=2)
    out = case.run()
    for i in range(len(pack)):
        bf16_gates(out[i], case.oracle(i), f"{kind} node {pack[i]}")


@pytest.mark.parametrize("kind,pack,resident", SMALL_PACKS)
def test_short_bf16_packs(kind, pack, resident):
    """Nodes of 96 queries run on the 128-query (4-wave) work-group shape."""
    case = AttnCase(SHORT, sc.SC_DTYPE_BF16, kind, pack, resident, seed=6)
    out = case.run()
    for i in range(len(pack)):
        bf16_gates(out[i], case.oracle(i), f"short {kind} node {pack[i]}")


@pytest.mark.parametrize("kind,pack,resident", SMALL_PACKS)
def test_narrow_bf16_packs(kind, pack, resident):
    """Nodes of 40 queries run on the 64-query (2-wave, 32-key tile) shape."""
    case = AttnCase(NARROW, sc.SC_DTYPE_BF16, kind, pack, resident, seed=12)
    out = case.run()
    for i in range(len(pack)):
        bf16_gates(out[i], case.oracle(i), f"narrow {kind} node {pack[i]}")


def test_narrow_long_windows_cut_into_pieces():
    """64-query nodes over 41 pages of 64 keys (2624 keys, 82 tiles of 32):
    the 36 units of three nodes are cut into key-range pieces (a workspace is
    needed) and merged; every row against the oracle."""
    geo = kv_stream(64, W=40)
    W = geo.W
    pack = [(41 * i + W, 4) for i in range(3)]
    resident = [(41 * i + r, 0) for i in range(3) for r in range(W)]
    case = AttnCase(geo, sc.SC_DTYPE_BF16, "clean", pack, resident, seed=13)
    out = case.run()
    assert case.workspace_bytes > 0
    for i in range(len(pack)):
        bf16_gates(out[i], case.oracle(i), f"narrow pieces node {pack[i]}")


@pytest.mark.parametrize("heads", [12, 16])
def test_narrow_many_units(heads):
    """64 one-frame nodes of 64 queries over 3 pages each: 768 units (12
    heads) run at once on the 64-query shape's 2-tile-in-flight ring; 1024
    (16 heads) take more than one round of it.  Nodes 0, 21, 42 and 63
    checked against the oracle."""
    geo = dataclasses.replace(kv_stream(64, W=2), heads=heads)
    pack = [(3 * i + 2, 4) for i in range(64)]
    resident = [(3 * i + r, 0) for i in range(64) for r in range(2)]
    case = AttnCase(geo, sc.SC_DTYPE_BF16, "clean", pack, resident, seed=14)
    out = case.run()
    assert case.workspace_bytes == 0
    for i in (0, 21, 42, 63):
        bf16_gates(out[i], case.oracle(i), f"narrow {heads} heads node {pack[i]}")


def test_wide_long_windows_cut_into_pieces():
    """128-query nodes over 41 pages of 128 keys (5248 keys): the 128-query
    shape, its 36 units cut into key-range pieces; every row against the
    oracle."""
    geo = kv_stream(128, W=40)
    W = geo.W
    pack = [(41 * i + W, 4) for i in range(3)]
    resident = [(41 * i + r, 0) for i in range(3) for r in range(W)]
    case = AttnCase(geo, sc.SC_DTYPE_BF16, "clean", pack, resident, seed=15)
    out = case.run()
    assert case.workspace_bytes > 0
    for i in range(len(pack)):
        bf16_gates(out[i], case.oracle(i), f"wide pieces node {pack[i]}")


@pytest.mark.parametrize("nq", [64, 128])
def test_kv_stream_shape(nq):
    """The short-context streaming shape (12 heads, one-frame chunks, 21
    pages per node): three nodes with disjoint windows, every row."""
    geo = kv_stream(nq)
    W = geo.W
    pack = [(21 * i + W, 4) for i in range(3)]
    resident = [(21 * i + r, 0) for i in range(3) for r in range(W)]
    case = AttnCase(geo, sc.SC_DTYPE_BF16, "clean", pack, resident, seed=7)
    out = case.run()
    for i in range(len(pack)):
        bf16_gates(out[i], case.oracle(i), f"kv stream nq={nq} node {pack[i]}")


def test_position_dependent_policy():
    """A chunk-dependent policy (Eq. 4's Phi_b and R_b,j: random per-chunk
    phi tables and offset masks) through the plan and the bf16 kernel."""
    import random
    rnd = random.Random(9)
    K, W, n = SMALL.K, SMALL.W, 10
    phi = [[[rnd.randint(0, K) for _ in range(W)] for _ in range(K + 1)] for _ in range(n)]
    mask = [[[int(rnd.random() < 0.7) for _ in range(W)] for _ in range(K + 1)] for _ in range(n)]
    kw = dict(phi_table=phi, r_mask=mask, n_chunks=n)
    pack = [(7, 1), (8, 3), (9, 4)]
    sel = select(oracle_policy("table", K, W, **kw), pack)
    resident = [s for s in sel.states if s not in pack]
    case = AttnCase(SMALL, sc.SC_DTYPE_BF16, "table", pack, resident, seed=10, policy_kw=kw)
    out = case.run()
    for i in range(len(pack)):
        bf16_gates(out[i], case.oracle(i), f"position-dependent node {pack[i]}")


def test_small_packed_matches_sequential():
    """The same nodes packed and one per call.  The split-key schedule cuts a
    node's key range where the pack's total work puts the work-group
    boundaries, so the two runs sum in different orders: they agree within
    the bf16 gates, not bitwise."""
    kind, pack, resident = SMALL_PACKS[0]
    case = AttnCase(SMALL, sc.SC_DTYPE_BF16, kind, pack, resident, seed=3)
    packed = case.run()
    # the same nodes one per call, ascending chunk (in-pack history comes
    # from the cache, appended by the earlier calls)
    for i, node in enumerate(pack):
        res = resident + pack[:i]
        alone = AttnCase(SMALL, sc.SC_DTYPE_BF16, kind, [node], res, seed=3)
        got = alone.run()[0]
        bf16_gates(got, packed[i], f"alone vs packed {node}")
        bf16_gates(got, alone.oracle(0), f"alone {node}")


def test_small_deterministic_and_pack_order_free():
    """Bitwise run-to-run determinism for one plan; a reversed pack agrees
    within the gates."""
    kind, pack, resident = SMALL_PACKS[1]
    a = AttnCase(SMALL, sc.SC_DTYPE_BF16, kind, pack, resident, seed=4)
    o1 = a.run()
    o2 = a.run()
    rev = AttnCase(SMALL, sc.SC_DTYPE_BF16, kind, pack[::-1], resident, seed=4).run()
    for i in range(len(pack)):
        assert np.array_equal(o1[i], o2[i])
        bf16_gates(rev[len(pack) - 1 - i], o1[i], f"reversed {pack[i]}")


def test_workspace_checked():
    """A workspace smaller than the plan needs is refused before any launch."""
    kind, pack, resident = SMALL_PACKS[0]
    case = AttnCase(SMALL, sc.SC_DTYPE_BF16, kind, pack, resident, seed=3)
    torch = torch_mod()
    need = sc.sc_attention_workspace_bytes(case.plan, case.cache)
    assert need > 0
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    with pytest.raises(sc.ScError) as e:
        sc.sc_attention(case.plan, case.cache, case.layer, case.q_dev, case.o_dev, case.scale,
                        ws, need - 1)
    assert e.value.code == sc.SC_EINVAL
    with pytest.raises(sc.ScError) as e:
        sc.sc_attention(case.plan, case.cache, case.layer, case.q_dev, case.o_dev, case.scale)
    assert e.value.code == sc.SC_EINVAL


def _probe_case(geo, kind, pack, resident):
    """V = one-hot(state id) in the first channels (exact in bf16)."""
    states = sorted(set(resident) | set(pack))
    sid = {s: k for k, s in enumerate(states)}

    def value_fn(st):
        v = np.zeros((geo.tokens_per_chunk, geo.heads, geo.head_dim), dtype=np.float32)
        v[:, :, sid[tuple(st)]] = 1.0
        return v
    return AttnCase(geo, sc.SC_DTYPE_BF16, kind, pack, resident, seed=5, value_fn=value_fn), states


@pytest.mark.parametrize("kind,pack,resident", SMALL_PACKS[:3])
def test_segment_probe_small(kind, pack, resident):
    case, states = _probe_case(SMALL, kind, pack, resident)
    out = case.run()
    for i in range(len(pack)):
        want = case.oracle(i)
        chosen = set(select(oracle_policy(kind, SMALL.K, SMALL.W), pack).segments(i))
        for k, st in enumerate(states):
            np.testing.assert_allclose(out[i][:, :, k], want[:, :, k], atol=2e-3)
            if st not in chosen:
                assert np.all(out[i][:, :, k] == 0.0), (pack[i], st)


def _corruptions(segs, geo):
    """Plausible planning mistakes, planted in the oracle's segment list."""
    c, j = segs[-1]
    out = {"drop_oldest": segs[1:], "level_off_by_one": [(sc_, min(l + 1, geo.K)) for sc_, l in segs[:-1]] + [segs[-1]]}
    out["future_chunk"] = segs + [(c + 1, j)]
    return out


def test_negative_controls_fail_gates():
    kind, pack, resident = SMALL_PACKS[0]
    extra = [(10, 4)] + [(c, min(l + 1, SMALL.K)) for c in range(10) for l in range(SMALL.K)]
    case = AttnCase(SMALL, sc.SC_DTYPE_BF16, kind, pack, resident + extra, seed=6,
                    n_slots=(len(resident) + len(extra) + len(pack) + 2) * SMALL.frames_per_chunk)
    out = case.run()
    sel = select(oracle_policy(kind, SMALL.K, SMALL.W), pack)
    node = 3
    segs = sel.segments(node)
    bf16_gates(out[node], case.oracle(node), "correct plan")
    for name, bad in _corruptions(segs, SMALL).items():
        bad = [s for s in bad if s in case.kv]
        want = case.oracle(node, segments=bad)
        with pytest.raises(AssertionError):
            bf16_gates(out[node], want, name)


@pytest.mark.parametrize("geo", [SMALL, SHORT, NARROW], ids=["256-query", "128-query", "64-query"])
def test_logits_far_above_first_tile(geo):
    """K channel 0 is 0 on each node's first page and 600 on most later
    pages (first page of every state for three-frame chunks; chunks 0..3,
    the first pages of this pack's nodes, for one-frame chunks), with Q
    channel 0 = 1: later logits sit about 76 (log2 units) above the maximum
    of a node's first key tile, past the kernel's 2^64 guard on probability
    sums, so the work items redo their keys in two exact passes.  The
    softmax is still the plain one: compared with the oracle."""
    kind, pack, resident = SMALL_PACKS[0]
    tpp = geo.tokens_per_page

    def key_fn(st, k):
        k = k.copy()
        k[:, :, 0] = 600.0
        if geo.frames_per_chunk > 1:
            k[:tpp, :, 0] = 0.0
        elif st[0] < 4:
            k[:, :, 0] = 0.0
        return k

    def query_fn(st, q):
        q = q.copy()
        q[:, :, 0] = 1.0
        return q
    case = AttnCase(geo, sc.SC_DTYPE_BF16, kind, pack, resident, seed=11, key_fn=key_fn,
                    query_fn=query_fn)
    out = case.run()
    for i in range(len(pack)):
        bf16_gates(out[i], case.oracle(i), f"large logits node {pack[i]}")


WAN_CASES = [cfg2_clean(4), cfg3_same(2), cfg4_prog(False), cfg4_prog(True)]


@pytest.mark.parametrize("wl", WAN_CASES, ids=[w.name for w in WAN_CASES])
def test_wan_sampled_rows(wl):
    case = AttnCase(WAN, sc.SC_DTYPE_BF16, wl.policy, wl.pack, wl.resident, seed=7)
    out = case.run()
    rows = sample_rows(WAN.tokens_per_chunk, 40, seed=len(wl.pack))
    for i in range(len(wl.pack)):
        got = out[i]
        assert np.all(np.isfinite(got)), "NaN from a poisoned slot or a bad tile"
        bf16_gates(got[rows], case.oracle(i, rows=rows), f"{wl.name} node {wl.pack[i]}")


def test_wan_segment_probe_prog():
    wl = cfg4_prog(True)
    case, states = _probe_case(WAN, wl.policy, wl.pack, wl.resident)
    out = case.run()
    rows = sample_rows(WAN.tokens_per_chunk, 16, seed=9)
    for i in range(len(wl.pack)):
        want = case.oracle(i, rows=rows)
        got = out[i][rows]
        chosen = set(select(oracle_policy(wl.policy, WAN.K, WAN.W), wl.pack).segments(i))
        for k, st in enumerate(states):
            np.testing.assert_allclose(got[:, :, k], want[:, :, k], atol=2e-3)
            if st not in chosen:
                assert np.all(out[i][:, :, k] == 0.0), (wl.pack[i], st)


def test_max_nodes_and_pages():
    """Pack limits of the attention kernel's plan arguments: 64 nodes run
    (the first, a middle and the last node checked against the oracle); a
    65th node, or more than 800 pages in one plan, is refused with
    SC_EUNSUPPORTED before any launch."""
    geo1 = dataclasses.replace(SHORT, W=1)
    pack = [(2 * i + 1, 4) for i in range(64)]
    resident = [(2 * i, 0) for i in range(64)]
    case = AttnCase(geo1, sc.SC_DTYPE_BF16, "clean", pack, resident, seed=8)
    out = case.run()
    for i in (0, 31, 63):
        bf16_gates(out[i], case.oracle(i), f"64-node pack node {pack[i]}")
    big = AttnCase(geo1, sc.SC_DTYPE_BF16, "clean", [(2 * i + 1, 4) for i in range(65)],
                   [(2 * i, 0) for i in range(65)], seed=8)
    with pytest.raises(sc.ScError) as e:
        big.run()
    assert e.value.code == sc.SC_EUNSUPPORTED
    # 64 nodes x 13 pages = 832 pages > 800
    geo12 = dataclasses.replace(SHORT, W=12)
    wide = AttnCase(geo12, sc.SC_DTYPE_BF16, "clean", [(12 + 13 * i, 4) for i in range(64)],
                    [(13 * i + r, 0) for i in range(64) for r in range(12)], seed=8)
    with pytest.raises(sc.ScError) as e:
        wide.run()
    assert e.value.code == sc.SC_EUNSUPPORTED
