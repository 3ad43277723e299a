"""Pins of the oracle's selection and availability logic (CPU only).

What fixes the expected values:
  * the worked example of Sec. 3.3 (K = 3, round two) -- golden fixture;
  * Eq. 5 applied by hand for a few nodes -- golden fixture;
  * Eq. 8, the pipeline availability constraint, for every diagonal pack and
    arbitrary policy tables (the oracle's availability rule is generic; the
    paper's constraint is specific to Eq. 7 packs);
  * causality (Sec. 3.2: future chunks are masked).
"""
import itertools
import os
import random

import pytest

from oracle.plan import CacheModel, PlanError, build_plan
from oracle.policy import CLEAN, PROG, SAME, TABLE, Policy, SelectionError, policy, select

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split("#")[0].strip() for ln in f if ln.split("#")[0].strip()]


def test_worked_example_k3():
    for ln in _lines("worked_example_k3.txt"):
        lhs, rhs = ln.split("->")
        name, c, j = lhs.split()
        pol = policy(name, K=3, W=1)
        sel = select(pol, [(0, 2), (1, 3)])
        cache = CacheModel(n_slots=16, pages_per_chunk=1)
        cache.append(0, (0, 3))                     # retained from round one
        rhs = rhs.split()
        if rhs[0] == "UNAVAILABLE":
            with pytest.raises(PlanError) as e:
                build_plan(sel, cache, 4)
            assert e.value.code == "EUNAVAILABLE"
            continue
        segs = sel.segments(1)
        assert segs[0] == (int(rhs[0]), int(rhs[1]))
        src = sel.seg_src[sel.seg_off[1]]
        assert (src >= 0) == (rhs[2] == "pack")
        build_plan(sel, cache, 4)                   # must succeed


def test_prog_segments_by_hand():
    pol = policy("prog", K=4, W=3)
    for ln in _lines("prog_segments_w3.txt"):
        lhs, rhs = ln.split(":")
        c, j = map(int, lhs.split())
        want = [tuple(map(int, t.strip("()").split(","))) for t in rhs.split()]
        assert select(pol, [(c, j)]).segments(0) == want


@pytest.mark.parametrize("K,W", [(1, 1), (2, 3), (3, 2), (4, 6), (6, 8)])
def test_policy_shapes(K, W):
    """Clean reads only level 0; same-level only j; prog decreases by one per
    step of distance and saturates at 0; every policy reads min(W, c) offsets."""
    for c in range(0, W + 3):
        for j in range(K + 1):
            for name in ("clean", "same", "prog"):
                segs = select(policy(name, K, W), [(c, j)]).segments(0)
                hist = segs[:-1]
                assert segs[-1] == (c, j)
                assert len(hist) == min(W, c)
                chunks = [s[0] for s in hist]
                assert chunks == list(range(c - min(W, c), c))
                levels = [s[1] for s in hist]
                if name == "clean":
                    assert set(levels) <= {0}
                elif name == "same":
                    assert set(levels) <= {j}
                else:
                    # nearest chunk first: j-1, j-2, ..., floored at 0
                    near_first = levels[::-1]
                    for r, lv in enumerate(near_first, start=1):
                        prev = j if r == 1 else near_first[r - 2]
                        assert lv == max(prev - 1, 0)


def test_causality_and_visibility():
    rnd = random.Random(0)
    for _ in range(200):
        K, W = rnd.randint(1, 5), rnd.randint(0, 6)
        nodes = rnd.sample([(c, j) for c in range(8) for j in range(K + 1)], rnd.randint(1, 6))
        for name in ("clean", "same", "prog"):
            sel = select(policy(name, K, W), nodes)
            for i, (c, j) in enumerate(sel.nodes):
                segs = sel.segments(i)
                assert all(sc < c for sc, _ in segs[:-1])          # no later chunk
                row = sel.vis[i]
                assert sum(row) == len(set(segs))
                for k, st in enumerate(sel.states):
                    assert row[k] == (1 if st in segs else 0)
            for s, src in enumerate(sel.seg_src):
                st = (sel.seg_chunk[s], sel.seg_level[s])
                assert (src >= 0) == (st in sel.nodes)
                if src >= 0:
                    assert sel.nodes[src] == st


def _diagonal(n, K, B, refresh=True):
    lo = 0 if refresh else 1
    # Eq. 7: chunk n at level K, chunk n-1 at K-1, ...; chunk n-K+j at level j
    return sorted((n - K + j, j) for j in range(lo, K + 1) if 0 <= n - K + j < B)


@pytest.mark.parametrize("K", [1, 2, 3, 4, 5, 6])
def test_eq8_availability_matches_paper(K):
    """For Eq. 7 packs (with the clean refresh node), a table policy plans
    successfully exactly when phi(j, r) >= max(j - r, 0) for every offset read
    (Eq. 8), given that all states of earlier rounds are retained."""
    rnd = random.Random(K)
    B, W = 3 * K + 4, K + 2
    for trial in range(40):
        phi = [[rnd.randint(0, K) for _ in range(W)] for _ in range(K + 1)]
        if trial % 4 == 0:
            phi = [[max(j - r, 0) for r in range(1, W + 1)] for j in range(K + 1)]
        pol = Policy(TABLE, K, W, phi_table=phi)
        for n in range(B + K):
            pack = _diagonal(n, K, B)
            cache = CacheModel(n_slots=(K + 1) * B, pages_per_chunk=1)
            for c in range(B):
                jc = K - (n - c)           # level of chunk c in round n
                if jc > K:
                    continue               # chunk not started yet
                lowest = 0 if jc < 0 else jc + 1   # completed, or in flight at jc
                for lv in range(lowest, K + 1):
                    cache.append(0, (c, lv))      # retained from earlier rounds
            ok = all(phi[j][r - 1] >= max(j - r, 0)
                     for (c, j) in pack for r in range(1, min(W, c) + 1))
            sel = select(pol, pack)
            try:
                build_plan(sel, cache, 1)
                got = True
            except PlanError as e:
                assert e.code == "EUNAVAILABLE"
                got = False
            assert got == ok, (n, pack, phi)


def test_clean_fails_in_diagonal_iff_window_reaches_inflight():
    """Clean history inside a pipelined pack is unavailable exactly when some
    node reads a chunk that is still in flight (r < j), Sec. 3.3 example."""
    K, W, B = 4, 6, 16
    for n in range(B + K):
        pack = _diagonal(n, K, B)
        cache = CacheModel(n_slots=4096, pages_per_chunk=1)
        for c in range(0, n - K):
            cache.append(0, (c, 0))
        need_inflight = any(1 <= r < j for (c, j) in pack for r in range(1, min(W, c) + 1))
        sel = select(policy("clean", K, W), pack)
        if need_inflight:
            with pytest.raises(PlanError):
                build_plan(sel, cache, 1)
        else:
            build_plan(sel, cache, 1)
        for name in ("prog",):
            cache2 = CacheModel(n_slots=4096, pages_per_chunk=1)
            for c in range(0, n - K):
                cache2.append(0, (c, 0))
            build_plan(select(policy(name, K, W), pack), cache2, 1)


def test_invalid_inputs():
    with pytest.raises(SelectionError):
        select(policy("prog", 0, 2), [(0, 0)])
    with pytest.raises(SelectionError):
        select(policy("prog", 4, -1), [(0, 0)])
    with pytest.raises(SelectionError):
        select(policy("prog", 4, 2), [(0, 5)])
    with pytest.raises(SelectionError):
        select(policy("prog", 4, 2), [(-1, 1)])
    with pytest.raises(SelectionError):
        select(policy("prog", 4, 2), [(1, 1), (1, 1)])
    with pytest.raises(SelectionError):
        select(Policy(TABLE, 2, 2, phi_table=[[0, 3], [0, 0], [0, 0]]), [(1, 1)])


def test_plan_pages_and_slots():
    """Pages follow segment order, frames ascending; pack states get the lowest
    free slots in pack order; capacity and release behave as a slot allocator."""
    K, W, ppc = 4, 2, 3
    cache = CacheModel(n_slots=20, pages_per_chunk=ppc)
    cache.append(0, (0, 0))        # slots 0,1,2
    cache.append(0, (1, 0))        # slots 3,4,5
    sel = select(policy("prog", K, W), [(2, 1), (3, 2)])
    plan = build_plan(sel, cache, 7)
    assert cache.slots[(2, 1)] == [6, 7, 8] and cache.slots[(3, 2)] == [9, 10, 11]
    # node (2,1): (0,0) (1,0) (2,1); node (3,2): (1,0) (2,1) (3,2)
    assert plan.page_off == [0, 9, 18]
    assert plan.page_slot[:9] == [0, 1, 2, 3, 4, 5, 6, 7, 8]
    assert plan.page_slot[9:] == [3, 4, 5, 6, 7, 8, 9, 10, 11]
    assert plan.page_frame[9:12] == [3, 4, 5]
    assert set(plan.page_tokens) == {7}
    cache.release((0, 0))
    assert cache.generation[0] == 1 and cache.free_slots()[:3] == [0, 1, 2]
    with pytest.raises(PlanError):
        cache.release((0, 0))
    with pytest.raises(PlanError):
        cache.append(0, (1, 0))    # layer 0 already written
    small = CacheModel(n_slots=5, pages_per_chunk=ppc)
    with pytest.raises(PlanError) as e:
        build_plan(select(policy("prog", K, W), [(0, 1), (1, 2)]), small, 7)
    assert e.value.code == "ECAPACITY" and small.slots == {}


def test_position_dependent_policy_by_hand():
    """Eq. 4 lets Phi_b and R_b,j depend on the chunk.  K = 2, W = 2, chunks
    0-1 read clean history and chunks 2-3 same-level history; chunk 3 at
    level 2 skips offset 1."""
    K, W = 2, 2
    clean = [[0, 0] for _ in range(K + 1)]
    same = [[j, j] for j in range(K + 1)]
    phi = [clean, clean, same, same]
    mask = [[[1, 1] for _ in range(K + 1)] for _ in range(4)]
    mask[3][2] = [0, 1]
    pol = Policy(3, K, W, phi_table=phi, r_mask=mask, n_chunks=4)
    assert select(pol, [(1, 2)]).segments(0) == [(0, 0), (1, 2)]
    assert select(pol, [(2, 1)]).segments(0) == [(0, 1), (1, 1), (2, 1)]
    assert select(pol, [(3, 1)]).segments(0) == [(1, 1), (2, 1), (3, 1)]
    assert select(pol, [(3, 2)]).segments(0) == [(1, 2), (3, 2)]
    with pytest.raises(SelectionError):
        select(pol, [(4, 0)])                                # beyond the tables


def test_chunk_constant_tables_equal_position_independent():
    """Repeating one (K+1) x W table for every chunk gives the
    position-independent policy exactly (tables of the three named policies
    included)."""
    rnd = random.Random(5)
    for _ in range(60):
        K, W, n = rnd.randint(1, 5), rnd.randint(0, 6), 10
        kind = rnd.choice(["clean", "same", "prog", "table"])
        if kind == "table":
            t = [[rnd.randint(0, K) for _ in range(W)] for _ in range(K + 1)]
        else:
            t = [[policy(kind, K, W).phi(j, r) for r in range(1, W + 1)] for j in range(K + 1)]
        base = Policy(3, K, W, phi_table=t)
        per_chunk = Policy(3, K, W, phi_table=[t] * n, n_chunks=n)
        pack = rnd.sample([(c, j) for c in range(n) for j in range(K + 1)], rnd.randint(1, 6))
        a, b = select(base, pack), select(per_chunk, pack)
        assert (a.seg_off, a.seg_chunk, a.seg_level, a.seg_src) == \
            (b.seg_off, b.seg_chunk, b.seg_level, b.seg_src)
        if kind != "table":
            c_ = select(policy(kind, K, W), pack)
            assert (c_.seg_chunk, c_.seg_level) == (b.seg_chunk, b.seg_level)
