"""Execution schedule through the C ABI vs the oracle, on the CPU.

Round packs of Eq. 7 (with and without the refresh node) must equal the
oracle's; the policy-general release rule (drop what no future node reads)
must keep every plan of the schedule available and, for progressive history,
release exactly what the oracle's progressive rule releases.
"""
import pytest

import paper_2609_22283_amd as sc
from oracle.pipeline import pipeline_rounds, serial_order
from oracle.plan import CacheModel, build_plan
from oracle.policy import policy, select


@pytest.mark.parametrize("K,B", [(1, 1), (2, 5), (3, 7), (4, 16), (6, 3)])
@pytest.mark.parametrize("refresh", [False, True])
def test_round_nodes_match_oracle(K, B, refresh):
    want = pipeline_rounds(B, K, refresh)
    assert sc.sc_pipeline_rounds(K, B, refresh) == len(want)
    for n, pack in enumerate(want):
        assert sc.sc_pipeline_round_nodes(K, B, refresh, n) == pack
    with pytest.raises(sc.ScError):
        sc.sc_pipeline_round_nodes(K, B, refresh, len(want))


def _host_cache(n_slots, ppc=1):
    return sc.sc_cache_create(0x100000, 1, 2, 128, 64, ppc, n_slots)


@pytest.mark.parametrize("kind", ["prog", "same"])
def test_release_rule_keeps_schedule_available(kind):
    """Run the whole pipelined schedule on host tables only: plan, then
    release what later rounds do not read.  No plan may fail, and the live
    state count stays bounded by the window."""
    K, B, W = 4, 16, 6
    cache = _host_cache(4096)
    rounds = pipeline_rounds(B, K, refresh=True)
    peak = 0
    for n, pack in enumerate(rounds):
        sc.sc_plan_build(sc.sc_selection_build(kind, K, W, pack), cache)
        peak = max(peak, 4096 - cache.free_slot_count())
        future = [node for p in rounds[n + 1:] for node in p]
        sc.sc_cache_release_unread(cache, kind, K, W, future)
    assert cache.free_slot_count() == 4096
    # progressive: W clean chunks + one round; same-level: W chunks per level
    assert peak <= (W + K + 1) * (K + 1)


def test_release_rule_equals_oracle_progressive():
    K, B, W = 4, 12, 6
    rounds = pipeline_rounds(B, K, refresh=True)
    cache = _host_cache(512)
    model = CacheModel(n_slots=512, pages_per_chunk=1)
    for n, pack in enumerate(rounds):
        sc.sc_plan_build(sc.sc_selection_build("prog", K, W, pack), cache)
        build_plan(select(policy("prog", K, W), pack), model, 64)
        future = [node for p in rounds[n + 1:] for node in p]
        sc.sc_cache_release_unread(cache, "prog", K, W, future)
        # the oracle's progressive rule (oracle/pipeline.py run_stack)
        nxt = rounds[n + 1] if n + 1 < len(rounds) else []
        oldest = min((c for c, _ in nxt), default=None)
        for (c, j) in pack:
            if j >= 1:
                model.release((c, j))
        for st in list(model.slots):
            if st[1] == 0 and (oldest is None or st[0] < oldest - W):
                model.release(st)
        assert sorted(model.slots) == sorted(st for st in model.slots if cache.contains(st))
        assert len(model.slots) == 512 - cache.free_slot_count()


def test_serial_schedule_with_release_is_available():
    """Fully serial execution (Eq. 2) under every policy, one node per plan."""
    K, B, W = 4, 8, 3
    order = serial_order(B, K, refresh=True)
    for kind in ("clean", "same", "prog"):
        cache = _host_cache(1024)
        for i, node in enumerate(order):
            sc.sc_plan_build(sc.sc_selection_build(kind, K, W, [node]), cache)
            sc.sc_cache_release_unread(cache, kind, K, W, order[i + 1:])
        assert cache.free_slot_count() == 1024


def test_release_rule_with_position_dependent_policy():
    """A policy that switches from same-level to progressive history after
    the first chunks (chunk-dependent tables; both are available under Eq. 8):
    the pipelined schedule, with the release rule evaluated under the same
    tables, keeps every plan available and ends with an empty cache."""
    K, B, W = 4, 10, 3
    same = [[j] * W for j in range(K + 1)]
    prog = [[max(j - r, 0) for r in range(1, W + 1)] for j in range(K + 1)]
    phi = [same if c < 4 else prog for c in range(B)]
    cache = _host_cache(1024)
    rounds = pipeline_rounds(B, K, refresh=True)
    for n, pack in enumerate(rounds):
        sc.sc_plan_build(sc.sc_selection_build("table", K, W, pack, phi_table=phi, n_chunks=B), cache)
        future = [node for p in rounds[n + 1:] for node in p]
        sc.sc_cache_release_unread(cache, "table", K, W, future, phi_table=phi, n_chunks=B)
    assert cache.free_slot_count() == 1024


@pytest.mark.parametrize("K,B,refresh", [(1, 1, False), (3, 5, True), (4, 16, True), (4, 16, False),
                                         (6, 3, True)])
def test_serial_order_matches_oracle(K, B, refresh):
    """Fully serial execution (Eq. 2): every update of chunk c before chunk
    c + 1, levels K .. 1, the refresh (c, 0) last."""
    from oracle.pipeline import serial_order
    n = sc.sc_serial_steps(K, B, refresh)
    got = [sc.sc_serial_step_node(K, B, refresh, i) for i in range(n)]
    assert got == serial_order(B, K, refresh)
    assert n == B * (K + 1 if refresh else K)
    for bad in (-1, n):
        with pytest.raises(sc.ScError) as e:
            sc.sc_serial_step_node(K, B, refresh, bad)
        assert e.value.code == sc.SC_EINVAL
