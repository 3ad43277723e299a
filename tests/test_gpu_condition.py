"""GPU parity of the condition path (the condition c of Eq. 1 read by
cross-attention) and of qk-norm, against the oracle.

Condition K/V pages: each projected value is rounded to bf16 once (V, plain
K) or twice (normalised K: the raw projection, then the scaled value), and
bf16 keeps 8 significant bits, so |gpu - oracle| <= n * 2^-8 * |oracle| plus
a floor of 2^-16 of the largest value for the fp32 accumulation.  Attention over a condition plan uses the same gates as the
pack attention.  Block outputs use the block gates; the block now has two
more bf16 roundings on the cross branch (the condition query and the
cross-attention output), both averaged over >= 256-term dot products before
they reach the residual stream, and one more on q and k with qk-norm (the
unnormalised value, then the scaled one: at most one extra half spacing).
"""
import math
import types

import numpy as np
import pytest

import paper_2609_22283_amd as sc
from oracle.attention import softmax_attention
from synth import TAG_GAIN, TAG_Q, normal
from synth.configs import SHORT, SMALL, WAN, cfg4_prog

from gpu_cases import ConditionCase, bf16_gates, from_device, gains, sample_rows, to_device, torch_mod
from test_gpu_block import BlockCase, _mod_table, block_gate, read_pages

pytestmark = pytest.mark.gpu


def rounding_gate(got, want, n_round, what):
    lim = n_round * 2.0 ** -8 * np.abs(want) + 2.0 ** -16 * np.abs(want).max()
    worst = float((np.abs(got - want) / lim).max())
    assert worst <= 1.0, f"{what}: worst error / bound {worst:.3g}"


def _page_geo(geo, L):
    return types.SimpleNamespace(heads=geo.heads, head_dim=geo.head_dim, tokens_per_page=L)


@pytest.mark.parametrize("k_norm", [False, True], ids=["plain", "k_norm"])
def test_condition_append_matches_oracle(k_norm):
    L = 200                                                  # not a multiple of 64
    cc = ConditionCase(SMALL, L, seed=21, n_cond=2, k_norm=k_norm)
    for i in range(2):
        k_got, v_got = read_pages(cc.pool, _page_geo(SMALL, L), 2, cc.cache.slots((i, 0)))
        rounding_gate(k_got, cc.kv[i][0], 2 if k_norm else 1, f"condition {i} K")
        rounding_gate(v_got, cc.kv[i][1], 1, f"condition {i} V")
    with pytest.raises(sc.ScError) as e:                     # layer already written
        sc.sc_condition_append(cc.cache, 0, (0, 0), cc.pool, cc.w_dev["w_k"], cc.w_dev["w_v"], None,
                               cc.ws, cc.ws_bytes)
    assert e.value.code == sc.SC_EEXIST


@pytest.mark.parametrize("nq,L,pages", [(300, 200, 1), (96, 200, 1), (300, 256, 2)],
                         ids=["256-query", "128-query", "two-page-condition"])
def test_attention_over_condition_plan(nq, L, pages):
    """Each pack node reads its own condition (two nodes share one), every
    query sees all L tokens; ragged L and ragged query counts; a condition
    spread over two page slots."""
    torch = torch_mod()
    cc = ConditionCase(SMALL, L, seed=22, n_cond=3, k_norm=True, pages=pages)
    conds = [0, 2, 1, 0]
    plan = cc.plan(conds, nq)
    H, d = SMALL.heads, SMALL.head_dim
    q_dev, q = to_device(normal((len(conds) * nq, H, d), (22, TAG_Q)), sc.SC_DTYPE_BF16)
    o = torch.empty_like(q_dev)
    ws_bytes = sc.sc_attention_workspace_bytes(plan, cc.cache)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    scale = 1.0 / math.sqrt(d)
    sc.sc_attention(plan, cc.cache, 0, q_dev, o, scale, ws, ws_bytes)
    torch.cuda.synchronize()
    got = from_device(o)
    for i, c in enumerate(conds):
        k, v = cc.kv[c]
        want = np.stack([softmax_attention(q[i * nq:(i + 1) * nq, h], k[:, h], v[:, h], scale)
                         for h in range(H)], axis=1)
        bf16_gates(got[i * nq:(i + 1) * nq], want, f"node {i} (condition {c})")


PACK = [(6, 0), (7, 1), (8, 2), (9, 3), (10, 4)]
RESIDENT = [(c, 0) for c in range(6)]


# bf16 roundings of a block output that the fp64 oracle does not make: the
# plain block's seven, plus q and k rounded again after the qk-norm (1); for
# cross-attention its RMSNorm output, query, cached condition K/V, attention
# output and residual (5); with its norms the query and the condition keys
# rounded again after them (2).  Folded RMSNorms (the query's always, the
# block's without modulation) never round their outputs, so these counts are
# upper bounds.
ROUNDINGS = {"qk": 8, "cross": 12, "cross_norm": 14, "all": 15}


@pytest.mark.parametrize("variant", ["qk", "cross", "cross_norm", "all"])
def test_small_block_qk_norm_and_cross(variant):
    """qk-norm alone; cross-attention without and with its query/key norms;
    everything together with level modulation.  Outputs and the cached
    (normalised) keys against the oracle; normalised keys reach |k| ~ 6, so
    they take the block's scale-relative gate."""
    qk = np.stack([gains(SMALL.hidden, (31, TAG_GAIN, s)) for s in range(2)])
    use_qk = variant in ("qk", "all")
    cross = None
    if variant != "qk":
        norms = variant != "cross"
        cross = ConditionCase(SMALL, 64 if variant == "cross" else 136, seed=32, q_norm=norms,
                              k_norm=norms)
    mod = _mod_table(SMALL, 33) if variant == "all" else None
    case = BlockCase(SMALL, "prog", PACK, RESIDENT, seed=34, mod=mod, qk=qk if use_qk else None,
                     cross=cross)
    got = case.run()
    want, new_kv = case.oracle()
    for i in range(len(PACK)):
        block_gate(got[i], want[i], f"{variant} node {PACK[i]}", ROUNDINGS[variant])
        k_got, v_got = read_pages(case.pool, SMALL, case.n_slots, case.cache.slots(PACK[i]))
        (block_gate if use_qk else bf16_gates)(k_got, new_kv[i][0], f"{variant} cached K")
        bf16_gates(v_got, new_kv[i][1], f"{variant} cached V")


def test_short_block_qk_norm_and_cross():
    """One-frame 96-token chunks: the 128-query attention shape for both the
    pack and the condition."""
    qk = np.stack([gains(SHORT.hidden, (35, TAG_GAIN, s)) for s in range(2)])
    cross = ConditionCase(SHORT, 72, seed=36, q_norm=True, k_norm=True)
    case = BlockCase(SHORT, "prog", PACK, RESIDENT, seed=37, qk=qk, cross=cross)
    got = case.run()
    want, _ = case.oracle()
    for i in range(len(PACK)):
        block_gate(got[i], want[i], f"short node {PACK[i]}", ROUNDINGS["all"])


def test_wan_block_qk_norm_and_cross_sampled_rows():
    """Wan-shaped block (hidden 1536, 12 heads) on the progressive pack with
    qk-norm and cross-attention to a 512-token condition, sampled rows."""
    wl = cfg4_prog(False)
    qk = np.stack([gains(WAN.hidden, (41, TAG_GAIN, s)) for s in range(2)])
    cross = ConditionCase(WAN, 512, seed=42, q_norm=True, k_norm=True)
    case = BlockCase(WAN, wl.policy, wl.pack, wl.resident, seed=43, qk=qk, cross=cross)
    got = case.run()
    rows = sample_rows(WAN.tokens_per_chunk, 24, seed=4)
    want, _ = case.oracle(rows=rows)
    for i in range(len(wl.pack)):
        block_gate(got[i][rows], want[i], f"wan qk+cross node {wl.pack[i]}", ROUNDINGS["all"])


def test_wan_width_qk_norm_256_token_tiles():
    """Wan widths with qk-norm over one 3584-token chunk (one 28 x 128
    frame): the QKV GEMM that also emits the sums of squares runs on
    256-token tiles here (252 tiles, one round), whose v tile is staged
    through LDS in two passes.  Sampled output rows, and the whole cached
    K (normalised) and V pages, against the oracle."""
    import dataclasses
    geo = dataclasses.replace(WAN, grid_h=28, grid_w=128, frames_per_chunk=1)
    qk = np.stack([gains(WAN.hidden, (44, TAG_GAIN, s)) for s in range(2)])
    case = BlockCase(geo, "clean", [(1, 4)], [(0, 0)], seed=45, qk=qk)
    got = case.run()
    rows = sample_rows(geo.tokens_per_chunk, 24, seed=6)
    want, new_kv = case.oracle(rows=rows)
    block_gate(got[0][rows], want[0], "wan-width qk-norm 3584-token node (1, 4)", ROUNDINGS["qk"])
    k_got, v_got = read_pages(case.pool, geo, case.n_slots, case.cache.slots((1, 4)))
    block_gate(k_got, new_kv[0][0], "3584-token cached K (qk-norm)")
    bf16_gates(v_got, new_kv[0][1], "3584-token cached V")
