"""Pins of the oracle's RoPE, RMSNorm, GELU, block and pipeline (CPU only).

RoPE and the block form are readings (the paper defines neither): their pins
are mathematical properties that any correct implementation of the stated
reading satisfies, plus special cases with closed forms.
"""
import math

import numpy as np
import pytest

from oracle.block import BlockShape, block_forward, gelu_tanh, rmsnorm
from oracle.pipeline import pipeline_rounds, run_stack, serial_order
from oracle.policy import policy, select
from oracle.rope import chunk_positions, rope
from synth import normal

DIMS = (12, 10, 10)


def _pos(n, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 60, size=(n, 3))


def test_rope_identity_at_origin_and_norm():
    x = normal((7, 3, 32), (1,)).astype(np.float64)
    np.testing.assert_array_equal(rope(x, np.zeros((7, 3), dtype=int), DIMS), x)
    y = rope(x, _pos(7, 0), DIMS)
    np.testing.assert_allclose(np.linalg.norm(y, axis=2), np.linalg.norm(x, axis=2), rtol=1e-13)
    # each channel pair keeps its own length (a rotation inside the pair)
    np.testing.assert_allclose(y[..., 0::2] ** 2 + y[..., 1::2] ** 2,
                               x[..., 0::2] ** 2 + x[..., 1::2] ** 2, rtol=1e-12, atol=1e-14)


def test_rope_relative_positions():
    """<R(p+s) q, R(p'+s) k> == <R(p) q, R(p') k> for any shift s of all axes."""
    q = normal((5, 2, 32), (2,)).astype(np.float64)
    k = normal((5, 2, 32), (3,)).astype(np.float64)
    p1, p2 = _pos(5, 1), _pos(5, 2)
    shift = np.array([[7, 3, 11]])
    a = np.einsum("nhd,mhd->hnm", rope(q, p1, DIMS), rope(k, p2, DIMS))
    b = np.einsum("nhd,mhd->hnm", rope(q, p1 + shift, DIMS), rope(k, p2 + shift, DIMS))
    np.testing.assert_allclose(a, b, atol=1e-11)


def test_rope_composes_and_first_pair_rotates_by_position():
    x = normal((4, 1, 32), (4,)).astype(np.float64)
    p1, p2 = _pos(4, 3), _pos(4, 4)
    np.testing.assert_allclose(rope(rope(x, p1, DIMS), p2, DIMS), rope(x, p1 + p2, DIMS), atol=1e-12)
    # the first pair of each axis has frequency 1: its angle moves by the position
    pos = np.array([[1, 0, 0], [0, 2, 0], [0, 0, 3], [0, 0, 0]])
    y = rope(x, pos, DIMS)
    starts = [0, DIMS[0] // 2, (DIMS[0] + DIMS[1]) // 2]
    for a, p in enumerate(starts):
        ang_x = np.arctan2(x[a, 0, 2 * p + 1], x[a, 0, 2 * p])
        ang_y = np.arctan2(y[a, 0, 2 * p + 1], y[a, 0, 2 * p])
        delta = (ang_y - ang_x - pos[a, a]) % (2 * math.pi)
        assert min(delta, 2 * math.pi - delta) < 1e-12


def test_chunk_positions():
    pos = chunk_positions(2, 3, 2, 4)
    assert pos.shape == (24, 3)
    assert list(pos[0]) == [6, 0, 0] and list(pos[5]) == [6, 1, 1] and list(pos[23]) == [8, 1, 3]


def test_rmsnorm_and_gelu():
    x = 3.0 * normal((10, 64), (5,)).astype(np.float64)
    r = rmsnorm(x)
    np.testing.assert_allclose(np.sqrt(np.mean(r * r, axis=1)), 1.0, rtol=1e-6)
    # tanh GELU vs the exact erf GELU: the approximation error is below 1e-3
    t = np.linspace(-8, 8, 4001)
    exact = np.array([0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in t])
    assert np.max(np.abs(gelu_tanh(t) - exact)) < 1e-3
    assert gelu_tanh(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(gelu_tanh(np.array([20.0, -20.0])), [20.0, 0.0], atol=1e-12)


def _tiny_shape():
    return BlockShape(hidden=32, heads=2, head_dim=16, mlp=48, frames_per_chunk=2,
                      grid_h=2, grid_w=3, rope_dims=(6, 6, 4))


def _weights(shp, layer, seed=0, zero_out=False):
    D, M = shp.hidden, shp.mlp
    w = {"w_qkv": normal((3 * D, D), (seed, 10, layer), 0.2).astype(np.float64),
         "w_o": normal((D, D), (seed, 11, layer), 0.2).astype(np.float64),
         "w_up": normal((M, D), (seed, 12, layer), 0.2).astype(np.float64),
         "w_down": normal((D, M), (seed, 13, layer), 0.2).astype(np.float64)}
    if zero_out:
        w["w_o"][:] = 0
        w["w_down"][:] = 0
    return w


def test_block_identity_with_zero_output_weights():
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(0, 4)])
    x = normal((shp.tokens_per_chunk, shp.hidden), (1, 4)).astype(np.float64)
    y, kv = block_forward(sel, lambda i: x, _weights(shp, 0, zero_out=True), None, shp)
    np.testing.assert_array_equal(y[0], x)


def test_block_single_token_attention_is_value_projection():
    """With one token per chunk and no history, attention returns that token's V."""
    shp = BlockShape(hidden=32, heads=2, head_dim=16, mlp=48, frames_per_chunk=1,
                     grid_h=1, grid_w=1, rope_dims=(6, 6, 4))
    w = _weights(shp, 0)
    w["w_up"][:] = 0                                   # MLP branch vanishes
    sel = select(policy("clean", 4, 0), [(3, 2)])
    x = normal((1, shp.hidden), (2,)).astype(np.float64)
    y, _ = block_forward(sel, lambda i: x, w, None, shp)
    h = rmsnorm(x)
    v = h @ w["w_qkv"][2 * shp.hidden:].T
    np.testing.assert_allclose(y[0], x + v @ w["w_o"].T, atol=1e-12)


def test_block_rows_subset_matches_full():
    shp = _tiny_shape()
    pack = [(1, 1), (2, 2)]
    sel = select(policy("prog", 4, 2), pack)
    xs = [normal((shp.tokens_per_chunk, shp.hidden), (3, i)).astype(np.float64) for i in range(2)]
    res = {(0, 0): tuple(normal((shp.tokens_per_chunk, 2, 16), (3, t, 0)).astype(np.float64) for t in (2, 3))}
    full, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), res.__getitem__, shp)
    rows = [0, 5, 11]
    part, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), res.__getitem__, shp, rows=rows)
    for i in range(2):
        np.testing.assert_array_equal(part[i], full[i][rows])


def _mod_table(shp, K, seed, neutral=False):
    """[K+1][6][hidden]: shift_a, scale_a, gate_a, shift_m, scale_m, gate_m."""
    m = np.zeros((K + 1, 6, shp.hidden))
    if neutral:
        m[:, 2] = 1.0
        m[:, 5] = 1.0
        return m
    for j in range(K + 1):
        for r in range(6):
            m[j, r] = normal((shp.hidden,), (seed, 30, j, r), 0.2).astype(np.float64)
        m[j, 2] += 1.0
        m[j, 5] += 1.0
    return m


def test_block_neutral_modulation_is_unconditioned_block():
    """shift = scale = 0 and gate = 1 at every level reproduce the
    unconditioned block exactly."""
    shp = _tiny_shape()
    pack = [(1, 1), (2, 2), (3, 3)]
    sel = select(policy("prog", 4, 2), pack)
    xs = [normal((shp.tokens_per_chunk, shp.hidden), (5, i)).astype(np.float64) for i in range(3)]
    res = {(0, 0): tuple(normal((shp.tokens_per_chunk, 2, 16), (5, t, 0)).astype(np.float64)
                         for t in (2, 3))}
    plain, kv0 = block_forward(sel, lambda i: xs[i], _weights(shp, 0), res.__getitem__, shp)
    neutral, kv1 = block_forward(sel, lambda i: xs[i], _weights(shp, 0), res.__getitem__, shp,
                                 mod=_mod_table(shp, 4, 0, neutral=True))
    for i in range(3):
        np.testing.assert_array_equal(neutral[i], plain[i])
        np.testing.assert_array_equal(kv0[i][0], kv1[i][0])


def test_block_modulation_gates():
    """Zero gates make the block the identity whatever the shifts and scales;
    with the MLP gate at zero, the residual update is linear in the attention
    gate; and the level of each node picks its own row."""
    shp = _tiny_shape()
    pack = [(0, 3), (1, 4)]
    sel = select(policy("prog", 4, 2), pack)
    xs = [normal((shp.tokens_per_chunk, shp.hidden), (6, i)).astype(np.float64) for i in range(2)]
    m = _mod_table(shp, 4, 1)
    m0 = m.copy()
    m0[:, 2] = 0.0
    m0[:, 5] = 0.0
    y, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), None, shp, mod=m0)
    for i in range(2):
        np.testing.assert_array_equal(y[i], xs[i])
    m1 = m.copy()
    m1[:, 5] = 0.0
    m2 = m1.copy()
    m2[:, 2] *= 2.0
    y1, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), None, shp, mod=m1)
    y2, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), None, shp, mod=m2)
    for i in range(2):
        np.testing.assert_allclose(y2[i] - xs[i], 2.0 * (y1[i] - xs[i]), rtol=1e-12, atol=1e-12)
    # changing the row of a level no pack node has leaves the outputs unchanged
    m3 = m.copy()
    m3[2] += 5.0
    ya, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), None, shp, mod=m)
    yb, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), None, shp, mod=m3)
    for i in range(2):
        np.testing.assert_array_equal(ya[i], yb[i])


def test_pipeline_counts():
    """K + B - 1 rounds and B*K updates (Sec. 3.3); with the refresh node
    K + B rounds and B*(K+1) forwards; first clean chunk after K rounds."""
    B, K = 16, 4
    r = pipeline_rounds(B, K, refresh=False)
    assert len(r) == K + B - 1 and sum(len(p) for p in r) == B * K
    assert sorted(n for p in r for n in p) == sorted((c, j) for c in range(B) for j in range(1, K + 1))
    finishing = [n for n, p in enumerate(r) if any(j == 1 for _, j in p)]
    assert finishing[0] == K - 1 and finishing == list(range(K - 1, K - 1 + B))
    rr = pipeline_rounds(B, K, refresh=True)
    assert len(rr) == K + B and sum(len(p) for p in rr) == B * (K + 1)
    assert max(len(p) for p in rr) == K + 1
    assert rr[10] == [(6, 0), (7, 1), (8, 2), (9, 3), (10, 4)]
    s = serial_order(B, K, refresh=False)
    assert len(s) == B * K and s[:K] == [(0, 4), (0, 3), (0, 2), (0, 1)]


def test_serial_and_pipelined_progressive_agree_bitwise():
    """Serial execution admits progressive history when states are retained
    (Sec. 3.3); the pipelined schedule computes the same updates."""
    shp = _tiny_shape()
    B, K, L = 5, 3, 2
    pol = policy("prog", K, 2)
    noise = lambda c, j: normal((shp.tokens_per_chunk, shp.hidden), (9, 20, c, j))
    weights = {l: _weights(shp, l) for l in range(L)}
    pipe, _, _ = run_stack(pipeline_rounds(B, K, True), pol, L, weights.__getitem__, noise, shp,
                           t_sched=(0.0, 0.5, 0.75, 1.0))
    ser, _, _ = run_stack([[n] for n in serial_order(B, K, True)], pol, L, weights.__getitem__, noise,
                          shp, t_sched=(0.0, 0.5, 0.75, 1.0), release=False)
    assert set(pipe) == set(ser) and len(pipe) == B * (K + 1)
    for node in pipe:
        assert np.array_equal(pipe[node], ser[node]), node


# ---- qk-norm and cross-attention to the condition (Wan block form) ----

def _pack_inputs(shp, seed, n=2):
    xs = [normal((shp.tokens_per_chunk, shp.hidden), (seed, i)).astype(np.float64) for i in range(n)]
    res = {(0, 0): tuple(normal((shp.tokens_per_chunk, 2, 16), (seed, t, 0)).astype(np.float64)
                         for t in (2, 3))}
    return xs, res


def _gains(shp, seed):
    return tuple(1.0 + normal((shp.hidden,), (seed, 40, s), 0.3).astype(np.float64) for s in range(2))


def test_qk_norm_removes_projection_scale():
    """With qk-norm the block no longer sees the scale of Wq and Wk (up to the
    eps of the norm); without it, the same rescale changes the output."""
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(1, 1), (2, 2)])
    xs, res = _pack_inputs(shp, 7)
    w = _weights(shp, 0)
    ws = {k: v.copy() for k, v in w.items()}
    ws["w_qkv"][:shp.hidden] *= 4.0
    ws["w_qkv"][shp.hidden:2 * shp.hidden] *= 0.25
    g = _gains(shp, 1)
    a, kva = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, qk_norm=g)
    b, kvb = block_forward(sel, lambda i: xs[i], ws, res.__getitem__, shp, qk_norm=g)
    c, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp)
    d, _ = block_forward(sel, lambda i: xs[i], ws, res.__getitem__, shp)
    for i in range(2):
        # eps / (mean square of the projection, about 1.3 here) bounds the change
        np.testing.assert_allclose(b[i], a[i], rtol=0, atol=1e-4)
        np.testing.assert_allclose(kvb[i][0], kva[i][0], rtol=0, atol=1e-4)
        assert np.max(np.abs(d[i] - c[i])) > 1e-2
        assert np.max(np.abs(a[i] - c[i])) > 1e-2


def test_qk_norm_gains_enter_as_a_product():
    """Gains constant over each RoPE pair commute with the rotation, so only
    g_q * g_k reaches the logits: (s g, g / s) equals (g, g) up to rounding,
    when the resident history's keys carry the same 1 / s."""
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(1, 1), (2, 2)])
    xs, res = _pack_inputs(shp, 8)
    k0, v0 = res[(0, 0)]
    res_s = {(0, 0): (k0 / 3.0, v0)}
    w = _weights(shp, 0)
    g = np.repeat(1.0 + normal((shp.hidden // 2,), (9, 41), 0.3).astype(np.float64), 2)
    a, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, qk_norm=(g, g))
    b, _ = block_forward(sel, lambda i: xs[i], w, res_s.__getitem__, shp,
                         qk_norm=(3.0 * g, g / 3.0))
    for i in range(2):
        np.testing.assert_allclose(b[i], a[i], rtol=1e-12, atol=1e-12)


def test_qk_norm_cached_keys_have_unit_rms_over_the_width():
    """With unit gains each cached key has mean square 1 over the whole hidden
    width (RoPE keeps lengths); the per-head mean squares differ, so the norm
    does not act head by head."""
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(0, 4)])
    xs, _ = _pack_inputs(shp, 9, n=1)
    one = np.ones(shp.hidden)
    _, kv = block_forward(sel, lambda i: xs[i], _weights(shp, 0), None, shp, qk_norm=(one, one))
    k = kv[0][0]
    ms = np.mean(k.reshape(k.shape[0], -1) ** 2, axis=1)
    np.testing.assert_allclose(ms, 1.0, rtol=1e-5)
    per_head = np.mean(k ** 2, axis=2)
    assert np.max(np.abs(per_head - 1.0)) > 1e-2


def _cross(shp, L, seed, g_q=None, g_k=None):
    from oracle.block import condition_kv
    D = shp.hidden
    ctx = normal((L, D), (seed, 50)).astype(np.float64)
    wk, wv = (normal((D, D), (seed, 51 + s), 0.2).astype(np.float64) for s in range(2))
    k, v = condition_kv(ctx, wk, wv, shp, g_k)
    return {"k": k, "v": v, "g_q": g_q,
            "w_q": normal((D, D), (seed, 53), 0.2).astype(np.float64),
            "w_o": normal((D, D), (seed, 54), 0.2).astype(np.float64)}


def test_cross_attention_with_zero_output_projection_is_the_plain_block():
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(1, 1), (2, 2)])
    xs, res = _pack_inputs(shp, 10)
    cr = _cross(shp, 5, 0)
    cr["w_o"][:] = 0.0
    a, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), res.__getitem__, shp)
    b, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), res.__getitem__, shp, cross=cr)
    for i in range(2):
        np.testing.assert_array_equal(b[i], a[i])


def _no_mlp(shp):
    w = _weights(shp, 0)
    w["w_down"][:] = 0.0
    return w


def test_cross_attention_single_and_constant_keys():
    """One condition token: every row adds v W_co^T.  Identical keys: every
    row adds mean(V) W_co^T (uniform weights).  The MLP is switched off so the
    block output is x' + cross term."""
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(1, 1), (2, 2)])
    xs, res = _pack_inputs(shp, 11)
    w = _no_mlp(shp)
    base, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp)
    one = _cross(shp, 1, 1)
    y1, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, cross=one)
    add1 = one["v"].reshape(1, -1) @ one["w_o"].T
    flat = _cross(shp, 6, 2)
    flat["k"] = np.repeat(flat["k"][:1], 6, axis=0)
    yc, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, cross=flat)
    addc = flat["v"].reshape(6, -1).mean(axis=0, keepdims=True) @ flat["w_o"].T
    for i in range(2):
        np.testing.assert_allclose(y1[i] - base[i], np.repeat(add1, len(xs[i]), 0), atol=1e-12)
        np.testing.assert_allclose(yc[i] - base[i], np.repeat(addc, len(xs[i]), 0), atol=1e-12)


def test_cross_attention_two_tokens_logistic_weights():
    """Two condition tokens: the weight of the first is the logistic function
    of the scaled logit difference, per head.  The cross query reads the
    self-attention residual x' (the plain block without MLP gives x')."""
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(0, 4)])
    xs, _ = _pack_inputs(shp, 12, n=1)
    w = _no_mlp(shp)
    cr = _cross(shp, 2, 3)
    y, _ = block_forward(sel, lambda i: xs[i], w, None, shp, cross=cr)
    x1, _ = block_forward(sel, lambda i: xs[i], w, None, shp)
    assert np.max(np.abs(x1[0] - xs[0])) > 1e-2
    q = (rmsnorm(x1[0]) @ cr["w_q"].T).reshape(-1, 2, 16)
    k, v = cr["k"], cr["v"]
    o = np.zeros_like(q)
    for h in range(2):
        dl = (q[:, h] @ (k[0, h] - k[1, h])) / 4.0        # 1/sqrt(16)
        p0 = 1.0 / (1.0 + np.exp(-dl))
        o[:, h] = p0[:, None] * v[0, h] + (1.0 - p0)[:, None] * v[1, h]
    np.testing.assert_allclose(y[0] - x1[0], o.reshape(len(q), -1) @ cr["w_o"].T, atol=1e-12)


def test_cross_attention_feeds_the_mlp():
    """Self-attention off (W_o = 0) and one condition token: the cross term is
    the constant a = v W_co^T, so the block on x equals the plain block on
    x + a (the MLP reads x + a)."""
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(0, 4)])
    xs, _ = _pack_inputs(shp, 15, n=1)
    w = _weights(shp, 0)
    w["w_o"][:] = 0.0
    one = _cross(shp, 1, 8)
    a = one["v"].reshape(1, -1) @ one["w_o"].T
    y, _ = block_forward(sel, lambda i: xs[i], w, None, shp, cross=one)
    ref, _ = block_forward(sel, lambda i: xs[i] + a, w, None, shp)
    np.testing.assert_allclose(y[0], ref[0], rtol=1e-12, atol=1e-12)


def test_cross_attention_zero_query_gain_is_uniform():
    """g_cq = 0 zeroes every cross logit: each row adds mean(V) W_co^T."""
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(1, 1), (2, 2)])
    xs, res = _pack_inputs(shp, 16)
    w = _no_mlp(shp)
    base, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp)
    cr = _cross(shp, 5, 9, g_q=np.zeros(shp.hidden), g_k=_gains(shp, 2)[1])
    y, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, cross=cr)
    add = cr["v"].reshape(5, -1).mean(axis=0, keepdims=True) @ cr["w_o"].T
    for i in range(2):
        np.testing.assert_allclose(y[i] - base[i], np.repeat(add, len(xs[i]), 0), atol=1e-12)


def test_cross_attention_ignores_condition_order_and_query_scale():
    """The condition has no positions: permuting its tokens leaves the block
    unchanged.  With the query norm (g_cq) the scale of W_cq drops out, and
    only g_cq * g_ck reaches the logits."""
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(1, 1), (2, 2)])
    xs, res = _pack_inputs(shp, 13)
    w = _weights(shp, 0)
    g_q, g_k = _gains(shp, 4)
    cr = _cross(shp, 7, 5, g_q=g_q, g_k=g_k)
    perm = np.random.default_rng(0).permutation(7)
    cp = dict(cr, k=cr["k"][perm], v=cr["v"][perm])
    cs = dict(cr, w_q=cr["w_q"] * 5.0)
    cg = _cross(shp, 7, 5, g_q=g_q * 4.0, g_k=g_k / 4.0)
    a, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, cross=cr)
    b, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, cross=cp)
    c, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, cross=cs)
    d, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, cross=cg)
    for i in range(2):
        np.testing.assert_allclose(b[i], a[i], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(c[i], a[i], rtol=0, atol=1e-5)
        np.testing.assert_allclose(d[i], a[i], rtol=1e-12, atol=1e-12)


def test_cross_and_qk_norm_rows_subset_matches_full():
    shp = _tiny_shape()
    sel = select(policy("prog", 4, 2), [(1, 1), (2, 2)])
    xs, res = _pack_inputs(shp, 14)
    g = _gains(shp, 6)
    cr = _cross(shp, 4, 7, g_q=g[0], g_k=g[1])
    full, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), res.__getitem__, shp,
                           qk_norm=g, cross=cr)
    rows = [1, 4, 10]
    part, _ = block_forward(sel, lambda i: xs[i], _weights(shp, 0), res.__getitem__, shp,
                            rows=rows, qk_norm=g, cross=cr)
    for i in range(2):
        np.testing.assert_array_equal(part[i], full[i][rows])


def test_condition_kv_is_linear_and_key_norm_is_scale_free():
    """V_c (and K_c without its norm) is linear in the condition; with the
    norm, K_c ignores the condition's scale (up to eps)."""
    from oracle.block import condition_kv
    shp = _tiny_shape()
    D = shp.hidden
    c1, c2 = (normal((4, D), (17, s)).astype(np.float64) for s in range(2))
    wk, wv = (normal((D, D), (17, 2 + s), 0.2).astype(np.float64) for s in range(2))
    k1, v1 = condition_kv(c1, wk, wv, shp)
    k2, v2 = condition_kv(c2, wk, wv, shp)
    k3, v3 = condition_kv(2.0 * c1 - 0.5 * c2, wk, wv, shp)
    np.testing.assert_allclose(v3, 2.0 * v1 - 0.5 * v2, atol=1e-12)
    np.testing.assert_allclose(k3, 2.0 * k1 - 0.5 * k2, atol=1e-12)
    g = _gains(shp, 3)[1]
    kn, vn = condition_kv(c1, wk, wv, shp, g)
    kb, vb = condition_kv(8.0 * c1, wk, wv, shp, g)
    np.testing.assert_allclose(kb, kn, rtol=2e-6)       # eps / mean square, halved
    np.testing.assert_allclose(vb, 8.0 * vn, atol=1e-12)
    np.testing.assert_array_equal(vn, v1)


def test_cross_attention_per_node_condition():
    """A per-node condition function gives each node the block it would get
    alone with that condition."""
    shp = _tiny_shape()
    pack = [(1, 1), (2, 2)]
    sel = select(policy("prog", 4, 2), pack)
    xs, res = _pack_inputs(shp, 18)
    w = _weights(shp, 0)
    crs = [_cross(shp, 5, 20), _cross(shp, 3, 21)]
    mixed, _ = block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp,
                             cross=lambda node: crs[node[0] - 1])
    for i in range(2):
        alone, _ = block_forward(sel, lambda k: xs[k], w, res.__getitem__, shp, cross=crs[i])
        np.testing.assert_array_equal(mixed[i], alone[i])
    one, _ = block_forward(sel, lambda k: xs[k], w, res.__getitem__, shp, cross=crs[0])
    assert np.max(np.abs(one[1] - mixed[1])) > 1e-3
