"""Pins of the oracle's attention (CPU only).

Expected values come from outside the oracle:
  * torch's scaled_dot_product_attention in float64 (a library routine) for
    plain attention and for a dense chunk-causal mask;
  * closed forms: zero keys give the mean of the visible values; one-hot
    values give the attention mass of each state;
  * the softmax definition: every row of probabilities sums to one.

The dense mask of the diagonal-pack test is built from chunk indices alone
(block-causal over one concatenated sequence, within the window), never from
the selection table, so it checks Eq. 4-6 and the pipelining claim of
Sec. 3.3 (the progressive diagonal pack is one joint causal forward).
"""
import math

import numpy as np
import pytest
import torch

from oracle.attention import node_attention, packed_attention, row_probabilities
from oracle.policy import policy, select
from synth import normal

SCALE = 1.0 / math.sqrt(16)


def _kv_store(states, n_tok, H, d, seed):
    store = {}
    for (c, l) in states:
        store[(c, l)] = (normal((n_tok, H, d), (seed, 2, c, l)).astype(np.float64),
                         normal((n_tok, H, d), (seed, 3, c, l)).astype(np.float64))
    return store


def _sdpa(q, k, v, mask=None):
    """torch reference, float64: q [Nq,H,d], k/v [Nk,H,d]."""
    qt = torch.from_numpy(np.ascontiguousarray(q.transpose(1, 0, 2)))
    kt = torch.from_numpy(np.ascontiguousarray(k.transpose(1, 0, 2)))
    vt = torch.from_numpy(np.ascontiguousarray(v.transpose(1, 0, 2)))
    m = None if mask is None else torch.from_numpy(mask)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=m, scale=SCALE)
    return o.numpy().transpose(1, 0, 2)


def test_first_chunk_is_plain_attention():
    H, d, n_tok = 2, 16, 24
    store = _kv_store([(0, 3)], n_tok, H, d, 1)
    q = normal((n_tok, H, d), (1, 1, 0, 3)).astype(np.float64)
    sel = select(policy("prog", 4, 3), [(0, 3)])
    o = node_attention(q, sel.segments(0), store.__getitem__, SCALE)
    k, v = store[(0, 3)]
    np.testing.assert_allclose(o, _sdpa(q, k, v), rtol=0, atol=1e-12)


@pytest.mark.parametrize("name", ["prog", "same"])
def test_pack_equals_block_causal_attention(name):
    """Diagonal prog pack (or level-synchronous same-level pack) == block-causal
    attention over one sequence [resident history; pack chunks in order]."""
    K, W, H, d, n_tok = 4, 3, 2, 16, 8
    first = 5
    if name == "prog":
        pack = [(first + i, i + 1) for i in range(K)]          # (5,1) (6,2) (7,3) (8,4)
        hist = [(c, 0) for c in range(first - W, first)]
    else:
        pack = [(first + i, 2) for i in range(K)]
        hist = [(c, 2) for c in range(first - W, first)]
    seq = hist + pack                                          # chunk-ascending
    store = _kv_store(seq, n_tok, H, d, 7)
    sel = select(policy(name, K, W), pack)
    qs = {i: normal((n_tok, H, d), (7, 1) + pack[i]).astype(np.float64) for i in range(len(pack))}
    got = packed_attention(sel, qs.__getitem__, store.__getitem__, SCALE)
    k_all = np.concatenate([store[s][0] for s in seq])
    v_all = np.concatenate([store[s][1] for s in seq])
    chunk_of_key = np.repeat([s[0] for s in seq], n_tok)
    for i, (c, j) in enumerate(pack):
        mask = (chunk_of_key <= c) & (chunk_of_key >= c - W)   # chunk-causal + window
        mask = np.broadcast_to(mask, (n_tok, len(chunk_of_key))).copy()
        want = _sdpa(qs[i], k_all, v_all, mask)
        np.testing.assert_allclose(got[i], want, rtol=0, atol=1e-12)


def test_zero_keys_average_visible_values():
    K, W, H, d, n_tok = 4, 2, 2, 16, 5
    pack = [(3, 1), (4, 2)]
    states = [(1, 0), (2, 0), (3, 1), (4, 2)]
    store = _kv_store(states, n_tok, H, d, 3)
    store = {s: (np.zeros_like(k), v) for s, (k, v) in store.items()}
    sel = select(policy("prog", K, W), pack)
    for i in range(len(pack)):
        q = normal((n_tok, H, d), (3, 1, i)).astype(np.float64)
        o = node_attention(q, sel.segments(i), store.__getitem__, SCALE)
        vis = np.concatenate([store[s][1] for s in sel.segments(i)])
        np.testing.assert_allclose(o, np.broadcast_to(vis.mean(axis=0), o.shape), atol=1e-13)


def test_one_hot_values_give_state_mass():
    """V = one-hot(state id): the output channel of a state is the attention mass
    on its tokens -- zero exactly for states the policy does not select."""
    K, W, H, n_tok = 4, 3, 2, 6
    all_states = [(c, l) for c in range(6) for l in range(K + 1)]
    d = len(all_states) + 2
    store = {}
    for sid, s in enumerate(all_states):
        k = normal((n_tok, H, d), (5, 2) + s).astype(np.float64)
        v = np.zeros((n_tok, H, d))
        v[:, :, sid] = 1.0
        store[s] = (k, v)
    pack = [(4, 1), (5, 2)]
    sel = select(policy("prog", K, W), pack)
    for i in range(len(pack)):
        q = normal((n_tok, H, d), (5, 1, i)).astype(np.float64)
        o = node_attention(q, sel.segments(i), store.__getitem__, 1.0 / math.sqrt(d))
        chosen = set(sel.segments(i))
        for sid, s in enumerate(all_states):
            if s not in chosen:
                assert np.all(o[:, :, sid] == 0.0)
        np.testing.assert_allclose(o[:, :, :len(all_states)].sum(axis=2), 1.0, atol=1e-13)
        # brute force the mass of each chosen state from its own logits
        for h in range(H):
            logits = {s: (q[:, h] @ store[s][0][:, h].T) / math.sqrt(d) for s in chosen}
            m = np.max(np.concatenate(list(logits.values()), axis=1), axis=1, keepdims=True)
            z = sum(np.exp(l - m).sum(axis=1) for l in logits.values())
            for s in chosen:
                mass = np.exp(logits[s] - m).sum(axis=1) / z
                np.testing.assert_allclose(o[:, h, all_states.index(s)], mass, atol=1e-13)


def test_row_sums_are_one():
    K, W, H, d, n_tok = 4, 3, 2, 16, 12
    pack = [(3, 4)]
    sel = select(policy("prog", K, W), pack)
    store = _kv_store(sel.segments(0), n_tok, H, d, 9)
    q = 4.0 * normal((n_tok, H, d), (9, 1)).astype(np.float64)     # sharp rows
    for h in range(H):
        p = row_probabilities(q, sel.segments(0), store.__getitem__, SCALE, h)
        assert np.all(np.abs(p.sum(axis=1) - 1.0) <= 1e-12)
        assert np.all(p >= 0)


def test_packed_equals_sequential_bitwise():
    K, W, H, d, n_tok = 4, 3, 2, 16, 8
    pack = [(5, 1), (6, 2), (7, 3), (8, 4)]
    states = sorted(set(s for i in range(4) for s in select(policy("prog", K, W), pack).segments(i)))
    store = _kv_store(states, n_tok, H, d, 11)
    qs = {i: normal((n_tok, H, d), (11, 1, i)).astype(np.float64) for i in range(4)}
    packed = packed_attention(select(policy("prog", K, W), pack), qs.__getitem__, store.__getitem__, SCALE)
    for i, node in enumerate(pack):
        alone = select(policy("prog", K, W), [node])
        o = node_attention(qs[i], alone.segments(0), store.__getitem__, SCALE)
        assert np.array_equal(o, packed[i])
