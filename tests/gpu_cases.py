"""Helpers for the GPU parity tests: seeded states, device buffers, gates.

Inputs come from ``synth`` only; expected values come from ``oracle`` only.
"""
from __future__ import annotations

import math
from typing import Dict, List, Tuple

import numpy as np

import paper_2609_22283_amd as sc
from oracle.attention import node_attention
from oracle.policy import policy as oracle_policy
from oracle.policy import select
from synth import TAG_K, TAG_Q, TAG_V, bf16_bits, bf16_value, normal, normal_parallel

BF16_MAX_ABS = 2e-2
BF16_MEAN_ABS = 2e-3
BF16_REL_FROB = 1e-2      # per (node, head); a dropped 1560-key page scores ~0.2
F32_MAX_ABS = 1e-4


def torch_mod():
    import torch
    return torch


def to_device(x: np.ndarray, dtype: int):
    """fp32 numpy -> device tensor in the cache dtype (bf16 rounded RNE);
    returns (tensor, the exact values as fp64 numpy)."""
    torch = torch_mod()
    if dtype == sc.SC_DTYPE_BF16:
        bits = bf16_bits(x)
        t = torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)
        return t, bf16_value(bits).astype(np.float64)
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
    return t, x.astype(np.float64)


def bits_to_device(bits: np.ndarray):
    """bf16 bit patterns (uint16 numpy) -> a bf16 device tensor."""
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def from_device(t) -> np.ndarray:
    torch = torch_mod()
    if t.dtype == torch.bfloat16:
        return bf16_value(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


class AttnCase:
    """A pack run through sc_attention with seeded Q/K/V, states appended
    without RoPE, and the whole pool poisoned with NaN beforehand (free and
    unreserved slots are NaN, so a stray page read shows up in the output)."""

    def __init__(self, geo, dtype, kind, pack, resident, seed=0, n_slots=None, value_fn=None,
                 n_layers=1, layer=0, policy_kw=None, key_fn=None, query_fn=None):
        torch = torch_mod()
        self.geo, self.dtype, self.kind, self.pack, self.seed = geo, dtype, kind, list(pack), seed
        self.policy_kw = dict(policy_kw or {})  # phi_table / r_mask / n_chunks
        self.layer = layer
        ppc, tpp = geo.frames_per_chunk, geo.tokens_per_page
        states = list(dict.fromkeys(list(resident) + list(pack)))
        n_slots = n_slots or (len(states) + 2) * ppc
        nbytes = sc.sc_cache_pool_bytes(n_layers, geo.heads, geo.head_dim, tpp, ppc, n_slots, dtype)
        self.pool = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
        self.cache = sc.sc_cache_create(self.pool, n_layers, geo.heads, geo.head_dim, tpp, ppc,
                                        n_slots, dtype)
        shape = (geo.tokens_per_chunk, geo.heads, geo.head_dim)
        big = geo.tokens_per_chunk * geo.heads * geo.head_dim > 1 << 20
        gen = normal_parallel if big else normal
        self.kv: Dict[Tuple[int, int], Tuple[np.ndarray, np.ndarray]] = {}
        self._dev = []
        self.key_fn = key_fn
        for st in resident:
            self._append(st, gen, shape, value_fn)
        self.sel = sc.sc_selection_build(kind, geo.K, geo.W, self.pack, **self.policy_kw)
        self.plan = sc.sc_plan_build(self.sel, self.cache)
        for st in self.pack:
            if st not in self.kv:
                self._append(st, gen, shape, value_fn)
        qs, self.q = [], {}
        for i, st in enumerate(self.pack):
            qf = gen(shape, (seed, TAG_Q) + st)
            qs.append(qf if query_fn is None else query_fn(st, qf))
        qt, qv = to_device(np.concatenate(qs, axis=0), dtype)
        self.q_dev = qt
        for i in range(len(self.pack)):
            self.q[i] = qv[i * geo.tokens_per_chunk:(i + 1) * geo.tokens_per_chunk]
        self.o_dev = torch.full_like(qt, float("nan"))
        self.scale = 1.0 / math.sqrt(geo.head_dim)

    def _append(self, st, gen, shape, value_fn):
        kf = gen(shape, (self.seed, TAG_K) + tuple(st))
        if self.key_fn is not None:
            kf = self.key_fn(st, kf)
        vf = gen(shape, (self.seed, TAG_V) + tuple(st)) if value_fn is None else value_fn(st)
        kd, kv = to_device(kf, self.dtype)
        vd, vv = to_device(vf, self.dtype)
        self.cache.append(self.layer, st, kd, vd)
        self._dev += [kd, vd]
        self.kv[tuple(st)] = (kv, vv)

    def run(self):
        torch = torch_mod()
        nws = sc.sc_attention_workspace_bytes(self.plan, self.cache)
        self.workspace_bytes = nws
        # stale contents must not matter: fill the workspace with NaN bytes
        ws = torch.full((max(nws, 1),), 0xFF, dtype=torch.uint8, device="cuda")
        sc.sc_attention(self.plan, self.cache, self.layer, self.q_dev, self.o_dev, self.scale,
                        ws, nws)
        torch.cuda.synchronize()
        out = from_device(self.o_dev)
        n = self.geo.tokens_per_chunk
        return {i: out[i * n:(i + 1) * n] for i in range(len(self.pack))}

    def oracle(self, i, rows=None, segments=None):
        segs = segments if segments is not None else select(
            oracle_policy(self.kind, self.geo.K, self.geo.W, **self.policy_kw), self.pack).segments(i)
        return node_attention(self.q[i], segs, self.kv.__getitem__, self.scale, rows)


def sample_rows(n: int, k: int = 48, seed: int = 0) -> np.ndarray:
    """Rows covering the first/last query tiles and tile boundaries plus a
    random sample."""
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 31, 32, 63, 64, 127, 128, n // 2, n - 129, n - 128, n - 65, n - 64, n - 33,
             n - 32, n - 2, n - 1]
    fixed = [r for r in fixed if 0 <= r < n]
    extra = rng.choice(n, size=min(k, n), replace=False)
    return np.unique(np.concatenate([fixed, extra]))


def bf16_gates(got: np.ndarray, want: np.ndarray, what: str):
    """max-abs, mean-abs and per-head relative Frobenius error of [N, H, d]."""
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    d = np.abs(got - want)
    assert d.max() <= BF16_MAX_ABS, f"{what}: max abs {d.max():.3g}"
    assert d.mean() <= BF16_MEAN_ABS, f"{what}: mean abs {d.mean():.3g}"
    for h in range(want.shape[1]):
        rel = np.linalg.norm(got[:, h] - want[:, h]) / np.linalg.norm(want[:, h])
        assert rel <= BF16_REL_FROB, f"{what}: head {h} relative error {rel:.3g}"
    return float(d.max()), float(d.mean())


def gains(hidden: int, key) -> np.ndarray:
    """RMSNorm gains around 1 (fp32 [hidden])."""
    return (1.0 + normal((hidden,), key, 0.3)).astype(np.float32)


class ConditionCase:
    """A condition cache of n_cond sequences of L tokens (one page each, one
    layer), filled through sc_condition_append, with the oracle's K_c/V_c
    (condition_kv on the same bf16 inputs) and the cross-attention weights.
    Weights are N(0, 1/hidden), so projections of unit-variance inputs have
    unit variance and the cross logits are O(1)."""

    def __init__(self, geo, L, seed, n_cond=1, q_norm=False, k_norm=False, pages=1):
        from oracle.block import BlockShape, condition_kv
        from synth import TAG_CTX, TAG_GAIN, TAG_W_CK, TAG_W_CO, TAG_W_CQ, TAG_W_CV
        torch = torch_mod()
        D = geo.hidden
        self.geo, self.L, self.n_cond = geo, L, n_cond
        tpp = L // pages                                  # a condition spans `pages` page slots
        nbytes = sc.sc_cache_pool_bytes(1, geo.heads, geo.head_dim, tpp, pages, n_cond * pages)
        self.pool = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
        self.cache = sc.sc_cache_create(self.pool, 1, geo.heads, geo.head_dim, tpp, pages, n_cond * pages)
        self.w_dev, self.w = {}, {}
        s = 1.0 / math.sqrt(D)
        for name, tag in (("w_q", TAG_W_CQ), ("w_k", TAG_W_CK), ("w_v", TAG_W_CV), ("w_o", TAG_W_CO)):
            self.w_dev[name], self.w[name] = to_device(normal((D, D), (seed, tag), s), sc.SC_DTYPE_BF16)
        self.g_q = gains(D, (seed, TAG_GAIN, 2)) if q_norm else None
        self.g_k = gains(D, (seed, TAG_GAIN, 3)) if k_norm else None
        self.g_q_dev = None if self.g_q is None else torch.from_numpy(self.g_q).cuda()
        g_k_dev = None if self.g_k is None else torch.from_numpy(self.g_k).cuda()
        shp = BlockShape(D, geo.heads, geo.head_dim, geo.mlp)
        ws_bytes = sc.sc_condition_workspace_bytes(self.cache)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        self.kv, keep = [], []
        for i in range(n_cond):
            ctx_dev, ctx = to_device(normal((L, D), (seed, TAG_CTX, i)), sc.SC_DTYPE_BF16)
            sc.sc_condition_append(self.cache, 0, (i, 0), ctx_dev, self.w_dev["w_k"], self.w_dev["w_v"],
                                   g_k_dev, ws, ws_bytes)
            g_k = None if self.g_k is None else self.g_k.astype(np.float64)
            self.kv.append(condition_kv(ctx, self.w["w_k"], self.w["w_v"], shp, g_k))
            keep.append(ctx_dev)
        torch.cuda.synchronize()
        self.g_k_dev, self.ws, self.ws_bytes = g_k_dev, ws, ws_bytes

    def plan(self, conds, nq):
        return sc.sc_plan_condition(self.cache, [(c, 0) for c in conds], nq)

    def cross_attn(self, n_nodes, nq, cond=0):
        self._plan = self.plan([cond] * n_nodes, nq)
        return sc.CrossAttn(self.w_dev["w_q"], self.w_dev["w_o"], self.cache, self._plan,
                            q_norm=self.g_q_dev)

    def oracle_dict(self, cond=0):
        return {"k": self.kv[cond][0], "v": self.kv[cond][1], "w_q": self.w["w_q"],
                "w_o": self.w["w_o"], "g_q": None if self.g_q is None else self.g_q.astype(np.float64)}
