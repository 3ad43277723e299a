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
