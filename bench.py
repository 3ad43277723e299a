#!/usr/bin/env python3
"""Steady-state packed progressive-history DiT step on one MI355X.

One step is one pass of the whole hot path over one pack of in-flight
nodes: the selection table, the plan (availability + page lists), one
Wan2.1-1.3B-shaped DiT block over the packed nodes (RMSNorm, QKV GEMM with
RoPE and the KV-cache append, packed paged attention, out-projection,
RMSNorm, MLP), the sampler step, and the release of the pack's noisy states.

Default workload ("cfg4"): the progressive-history diagonal
[(6,1), (7,2), (8,3), (9,4)] (levels 0 = clean .. 4 = noise) over clean
history chunks 0..5 cached in 1560-token pages; every node attends to its
own chunk plus 6 prior chunks (21 latent frames, 32760 keys).  Inputs are
seeded synthetic tensors (N(0,1) activations and cached K/V, N(0, 0.02)
weights), all resident in HBM before timing.

Prints one JSON line.  ``value`` is latent frames/s per DiT block:
3 latent frames per chunk, K + 1 = 5 node forwards per chunk.

``full_block`` in the same line times the fuller Wan block form on the same
pack: per-level modulation (adaLN table), qk-norm, and cross-attention to a
512-token condition whose K/V were projected and cached once beforehand
(they depend on the condition only, not on the step).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
METRIC = "steady-state latent frames/s per DiT block + attention TFLOP/s (% bf16 MFMA peak)"
# Input times t_0 .. t_4 of the four denoising levels (level 0 clean): the
# training configuration table's schedule 1, 15/16, 5/6, 5/8, noisiest first.
T_SCHEDULE_K4 = (0.0, 5.0 / 8.0, 5.0 / 6.0, 15.0 / 16.0, 1.0)
# HBM bytes per attn_bf16_kernel launch at the default workload: rocprofv3
# FETCH_SIZE and WRITE_SIZE per dispatch, scaled by what the same counters
# read for a plain 256 MiB copy (x2.0 fetch, x1.0 write).  Valid only for the
# kernel sources it was measured on (hash below); otherwise reported as null.
ATTN_TRAFFIC = {"sources_sha1": "c261a262610c20a9c596a956e8688d36f375a5bb",
                "fetch_bytes": 1.3516e+09, "write_bytes": 2.0062e+08}


def attn_traffic():
    import hashlib
    h = hashlib.sha1()
    for f in ("attention.hip", "device.h", "divmagic.h"):
        with open(os.path.join(ROOT, "paper_2609_22283_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != ATTN_TRAFFIC["sources_sha1"]:
        return None
    return round(ATTN_TRAFFIC["fetch_bytes"] + ATTN_TRAFFIC["write_bytes"], -6)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def workload(name):
    from synth.configs import cfg2_clean, cfg3_same, cfg4_prog
    return {"cfg4": cfg4_prog(False), "cfg4R": cfg4_prog(True), "cfg3": cfg3_same(2),
            "cfg2": cfg2_clean(4)}[name]


COND_TOKENS = 512    # condition (text) tokens of the full block form
FULL_FORM = f"level modulation, qk-norm, cross-attention to {COND_TOKENS} condition tokens"


class Setup:
    """Device-resident inputs of one packed block step; ``full`` adds the
    modulation table, qk-norm gains and a cached 512-token condition."""

    def __init__(self, wl, seed=0, full=False):
        import numpy as np
        import torch

        import paper_2609_22283_amd as sc
        from synth import (TAG_CTX, TAG_GAIN, TAG_K, TAG_NOISE, TAG_V, TAG_W_CK, TAG_W_CO, TAG_W_CQ,
                           TAG_W_CV, TAG_W_DOWN, TAG_W_O, TAG_W_QKV, TAG_W_UP, TAG_X, bf16_bits,
                           normal, normal_parallel)
        from synth.configs import WAN as g

        self.sc, self.torch, self.g, self.wl = sc, torch, g, wl
        ppc, tpp, n = g.frames_per_chunk, g.tokens_per_page, g.tokens_per_chunk
        self.n = n

        def dev(x):
            return torch.from_numpy(bf16_bits(x).view(np.int16)).cuda().view(torch.bfloat16)

        n_slots = (len(wl.resident) + 2 * len(wl.pack) + 2) * ppc
        nbytes = sc.sc_cache_pool_bytes(1, g.heads, g.head_dim, tpp, ppc, n_slots)
        self.pool = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        self.cache = sc.sc_cache_create(self.pool, 1, g.heads, g.head_dim, tpp, ppc, n_slots)
        rt = torch.empty(sc.sc_rope_table_bytes(g.grid_h, g.grid_w, g.rope_dims, 256),
                         dtype=torch.uint8, device="cuda")
        self.rope = sc.sc_rope_table_build(rt, g.grid_h, g.grid_w, g.rope_dims, 256, g.theta)
        shape = (n, g.heads, g.head_dim)
        for st in wl.resident:
            k = dev(normal_parallel(shape, (seed, TAG_K) + st))
            v = dev(normal_parallel(shape, (seed, TAG_V) + st))
            self.cache.append(0, st, k, v, rope=self.rope)
        torch.cuda.synchronize()
        D, M = g.hidden, g.mlp
        self.w = [dev(normal_parallel(s, (seed, tag, 0), 0.02)) for s, tag in
                  [((3 * D, D), TAG_W_QKV), ((D, D), TAG_W_O), ((M, D), TAG_W_UP), ((D, M), TAG_W_DOWN)]]
        self.bw = sc.BlockWeights(D, g.heads, g.head_dim, M, *self.w)
        self.full = full
        if full:
            def f32(x):
                return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
            mod = np.stack([np.stack([normal((D,), (seed, 30, j, r), 0.2) for r in range(6)])
                            for j in range(g.K + 1)])
            mod[:, 2] += 1.0
            mod[:, 5] += 1.0
            self.mod = f32(mod)
            self.qk = f32(1.0 + np.stack([normal((D,), (seed, TAG_GAIN, s), 0.3) for s in range(4)]))
            self.wc = {k: dev(normal_parallel((D, D), (seed, tag), 0.02)) for k, tag in
                       [("w_q", TAG_W_CQ), ("w_k", TAG_W_CK), ("w_v", TAG_W_CV), ("w_o", TAG_W_CO)]}
            L = COND_TOKENS
            cb = sc.sc_cache_pool_bytes(1, g.heads, g.head_dim, L, 1, 1)
            self.cond_pool = torch.empty(cb, dtype=torch.uint8, device="cuda")
            self.cond = sc.sc_cache_create(self.cond_pool, 1, g.heads, g.head_dim, L, 1, 1)
            cws = sc.sc_condition_workspace_bytes(self.cond)
            ws = torch.empty(cws, dtype=torch.uint8, device="cuda")
            ctx = dev(normal_parallel((L, D), (seed, TAG_CTX, 0)))
            sc.sc_condition_append(self.cond, 0, (0, 0), ctx, self.wc["w_k"], self.wc["w_v"],
                                   self.qk[3], ws, cws)
            torch.cuda.synchronize()
            del ws, ctx
        T = len(wl.pack) * n
        self.x = dev(np.concatenate([normal_parallel((n, D), (seed, TAG_X) + st) for st in wl.pack]))
        self.noise = dev(np.concatenate([normal_parallel((n, D), (seed, TAG_NOISE) + st)
                                         for st in wl.pack]))
        self.ws_bytes = sc.sc_block_workspace_bytes(self.block_weights(len(wl.pack)), T)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device="cuda")
        self.t_sched = T_SCHEDULE_K4
        torch.cuda.synchronize()

    def block_weights(self, n_nodes):
        """The block's weights for a pack of n_nodes (the full form also plans
        the pack's reads of the condition)."""
        if not self.full:
            return self.bw
        sc, g = self.sc, self.g
        plan_c = sc.sc_plan_condition(self.cond, [(0, 0)] * n_nodes, g.tokens_per_chunk)
        cross = sc.CrossAttn(self.wc["w_q"], self.wc["w_o"], self.cond, plan_c, q_norm=self.qk[2])
        return sc.BlockWeights(g.hidden, g.heads, g.head_dim, g.mlp, *self.w, mod=self.mod,
                               qk_norm=self.qk[0:2], cross=cross)

    def packed_step(self):
        sc, g, wl = self.sc, self.g, self.wl
        sel = sc.sc_selection_build(wl.policy, g.K, g.W, wl.pack)
        plan = sc.sc_plan_build(sel, self.cache)
        sc.sc_block_forward(self.block_weights(len(wl.pack)), self.cache, 0, plan, self.x, self.rope,
                            self.ws, self.ws_bytes)
        sc.sc_sampler_step(wl.pack, self.t_sched, g.K, self.x, self.x, self.noise,
                           self.n * g.hidden)
        for st in wl.pack:
            self.cache.release(st)

    def sequential_step(self):
        """The same nodes one forward each, ascending chunk (history produced
        by an earlier node of the pack is read back from the cache)."""
        sc, g, wl = self.sc, self.g, self.wl
        D = g.hidden
        order = sorted(range(len(wl.pack)), key=lambda i: wl.pack[i])
        for i in order:
            node = wl.pack[i]
            sel = sc.sc_selection_build(wl.policy, g.K, g.W, [node])
            plan = sc.sc_plan_build(sel, self.cache)
            xi = self.x[i * self.n:(i + 1) * self.n]
            sc.sc_block_forward(self.block_weights(1), self.cache, 0, plan, xi, self.rope, self.ws,
                                self.ws_bytes)
            sc.sc_sampler_step([node], self.t_sched, g.K, xi, xi,
                               self.noise[i * self.n:(i + 1) * self.n], self.n * D)
        for st in wl.pack:
            self.cache.release(st)


def time_steps(setup, fn, steps, warmup, timer=False):
    torch, sc = setup.torch, setup.sc
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    if timer:
        sc.sc_timer_enable(True)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / steps
    kernels = {}
    if timer:
        for kind in ("attention", "attention_combine", "gemm_qkv", "gemm_out", "gemm_up",
                     "gemm_down", "rmsnorm", "row_scale", "sampler", "qk_norm", "cross_attention",
                     "gemm_cross_q", "gemm_cross_out"):
            n, tot = sc.sc_timer_read(kind)
            if n:
                kernels[kind] = (n, tot / n)
        sc.sc_timer_enable(False)
    return ms, wall / steps * 1e3, kernels


def mfma_ceiling(iters=4000, launches=5):
    """Sustained rate of the library's matrix-core probe (back-to-back
    16x16x32 bf16 MFMAs from registers, no memory traffic), with random and
    with constant operands: TFLOP/s each, measured right after the timed
    steps.  The gap between the two shows the data-dependent, power-limited
    clock; it is context for the roofline, not a bound."""
    import torch

    import paper_2609_22283_amd as sc
    nb = sc.sc_probe_mfma_out_bytes()
    out = torch.empty(nb, dtype=torch.uint8, device="cuda")
    res = {}
    for rnd in (True, False):
        sc.sc_probe_mfma(rnd, iters, out, nb)                 # warm-up launch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fl = sum(sc.sc_probe_mfma(rnd, iters, out, nb) for _ in range(launches))
        e1.record()
        torch.cuda.synchronize()
        res["random" if rnd else "constant"] = round(fl / (e0.elapsed_time(e1) * 1e-3) / 1e12, 1)
    return res


def segment_counts(wl, g):
    """Segments (chunk-states) each pack node reads, from the library's table."""
    import paper_2609_22283_amd as sc
    off, _, _, _ = sc.sc_selection_build(wl.policy, g.K, g.W, wl.pack).tables()
    return [off[i + 1] - off[i] for i in range(len(wl.pack))]


def attention_flops(wl, g):
    """4 d H sum_i Nq_i Nk_i over the pairs the selection table makes visible."""
    nq = g.tokens_per_chunk
    return 4.0 * g.head_dim * g.heads * sum(nq * (s * nq) for s in segment_counts(wl, g))


def gemm_flops(n_tokens, g):
    D, M = g.hidden, g.mlp
    return 2.0 * n_tokens * (D * 3 * D + D * D + D * M + M * D)


def cpu_baseline(wl, seed=0, row_stride=8, trials=3):
    """The oracle's block on this workload, timed on the host's cores.

    Bounded sample: K/V projections for every token of every pack node (every
    query row reads them), then query-side work (Q, attention, out-projection,
    MLP) for every ``row_stride``-th row only; the query-side time is scaled
    by the row ratio (rows are independent).  The median of ``trials``
    timings.  The oracle runs as it stands: numpy with its BLAS thread pool,
    everything else in one process."""
    import numpy as np

    from oracle.block import BlockShape, block_forward, project_kv
    from oracle.policy import policy, select
    from oracle.rope import chunk_positions, rope
    from synth import (TAG_K, TAG_V, TAG_W_DOWN, TAG_W_O, TAG_W_QKV, TAG_W_UP, TAG_X, bf16_round,
                       normal_parallel)
    from synth.configs import WAN as g

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    n = g.tokens_per_chunk
    shp = BlockShape(g.hidden, g.heads, g.head_dim, g.mlp, g.frames_per_chunk, g.grid_h, g.grid_w,
                     g.rope_dims, g.theta)
    D, M = g.hidden, g.mlp
    w = {k: bf16_round(normal_parallel(s, (seed, tag, 0), 0.02)).astype(np.float64) for k, s, tag in
         [("w_qkv", (3 * D, D), TAG_W_QKV), ("w_o", (D, D), TAG_W_O), ("w_up", (M, D), TAG_W_UP),
          ("w_down", (D, M), TAG_W_DOWN)]}
    res = {}
    for st in wl.resident:
        k = bf16_round(normal_parallel((n, g.heads, g.head_dim), (seed, TAG_K) + st))
        v = bf16_round(normal_parallel((n, g.heads, g.head_dim), (seed, TAG_V) + st))
        pos = chunk_positions(st[0], g.frames_per_chunk, g.grid_h, g.grid_w)
        res[st] = (rope(k, pos, g.rope_dims, g.theta), v.astype(np.float64))
    xs = [bf16_round(normal_parallel((n, D), (seed, TAG_X) + st)).astype(np.float64) for st in wl.pack]
    sel = select(policy(wl.policy, g.K, g.W), wl.pack)
    rows = np.arange(0, n, row_stride)
    runs = []
    for _ in range(trials):
        t0 = time.perf_counter()
        for i, (c, j) in enumerate(wl.pack):
            project_kv(xs[i], c, w["w_qkv"], shp)
        t_kv = time.perf_counter() - t0
        t0 = time.perf_counter()
        block_forward(sel, lambda i: xs[i], w, res.__getitem__, shp, rows=rows)
        t_all = time.perf_counter() - t0
        t_rows = max(t_all - t_kv, 0.0)    # block_forward repeats the K/V projections
        runs.append((t_kv + t_rows * (n / len(rows)), t_kv, t_rows))
    est, t_kv, t_rows = sorted(runs)[len(runs) // 2]
    node_fwd_per_s = len(wl.pack) / est
    return {"value": 3.0 * node_fwd_per_s / (g.K + 1), "unit": "latent frames/s per DiT block",
            "cores": len(os.sched_getaffinity(0)), "blas_threads": int(threads), "kind": "oracle",
            "sample": (f"one block over all {len(wl.pack)} pack nodes, median of {trials} trials: "
                       f"K/V projections of all {n} tokens per node timed in full ({t_kv:.1f} s), "
                       f"query-side work on every {row_stride}th row ({len(rows)} rows/node, "
                       f"{t_rows:.1f} s) scaled x{n / len(rows):.2f}; estimated {est:.1f} s per step")}


def stack_weights(n_layers, seed=0, full=False):
    """bf16 device weights of an n-layer Wan-shaped stack (N(0, 0.02)).  With
    ``full``: per-layer modulation tables, qk-norm gains and cross-attention
    weights, and a condition cache holding a 512-token condition's K/V for
    every layer; returns (layers, keep, condition dict or None)."""
    import concurrent.futures as cf

    import numpy as np
    import torch

    import paper_2609_22283_amd as sc
    from synth import (TAG_CTX, TAG_GAIN, TAG_W_CK, TAG_W_CO, TAG_W_CQ, TAG_W_CV, TAG_W_DOWN, TAG_W_O,
                       TAG_W_QKV, TAG_W_UP, bf16_bits, normal)
    from synth.configs import WAN as g

    D, M = g.hidden, g.mlp
    shapes = [("w_qkv", (3 * D, D), TAG_W_QKV), ("w_o", (D, D), TAG_W_O),
              ("w_up", (M, D), TAG_W_UP), ("w_down", (D, M), TAG_W_DOWN)]
    if full:
        shapes += [("w_cq", (D, D), TAG_W_CQ), ("w_ck", (D, D), TAG_W_CK), ("w_cv", (D, D), TAG_W_CV),
                   ("w_co", (D, D), TAG_W_CO)]
    jobs = [(l, name, shp, tag) for l in range(n_layers) for name, shp, tag in shapes]

    def make(job):
        l, name, shp, tag = job
        return job, bf16_bits(normal(shp, (seed, tag, l), 0.02))

    dev = {}
    with cf.ThreadPoolExecutor(min(16, len(os.sched_getaffinity(0)))) as ex:
        for (l, name, _, _), bits in ex.map(make, jobs):
            dev[(l, name)] = torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)
    if not full:
        layers = [sc.BlockWeights(D, g.heads, g.head_dim, M, dev[(l, "w_qkv")], dev[(l, "w_o")],
                                  dev[(l, "w_up")], dev[(l, "w_down")]) for l in range(n_layers)]
        return layers, dev, None

    def f32(x):
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
    layers, cross = [], []
    L = COND_TOKENS
    cb = sc.sc_cache_pool_bytes(n_layers, g.heads, g.head_dim, L, 1, 1)
    dev["cond_pool"] = torch.empty(cb, dtype=torch.uint8, device="cuda")
    cond = sc.sc_cache_create(dev["cond_pool"], n_layers, g.heads, g.head_dim, L, 1, 1)
    cws = sc.sc_condition_workspace_bytes(cond)
    ws = torch.empty(cws, dtype=torch.uint8, device="cuda")
    ctx = torch.from_numpy(bf16_bits(normal((L, D), (seed, TAG_CTX, 0))).view(np.int16)).cuda().view(torch.bfloat16)
    for l in range(n_layers):
        mod = np.stack([np.stack([normal((D,), (seed, 30, l, j, r), 0.2) for r in range(6)])
                        for j in range(g.K + 1)])
        mod[:, 2] += 1.0
        mod[:, 5] += 1.0
        gains = f32(1.0 + np.stack([normal((D,), (seed, TAG_GAIN, l, k), 0.3) for k in range(4)]))
        dev[(l, "mod")], dev[(l, "gains")] = f32(mod), gains
        layers.append(sc.BlockWeights(D, g.heads, g.head_dim, M, dev[(l, "w_qkv")], dev[(l, "w_o")],
                                      dev[(l, "w_up")], dev[(l, "w_down")], mod=dev[(l, "mod")],
                                      qk_norm=gains[0:2]))
        cross.append((dev[(l, "w_cq")], dev[(l, "w_co")], gains[2]))
        sc.sc_condition_append(cond, l, (0, 0), ctx, dev[(l, "w_ck")], dev[(l, "w_cv")], gains[3], ws, cws)
    torch.cuda.synchronize()
    return layers, dev, {"cache": cond, "cross": cross}


def bench_kv_stream(args):
    """Short-context K/V streaming: nodes of 64 or 128 queries (one latent
    frame of 8x8 or 8x16 tokens, Wan heads 12 x 128) attending to P = 1..21
    pages each, windows disjoint between nodes so every page is read by one
    node only.  Arithmetic intensity is about Nq FLOP per byte of K/V, below
    the bf16 ridge, so the attention streams K/V at HBM speed.  Reports, per
    (Nq, P): the time per launch of back-to-back launches (and with events
    around each launch), algorithmic bytes (K/V of the visible pages, Q, O)
    and GB/s against 8 TB/s; beside them, the plain streaming-read rate of
    the same GPU (sc_probe_read) over 4 GiB (HBM) and 128 MiB (within the
    256 MB last-level cache)."""
    import numpy as np
    import torch

    import paper_2609_22283_amd as sc
    from synth import TAG_K, TAG_Q, TAG_V, bf16_bits, normal_parallel
    from synth.configs import kv_stream

    def dev(x):
        return torch.from_numpy(bf16_bits(x).view(np.int16)).cuda().view(torch.bfloat16)

    rows = []
    # the plain streaming-read ceiling of this GPU, beyond and within the
    # last-level cache (256 MB)
    ceiling = {}
    big = torch.empty(4 << 30, dtype=torch.uint8, device="cuda")
    word = torch.zeros(1, dtype=torch.int32, device="cuda")
    for mib in (4096, 128):
        nbytes = mib << 20
        for _ in range(3):
            sc.sc_probe_read(big, nbytes, word)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            sc.sc_probe_read(big, nbytes, word)
        e1.record()
        torch.cuda.synchronize()
        ceiling[f"read_{mib}_mib_gb_s"] = round(nbytes / (e0.elapsed_time(e1) / args.steps * 1e-3) / 1e9, 1)
    del big
    log(f"[bench] streaming-read probe: {ceiling}")
    for nq in (64, 128):
        g = kv_stream(nq)
        shape = (nq, g.heads, g.head_dim)
        # a small set of distinct random pages, reused round-robin (values
        # only set the arithmetic's data; every page is its own HBM slot)
        bank_k = [dev(normal_parallel(shape, (0, TAG_K, nq, b))) for b in range(16)]
        bank_v = [dev(normal_parallel(shape, (0, TAG_V, nq, b))) for b in range(16)]
        for P in (1, 2, 4, 8, 16, 21):
            n_nodes = min(64, 800 // P)
            W = P - 1
            pack = [(21 * i + W, 4) for i in range(n_nodes)]
            resident = [(21 * i + r, 0) for i in range(n_nodes) for r in range(W)]
            n_slots = len(pack) + len(resident) + 2
            pool = torch.empty(sc.sc_cache_pool_bytes(1, g.heads, g.head_dim, nq, 1, n_slots),
                               dtype=torch.uint8, device="cuda")
            cache = sc.sc_cache_create(pool, 1, g.heads, g.head_dim, nq, 1, n_slots)
            for k, st in enumerate(resident + pack):
                cache.append(0, st, bank_k[k % 16], bank_v[(k + 5) % 16])
            plan = sc.sc_plan_build(sc.sc_selection_build("clean", g.K, W, pack), cache)
            q = dev(normal_parallel((n_nodes * nq, g.heads, g.head_dim), (0, TAG_Q, nq, P)))
            o = torch.empty_like(q)
            nws = sc.sc_attention_workspace_bytes(plan, cache)
            ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda")
            scale = g.head_dim ** -0.5
            for _ in range(3):
                sc.sc_attention(plan, cache, 0, q, o, scale, ws, nws)
            torch.cuda.synchronize()
            # (a) back-to-back launches between two events: the time per
            # launch of a stream of them
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(args.steps):
                sc.sc_attention(plan, cache, 0, q, o, scale, ws, nws)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / args.steps
            # (b) events around each launch (main kernel plus combine)
            sc.sc_timer_enable(True)
            for _ in range(args.steps):
                sc.sc_attention(plan, cache, 0, q, o, scale, ws, nws)
            n, tot = sc.sc_timer_read("attention")
            nc, totc = sc.sc_timer_read("attention_combine")
            sc.sc_timer_enable(False)
            ms_each = (tot + totc) / n
            kv_bytes = n_nodes * P * g.heads * nq * g.head_dim * 2 * 2
            qo_bytes = 2 * n_nodes * nq * g.heads * g.head_dim * 2
            flops = 4.0 * g.head_dim * g.heads * n_nodes * nq * P * nq
            gbs = (kv_bytes + qo_bytes) / (ms * 1e-3) / 1e9
            rows.append({"nq": nq, "pages": P, "nodes": n_nodes, "ms": round(ms, 4),
                         "ms_event_each": round(ms_each, 4),
                         "kv_mb": round(kv_bytes / 1e6, 1), "gb_s": round(gbs, 1),
                         "gb_s_event_each": round((kv_bytes + qo_bytes) / (ms_each * 1e-3) / 1e9, 1),
                         "frac_hbm": round(gbs / PEAK_HBM_GBS, 3),
                         "tflops": round(flops / (ms * 1e-3) / 1e12, 1)})
            log(f"[bench] kv stream nq={nq} pages={P} nodes={n_nodes}: {ms:.4f} ms per launch "
                f"back to back ({ms_each:.4f} with events around each), {gbs:.0f} GB/s, "
                f"{rows[-1]['tflops']} TFLOP/s")
            del cache, pool
    return rows, ceiling


def bench_stack(args):
    """cfg5: the 30-block stack run as a pipeline over B chunks (K = 4, W = 6;
    B = 16 by default, 40 for the paper's 477-frame streams).

    Steady-state rounds are those with a full pack (4 denoising nodes + the
    refresh node) whose oldest node already has a full 6-chunk window; each
    produces one clean chunk (3 latent frames).  Modes: packed (one forward
    per round), sequential (the same nodes one forward each), and the clean
    serial baseline of the paper's latency table (clean history, chunk by
    chunk, 5 forwards per chunk).  The same-level pipeline (Eq. 7 with the
    same-level policy: every level's recent window stays cached) is timed
    packed as well."""
    import numpy as np
    import torch

    import paper_2609_22283_amd as sc
    from paper_2609_22283_amd.pipeline import StackPipeline
    from synth import TAG_NOISE, bf16_bits, normal
    from synth.configs import WAN as g

    L, B, K, W = args.layers, args.chunks, g.K, g.W
    n, D = g.tokens_per_chunk, g.hidden
    t0 = time.perf_counter()
    layers, keep, condition = stack_weights(L, full=args.form == "full")
    noise = torch.empty((B, K + 2, n, D), dtype=torch.bfloat16, device="cuda")
    import concurrent.futures as cf

    def draw(cj):
        return cj, bf16_bits(normal((n, D), (0, TAG_NOISE) + cj))
    with cf.ThreadPoolExecutor(min(16, len(os.sched_getaffinity(0)))) as ex:
        for (c, j), bits in ex.map(draw, [(c, j) for c in range(B) for j in range(K + 2)]):
            noise[c, j].copy_(torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16))
    rt = torch.empty(sc.sc_rope_table_bytes(g.grid_h, g.grid_w, g.rope_dims, 3 * B + 3),
                     dtype=torch.uint8, device="cuda")
    rope = sc.sc_rope_table_build(rt, g.grid_h, g.grid_w, g.rope_dims, 3 * B + 3, g.theta)
    # progressive: W clean chunks + one round in flight; same-level: a W-chunk
    # window per level (K + 1 levels) + one round in flight
    n_slots = ((K + 1) * (W + 1) + K + 2) * g.frames_per_chunk
    nbytes = sc.sc_cache_pool_bytes(L, g.heads, g.head_dim, g.tokens_per_page, g.frames_per_chunk,
                                    n_slots)
    pool = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    log(f"[bench] cfg5 setup {time.perf_counter() - t0:.1f} s: {L} layers, pool {nbytes / 2**30:.1f} GiB")

    def pipeline(policy):
        cache = sc.sc_cache_create(pool, L, g.heads, g.head_dim, g.tokens_per_page,
                                   g.frames_per_chunk, n_slots)
        xs = noise[:, K + 1].clone()
        return StackPipeline(layers=layers, cache=cache, rope=rope, xs=xs, noise=noise,
                             policy=policy, K=K, W=W, B=B, t_sched=T_SCHEDULE_K4,
                             refresh=True, condition=condition)

    # steady rounds: full pack, full window; at most 20 of them, as the
    # paper's latency table measures 20 steady output chunks
    steady = [r for r in range(K + B) if r - K >= W and r < B][:20]
    res = {"trials": args.trials, "steady_rounds": [steady[0], steady[-1]], "per_trial": {}}

    def trials(key, run_once):
        vals = [run_once() for _ in range(args.trials)]
        res["per_trial"][key] = [round(v, 3) for v in vals]
        res[key] = float(np.median(vals))
        log(f"[bench] cfg5 {key}: {res[key]:.2f} ms (median of {args.trials} trials of the median "
            f"steady round, rounds {steady[0]}..{steady[-1]}; trials {res['per_trial'][key]})")

    for key, mode, policy in (("packed", "packed", "prog"), ("sequential", "sequential", "prog"),
                              ("same_packed", "packed", "same")):
        def once(mode=mode, policy=policy):
            ms = pipeline(policy).run(mode, time_rounds=True)
            return float(np.median([ms[r] for r in steady]))
        trials(key, once)
        if key == "packed":  # kernel averages from a further run with the kernel timer on
            pt = pipeline(policy)
            pt.run(mode, kernel_timer_rounds=(steady[0], steady[-1]))
            n_attn, attn_tot = pt.kernel_times["attention"]
            del pt
            res["attn_ms_per_launch"] = attn_tot / max(1, n_attn)
            res["attn_launches"] = n_attn

    def clean_once():
        ms = pipeline("clean").run("serial", time_rounds=True)      # one entry per node
        per_chunk = [sum(ms[c * (K + 1):(c + 1) * (K + 1)]) for c in range(B)]
        return float(np.median([per_chunk[c] for c in range(W, min(B, W + 20))]))
    trials("clean_serial", clean_once)
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10,
                    help="untimed steps first: the first ~6 launches run while the clock ramps")
    ap.add_argument("--workload", default="cfg4",
                    choices=["cfg4", "cfg4R", "cfg3", "cfg2", "cfg5", "kvstream"])
    ap.add_argument("--layers", type=int, default=30, help="cfg5: blocks in the stack")
    ap.add_argument("--trials", type=int, default=3,
                    help="cfg5: trials per mode (the median is reported)")
    ap.add_argument("--chunks", type=int, default=16,
                    help="cfg5: chunks in the stream (40 = the paper's 477-frame videos)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sequential", action="store_true")
    ap.add_argument("--no-probe", action="store_true", help="skip the matrix-core ceiling probe")
    ap.add_argument("--form", default="plain", choices=["plain", "full"],
                    help="block form of the main measurement: plain (RMSNorm, RoPE, attention, "
                         "MLP) or full (plus level modulation, qk-norm, cross-attention)")
    ap.add_argument("--no-full-block", action="store_true",
                    help="with --form plain: skip the extra timing of the full block form")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only copy a 256 MiB device buffer 4 times (calibrates the HBM byte "
                         "counters of a profiler run) and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(collectives and sharding are out of scope); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_probe:
        src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": 256 << 20, "copies": 4}), flush=True)
        return
    if args.workload == "kvstream":
        rows, ceiling = bench_kv_stream(args)
        best = max(rows, key=lambda r: r["gb_s"])
        print(json.dumps({
            "metric": "short-context K/V streaming rate of the packed attention",
            "value": best["gb_s"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": 3,
            "higher_is_better": True, "dtype": "bf16", "data": "synthetic (seeded N(0,1))",
            "config": {"workload": "kvstream: 12x128 heads, one-frame chunks of 64 or 128 tokens, "
                                   "1..21 pages per node, disjoint windows", "parallelism": "single GPU"},
            "roofline": {"bound": "hbm", "achieved": best["gb_s"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(best["gb_s"] / PEAK_HBM_GBS, 4), "traffic": None,
                         "kernel": "attn_bf16_kernel"},
            "read_probe": ceiling, "sweep": rows}), flush=True)
        return
    if args.workload == "cfg5":
        from synth.configs import WAN as g
        r = bench_stack(args)
        wl5 = workload("cfg4R")                    # the steady round's pack and windows
        a_flops = attention_flops(wl5, g)
        attn_tflops = a_flops / (r["attn_ms_per_launch"] * 1e-3) / 1e12
        value = 3.0 / (r["packed"] * 1e-3) * args.layers
        result = {
            "metric": METRIC, "value": round(value, 3), "unit": "latent frames/s per DiT block",
            "n_gpus": 1, "steps": 20, "warmup": 0, "ms_per_step": round(r["packed"], 3),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded noise, N(0,0.02) weights)",
            "config": {"workload": f"cfg5: {args.layers}-block Wan-shaped stack, progressive "
                                   f"pipeline, {args.chunks} chunks x 3 latent frames, K=4, W=6, refresh",
                       "layers": args.layers, "chunks": args.chunks,
                       "block_form": FULL_FORM if args.form == "full" else "plain",
                       "parallelism": "single GPU"},
            "stack_latent_frames_per_s": round(3.0 / (r["packed"] * 1e-3), 3),
            "sequential_ms_per_round": round(r["sequential"], 3),
            "same_level_packed_ms_per_round": round(r["same_packed"], 3),
            "clean_serial_ms_per_chunk": round(r["clean_serial"], 3),
            "packed_vs_sequential": round(r["sequential"] / r["packed"], 3),
            "prog_pipeline_vs_clean_serial": round(r["clean_serial"] / r["packed"], 3),
            "trials": r["trials"], "steady_rounds": r["steady_rounds"], "per_trial_ms": r["per_trial"],
            "attention_tflops": round(attn_tflops, 1),
            "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 1), "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                         "traffic": None, "kernel": "attn_bf16_kernel"},
        }
        if not args.no_cpu_baseline:
            cb = cpu_baseline(wl5)
            cb["sample"] += "; one block of the 5-node steady round (per-block rate)"
            result["cpu_baseline"] = cb
        print(json.dumps(result), flush=True)
        return
    wl = workload(args.workload)
    log(f"[bench] workload {wl.name}: pack {wl.pack}, resident {len(wl.resident)} states")
    setup = Setup(wl, full=args.form == "full")
    g = setup.g
    # the step time without the kernel timer (its two event records per
    # launch are measurement, not product); per-kernel averages from a second
    # pass of the same steps with the timer on
    ms, wall_ms, _ = time_steps(setup, setup.packed_step, args.steps, args.warmup)
    _, _, kernels = time_steps(setup, setup.packed_step, args.steps, 1, timer=True)
    log(f"[bench] packed: {ms:.3f} ms/step (host wall {wall_ms:.3f})")
    seq_ms = None
    if not args.no_sequential:
        seq_ms, _, _ = time_steps(setup, setup.sequential_step, max(3, args.steps // 2), 1)
        log(f"[bench] sequential: {seq_ms:.3f} ms/step")

    n_nodes = len(wl.pack)
    T = n_nodes * g.tokens_per_chunk
    a_flops = attention_flops(wl, g)
    g_flops = gemm_flops(T, g)
    attn_n, attn_ms = kernels.get("attention", (0, float("nan")))
    attn_tflops = a_flops / (attn_ms * 1e-3) / 1e12
    gemm_ms = sum(kernels[k][1] for k in ("gemm_qkv", "gemm_out", "gemm_up", "gemm_down") if k in kernels)
    node_fwd_per_s = n_nodes / (ms * 1e-3)
    value = 3.0 * node_fwd_per_s / (g.K + 1)
    result = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "latent frames/s per DiT block",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations and cached K/V, N(0,0.02) weights)",
        "config": {"workload": f"{wl.name}: {wl.description}", "nodes": wl.pack,
                   "policy": wl.policy, "tokens_per_node": g.tokens_per_chunk,
                   "keys_per_node": [s * g.tokens_per_chunk for s in segment_counts(wl, g)],
                   "hidden": g.hidden, "heads": g.heads,
                   "head_dim": g.head_dim, "mlp": g.mlp, "page_tokens": g.tokens_per_page,
                   "block_form": FULL_FORM if args.form == "full" else "plain",
                   "parallelism": "single GPU"},
        "attention_tflops": round(attn_tflops, 1),
        "attention_pct_peak": round(100.0 * attn_tflops / PEAK_BF16_TFLOPS, 2),
        "attention_ms": round(attn_ms, 4),
        "attention_combine_ms": round(kernels["attention_combine"][1], 4) if "attention_combine" in kernels else 0.0,
        "gemm_tflops": round(g_flops / (gemm_ms * 1e-3) / 1e12, 1) if gemm_ms else None,
        "kernel_avg_ms": {k: round(v[1], 4) for k, v in kernels.items()},
        "sequential_ms_per_step": round(seq_ms, 4) if seq_ms else None,
        "packed_vs_sequential": round(seq_ms / ms, 3) if seq_ms else None,
        "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 1), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": attn_traffic() if wl.name == "cfg4-prog" else None,
                     "kernel": "attn_bf16_kernel",
                     "algorithmic_per_launch": f"{a_flops:.4e} FLOP"},
    }
    if args.form == "plain" and not args.no_full_block:
        del setup
        full = Setup(wl, full=True)
        fms, _, _ = time_steps(full, full.packed_step, args.steps, args.warmup)
        _, _, fk = time_steps(full, full.packed_step, args.steps, 1, timer=True)
        log(f"[bench] full block form: {fms:.3f} ms/step")
        fseq = None
        if not args.no_sequential:
            fseq, _, _ = time_steps(full, full.sequential_step, max(3, args.steps // 2), 1)
            log(f"[bench] full block form, sequential: {fseq:.3f} ms/step")
        del full
        result["full_block"] = {
            "form": FULL_FORM,
            "ms_per_step": round(fms, 4),
            "value": round(3.0 * n_nodes / (fms * 1e-3) / (g.K + 1), 3),
            "unit": "latent frames/s per DiT block",
            "sequential_ms_per_step": round(fseq, 4) if fseq else None,
            "packed_vs_sequential": round(fseq / fms, 3) if fseq else None,
            "kernel_avg_ms": {k: round(v[1], 4) for k, v in fk.items()},
        }
    if not args.no_probe:
        ceil = mfma_ceiling()
        log(f"[bench] matrix-core probe: {ceil} TFLOP/s")
        result["mfma_sustained_tflops"] = ceil
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host (bounded sample)...")
        result["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
