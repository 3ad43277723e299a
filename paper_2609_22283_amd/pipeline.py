"""Round driver of the streaming schedule (Sec. 3.3), on top of the C ABI.

Each chunk's current latent state lives in ``xs[c]`` ([tokens, hidden]
bf16), initialised with the chunk's starting noise x^K.  A forward gathers the
states of its nodes into a staging buffer (node order), runs the block stack
(``sc_stack_forward``), and the sampler writes x^{j-1} back into ``xs[c]``
(``sc_sampler_step``); the refresh node (c, 0) only leaves its K/V in the cache.
After every round the states no later node reads are released
(``sc_cache_release_unread``).  Modes:

  packed      Eq. 7 rounds (plus the refresh node), one forward per round
  sequential  the same rounds, one forward per node, oldest chunk first
  serial      Eq. 2 order, one forward per node, chunk by chunk

With ``condition`` set, every block also cross-attends to a cached
condition sequence (the condition c of Eq. 1): per forward, a condition plan
maps each pack node to the condition its chunk reads (``condition_of``), and
each layer's weights are bound to that plan.

Every computation runs in the library; this module sequences calls and moves
device buffers.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

from . import binding as sc


class StackPipeline:
    def __init__(self, *, layers: Sequence["sc.BlockWeights"], cache: "sc.Cache", rope: "sc.Rope",
                 xs, noise, policy: str, K: int, W: int, B: int, t_sched: Sequence[float],
                 refresh: bool = True, stream=None, condition=None):
        """``condition``: optional dict with ``cache`` (an sc.Cache holding the
        condition K/V of every layer), ``cross`` (per layer: (w_q, w_o,
        q_norm or None)) and ``condition_of`` (chunk -> cached condition
        state; default (0, 0))."""
        import torch
        self.torch = torch
        self.layers, self.cache, self.rope = list(layers), cache, rope
        self.xs, self.noise = xs, noise            # [B, n, hidden], [B, K + 2, n, hidden]
        self.policy, self.K, self.W, self.B = policy, K, W, B
        self.t_sched, self.refresh, self.stream = tuple(t_sched), refresh, stream
        self.condition = condition
        self.n_tok, self.hidden = xs.shape[1], xs.shape[2]
        max_pack = K + 1
        self.stage = torch.empty((max_pack * self.n_tok, self.hidden), dtype=xs.dtype, device=xs.device)
        self.ws_bytes = sc.sc_block_workspace_bytes(self.layers[0], max_pack * self.n_tok)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=xs.device)

    # ----------------------------------------------------------- schedules
    def rounds(self) -> List[List[Tuple[int, int]]]:
        n = sc.sc_pipeline_rounds(self.K, self.B, self.refresh)
        return [sc.sc_pipeline_round_nodes(self.K, self.B, self.refresh, r) for r in range(n)]

    def serial_nodes(self) -> List[Tuple[int, int]]:
        n = sc.sc_serial_steps(self.K, self.B, self.refresh)
        return [sc.sc_serial_step_node(self.K, self.B, self.refresh, i) for i in range(n)]

    # ------------------------------------------------------------ forwards
    def forward(self, nodes: Sequence[Tuple[int, int]], layer_hook=None) -> None:
        """One packed forward of ``nodes`` through every layer, then the sampler.

        ``layer_hook(layer, phase, x, plan, layers)``, when given, observes the
        forward layer by layer: it is called with phase "in" before and "out"
        after each layer's block is enqueued (x: the pack's activations,
        layers: the block weights in use).  The layers then run one
        sc_block_forward call each instead of one sc_stack_forward call;
        the work is the same."""
        n = self.n_tok
        sel = sc.sc_selection_build(self.policy, self.K, self.W, nodes)
        plan = sc.sc_plan_build(sel, self.cache)
        for i, (c, _) in enumerate(nodes):
            self.stage[i * n:(i + 1) * n].copy_(self.xs[c])
        x = self.stage[:len(nodes) * n]
        layers = self.layers
        if self.condition is not None:
            cond = self.condition
            of = cond.get("condition_of") or (lambda c: (0, 0))
            plan_c = sc.sc_plan_condition(cond["cache"], [of(c) for c, _ in nodes], n)
            layers = [w.with_cross(sc.CrossAttn(wq, wo, cond["cache"], plan_c, q_norm=qn))
                      for w, (wq, wo, qn) in zip(self.layers, cond["cross"])]
        if layer_hook is None:
            sc.sc_stack_forward(layers, self.cache, plan, x, self.rope, self.ws, self.ws_bytes,
                                self.stream)
        else:
            for l, w in enumerate(layers):
                layer_hook(l, "in", x, plan, layers)
                sc.sc_block_forward(w, self.cache, l, plan, x, self.rope, self.ws, self.ws_bytes,
                                    self.stream)
                layer_hook(l, "out", x, plan, layers)
        for i, (c, j) in enumerate(nodes):
            if j >= 1:
                sc.sc_sampler_step([(c, j)], self.t_sched, self.K, self.xs[c],
                                   self.stage[i * n:(i + 1) * n], self.noise[c, j],
                                   n * self.hidden, self.stream)

    def run(self, mode: str = "packed", time_rounds: bool = False,
            kernel_timer_rounds: Tuple[int, int] = None, layer_hooks=None,
            stop_after: int = None) -> List[float]:
        """Run the whole schedule; returns per-round (or per-node for serial)
        milliseconds when ``time_rounds``.  With ``kernel_timer_rounds =
        (first, last)`` the library's kernel timer records the launches of
        those rounds; ``self.kernel_times`` then maps kernel kinds to
        (launches, total ms).  ``layer_hooks`` maps a round (a forward in
        serial mode) to a layer hook of its forwards (see ``forward``);
        ``stop_after`` ends the run after that round."""
        torch = self.torch
        times = []
        self.kernel_times = {}
        if mode == "serial":
            units = [[node] for node in self.serial_nodes()]
            groups = [[u] for u in units]
        else:
            units = self.rounds()
            groups = [[u] if mode == "packed" else [[node] for node in u] for u in units]
        flat = [node for u in units for node in u]
        done = 0
        for g, group in enumerate(groups):
            if kernel_timer_rounds and g == kernel_timer_rounds[0]:
                sc.sc_timer_enable(True)
            if time_rounds:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
            for nodes in group:
                self.forward(nodes, (layer_hooks or {}).get(g))
                done += len(nodes)
            sc.sc_cache_release_unread(self.cache, self.policy, self.K, self.W, flat[done:])
            if time_rounds:
                e1.record()
                times.append((e0, e1))
            if kernel_timer_rounds and g == kernel_timer_rounds[1]:
                for kind in ("attention", "attention_combine", "gemm_qkv", "gemm_out", "gemm_up",
                             "gemm_down", "qk_norm", "cross_attention", "gemm_cross_q", "gemm_cross_out"):
                    self.kernel_times[kind] = sc.sc_timer_read(kind)
                sc.sc_timer_enable(False)
            if stop_after is not None and g == stop_after:
                break
        if time_rounds:
            torch.cuda.synchronize()
            return [a.elapsed_time(b) for a, b in times]
        return []
