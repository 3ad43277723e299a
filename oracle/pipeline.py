"""Serial and pipelined execution with the sampler -- oracle, test infrastructure only.

Sec. 3.3.  Fully serial execution (Eq. 2) finishes all K updates of chunk c
before chunk c + 1 starts.  The pipeline of Eq. 7 admits one new chunk per
round and advances every active chunk by one level: round n holds the
states x_n^K, x_{n-1}^{K-1}, ..., x_{n-K+1}^1 (0-based chunks here), chunks
outside 0..B-1 omitted.  It spans K + B - 1 rounds and still performs B*K
denoising updates.

Clean-state refresh (a reading: the paper states one clean-state KV refresh
per chunk but not where it runs).  The refresh of chunk c is the node (c, 0):
a forward over the clean state whose output is discarded and whose K/V become
the chunk's clean history.  In the pipeline it joins round n as the node
(n - K, 0), so a round packs [(n-K, 0), (n-K+1, 1), ..., (n, K)] and the
schedule spans K + B rounds with B*(K+1) node forwards.

Sampler (Eq. 1, a reading; parity unpinned beyond x^0 = y at t_0 = 0): the
network predicts the clean state and the next state is re-noised to the next
input time, x^{j-1} = (1 - t_{j-1}) * y + t_{j-1} * xi_{c,j}; the initial
state is x^K = xi_{c,K+1}.  Input times for K = 4 are t = (0, 5/8, 5/6, 15/16, 1)
(the four-step schedule of the training configuration table).
"""
from __future__ import annotations

from typing import Callable, Dict, List, Tuple

import numpy as np

from .block import block_forward
from .policy import Policy, select
from .plan import CacheModel, build_plan

T_SCHEDULE_K4 = (0.0, 5.0 / 8.0, 5.0 / 6.0, 15.0 / 16.0, 1.0)


def pipeline_rounds(B: int, K: int, refresh: bool) -> List[List[Tuple[int, int]]]:
    """Node lists of every round, oldest chunk first (Eq. 7, plus refresh)."""
    rounds = []
    n_rounds = K + B if refresh else K + B - 1
    lowest = 0 if refresh else 1
    for n in range(n_rounds):
        pack = []
        for j in range(lowest, K + 1):
            c = n - K + j
            if 0 <= c < B:
                pack.append((c, j))
        pack.sort()
        rounds.append(pack)
    return rounds


def serial_order(B: int, K: int, refresh: bool) -> List[Tuple[int, int]]:
    """Eq. 2: all updates of chunk 0, then chunk 1, ... (refresh last in a chunk)."""
    order = []
    for c in range(B):
        for j in range(K, 0, -1):
            order.append((c, j))
        if refresh:
            order.append((c, 0))
    return order


def sampler_step(y: np.ndarray, xi: np.ndarray, t_prev: float) -> np.ndarray:
    """x^{j-1} = (1 - t_{j-1}) y + t_{j-1} xi."""
    return (1.0 - t_prev) * np.asarray(y, dtype=np.float64) + t_prev * np.asarray(xi, dtype=np.float64)


def run_stack(packs: List[List[Tuple[int, int]]], pol: Policy, n_layers: int,
              weights_of: Callable[[int], Dict[str, np.ndarray]], noise_of: Callable[[int, int], np.ndarray],
              shp, t_sched=T_SCHEDULE_K4, release: bool = True, n_slots: int = 4096,
              options_of: Callable[[int], Dict] = None):
    """Run the packs in order through an ``n_layers`` block stack.

    Each pack is one forward: every node reads its selected states through
    the model cache (resident ones from earlier packs, in-pack ones from this
    forward, layer by layer).  Returns ({(c, j): y}, cache model, plans).
    Under ``release`` the states that no later pack reads are dropped after
    each pack: levels >= 1 of the pack, and clean chunks older than the next
    pack's window (prog policy; other policies keep everything).
    ``options_of(layer)`` gives that layer's optional block_forward keywords
    (mod, qk_norm, cross).
    """
    K = pol.K
    x_state: Dict[Tuple[int, int], np.ndarray] = {}
    kv: Dict[Tuple[Tuple[int, int], int], Tuple[np.ndarray, np.ndarray]] = {}
    cache = CacheModel(n_slots=n_slots, pages_per_chunk=shp.frames_per_chunk, n_layers=n_layers)
    outputs, plans = {}, []
    for p, pack in enumerate(packs):
        sel = select(pol, pack)
        plans.append(build_plan(sel, cache, shp.grid_h * shp.grid_w))
        xs = []
        for (c, j) in pack:
            if (c, j) not in x_state:
                assert j == K, "only the first update of a chunk starts from noise"
                x_state[(c, j)] = np.asarray(noise_of(c, K + 1), dtype=np.float64)
            xs.append(x_state[(c, j)])
        for layer in range(n_layers):
            y, new_kv = block_forward(sel, lambda i: xs[i], weights_of(layer),
                                      lambda st, l=layer: kv[(st, l)], shp,
                                      **(options_of(layer) if options_of else {}))
            for i, node in enumerate(pack):
                kv[(node, layer)] = new_kv[i]
                cache.append(layer, node)
            xs = [y[i] for i in range(len(pack))]
        for i, (c, j) in enumerate(pack):
            outputs[(c, j)] = xs[i]
            if j >= 1:
                x_state[(c, j - 1)] = sampler_step(xs[i], noise_of(c, j), t_sched[j - 1])
        if release and pol.kind == 2:
            nxt = packs[p + 1] if p + 1 < len(packs) else []
            oldest = min((c for c, _ in nxt), default=None)
            for (c, j) in pack:
                if j >= 1:
                    cache.release((c, j))
            for st in list(cache.slots):
                if st[1] == 0 and (oldest is None or st[0] < oldest - pol.W):
                    cache.release(st)
    return outputs, cache, plans
