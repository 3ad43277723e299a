"""Availability and page resolution over a paged KV cache -- oracle, test infrastructure only.

The effective context C of a node is the cached representation (keys and
values) of each selected state (Sec. 3.2, "Effective context and
visibility"); its visibility mask (Eq. 6) is 0 on exactly those tokens and
-inf elsewhere.  Here that mask is kept in list form: the ordered pages of
each node.

Availability (Sec. 3.3, "Restrictions on context selection", and Eq. 8): a
selected historical state must already exist and its features must be
readable.  A state is readable when it is resident in the cache, or when a
node of the same pack produces it in this call -- a joint causal forward
computes an older chunk's features before the newer chunk reads them.
Anything else is unavailable.

Cache model.  One page holds one latent frame of one state (all heads, keys
and values) for every layer; a state of chunk c occupies ``pages_per_chunk``
page slots.  Slots are taken lowest-free-first, frames ascending, and a plan
reserves slots for the pack nodes that are not yet cached, in pack order.
This model only fixes slot numbers so tables can be compared bit for bit;
attention results never depend on them.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Set, Tuple

from .policy import Selection


class PlanError(RuntimeError):
    def __init__(self, code: str, msg: str = ""):
        super().__init__(f"{code}: {msg}")
        self.code = code


@dataclass
class CacheModel:
    n_slots: int
    pages_per_chunk: int
    n_layers: int = 1
    slots: Dict[Tuple[int, int], List[int]] = field(default_factory=dict)
    written: Dict[Tuple[int, int], Set[int]] = field(default_factory=dict)
    generation: List[int] = field(default_factory=list)

    def __post_init__(self):
        self.generation = [0] * self.n_slots

    def free_slots(self) -> List[int]:
        used = {s for v in self.slots.values() for s in v}
        return [s for s in range(self.n_slots) if s not in used]

    def contains(self, state) -> bool:
        return tuple(state) in self.slots

    def _allocate(self, state) -> List[int]:
        free = self.free_slots()
        if len(free) < self.pages_per_chunk:
            raise PlanError("ECAPACITY", f"no room for state {state}")
        self.slots[tuple(state)] = free[: self.pages_per_chunk]
        self.written[tuple(state)] = set()
        return self.slots[tuple(state)]

    def append(self, layer: int, state) -> List[int]:
        """Record that ``state``'s K/V for ``layer`` were written."""
        state = tuple(state)
        if state not in self.slots:
            self._allocate(state)
        if layer in self.written[state]:
            raise PlanError("EEXIST", f"state {state} layer {layer} already written")
        self.written[state].add(layer)
        return self.slots[state]

    def release(self, state) -> None:
        state = tuple(state)
        if state not in self.slots:
            raise PlanError("ENOTFOUND", f"state {state} not cached")
        for s in self.slots.pop(state):
            self.generation[s] += 1
        self.written.pop(state, None)


@dataclass
class Plan:
    page_off: List[int]
    page_slot: List[int]
    page_tokens: List[int]
    page_frame: List[int]
    page_chunk: List[int]
    page_level: List[int]


def build_plan(sel: Selection, cache: CacheModel, tokens_per_page: int) -> Plan:
    """Resolve a selection table to per-node page lists, reserving pack slots.

    Raises PlanError("EUNAVAILABLE") when a selected state is neither cached
    nor produced by the pack, and PlanError("ECAPACITY") when the pack's own
    states do not fit.  On error the cache is left unchanged.
    """
    n = len(sel.nodes)
    for i in range(n):
        lo, hi = sel.seg_off[i], sel.seg_off[i + 1]
        for s in range(lo, hi):
            state = (sel.seg_chunk[s], sel.seg_level[s])
            if sel.seg_src[s] < 0 and not cache.contains(state):
                raise PlanError("EUNAVAILABLE", f"node {sel.nodes[i]} reads {state}")
    missing = [node for node in sel.nodes if not cache.contains(node)]
    if len(cache.free_slots()) < len(missing) * cache.pages_per_chunk:
        raise PlanError("ECAPACITY", "pack states do not fit")
    for node in missing:
        cache._allocate(node)
    plan = Plan([0], [], [], [], [], [])
    ppc = cache.pages_per_chunk
    for i in range(n):
        for (c, l) in sel.segments(i):
            slots = cache.slots[(c, l)]
            for f in range(ppc):
                plan.page_slot.append(slots[f])
                plan.page_tokens.append(tokens_per_page)
                plan.page_frame.append(c * ppc + f)
                plan.page_chunk.append(c)
                plan.page_level.append(l)
        plan.page_off.append(len(plan.page_slot))
    return plan
