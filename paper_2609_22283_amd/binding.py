"""ctypes binding of libstreamctx.so: same names as the C ABI, marshalling only.

Device buffers are passed as torch tensors (their ``data_ptr()``) or raw
integer addresses; streams as ``torch.cuda.Stream`` objects, raw integers or
``None`` (the current torch stream when CUDA is initialised, else the null
stream).  Errors come back as ``ScError`` carrying the C status code and the
library's message.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import List, Optional, Sequence, Tuple

__all__ = [
    "ScError", "lib", "library_path", "SC_OK", "SC_EINVAL", "SC_EUNAVAILABLE", "SC_ECAPACITY",
    "SC_EEXIST", "SC_ENOTFOUND", "SC_ESTALE", "SC_EDEVICE", "SC_EUNSUPPORTED",
    "SC_POLICY_CLEAN", "SC_POLICY_SAME", "SC_POLICY_PROG", "SC_POLICY_TABLE",
    "SC_DTYPE_BF16", "SC_DTYPE_F32", "POLICY_KINDS", "EXPORTED_SYMBOLS", "ABI_VERSION",
    "sc_abi_version", "sc_selection_build", "sc_cache_pool_bytes", "sc_cache_create",
    "sc_rope_table_bytes", "sc_rope_table_build", "sc_plan_build", "sc_attention",
    "sc_attention_workspace_bytes", "sc_block_workspace_bytes", "sc_block_forward", "sc_sampler_step",
    "sc_timer_enable", "sc_timer_read", "sc_probe_mfma_out_bytes", "sc_probe_mfma", "sc_probe_read",
    "Selection", "Cache", "Plan", "Rope", "BlockWeights", "CrossAttn",
    "sc_plan_condition", "sc_condition_workspace_bytes", "sc_condition_append",
    "sc_pipeline_rounds", "sc_pipeline_round_nodes", "sc_cache_release_unread", "sc_stack_forward",
    "sc_serial_steps", "sc_serial_step_node", "sc_block_workspace_views",
    "sc_attention_noalloc", "sc_attention_noalloc_scratch_bytes",
]

SC_OK, SC_EINVAL, SC_EUNAVAILABLE, SC_ECAPACITY = 0, -1, -2, -3
SC_EEXIST, SC_ENOTFOUND, SC_ESTALE, SC_EDEVICE, SC_EUNSUPPORTED = -4, -5, -6, -7, -8
SC_POLICY_CLEAN, SC_POLICY_SAME, SC_POLICY_PROG, SC_POLICY_TABLE = 0, 1, 2, 3
SC_DTYPE_BF16, SC_DTYPE_F32 = 0, 1
POLICY_KINDS = {"clean": 0, "same": 1, "prog": 2, "table": 3}

# Every function the headers under include/ declare (checked by the CPU tests).
EXPORTED_SYMBOLS = [
    "sc_abi_version", "sc_last_error", "sc_status_name",
    "sc_selection_build", "sc_selection_get", "sc_visibility_get", "sc_selection_free",
    "sc_cache_pool_bytes", "sc_cache_create", "sc_cache_free", "sc_cache_contains",
    "sc_cache_slots", "sc_cache_free_slot_count", "sc_cache_release", "sc_cache_append",
    "sc_rope_table_bytes", "sc_rope_table_build",
    "sc_plan_build", "sc_plan_get", "sc_plan_free", "sc_plan_condition",
    "sc_condition_workspace_bytes", "sc_condition_append",
    "sc_attention_workspace_bytes", "sc_attention",
    "sc_block_workspace_bytes", "sc_block_forward", "sc_sampler_step",
    "sc_timer_enable", "sc_timer_read", "sc_probe_mfma_out_bytes", "sc_probe_mfma", "sc_probe_read",
    "sc_pipeline_rounds", "sc_pipeline_round_nodes", "sc_cache_release_unread", "sc_stack_forward",
    "sc_serial_steps", "sc_serial_step_node", "sc_block_workspace_views",
    "sc_attention_noalloc", "sc_attention_noalloc_scratch_bytes",
]

# The library and PyTorch must share one HIP runtime: torch ships its own
# libamdhip64 (same SONAME as /opt/rocm's).  Loading torch first makes the
# dynamic linker bind the library to torch's copy, so device pointers and
# streams created by torch are valid inside the library.  Loading the
# library first would bring up a second HIP/HSA runtime in the process.
try:
    import torch as _torch  # noqa: F401
except ImportError:  # a non-torch host process uses the system HIP runtime
    _torch = None

library_path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libstreamctx.so")
if not os.path.exists(library_path):
    raise ImportError(f"{library_path} is missing: build it with __graft_entry__.build() "
                      "(there is no fallback implementation)")
lib = C.CDLL(library_path)


class ScError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(msg)
        self.code = code


class sc_node(C.Structure):
    _fields_ = [("chunk", C.c_int32), ("level", C.c_int32)]


class sc_policy(C.Structure):
    _fields_ = [("kind", C.c_int32), ("K", C.c_int32), ("W", C.c_int32),
                ("phi_table", C.POINTER(C.c_int8)), ("r_mask", C.POINTER(C.c_uint8)),
                ("n_chunks", C.c_int32)]


class sc_cache_desc(C.Structure):
    _fields_ = [(n, C.c_int32) for n in
                ("n_layers", "n_heads", "head_dim", "tokens_per_page", "pages_per_chunk", "n_slots",
                 "dtype")]


class sc_rope_desc(C.Structure):
    _fields_ = [("grid_h", C.c_int32), ("grid_w", C.c_int32), ("dim_t", C.c_int32),
                ("dim_h", C.c_int32), ("dim_w", C.c_int32), ("max_frames", C.c_int32),
                ("theta", C.c_float)]


class sc_rope(C.Structure):
    _fields_ = [("desc", sc_rope_desc), ("dev_table", C.c_void_p)]


class sc_cross_attn(C.Structure):
    _fields_ = [("w_q", C.c_void_p), ("w_o", C.c_void_p), ("q_norm", C.c_void_p),
                ("cache", C.c_void_p), ("plan", C.c_void_p)]


class sc_block_weights(C.Structure):
    _fields_ = [("hidden", C.c_int32), ("n_heads", C.c_int32), ("head_dim", C.c_int32),
                ("mlp", C.c_int32), ("w_qkv", C.c_void_p), ("w_o", C.c_void_p),
                ("w_up", C.c_void_p), ("w_down", C.c_void_p), ("mod", C.c_void_p),
                ("mod_levels", C.c_int32), ("qk_norm", C.c_void_p),
                ("cross", C.POINTER(sc_cross_attn))]


_P = C.c_void_p
_I32P = C.POINTER(C.c_int32)
_SIG = {
    "sc_abi_version": (C.c_int, []),
    "sc_last_error": (C.c_char_p, []),
    "sc_status_name": (C.c_char_p, [C.c_int]),
    "sc_selection_build": (C.c_int, [C.POINTER(sc_policy), C.POINTER(sc_node), C.c_int32, C.POINTER(_P)]),
    "sc_selection_get": (C.c_int, [_P, _I32P, _I32P] + [C.POINTER(_I32P)] * 4),
    "sc_visibility_get": (C.c_int, [_P, _I32P, C.POINTER(C.POINTER(sc_node)),
                                    C.POINTER(C.POINTER(C.c_uint8))]),
    "sc_selection_free": (None, [_P]),
    "sc_cache_pool_bytes": (C.c_size_t, [C.POINTER(sc_cache_desc)]),
    "sc_cache_create": (C.c_int, [C.POINTER(sc_cache_desc), _P, C.POINTER(_P)]),
    "sc_cache_free": (None, [_P]),
    "sc_cache_contains": (C.c_int, [_P, sc_node, C.c_int32]),
    "sc_cache_slots": (C.c_int, [_P, sc_node, _I32P]),
    "sc_cache_free_slot_count": (C.c_int, [_P]),
    "sc_cache_release": (C.c_int, [_P, sc_node]),
    "sc_cache_append": (C.c_int, [_P, C.c_int32, sc_node, _P, _P, C.POINTER(sc_rope), _P]),
    "sc_rope_table_bytes": (C.c_size_t, [C.POINTER(sc_rope_desc)]),
    "sc_rope_table_build": (C.c_int, [C.POINTER(sc_rope_desc), _P, _P]),
    "sc_plan_build": (C.c_int, [_P, _P, C.POINTER(_P)]),
    "sc_plan_get": (C.c_int, [_P, _I32P, _I32P] + [C.POINTER(_I32P)] * 4),
    "sc_plan_free": (None, [_P]),
    "sc_plan_condition": (C.c_int, [_P, C.POINTER(sc_node), C.c_int32, C.c_int32, C.POINTER(_P)]),
    "sc_condition_workspace_bytes": (C.c_size_t, [_P]),
    "sc_condition_append": (C.c_int, [_P, C.c_int32, sc_node, _P, _P, _P, _P, _P, C.c_size_t, _P]),
    "sc_attention_workspace_bytes": (C.c_size_t, [_P, _P]),
    "sc_attention": (C.c_int, [_P, _P, C.c_int32, _P, _P, C.c_float, _P, C.c_size_t, _P]),
    "sc_block_workspace_bytes": (C.c_size_t, [C.POINTER(sc_block_weights), C.c_int32]),
    "sc_block_forward": (C.c_int, [C.POINTER(sc_block_weights), _P, C.c_int32, _P, _P,
                                   C.POINTER(sc_rope), _P, C.c_size_t, _P]),
    "sc_sampler_step": (C.c_int, [C.POINTER(sc_node), C.c_int32, C.POINTER(C.c_float), C.c_int32,
                                  _P, _P, _P, C.c_int64, _P]),
    "sc_timer_enable": (C.c_int, [C.c_int]),
    "sc_timer_read": (C.c_int, [C.c_char_p, _I32P, C.POINTER(C.c_double)]),
    "sc_probe_mfma_out_bytes": (C.c_size_t, []),
    "sc_probe_mfma": (C.c_int, [C.c_int32, C.c_int32, _P, C.c_size_t, C.POINTER(C.c_double), _P]),
    "sc_probe_read": (C.c_int, [_P, C.c_size_t, _P, _P]),
    "sc_pipeline_rounds": (C.c_int, [C.c_int32, C.c_int32, C.c_int32]),
    "sc_pipeline_round_nodes": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                          C.POINTER(sc_node), _I32P]),
    "sc_cache_release_unread": (C.c_int, [_P, C.POINTER(sc_policy), C.POINTER(sc_node), C.c_int32]),
    "sc_stack_forward": (C.c_int, [C.POINTER(sc_block_weights), C.c_int32, _P, _P, _P,
                                   C.POINTER(sc_rope), _P, C.c_size_t, _P]),
    "sc_attention_noalloc": (C.c_int, [_P, _P, C.c_int32, _P, _P, C.c_float, _P]),
    "sc_attention_noalloc_scratch_bytes": (C.c_size_t, []),
    "sc_serial_steps": (C.c_int, [C.c_int32, C.c_int32, C.c_int32]),
    "sc_serial_step_node": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.POINTER(sc_node)]),
    "sc_block_workspace_views": (C.c_int, [C.POINTER(sc_block_weights), C.c_int32, C.POINTER(C.c_size_t),
                                           C.POINTER(C.c_size_t)]),
}
# ABI version this binding marshals for (SC_ABI_VERSION of the header)
ABI_VERSION = 7
if not hasattr(lib, "sc_abi_version") or lib.sc_abi_version() != ABI_VERSION:
    raise ImportError(f"{library_path} does not implement ABI version {ABI_VERSION}; rebuild it "
                      "(__graft_entry__.build())")
for _name, (_res, _args) in _SIG.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def _check(rc: int) -> int:
    if rc < 0:
        raise ScError(rc, lib.sc_last_error().decode())
    return rc


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s) -> Optional[int]:
    if s is None:
        try:
            import torch
            if torch.cuda.is_initialized():
                return torch.cuda.current_stream().cuda_stream
        except Exception:
            pass
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def sc_abi_version() -> int:
    return lib.sc_abi_version()


# ------------------------------------------------------------------ selection
class Selection:
    def __init__(self, handle):
        self._h = C.c_void_p(handle)

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value:
            lib.sc_selection_free(self._h)
            self._h = None

    @property
    def handle(self):
        return self._h

    def tables(self):
        """(seg_off, seg_chunk, seg_level, seg_src) as Python lists."""
        n, ns = C.c_int32(), C.c_int32()
        arr = [_I32P() for _ in range(4)]
        _check(lib.sc_selection_get(self._h, C.byref(n), C.byref(ns), *[C.byref(a) for a in arr]))
        lens = [n.value + 1, ns.value, ns.value, ns.value]
        return tuple([arr[i][k] for k in range(lens[i])] for i in range(4))

    def visibility(self):
        n_states = C.c_int32()
        st = C.POINTER(sc_node)()
        vis = C.POINTER(C.c_uint8)()
        _check(lib.sc_visibility_get(self._h, C.byref(n_states), C.byref(st), C.byref(vis)))
        states = [(st[k].chunk, st[k].level) for k in range(n_states.value)]
        n = len(self.tables()[0]) - 1
        rows = [[vis[i * n_states.value + k] for k in range(n_states.value)] for i in range(n)]
        return states, rows


def _flatten(t):
    """Nested [c][j][r] or [j][r] table -> flat list (row-major)."""
    if isinstance(t, (list, tuple)) and t and isinstance(t[0], (list, tuple)):
        return [v for row in t for v in _flatten(row)]
    return [int(v) for v in t]


def _policy_struct(kind, K, W, phi_table=None, r_mask=None, n_chunks=0):
    """phi_table / r_mask: [K+1][W], or [n_chunks][K+1][W] when n_chunks > 0
    (position-dependent policy)."""
    pol = sc_policy()
    pol.kind = POLICY_KINDS[kind] if isinstance(kind, str) else int(kind)
    pol.K, pol.W, pol.n_chunks = int(K), int(W), int(n_chunks)
    keep = []
    if phi_table is not None:
        flat = _flatten(phi_table)
        buf = (C.c_int8 * max(1, len(flat)))(*flat)
        keep.append(buf)
        pol.phi_table = C.cast(buf, C.POINTER(C.c_int8))
    if r_mask is not None:
        flat = _flatten(r_mask)
        buf = (C.c_uint8 * max(1, len(flat)))(*flat)
        keep.append(buf)
        pol.r_mask = C.cast(buf, C.POINTER(C.c_uint8))
    return pol, keep


def sc_selection_build(kind, K, W, nodes: Sequence[Tuple[int, int]], phi_table=None,
                       r_mask=None, n_chunks=0) -> Selection:
    pol, keep = _policy_struct(kind, K, W, phi_table, r_mask, n_chunks)
    arr = (sc_node * max(1, len(nodes)))(*[sc_node(int(c), int(j)) for c, j in nodes])
    out = C.c_void_p()
    _check(lib.sc_selection_build(C.byref(pol), arr, len(nodes), C.byref(out)))
    del keep
    return Selection(out.value)


# ---------------------------------------------------------------------- cache
def _desc(n_layers, n_heads, head_dim, tokens_per_page, pages_per_chunk, n_slots, dtype):
    return sc_cache_desc(n_layers, n_heads, head_dim, tokens_per_page, pages_per_chunk, n_slots, dtype)


def sc_cache_pool_bytes(n_layers, n_heads, head_dim, tokens_per_page, pages_per_chunk, n_slots,
                        dtype=SC_DTYPE_BF16) -> int:
    d = _desc(n_layers, n_heads, head_dim, tokens_per_page, pages_per_chunk, n_slots, dtype)
    return lib.sc_cache_pool_bytes(C.byref(d))


class Cache:
    """Handle on a paged KV cache whose pool is caller device memory."""

    def __init__(self, handle, desc, pool):
        self._h = C.c_void_p(handle)
        self.desc = desc
        self.pool = pool  # keeps the caller's buffer alive

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value:
            lib.sc_cache_free(self._h)
            self._h = None

    @property
    def handle(self):
        return self._h

    def contains(self, state, layer: int = -1) -> bool:
        return bool(_check(lib.sc_cache_contains(self._h, sc_node(*state), layer)))

    def slots(self, state) -> List[int]:
        buf = (C.c_int32 * self.desc.pages_per_chunk)()
        _check(lib.sc_cache_slots(self._h, sc_node(*state), buf))
        return list(buf)

    def free_slot_count(self) -> int:
        return _check(lib.sc_cache_free_slot_count(self._h))

    def release(self, state) -> None:
        _check(lib.sc_cache_release(self._h, sc_node(*state)))

    def append(self, layer: int, state, k, v, rope: "Rope" = None, stream=None) -> None:
        rp = C.byref(rope.struct) if rope is not None else None
        _check(lib.sc_cache_append(self._h, layer, sc_node(*state), _ptr(k), _ptr(v), rp,
                                   _stream(stream)))


def sc_cache_create(pool, n_layers, n_heads, head_dim, tokens_per_page, pages_per_chunk, n_slots,
                    dtype=SC_DTYPE_BF16) -> Cache:
    d = _desc(n_layers, n_heads, head_dim, tokens_per_page, pages_per_chunk, n_slots, dtype)
    out = C.c_void_p()
    _check(lib.sc_cache_create(C.byref(d), _ptr(pool), C.byref(out)))
    return Cache(out.value, d, pool)


# ----------------------------------------------------------------------- rope
class Rope:
    def __init__(self, desc: sc_rope_desc, table):
        self.table = table
        self.struct = sc_rope(desc, _ptr(table))


def _rope_desc(grid_h, grid_w, dims, max_frames, theta):
    return sc_rope_desc(grid_h, grid_w, dims[0], dims[1], dims[2], max_frames, theta)


def sc_rope_table_bytes(grid_h, grid_w, dims, max_frames, theta=10000.0) -> int:
    d = _rope_desc(grid_h, grid_w, dims, max_frames, theta)
    return lib.sc_rope_table_bytes(C.byref(d))


def sc_rope_table_build(table, grid_h, grid_w, dims, max_frames, theta=10000.0, stream=None) -> Rope:
    d = _rope_desc(grid_h, grid_w, dims, max_frames, theta)
    _check(lib.sc_rope_table_build(C.byref(d), _ptr(table), _stream(stream)))
    return Rope(d, table)


# ----------------------------------------------------------------------- plan
class Plan:
    def __init__(self, handle, cache):
        self._h = C.c_void_p(handle)
        self.cache = cache

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value:
            lib.sc_plan_free(self._h)
            self._h = None

    @property
    def handle(self):
        return self._h

    def tables(self):
        """(page_off, page_slot, page_tokens, page_frame) as Python lists."""
        n, npg = C.c_int32(), C.c_int32()
        arr = [_I32P() for _ in range(4)]
        _check(lib.sc_plan_get(self._h, C.byref(n), C.byref(npg), *[C.byref(a) for a in arr]))
        lens = [n.value + 1, npg.value, npg.value, npg.value]
        return tuple([arr[i][k] for k in range(lens[i])] for i in range(4))


def sc_plan_build(sel: Selection, cache: Cache) -> Plan:
    out = C.c_void_p()
    _check(lib.sc_plan_build(sel.handle, cache.handle, C.byref(out)))
    return Plan(out.value, cache)


def sc_plan_condition(cache: Cache, conditions, nq: int) -> Plan:
    """Plan in which pack node i reads every page of the cached condition
    state conditions[i], with nq query rows per node."""
    arr = (sc_node * max(1, len(conditions)))(*[sc_node(int(c), int(j)) for c, j in conditions])
    out = C.c_void_p()
    _check(lib.sc_plan_condition(cache.handle, arr, len(conditions), nq, C.byref(out)))
    return Plan(out.value, cache)


def sc_condition_workspace_bytes(cache: Cache) -> int:
    return lib.sc_condition_workspace_bytes(cache.handle)


def sc_condition_append(cache: Cache, layer: int, state, ctx, w_k, w_v, k_norm, ws, ws_bytes: int,
                        stream=None) -> None:
    _check(lib.sc_condition_append(cache.handle, layer, sc_node(*state), _ptr(ctx), _ptr(w_k),
                                   _ptr(w_v), _ptr(k_norm), _ptr(ws), ws_bytes, _stream(stream)))


def sc_attention_workspace_bytes(plan: Plan, cache: Cache) -> int:
    return lib.sc_attention_workspace_bytes(plan.handle, cache.handle)


def sc_attention(plan: Plan, cache: Cache, layer: int, q, o, scale: float, ws=None,
                 ws_bytes: int = 0, stream=None) -> None:
    _check(lib.sc_attention(plan.handle, cache.handle, layer, _ptr(q), _ptr(o), scale, _ptr(ws),
                            ws_bytes, _stream(stream)))


# ---------------------------------------------------------------------- block
def sc_attention_noalloc(plan: Plan, cache: Cache, layer: int, q, o, scale: float, stream=None) -> None:
    """sc_attention with the library's own scratch (no workspace argument)."""
    _check(lib.sc_attention_noalloc(plan.handle, cache.handle, layer, _ptr(q), _ptr(o), scale,
                                    _stream(stream)))


def sc_attention_noalloc_scratch_bytes() -> int:
    return lib.sc_attention_noalloc_scratch_bytes()


class CrossAttn:
    """Cross-attention of a block to a condition cache: device weights w_q,
    w_o, optional fp32 query gain q_norm, the condition cache and its plan
    (sc_plan_condition)."""

    def __init__(self, w_q, w_o, cache: "Cache", plan: "Plan", q_norm=None):
        self.refs = (w_q, w_o, q_norm, cache, plan)
        self.struct = sc_cross_attn(_ptr(w_q), _ptr(w_o), _ptr(q_norm), cache.handle.value,
                                    plan.handle.value)


class BlockWeights:
    """Device weights of one block; ``mod`` is the optional fp32 per-level
    modulation table [levels][6][hidden] (noise-level conditioning),
    ``qk_norm`` the optional fp32 gains [2][hidden] of q and k, ``cross``
    the optional CrossAttn."""

    def __init__(self, hidden, n_heads, head_dim, mlp, w_qkv, w_o, w_up, w_down, mod=None,
                 qk_norm=None, cross: Optional[CrossAttn] = None):
        self.tensors = (w_qkv, w_o, w_up, w_down, mod, qk_norm, cross)
        levels = 0 if mod is None else int(mod.shape[0])
        cp = C.pointer(cross.struct) if cross is not None else None
        self.args = (hidden, n_heads, head_dim, mlp, w_qkv, w_o, w_up, w_down, mod, qk_norm)
        self.struct = sc_block_weights(hidden, n_heads, head_dim, mlp, _ptr(w_qkv), _ptr(w_o),
                                       _ptr(w_up), _ptr(w_down), _ptr(mod), levels, _ptr(qk_norm), cp)

    def with_cross(self, cross: Optional[CrossAttn]) -> "BlockWeights":
        """The same block reading the condition through ``cross`` (a plan
        per pack: the condition plan names the pack's nodes)."""
        hidden, n_heads, head_dim, mlp, w_qkv, w_o, w_up, w_down, mod, qk_norm = self.args
        return BlockWeights(hidden, n_heads, head_dim, mlp, w_qkv, w_o, w_up, w_down, mod=mod,
                            qk_norm=qk_norm, cross=cross)


def sc_block_workspace_bytes(w: BlockWeights, n_tokens: int) -> int:
    return lib.sc_block_workspace_bytes(C.byref(w.struct), n_tokens)


def sc_block_forward(w: BlockWeights, cache: Cache, layer: int, plan: Plan, x, rope: Rope, ws,
                     ws_bytes: int, stream=None) -> None:
    _check(lib.sc_block_forward(C.byref(w.struct), cache.handle, layer, plan.handle, _ptr(x),
                                C.byref(rope.struct) if rope is not None else None, _ptr(ws),
                                ws_bytes, _stream(stream)))


def sc_block_workspace_views(w: BlockWeights, n_tokens: int) -> Tuple[int, int]:
    """Byte offsets (q, o) of the last block's rotated queries and attention
    output inside its workspace (bf16 [n_tokens, hidden] each)."""
    q, o = C.c_size_t(), C.c_size_t()
    _check(lib.sc_block_workspace_views(C.byref(w.struct), n_tokens, C.byref(q), C.byref(o)))
    return q.value, o.value


def sc_sampler_step(nodes, t: Sequence[float], K: int, out, y, noise, elems_per_node: int,
                    stream=None) -> None:
    arr = (sc_node * max(1, len(nodes)))(*[sc_node(int(c), int(j)) for c, j in nodes])
    tt = (C.c_float * len(t))(*[float(v) for v in t])
    _check(lib.sc_sampler_step(arr, len(nodes), tt, K, _ptr(out), _ptr(y), _ptr(noise),
                               elems_per_node, _stream(stream)))


def sc_timer_enable(on: bool = True) -> None:
    _check(lib.sc_timer_enable(1 if on else 0))


def sc_timer_read(kind: str):
    """(launches, total milliseconds) of one kernel kind since enabling."""
    n, ms = C.c_int32(), C.c_double()
    _check(lib.sc_timer_read(kind.encode(), C.byref(n), C.byref(ms)))
    return n.value, ms.value


def sc_probe_mfma_out_bytes() -> int:
    return lib.sc_probe_mfma_out_bytes()


def sc_probe_mfma(random_operands: bool, iters: int, out, out_bytes: int, stream=None) -> float:
    """Launch the matrix-core probe; returns the FLOPs it performs."""
    fl = C.c_double()
    _check(lib.sc_probe_mfma(1 if random_operands else 0, iters, _ptr(out), out_bytes, C.byref(fl),
                             _stream(stream)))
    return fl.value


def sc_probe_read(buf, nbytes: int, out, stream=None) -> None:
    """Launch the streaming-read probe over the first nbytes of buf."""
    _check(lib.sc_probe_read(_ptr(buf), nbytes, _ptr(out), _stream(stream)))


# ------------------------------------------------------------------- schedule
def sc_pipeline_rounds(K: int, B: int, refresh: bool) -> int:
    return _check(lib.sc_pipeline_rounds(K, B, 1 if refresh else 0))


def sc_pipeline_round_nodes(K: int, B: int, refresh: bool, n: int):
    """Nodes of pipelined round n (Eq. 7, plus the refresh node), oldest first."""
    buf = (sc_node * (K + 1))()
    m = C.c_int32()
    _check(lib.sc_pipeline_round_nodes(K, B, 1 if refresh else 0, n, buf, C.byref(m)))
    return [(buf[i].chunk, buf[i].level) for i in range(m.value)]


def sc_serial_steps(K: int, B: int, refresh: bool) -> int:
    return _check(lib.sc_serial_steps(K, B, 1 if refresh else 0))


def sc_serial_step_node(K: int, B: int, refresh: bool, n: int) -> Tuple[int, int]:
    """Node of forward n of fully serial execution (Eq. 2)."""
    nd = sc_node()
    _check(lib.sc_serial_step_node(K, B, 1 if refresh else 0, n, C.byref(nd)))
    return nd.chunk, nd.level


def sc_cache_release_unread(cache: "Cache", kind, K, W, future, phi_table=None, r_mask=None,
                            n_chunks=0) -> int:
    """Release every cached state none of the future nodes reads; returns the count."""
    pol, keep = _policy_struct(kind, K, W, phi_table, r_mask, n_chunks)
    arr = (sc_node * max(1, len(future)))(*[sc_node(int(c), int(j)) for c, j in future])
    n = _check(lib.sc_cache_release_unread(cache.handle, C.byref(pol), arr, len(future)))
    del keep
    return n


def sc_stack_forward(layers, cache: "Cache", plan: "Plan", x, rope: "Rope", ws, ws_bytes: int,
                     stream=None) -> None:
    """All layers of a block stack over one pack (layers: list of BlockWeights)."""
    arr = (sc_block_weights * len(layers))(*[w.struct for w in layers])
    _check(lib.sc_stack_forward(arr, len(layers), cache.handle, plan.handle, _ptr(x),
                                C.byref(rope.struct) if rope is not None else None, _ptr(ws),
                                ws_bytes, _stream(stream)))
