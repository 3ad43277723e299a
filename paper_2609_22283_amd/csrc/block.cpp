// One DiT block over a pack of nodes: launch sequence and argument checks.
// RMSNorm -> QKV GEMM (+RoPE, q out, k/v into the pack's page slots) ->
// packed attention -> out-projection (+residual) -> RMSNorm -> MLP up (+GELU)
// -> MLP down (+residual).  Stream order makes "append before attend" hold,
// which is what lets a node read the K/V an older pack node computes in the
// same forward (the joint causal forward of Sec. 3.3).
#include <cstring>

#include "gemm.h"
#include "internal.h"

using namespace sc;

static size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

extern "C" size_t sc_block_workspace_bytes(const sc_block_weights* w, int32_t n_tokens) {
  if (!w || n_tokens <= 0) return 0;
  const size_t T = (size_t)n_tokens;
  return align256(T * w->hidden * 2) * 3 + align256(T * w->mlp * 2) + attention_workspace_bound();
}

extern "C" int sc_block_forward(const sc_block_weights* w, sc_cache* c, int32_t layer,
                                const sc_plan* p, void* x, const sc_rope* rope, void* ws,
                                size_t ws_bytes, sc_stream stream_) {
  if (!w || !c || !p || !x || !ws) return fail(SC_EINVAL, "null argument");
  if (!w->w_qkv || !w->w_o || !w->w_up || !w->w_down) return fail(SC_EINVAL, "null weight");
  const sc_cache_desc& d = c->d;
  if (d.dtype != SC_DTYPE_BF16) return fail(SC_EUNSUPPORTED, "block forward is bf16 only");
  if (w->n_heads != d.n_heads || w->head_dim != d.head_dim || w->hidden != d.n_heads * d.head_dim)
    return fail(SC_EINVAL, "weights (%d heads x %d, hidden %d) do not match the cache", w->n_heads,
                w->head_dim, w->hidden);
  if (p->cache != c) return fail(SC_EINVAL, "plan was built for another cache");
  if (layer < 0 || layer >= d.n_layers) return fail(SC_EINVAL, "layer %d out of range", layer);
  const int32_t n = (int32_t)p->nodes.size();
  if (n == 0) return SC_OK;
  if (n > kGemmMaxNodes || n * d.pages_per_chunk > kGemmMaxNodePages)
    return fail(SC_EUNSUPPORTED, "pack too large for the QKV epilogue (%d nodes)", n);
  const int32_t T = n * p->nq;
  if (w->mod) {
    if (reinterpret_cast<uintptr_t>(w->mod) & 15) return fail(SC_EINVAL, "modulation table must be 16-byte aligned");
    for (int32_t i = 0; i < n; ++i)
      if (p->nodes[i].level >= w->mod_levels)
        return fail(SC_EINVAL, "node (%d,%d) has no row in a %d-level modulation table",
                    p->nodes[i].chunk, p->nodes[i].level, w->mod_levels);
  }
  NormMod nm_a;
  std::memset(&nm_a, 0, sizeof nm_a);
  nm_a.mod = w->mod;
  nm_a.nq = p->nq;
  for (int32_t i = 0; i < n; ++i) nm_a.node_level[i] = p->nodes[i].level;
  NormMod nm_m = nm_a;
  nm_m.which = 1;
  if (ws_bytes < sc_block_workspace_bytes(w, T))
    return fail(SC_EINVAL, "workspace of %zu bytes, need %zu", ws_bytes, sc_block_workspace_bytes(w, T));
  if (rope) {
    const sc_rope_desc& r = rope->desc;
    if (!rope->dev_table || r.grid_h * r.grid_w != d.tokens_per_page ||
        r.dim_t + r.dim_h + r.dim_w != d.head_dim)
      return fail(SC_EINVAL, "rope descriptor does not match the cache geometry");
  }
  // pages of states the pack does not produce must be written at this layer;
  // the pack's own states must not be (they are written here)
  GemmEpilogue ep;
  std::memset(&ep, 0, sizeof ep);
  for (int32_t i = 0; i < n; ++i) {
    auto it = c->states.find(StateKey(p->nodes[i].chunk, p->nodes[i].level));
    if (it == c->states.end())
      return fail(SC_ESTALE, "pack state (%d,%d) no longer cached", p->nodes[i].chunk, p->nodes[i].level);
    if (it->second.written[layer])
      return fail(SC_EEXIST, "pack state (%d,%d) already written at layer %d", p->nodes[i].chunk,
                  p->nodes[i].level, layer);
    if (rope && (p->nodes[i].chunk + 1) * d.pages_per_chunk > rope->desc.max_frames)
      return fail(SC_EINVAL, "chunk %d beyond the rope table", p->nodes[i].chunk);
    ep.node_chunk[i] = p->nodes[i].chunk;
    for (int32_t f = 0; f < d.pages_per_chunk; ++f)
      ep.node_slot[i * d.pages_per_chunk + f] = it->second.slots[f];
  }
  for (size_t q = 0; q < p->page_slot.size(); ++q) {
    int32_t s = p->page_slot[q];
    if (!c->used[s] || c->gen[s] != p->page_gen[q])
      return fail(SC_ESTALE, "slot %d was released after the plan was built", s);
    const StateKey& key = p->page_state[q];
    bool in_pack = false;
    for (int32_t i = 0; i < n; ++i)
      if (p->nodes[i].chunk == key.first && p->nodes[i].level == key.second) in_pack = true;
    if (!in_pack && !c->states.at(key).written[layer])
      return fail(SC_EUNAVAILABLE, "state (%d,%d) has no K/V at layer %d", key.first, key.second, layer);
  }

  hipStream_t stream = static_cast<hipStream_t>(stream_);
  char* wsb = static_cast<char*>(ws);
  uint16_t* hn = reinterpret_cast<uint16_t*>(wsb);
  uint16_t* qb = reinterpret_cast<uint16_t*>(wsb + align256((size_t)T * w->hidden * 2));
  uint16_t* ob = reinterpret_cast<uint16_t*>(wsb + 2 * align256((size_t)T * w->hidden * 2));
  uint16_t* ub = reinterpret_cast<uint16_t*>(wsb + 3 * align256((size_t)T * w->hidden * 2));
  char* attn_ws = wsb + 3 * align256((size_t)T * w->hidden * 2) + align256((size_t)T * w->mlp * 2);
  uint16_t* xb = static_cast<uint16_t*>(x);
  const int32_t D = w->hidden;

  ep.q_out = qb;
  ep.layer_base = c->pool + (size_t)layer * d.n_slots * c->slot_bytes;
  ep.slot_bytes = c->slot_bytes;
  ep.kv_half = c->kv_half;
  ep.hidden = D;
  ep.head_dim = d.head_dim;
  ep.nq = p->nq;
  ep.tpp = d.tokens_per_page;
  ep.ppc = d.pages_per_chunk;
  if (rope) {
    RopeLayout L = rope_layout(&rope->desc);
    ep.grid_w = rope->desc.grid_w;
    ep.rope_table = static_cast<const float2*>(rope->dev_table);
    ep.pairs_t = L.pairs_t;
    ep.pairs_h = L.pairs_h;
    ep.pairs_w = L.pairs_w;
    ep.rope_off_h = L.off_h;
    ep.rope_off_w = L.off_w;
  } else {
    ep.grid_w = 1;
  }

  int rc;
  if ((rc = launch_rmsnorm(xb, hn, T, D, nm_a, stream)) != SC_OK) return rc;
  if ((rc = launch_gemm(EPI_QKV, TK_GEMM_QKV, static_cast<const uint16_t*>(w->w_qkv), hn, 3 * D, T, D, ep, stream)) != SC_OK)
    return rc;
  for (int32_t i = 0; i < n; ++i)
    c->states.at(StateKey(p->nodes[i].chunk, p->nodes[i].level)).written[layer] = 1;
  if ((rc = launch_attention(p, c, layer, qb, ob, 1.0f / std::sqrt((float)d.head_dim), attn_ws,
                             attention_workspace_bound(), stream)) != SC_OK)
    return rc;
  GemmEpilogue e2;
  std::memset(&e2, 0, sizeof e2);
  e2.out = xb;
  e2.ld_out = D;
  e2.nq = p->nq;
  e2.mod = w->mod;
  e2.gate_row = 2;  // gate_a
  for (int32_t i = 0; i < n; ++i) e2.node_level[i] = p->nodes[i].level;
  if ((rc = launch_gemm(EPI_RESIDUAL, TK_GEMM_OUT, static_cast<const uint16_t*>(w->w_o), ob, D, T, D, e2, stream)) != SC_OK)
    return rc;
  if ((rc = launch_rmsnorm(xb, hn, T, D, nm_m, stream)) != SC_OK) return rc;
  GemmEpilogue e3;
  std::memset(&e3, 0, sizeof e3);
  e3.out = ub;
  e3.ld_out = w->mlp;
  if ((rc = launch_gemm(EPI_GELU, TK_GEMM_UP, static_cast<const uint16_t*>(w->w_up), hn, w->mlp, T, D, e3, stream)) != SC_OK)
    return rc;
  GemmEpilogue e4 = e2;
  e4.gate_row = 5;  // gate_m
  if ((rc = launch_gemm(EPI_RESIDUAL, TK_GEMM_DOWN, static_cast<const uint16_t*>(w->w_down), ub, D, T, w->mlp, e4, stream)) != SC_OK)
    return rc;
  return SC_OK;
}
