// One DiT block over a pack of nodes: launch sequence and argument checks.
// RMSNorm -> QKV GEMM (+RoPE, q out, k/v into the pack's page slots)
// [-> qk-norm scaling] -> packed attention -> out-projection (+residual)
// [-> RMSNorm -> condition query GEMM [-> its norm] -> attention over the
// condition cache -> condition out-projection (+residual)] -> RMSNorm ->
// MLP up (+GELU) -> MLP down (+residual).  Stream order makes "append before
// attend" hold, which is what lets a node read the K/V an older pack node
// computes in the same forward (the joint causal forward of Sec. 3.3).
// Also the condition's K/V projection (sc_condition_append).
#include <cstring>

#include "gemm.h"
#include "internal.h"

using namespace sc;

static size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

constexpr float kNormEps = 1e-6f;

// workspace: normalised input (or the folded RMSNorms' per-token factors) | q |
// attention output | MLP hidden | attention partials | partial sums of squares
extern "C" size_t sc_block_workspace_bytes(const sc_block_weights* w, int32_t n_tokens) {
  if (!w || n_tokens <= 0) return 0;
  const size_t T = (size_t)n_tokens;
  return align256(T * w->hidden * 2) * 3 + align256(T * w->mlp * 2) + attention_workspace_bound() +
         align256(T * (2 * w->hidden / kSsPartWidth) * 4);
}

extern "C" int sc_block_workspace_views(const sc_block_weights* w, int32_t n_tokens, size_t* q_offset,
                                        size_t* o_offset) {
  if (!w || n_tokens <= 0 || !q_offset || !o_offset) return fail(SC_EINVAL, "null argument or no tokens");
  const size_t act = align256((size_t)n_tokens * w->hidden * 2);
  *q_offset = act;
  *o_offset = 2 * act;
  return SC_OK;
}

static bool misaligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) & 15; }

// Checks of the optional cross-attention against the block's pack plan.
static int cross_check(const sc_cross_attn* cr, const sc_cache* c, const sc_plan* p, int32_t layer) {
  if (!cr->w_q || !cr->w_o || !cr->cache || !cr->plan)
    return fail(SC_EINVAL, "cross-attention needs w_q, w_o, a condition cache and its plan");
  const sc_cache_desc& e = cr->cache->d;
  if (e.dtype != SC_DTYPE_BF16 || e.n_heads != c->d.n_heads || e.head_dim != c->d.head_dim)
    return fail(SC_EINVAL, "condition cache (%d heads x %d, dtype %d) does not match the block",
                e.n_heads, e.head_dim, e.dtype);
  if (cr->plan->nodes.size() != p->nodes.size() || cr->plan->nq != p->nq)
    return fail(SC_EINVAL, "condition plan has %zu nodes of %d queries, the pack %zu of %d",
                cr->plan->nodes.size(), cr->plan->nq, p->nodes.size(), p->nq);
  if (cr->q_norm && misaligned16(cr->q_norm))
    return fail(SC_EINVAL, "condition query gain must be 16-byte aligned");
  int rc = attention_check(cr->plan, cr->cache);  // shape support first, then state
  if (rc != SC_OK) return rc;
  return plan_check(cr->plan, cr->cache, layer);
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
  // every projection's shape is checked before the first launch
  if (w->hidden % 256 || w->mlp <= 0 || w->mlp % 256)
    return fail(SC_EUNSUPPORTED, "block GEMMs need hidden and mlp multiples of 256 (got %d, %d)", w->hidden,
                w->mlp);
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
  if (misaligned16(ws)) return fail(SC_EINVAL, "workspace must be 16-byte aligned");
  if (w->qk_norm && misaligned16(w->qk_norm)) return fail(SC_EINVAL, "qk-norm gains must be 16-byte aligned");
  int rc = attention_check(p, c);
  if (rc != SC_OK) return rc;
  if (w->cross && (rc = cross_check(w->cross, c, p, layer)) != SC_OK) return rc;
  if (rope) {
    const sc_rope_desc& r = rope->desc;
    if (!rope->dev_table || r.grid_h * r.grid_w != d.tokens_per_page ||
        r.dim_t + r.dim_h + r.dim_w != d.head_dim || (r.dim_t | r.dim_h | r.dim_w) & 1)
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
  float* ssb = reinterpret_cast<float*>(attn_ws + attention_workspace_bound());
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

  if (w->qk_norm) {
    ep.ss_part = ssb;
    ep.n_part = 2 * D / kSsPartWidth;
    ep.qk_gain = w->qk_norm;
  }

  // Without modulation the pre-attention RMSNorm folds into the QKV GEMM:
  // one pass over x writes each token's 1 / rms (into hn's region), and the
  // QKV epilogue scales the token's accumulators by it, reading the raw rows.
  const uint16_t* qkv_in = hn;
  if (!w->mod) {
    float* rsa = reinterpret_cast<float*>(hn);
    if ((rc = launch_row_rms(xb, T, D, rsa, stream)) != SC_OK) return rc;
    ep.row_scale = rsa;
    qkv_in = xb;
  } else if ((rc = launch_rmsnorm(xb, hn, T, D, nm_a, stream)) != SC_OK) {
    return rc;
  }
  if ((rc = launch_gemm(EPI_QKV, TK_GEMM_QKV, static_cast<const uint16_t*>(w->w_qkv), qkv_in, 3 * D, T, D, ep, stream)) != SC_OK)
    return rc;
  if (w->qk_norm) {  // 1 / rms of q (token-major) and of k (in the page slots)
    NormScale ns;
    std::memset(&ns, 0, sizeof ns);
    ns.part = ssb;
    ns.n_part = 2 * D / kSsPartWidth;
    ns.D = D;
    ns.eps = kNormEps;
    ns.rows = qb;
    ns.ld = D;
    ns.layer_base = ep.layer_base;
    ns.slot_bytes = ep.slot_bytes;
    ns.nq = p->nq;
    ns.tpp = d.tokens_per_page;
    ns.ppc = d.pages_per_chunk;
    ns.head_dim = d.head_dim;
    std::memcpy(ns.node_slot, ep.node_slot, sizeof ns.node_slot);
    if ((rc = launch_norm_scale(T, ns, stream)) != SC_OK) return rc;
  }
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
  // Without modulation the MLP's RMSNorm folds into its first GEMM: the last
  // residual GEMM before it stores per-64-feature sums of squares of the rows
  // it writes (part-major in ssb), a per-token kernel turns them into 1 / rms
  // (into hn's region, unused then), and the GELU epilogue scales each
  // token's accumulators by it, reading the raw rows x.
  const bool fold_mlp_norm = !w->mod;
  if (fold_mlp_norm && !w->cross) e2.ss_part = ssb;
  if ((rc = launch_gemm(EPI_RESIDUAL, TK_GEMM_OUT, static_cast<const uint16_t*>(w->w_o), ob, D, T, D, e2, stream)) != SC_OK)
    return rc;
  if (const sc_cross_attn* cr = w->cross) {
    // the query's RMSNorm (no modulation) folded into its GEMM, the factors
    // in hn's region (free once the QKV GEMM has read it)
    float* rsq = reinterpret_cast<float*>(hn);
    if ((rc = launch_row_rms(xb, T, D, rsq, stream)) != SC_OK) return rc;
    GemmEpilogue ec;
    std::memset(&ec, 0, sizeof ec);
    ec.out = qb;
    ec.ld_out = D;
    ec.row_scale = rsq;
    if (cr->q_norm) {
      ec.ss_part = ssb;
      ec.n_part = D / kSsPartWidth;
    }
    if ((rc = launch_gemm(EPI_STORE, TK_GEMM_CROSS_Q, static_cast<const uint16_t*>(cr->w_q), xb, D, T, D, ec, stream)) != SC_OK)
      return rc;
    if (cr->q_norm) {
      NormScale ns;
      std::memset(&ns, 0, sizeof ns);
      ns.part = ssb;
      ns.n_part = D / kSsPartWidth;
      ns.D = D;
      ns.eps = kNormEps;
      ns.rows = qb;
      ns.ld = D;
      ns.gain = cr->q_norm;
      if ((rc = launch_norm_scale(T, ns, stream)) != SC_OK) return rc;
    }
    {
      TimerAlias alias(TK_ATTENTION, TK_CROSS_ATTENTION);
      if ((rc = launch_attention(cr->plan, cr->cache, layer, qb, ob, 1.0f / std::sqrt((float)d.head_dim),
                                 attn_ws, attention_workspace_bound(), stream)) != SC_OK)
        return rc;
    }
    GemmEpilogue eo;
    std::memset(&eo, 0, sizeof eo);
    eo.out = xb;
    eo.ld_out = D;
    eo.nq = p->nq;
    if (fold_mlp_norm) eo.ss_part = ssb;
    if ((rc = launch_gemm(EPI_RESIDUAL, TK_GEMM_CROSS_OUT, static_cast<const uint16_t*>(cr->w_o), ob, D, T, D, eo, stream)) != SC_OK)
      return rc;
  }
  GemmEpilogue e3;
  std::memset(&e3, 0, sizeof e3);
  e3.out = ub;
  e3.ld_out = w->mlp;
  const uint16_t* mlp_in = hn;
  if (fold_mlp_norm) {
    float* rsb = reinterpret_cast<float*>(hn);
    if ((rc = launch_row_scale(ssb, D / kSsPartWidth, T, D, kNormEps, rsb, stream)) != SC_OK) return rc;
    e3.row_scale = rsb;
    mlp_in = xb;
  } else if ((rc = launch_rmsnorm(xb, hn, T, D, nm_m, stream)) != SC_OK) {
    return rc;
  }
  if ((rc = launch_gemm(EPI_GELU, TK_GEMM_UP, static_cast<const uint16_t*>(w->w_up), mlp_in, w->mlp, T, D, e3, stream)) != SC_OK)
    return rc;
  GemmEpilogue e4 = e2;
  e4.ss_part = nullptr;
  e4.gate_row = 5;  // gate_m
  if ((rc = launch_gemm(EPI_RESIDUAL, TK_GEMM_DOWN, static_cast<const uint16_t*>(w->w_down), ub, D, T, w->mlp, e4, stream)) != SC_OK)
    return rc;
  // only now are the pack's K/V of this layer complete: a failed call leaves
  // them unwritten, so the caller can run the block again
  for (int32_t i = 0; i < n; ++i)
    set_written(c, c->states.at(StateKey(p->nodes[i].chunk, p->nodes[i].level)), layer, 1);
  return SC_OK;
}

extern "C" size_t sc_condition_workspace_bytes(const sc_cache* c) {
  if (!c) return 0;
  const size_t L = (size_t)c->d.tokens_per_page * c->d.pages_per_chunk;
  const size_t D = (size_t)c->d.n_heads * c->d.head_dim;
  return 2 * align256(L * D * 2) + align256(L * (D / kSsPartWidth) * 4);
}

extern "C" int sc_condition_append(sc_cache* c, int32_t layer, sc_node st, const void* ctx,
                                   const void* w_k, const void* w_v, const float* k_norm, void* ws,
                                   size_t ws_bytes, sc_stream stream_) {
  if (!c || !ctx || !w_k || !w_v || !ws) return fail(SC_EINVAL, "null argument");
  const sc_cache_desc& d = c->d;
  if (d.dtype != SC_DTYPE_BF16) return fail(SC_EUNSUPPORTED, "condition projection is bf16 only");
  const int32_t D = d.n_heads * d.head_dim;
  const int32_t L = d.tokens_per_page * d.pages_per_chunk;
  if (d.head_dim != 128 || D % 256)
    return fail(SC_EUNSUPPORTED, "condition projection needs head_dim 128 and hidden %% 256 == 0");
  if (layer < 0 || layer >= d.n_layers) return fail(SC_EINVAL, "layer %d out of range", layer);
  if (st.chunk < 0 || st.level < 0) return fail(SC_EINVAL, "bad state (%d,%d)", st.chunk, st.level);
  auto it = c->states.find(StateKey(st.chunk, st.level));
  if (it != c->states.end() && it->second.written[layer])
    return fail(SC_EEXIST, "state (%d,%d) layer %d already written", st.chunk, st.level, layer);
  if (it == c->states.end() && sc_cache_free_slot_count(c) < d.pages_per_chunk)
    return fail(SC_ECAPACITY, "no free slots for condition (%d,%d)", st.chunk, st.level);
  if (ws_bytes < sc_condition_workspace_bytes(c))
    return fail(SC_EINVAL, "workspace of %zu bytes, need %zu", ws_bytes, sc_condition_workspace_bytes(c));
  if (misaligned16(ws) || (k_norm && misaligned16(k_norm)))
    return fail(SC_EINVAL, "workspace and key gain must be 16-byte aligned");
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  char* wsb = static_cast<char*>(ws);
  uint16_t* kb = reinterpret_cast<uint16_t*>(wsb);
  uint16_t* vb = reinterpret_cast<uint16_t*>(wsb + align256((size_t)L * D * 2));
  float* ssb = reinterpret_cast<float*>(wsb + 2 * align256((size_t)L * D * 2));
  const uint16_t* xb = static_cast<const uint16_t*>(ctx);
  GemmEpilogue e;
  std::memset(&e, 0, sizeof e);
  e.out = kb;
  e.ld_out = D;
  if (k_norm) {
    e.ss_part = ssb;
    e.n_part = D / kSsPartWidth;
  }
  int rc;
  if ((rc = launch_gemm(EPI_STORE, TK_GEMM_CONDITION, static_cast<const uint16_t*>(w_k), xb, D, L, D, e, stream)) != SC_OK)
    return rc;
  if (k_norm) {
    NormScale ns;
    std::memset(&ns, 0, sizeof ns);
    ns.part = ssb;
    ns.n_part = D / kSsPartWidth;
    ns.D = D;
    ns.eps = kNormEps;
    ns.rows = kb;
    ns.ld = D;
    ns.gain = k_norm;
    if ((rc = launch_norm_scale(L, ns, stream)) != SC_OK) return rc;
  }
  e.out = vb;
  e.ss_part = nullptr;
  if ((rc = launch_gemm(EPI_STORE, TK_GEMM_CONDITION, static_cast<const uint16_t*>(w_v), xb, D, L, D, e, stream)) != SC_OK)
    return rc;
  return sc_cache_append(c, layer, st, kb, vb, nullptr, stream_);
}
