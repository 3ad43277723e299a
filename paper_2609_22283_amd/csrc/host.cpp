// Host core: error reporting, selection table (Sec. 3.2, Eq. 4-5), paged
// cache metadata (Sec. 3.2 "Effective context"), plan with availability
// (Sec. 3.3 "Restrictions on context selection", Eq. 8).
#include <algorithm>
#include <cstdio>
#include <cstring>
#include <new>
#include <set>

#include "internal.h"

namespace sc {

static thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = std::string(sc_status_name(code)) + ": " + buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(SC_EDEVICE, "%s failed: %s", what, hipGetErrorString(e));
}

int plan_check(const sc_plan* plan, const sc_cache* cache, int32_t layer) {
  if (plan->cache != cache) return fail(SC_EINVAL, "plan was built for another cache");
  if (layer < 0 || layer >= cache->d.n_layers)
    return fail(SC_EINVAL, "layer %d outside [0, %d)", layer, cache->d.n_layers);
  for (size_t p = 0; p < plan->page_slot.size(); ++p) {
    int32_t s = plan->page_slot[p];
    if (!cache->used[s] || cache->gen[s] != plan->page_gen[p])
      return fail(SC_ESTALE, "slot %d was released after the plan was built", s);
  }
  // every slot is still the one planned (above), so its flag is its state's
  const uint8_t* wr = cache->slot_written.data() + (size_t)layer * cache->d.n_slots;
  for (size_t p = 0; p < plan->page_slot.size(); ++p)
    if (!wr[plan->page_slot[p]])
      return fail(SC_EUNAVAILABLE, "state (%d,%d) has no K/V at layer %d",
                  plan->page_state[p].first, plan->page_state[p].second, layer);
  return SC_OK;
}

void set_written(sc_cache* cache, StateEntry& e, int32_t layer, uint8_t v) {
  e.written[layer] = v;
  for (int32_t s : e.slots) cache->slot_written[(size_t)layer * cache->d.n_slots + s] = v;
}

int policy_check(const sc_policy* p) {
  if (p->kind < SC_POLICY_CLEAN || p->kind > SC_POLICY_TABLE)
    return fail(SC_EINVAL, "unknown policy kind %d", p->kind);
  if (p->K < 1 || p->W < 0 || p->n_chunks < 0)
    return fail(SC_EINVAL, "need K >= 1, W >= 0, n_chunks >= 0 (K=%d W=%d n_chunks=%d)", p->K, p->W,
                p->n_chunks);
  if (p->kind == SC_POLICY_TABLE && p->W > 0) {
    if (!p->phi_table) return fail(SC_EINVAL, "table policy without phi table");
    const int64_t n = (int64_t)std::max(p->n_chunks, 1) * (p->K + 1) * p->W;
    for (int64_t i = 0; i < n; ++i)
      if (p->phi_table[i] < 0 || p->phi_table[i] > p->K)
        return fail(SC_EINVAL, "phi table entry %d outside [0, K]", (int)p->phi_table[i]);
  }
  return SC_OK;
}

static int64_t policy_index(const sc_policy* p, int32_t c, int32_t j, int32_t r) {
  const int64_t row = p->n_chunks > 0 ? (int64_t)c * (p->K + 1) + j : j;
  return row * p->W + (r - 1);
}

bool policy_selects(const sc_policy* p, int32_t c, int32_t j, int32_t r) {
  return !p->r_mask || p->r_mask[policy_index(p, c, j, r)] != 0;
}

int32_t policy_level(const sc_policy* p, int32_t c, int32_t j, int32_t r) {
  switch (p->kind) {
    case SC_POLICY_CLEAN: return 0;
    case SC_POLICY_SAME: return j;
    case SC_POLICY_PROG: return j - r > 0 ? j - r : 0;
    default: return p->phi_table[policy_index(p, c, j, r)];
  }
}

RopeLayout rope_layout(const sc_rope_desc* d) {
  RopeLayout L;
  L.pairs_t = d->dim_t / 2;
  L.pairs_h = d->dim_h / 2;
  L.pairs_w = d->dim_w / 2;
  L.off_t = 0;
  L.off_h = (int64_t)d->max_frames * L.pairs_t;
  L.off_w = L.off_h + (int64_t)d->grid_h * L.pairs_h;
  L.total = L.off_w + (int64_t)d->grid_w * L.pairs_w;
  return L;
}

}  // namespace sc

using namespace sc;

extern "C" {

int sc_abi_version(void) { return SC_ABI_VERSION; }

const char* sc_last_error(void) { return g_last_error.c_str(); }

const char* sc_status_name(int status) {
  switch (status) {
    case SC_OK: return "SC_OK";
    case SC_EINVAL: return "SC_EINVAL";
    case SC_EUNAVAILABLE: return "SC_EUNAVAILABLE";
    case SC_ECAPACITY: return "SC_ECAPACITY";
    case SC_EEXIST: return "SC_EEXIST";
    case SC_ENOTFOUND: return "SC_ENOTFOUND";
    case SC_ESTALE: return "SC_ESTALE";
    case SC_EDEVICE: return "SC_EDEVICE";
    case SC_EUNSUPPORTED: return "SC_EUNSUPPORTED";
    default: return "SC_E?";
  }
}

// ---------------------------------------------------------------- selection

int sc_selection_build(const sc_policy* p, const sc_node* nodes, int32_t n, sc_selection** out) {
  if (!p || !out || n < 0 || (n > 0 && !nodes)) return fail(SC_EINVAL, "null argument");
  *out = nullptr;
  int rc = policy_check(p);
  if (rc != SC_OK) return rc;
  std::map<StateKey, int32_t> index_of;
  for (int32_t i = 0; i < n; ++i) {
    if (nodes[i].chunk < 0 || (p->n_chunks > 0 && nodes[i].chunk >= p->n_chunks) ||
        nodes[i].level < 0 || nodes[i].level > p->K)
      return fail(SC_EINVAL, "node %d = (%d,%d) outside chunk in [0, n_chunks), level in [0, K]", i,
                  nodes[i].chunk, nodes[i].level);
    if (!index_of.emplace(StateKey(nodes[i].chunk, nodes[i].level), i).second)
      return fail(SC_EINVAL, "duplicate node (%d,%d)", nodes[i].chunk, nodes[i].level);
  }
  sc_selection* s = new (std::nothrow) sc_selection;
  if (!s) return fail(SC_EINVAL, "out of host memory");
  s->nodes.assign(nodes, nodes + n);
  s->seg_off.push_back(0);
  std::set<StateKey> distinct;
  auto emit = [&](int32_t c, int32_t l) {
    s->seg_chunk.push_back(c);
    s->seg_level.push_back(l);
    auto it = index_of.find(StateKey(c, l));
    s->seg_src.push_back(it == index_of.end() ? -1 : it->second);
    distinct.insert(StateKey(c, l));
  };
  for (int32_t i = 0; i < n; ++i) {
    const int32_t c = nodes[i].chunk, j = nodes[i].level;
    const int32_t rmax = std::min(p->W, c);
    for (int32_t r = rmax; r >= 1; --r) {  // oldest history chunk first
      if (!policy_selects(p, c, j, r)) continue;
      emit(c - r, policy_level(p, c, j, r));
    }
    emit(c, j);  // the node's own chunk at its own level
    s->seg_off.push_back((int32_t)s->seg_chunk.size());
  }
  for (const auto& k : distinct) s->states.push_back(sc_node{k.first, k.second});
  const size_t ns = s->states.size();
  s->vis.assign((size_t)n * ns, 0);
  for (int32_t i = 0; i < n; ++i)
    for (int32_t g = s->seg_off[i]; g < s->seg_off[i + 1]; ++g) {
      StateKey key(s->seg_chunk[g], s->seg_level[g]);
      size_t k = std::distance(distinct.begin(), distinct.find(key));
      s->vis[(size_t)i * ns + k] = 1;
    }
  *out = s;
  return SC_OK;
}

int sc_selection_get(const sc_selection* s, int32_t* n_nodes, int32_t* n_segments,
                     const int32_t** seg_off, const int32_t** seg_chunk, const int32_t** seg_level,
                     const int32_t** seg_src) {
  if (!s) return fail(SC_EINVAL, "null selection");
  if (n_nodes) *n_nodes = (int32_t)s->nodes.size();
  if (n_segments) *n_segments = (int32_t)s->seg_chunk.size();
  if (seg_off) *seg_off = s->seg_off.data();
  if (seg_chunk) *seg_chunk = s->seg_chunk.data();
  if (seg_level) *seg_level = s->seg_level.data();
  if (seg_src) *seg_src = s->seg_src.data();
  return SC_OK;
}

int sc_visibility_get(const sc_selection* s, int32_t* n_states, const sc_node** states,
                      const uint8_t** vis) {
  if (!s) return fail(SC_EINVAL, "null selection");
  if (n_states) *n_states = (int32_t)s->states.size();
  if (states) *states = s->states.data();
  if (vis) *vis = s->vis.data();
  return SC_OK;
}

void sc_selection_free(sc_selection* s) { delete s; }

// -------------------------------------------------------------------- cache

static int validate_desc(const sc_cache_desc* d) {
  if (!d) return fail(SC_EINVAL, "null cache descriptor");
  if (d->n_layers < 1 || d->n_heads < 1 || d->n_slots < 1 || d->pages_per_chunk < 1)
    return fail(SC_EINVAL, "n_layers, n_heads, n_slots, pages_per_chunk must be >= 1");
  if (d->tokens_per_page < 8 || d->tokens_per_page % 8 != 0)
    return fail(SC_EINVAL, "tokens_per_page must be a positive multiple of 8 (got %d)",
                d->tokens_per_page);
  if (d->dtype != SC_DTYPE_BF16 && d->dtype != SC_DTYPE_F32)
    return fail(SC_EINVAL, "unknown dtype %d", d->dtype);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(SC_EUNSUPPORTED, "head_dim must be 64 or 128 (got %d)", d->head_dim);
  return SC_OK;
}

static size_t slot_bytes(const sc_cache_desc* d) {
  return 2ull * d->n_heads * d->tokens_per_page * d->head_dim * dtype_size(d->dtype);
}

size_t sc_cache_pool_bytes(const sc_cache_desc* d) {
  if (validate_desc(d) != SC_OK) return 0;
  return slot_bytes(d) * (size_t)d->n_slots * (size_t)d->n_layers;
}

int sc_cache_create(const sc_cache_desc* d, void* pool, sc_cache** out) {
  if (!out) return fail(SC_EINVAL, "null output");
  *out = nullptr;
  int rc = validate_desc(d);
  if (rc != SC_OK) return rc;
  sc_cache* c = new (std::nothrow) sc_cache;
  if (!c) return fail(SC_EINVAL, "out of host memory");
  c->d = *d;
  c->pool = static_cast<char*>(pool);
  c->slot_bytes = slot_bytes(d);
  c->kv_half = c->slot_bytes / 2;
  c->used.assign(d->n_slots, 0);
  c->gen.assign(d->n_slots, 0);
  c->owner.assign(d->n_slots, StateKey(-1, -1));
  c->slot_written.assign((size_t)d->n_layers * d->n_slots, 0);
  *out = c;
  return SC_OK;
}

void sc_cache_free(sc_cache* c) { delete c; }

int sc_cache_contains(const sc_cache* c, sc_node st, int32_t layer) {
  if (!c) return fail(SC_EINVAL, "null cache");
  auto it = c->states.find(StateKey(st.chunk, st.level));
  if (it == c->states.end()) return 0;
  if (layer < 0) return 1;
  if (layer >= c->d.n_layers) return fail(SC_EINVAL, "layer %d out of range", layer);
  return it->second.written[layer] ? 1 : 0;
}

int sc_cache_slots(const sc_cache* c, sc_node st, int32_t* slots) {
  if (!c || !slots) return fail(SC_EINVAL, "null argument");
  auto it = c->states.find(StateKey(st.chunk, st.level));
  if (it == c->states.end()) return fail(SC_ENOTFOUND, "state (%d,%d) not cached", st.chunk, st.level);
  std::copy(it->second.slots.begin(), it->second.slots.end(), slots);
  return SC_OK;
}

int sc_cache_free_slot_count(const sc_cache* c) {
  if (!c) return fail(SC_EINVAL, "null cache");
  return (int)std::count(c->used.begin(), c->used.end(), 0);
}

// Lowest-free-first allocation of one state's pages (frames ascending).
static int allocate_state(sc_cache* c, StateKey key) {
  std::vector<int32_t> got;
  for (int32_t s = 0; s < c->d.n_slots && (int32_t)got.size() < c->d.pages_per_chunk; ++s)
    if (!c->used[s]) got.push_back(s);
  if ((int32_t)got.size() < c->d.pages_per_chunk)
    return fail(SC_ECAPACITY, "no free slots for state (%d,%d)", key.first, key.second);
  for (int32_t s : got) {
    c->used[s] = 1;
    c->owner[s] = key;
    for (int32_t l = 0; l < c->d.n_layers; ++l) c->slot_written[(size_t)l * c->d.n_slots + s] = 0;
  }
  StateEntry e;
  e.slots = got;
  e.written.assign(c->d.n_layers, 0);
  c->states.emplace(key, std::move(e));
  return SC_OK;
}

int sc_cache_release(sc_cache* c, sc_node st) {
  if (!c) return fail(SC_EINVAL, "null cache");
  auto it = c->states.find(StateKey(st.chunk, st.level));
  if (it == c->states.end()) return fail(SC_ENOTFOUND, "state (%d,%d) not cached", st.chunk, st.level);
  for (int32_t s : it->second.slots) {
    c->used[s] = 0;
    c->gen[s] += 1;
    c->owner[s] = StateKey(-1, -1);
    for (int32_t l = 0; l < c->d.n_layers; ++l) c->slot_written[(size_t)l * c->d.n_slots + s] = 0;
  }
  c->states.erase(it);
  return SC_OK;
}

int sc_cache_append(sc_cache* c, int32_t layer, sc_node st, const void* k, const void* v,
                    const sc_rope* rope, sc_stream stream) {
  if (!c || !k || !v) return fail(SC_EINVAL, "null argument");
  if (layer < 0 || layer >= c->d.n_layers) return fail(SC_EINVAL, "layer %d out of range", layer);
  if (st.chunk < 0 || st.level < 0) return fail(SC_EINVAL, "bad state (%d,%d)", st.chunk, st.level);
  if (rope) {
    const sc_rope_desc& r = rope->desc;
    if (!rope->dev_table || r.grid_h * r.grid_w != c->d.tokens_per_page ||
        r.dim_t + r.dim_h + r.dim_w != c->d.head_dim || (r.dim_t | r.dim_h | r.dim_w) & 1)
      return fail(SC_EINVAL, "rope descriptor does not match the cache geometry");
    if ((st.chunk + 1) * c->d.pages_per_chunk > r.max_frames)
      return fail(SC_EINVAL, "chunk %d beyond the rope table's %d frames", st.chunk, r.max_frames);
  }
  StateKey key(st.chunk, st.level);
  auto it = c->states.find(key);
  if (it != c->states.end() && it->second.written[layer])
    return fail(SC_EEXIST, "state (%d,%d) layer %d already written", st.chunk, st.level, layer);
  bool fresh = false;
  if (it == c->states.end()) {
    int rc = allocate_state(c, key);
    if (rc != SC_OK) return rc;
    it = c->states.find(key);
    fresh = true;
  }
  int rc = launch_append(c, layer, it->second.slots.data(), st.chunk, k, v, rope,
                         static_cast<hipStream_t>(stream));
  if (rc != SC_OK) {
    if (fresh) sc_cache_release(c, st);
    return rc;
  }
  set_written(c, it->second, layer, 1);
  return SC_OK;
}

// --------------------------------------------------------------------- plan

int sc_plan_build(const sc_selection* s, sc_cache* c, sc_plan** out) {
  if (!s || !c || !out) return fail(SC_EINVAL, "null argument");
  *out = nullptr;
  const int32_t n = (int32_t)s->nodes.size();
  for (int32_t i = 0; i < n; ++i)
    for (int32_t g = s->seg_off[i]; g < s->seg_off[i + 1]; ++g)
      if (s->seg_src[g] < 0 && !c->states.count(StateKey(s->seg_chunk[g], s->seg_level[g])))
        return fail(SC_EUNAVAILABLE, "node (%d,%d) reads state (%d,%d): not cached, not in the pack",
                    s->nodes[i].chunk, s->nodes[i].level, s->seg_chunk[g], s->seg_level[g]);
  int32_t missing = 0;
  for (const auto& nd : s->nodes)
    if (!c->states.count(StateKey(nd.chunk, nd.level))) ++missing;
  if ((int64_t)missing * c->d.pages_per_chunk > sc_cache_free_slot_count(c))
    return fail(SC_ECAPACITY, "%d pack states need %d slots, %d free", missing,
                missing * c->d.pages_per_chunk, sc_cache_free_slot_count(c));
  for (const auto& nd : s->nodes) {
    StateKey key(nd.chunk, nd.level);
    if (!c->states.count(key)) {
      int rc = allocate_state(c, key);
      if (rc != SC_OK) return rc;  // unreachable: capacity checked above
    }
  }
  sc_plan* p = new (std::nothrow) sc_plan;
  if (!p) return fail(SC_EINVAL, "out of host memory");
  p->nodes = s->nodes;
  p->cache = c;
  p->nq = c->d.tokens_per_page * c->d.pages_per_chunk;
  p->page_off.push_back(0);
  const int32_t ppc = c->d.pages_per_chunk;
  for (int32_t i = 0; i < n; ++i) {
    for (int32_t g = s->seg_off[i]; g < s->seg_off[i + 1]; ++g) {
      StateKey key(s->seg_chunk[g], s->seg_level[g]);
      const StateEntry& e = c->states.at(key);
      for (int32_t f = 0; f < ppc; ++f) {
        p->page_slot.push_back(e.slots[f]);
        p->page_tokens.push_back(c->d.tokens_per_page);
        p->page_frame.push_back(key.first * ppc + f);
        p->page_gen.push_back(c->gen[e.slots[f]]);
        p->page_state.push_back(key);
      }
    }
    p->page_off.push_back((int32_t)p->page_slot.size());
  }
  *out = p;
  return SC_OK;
}

int sc_plan_get(const sc_plan* p, int32_t* n_nodes, int32_t* n_pages, const int32_t** page_off,
                const int32_t** page_slot, const int32_t** page_tokens, const int32_t** page_frame) {
  if (!p) return fail(SC_EINVAL, "null plan");
  if (n_nodes) *n_nodes = (int32_t)p->nodes.size();
  if (n_pages) *n_pages = (int32_t)p->page_slot.size();
  if (page_off) *page_off = p->page_off.data();
  if (page_slot) *page_slot = p->page_slot.data();
  if (page_tokens) *page_tokens = p->page_tokens.data();
  if (page_frame) *page_frame = p->page_frame.data();
  return SC_OK;
}

void sc_plan_free(sc_plan* p) { delete p; }

int sc_plan_condition(sc_cache* c, const sc_node* conds, int32_t n, int32_t nq, sc_plan** out) {
  if (!c || !conds || !out) return fail(SC_EINVAL, "null argument");
  *out = nullptr;
  if (n < 1 || nq < 1) return fail(SC_EINVAL, "need n >= 1 and nq >= 1 (n=%d nq=%d)", n, nq);
  for (int32_t i = 0; i < n; ++i)
    if (!c->states.count(StateKey(conds[i].chunk, conds[i].level)))
      return fail(SC_ENOTFOUND, "condition state (%d,%d) not in the cache", conds[i].chunk,
                  conds[i].level);
  sc_plan* p = new (std::nothrow) sc_plan;
  if (!p) return fail(SC_EINVAL, "out of host memory");
  p->nodes.assign(conds, conds + n);
  p->cache = c;
  p->nq = nq;
  p->page_off.push_back(0);
  const int32_t ppc = c->d.pages_per_chunk;
  for (int32_t i = 0; i < n; ++i) {
    const StateKey key(conds[i].chunk, conds[i].level);
    const StateEntry& e = c->states.at(key);
    for (int32_t f = 0; f < ppc; ++f) {
      p->page_slot.push_back(e.slots[f]);
      p->page_tokens.push_back(c->d.tokens_per_page);
      p->page_frame.push_back(f);
      p->page_gen.push_back(c->gen[e.slots[f]]);
      p->page_state.push_back(key);
    }
    p->page_off.push_back((int32_t)p->page_slot.size());
  }
  *out = p;
  return SC_OK;
}

// ---------------------------------------------------------------- attention

size_t sc_attention_workspace_bytes(const sc_plan* p, const sc_cache* c) {
  if (!p || !c || p->cache != c) return 0;
  return attention_workspace_bytes(p, c);
}

int sc_attention(const sc_plan* p, const sc_cache* c, int32_t layer, const void* q, void* o,
                 float scale, void* ws, size_t ws_bytes, sc_stream stream) {
  if (!p || !c || !q || !o) return fail(SC_EINVAL, "null argument");
  int rc = plan_check(p, c, layer);
  if (rc != SC_OK) return rc;
  if (p->nodes.empty()) return SC_OK;
  return launch_attention(p, c, layer, q, o, scale, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

// --------------------------------------------------------------------- rope

size_t sc_rope_table_bytes(const sc_rope_desc* d) {
  if (!d) return 0;
  return (size_t)rope_layout(d).total * 2 * sizeof(float);
}

int sc_rope_table_build(const sc_rope_desc* d, void* table, sc_stream stream) {
  if (!d || !table) return fail(SC_EINVAL, "null argument");
  if (d->grid_h < 1 || d->grid_w < 1 || d->max_frames < 1 || d->dim_t < 0 || d->dim_h < 0 ||
      d->dim_w < 0 || (d->dim_t | d->dim_h | d->dim_w) & 1 || !(d->theta > 0.0f))
    return fail(SC_EINVAL, "bad rope descriptor");
  return launch_rope_table(d, table, static_cast<hipStream_t>(stream));
}

}  // extern "C"
