// Execution schedule (Sec. 3.3, Eq. 7): round packs, retention, stack forward.
#include <set>

#include "internal.h"

using namespace sc;

extern "C" int sc_pipeline_rounds(int32_t K, int32_t B, int32_t refresh) {
  if (K < 1 || B < 1) return fail(SC_EINVAL, "need K >= 1 and B >= 1");
  return refresh ? K + B : K + B - 1;
}

extern "C" int sc_pipeline_round_nodes(int32_t K, int32_t B, int32_t refresh, int32_t n, sc_node* out,
                                       int32_t* n_out) {
  if (!out || !n_out) return fail(SC_EINVAL, "null argument");
  const int rounds = sc_pipeline_rounds(K, B, refresh);
  if (rounds < 0) return rounds;
  if (n < 0 || n >= rounds) return fail(SC_EINVAL, "round %d outside [0, %d)", n, rounds);
  int32_t m = 0;
  // chunk n - K + j at level j; ascending j is ascending chunk (oldest first)
  for (int32_t j = refresh ? 0 : 1; j <= K; ++j) {
    const int32_t c = n - K + j;
    if (c >= 0 && c < B) out[m++] = sc_node{c, j};
  }
  *n_out = m;
  return SC_OK;
}

extern "C" int sc_serial_steps(int32_t K, int32_t B, int32_t refresh) {
  if (K < 1 || B < 1) return fail(SC_EINVAL, "need K >= 1 and B >= 1");
  return B * (refresh ? K + 1 : K);
}

extern "C" int sc_serial_step_node(int32_t K, int32_t B, int32_t refresh, int32_t n, sc_node* out) {
  if (!out) return fail(SC_EINVAL, "null argument");
  const int steps = sc_serial_steps(K, B, refresh);
  if (steps < 0) return steps;
  if (n < 0 || n >= steps) return fail(SC_EINVAL, "step %d outside [0, %d)", n, steps);
  // chunk by chunk; within a chunk the levels K .. 1, then the refresh (c, 0)
  const int32_t per = refresh ? K + 1 : K;
  out->chunk = n / per;
  out->level = K - n % per;
  return SC_OK;
}

extern "C" int sc_cache_release_unread(sc_cache* c, const sc_policy* p, const sc_node* future,
                                       int32_t n_future) {
  if (!c || !p || (n_future > 0 && !future)) return fail(SC_EINVAL, "null argument");
  int rc = policy_check(p);
  if (rc != SC_OK) return rc;
  std::set<StateKey> needed;
  for (int32_t i = 0; i < n_future; ++i) {
    const int32_t cc = future[i].chunk, j = future[i].level;
    if (cc < 0 || (p->n_chunks > 0 && cc >= p->n_chunks) || j < 0 || j > p->K)
      return fail(SC_EINVAL, "bad future node (%d,%d)", cc, j);
    for (int32_t r = 1; r <= p->W && r <= cc; ++r)
      if (policy_selects(p, cc, j, r)) needed.insert(StateKey(cc - r, policy_level(p, cc, j, r)));
  }
  std::vector<StateKey> drop;
  for (const auto& kv : c->states)
    if (!needed.count(kv.first)) drop.push_back(kv.first);
  for (const auto& k : drop) {
    rc = sc_cache_release(c, sc_node{k.first, k.second});
    if (rc != SC_OK) return rc;
  }
  return (int)drop.size();
}

extern "C" int sc_stack_forward(const sc_block_weights* layers, int32_t n_layers, sc_cache* cache,
                                const sc_plan* plan, void* x, const sc_rope* rope, void* ws,
                                size_t ws_bytes, sc_stream stream) {
  if (!layers || n_layers < 1) return fail(SC_EINVAL, "need at least one layer");
  if (!cache || n_layers > cache->d.n_layers)
    return fail(SC_EINVAL, "%d layers but the cache holds %d", n_layers, cache ? cache->d.n_layers : 0);
  for (int32_t l = 0; l < n_layers; ++l) {
    int rc = sc_block_forward(&layers[l], cache, l, plan, x, rope, ws, ws_bytes, stream);
    if (rc != SC_OK) {
      // layers before l are complete, but the forward as a whole is not:
      // mark none of the pack's layers written so the caller can rerun it
      for (int32_t e = 0; e < l; ++e)
        for (const sc_node& nd : plan->nodes) {
          auto it = cache->states.find(StateKey(nd.chunk, nd.level));
          if (it != cache->states.end()) set_written(cache, it->second, e, 0);
        }
      return rc;
    }
  }
  return SC_OK;
}
