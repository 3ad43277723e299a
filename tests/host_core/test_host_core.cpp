// Host core of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer
// (CPU only; the device launchers are stubs, see device_stubs.cpp).
//
// Covers the selection table (Sec. 3.2, Eq. 4-5: causality, self segment,
// in-pack sources, visibility), the paged cache (slot allocation, written
// flags, release and generations), plans (availability, Eq. 8; stale plans),
// the schedule (Eq. 7 rounds, Eq. 2 serial order, the release rule), and the
// block and stack orchestration's error paths: a launch failing at any point
// of a block leaves the pack's states unwritten, and a stack failing in its
// second layer leaves the first layer unwritten too.  Also the magic
// dividers the kernels split token indices with: exact quotients for every
// divisor up to 4096 and the workload's own.  Exit status 0 when every check
// holds; the sanitizers abort on the first memory or UB error.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../include/streamctx.h"
#include "../../paper_2609_22283_amd/csrc/divmagic.h"

extern int g_launches;
extern int g_fail_at;

static int g_failed = 0;
#define CHECK(cond)                                                      \
  do {                                                                   \
    if (!(cond)) {                                                       \
      std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++g_failed;                                                        \
    }                                                                    \
  } while (0)

static sc_policy policy(int kind, int K, int W) {
  sc_policy p;
  std::memset(&p, 0, sizeof p);
  p.kind = kind;
  p.K = K;
  p.W = W;
  return p;
}

// A fake device address: the host core stores and offsets device pointers
// but never dereferences them, and the stub launchers touch nothing.
static void* fake(uintptr_t a) { return reinterpret_cast<void*>(a); }

static void test_selection() {
  for (int kind = 0; kind < 3; ++kind) {
    sc_policy p = policy(kind, 4, 6);
    std::vector<sc_node> pack = {{6, 1}, {7, 2}, {8, 3}, {9, 4}};
    if (kind == SC_POLICY_SAME) pack = {{6, 2}, {7, 2}, {8, 2}, {9, 2}};
    sc_selection* sel = nullptr;
    CHECK(sc_selection_build(&p, pack.data(), (int32_t)pack.size(), &sel) == SC_OK);
    int32_t n = 0, ns = 0;
    const int32_t *off, *ch, *lv, *src;
    CHECK(sc_selection_get(sel, &n, &ns, &off, &ch, &lv, &src) == SC_OK);
    CHECK(n == 4 && off[0] == 0 && off[n] == ns);
    for (int32_t i = 0; i < n; ++i) {
      CHECK(off[i + 1] - off[i] == 7);  // six history chunks and the node itself
      for (int32_t s = off[i]; s < off[i + 1] - 1; ++s) CHECK(ch[s] < pack[i].chunk);
      const int32_t self = off[i + 1] - 1;
      CHECK(ch[self] == pack[i].chunk && lv[self] == pack[i].level && src[self] == i);
      for (int32_t s = off[i]; s < off[i + 1]; ++s)
        if (src[s] >= 0) CHECK(pack[src[s]].chunk == ch[s] && pack[src[s]].level == lv[s]);
    }
    int32_t nst = 0;
    const sc_node* states;
    const uint8_t* vis;
    CHECK(sc_visibility_get(sel, &nst, &states, &vis) == SC_OK);
    int32_t ones = 0;
    for (int32_t k = 0; k < n * nst; ++k) ones += vis[k];
    CHECK(ones == ns);
    sc_selection_free(sel);
  }
  // errors
  sc_policy bad = policy(SC_POLICY_PROG, 0, 6);
  sc_node one = {1, 1};
  sc_selection* sel = nullptr;
  CHECK(sc_selection_build(&bad, &one, 1, &sel) == SC_EINVAL && sel == nullptr);
  CHECK(std::strlen(sc_last_error()) > 0);
  sc_policy p = policy(SC_POLICY_PROG, 4, 6);
  sc_node dup[2] = {{3, 2}, {3, 2}};
  CHECK(sc_selection_build(&p, dup, 2, &sel) == SC_EINVAL);
  sc_node lvl = {3, 5};
  CHECK(sc_selection_build(&p, &lvl, 1, &sel) == SC_EINVAL);
  int8_t phi[5 * 2] = {0, 0, 1, 0, 2, 1, 3, 2, 9, 0};  // one entry above K
  sc_policy t = policy(SC_POLICY_TABLE, 4, 2);
  t.phi_table = phi;
  CHECK(sc_selection_build(&t, &one, 1, &sel) == SC_EINVAL);
  for (int code = 0; code >= -8; --code) CHECK(sc_status_name(code) != nullptr);
}

struct Cache {
  sc_cache* c = nullptr;
  sc_cache_desc d;
  Cache(int layers, int slots) {
    d = {layers, 2, 128, 104, 3, slots, SC_DTYPE_BF16};
    CHECK(sc_cache_pool_bytes(&d) > 0);
    CHECK(sc_cache_create(&d, fake(0x10000000), &c) == SC_OK);
  }
  ~Cache() { sc_cache_free(c); }
  void append_all_layers(sc_node st) {
    for (int l = 0; l < d.n_layers; ++l)
      CHECK(sc_cache_append(c, l, st, fake(0x20000000), fake(0x30000000), nullptr, nullptr) == SC_OK);
  }
};

static void test_cache_and_plan() {
  Cache cc(1, 30);
  for (int ch = 0; ch < 6; ++ch) cc.append_all_layers({ch, 0});
  CHECK(sc_cache_free_slot_count(cc.c) == 30 - 18);
  CHECK(sc_cache_contains(cc.c, {2, 0}, 0) == 1 && sc_cache_contains(cc.c, {2, 1}, -1) == 0);
  CHECK(sc_cache_append(cc.c, 0, {2, 0}, fake(0x20000000), fake(0x30000000), nullptr, nullptr) == SC_EEXIST);
  int32_t slots[3];
  CHECK(sc_cache_slots(cc.c, {1, 0}, slots) == SC_OK && slots[0] == 3 && slots[2] == 5);
  CHECK(sc_cache_slots(cc.c, {1, 1}, slots) == SC_ENOTFOUND);

  sc_policy p = policy(SC_POLICY_PROG, 4, 6);
  sc_node pack[4] = {{6, 1}, {7, 2}, {8, 3}, {9, 4}};
  sc_selection* sel = nullptr;
  CHECK(sc_selection_build(&p, pack, 4, &sel) == SC_OK);
  sc_plan* plan = nullptr;
  CHECK(sc_plan_build(sel, cc.c, &plan) == SC_OK);
  int32_t n = 0, np = 0;
  const int32_t *off, *ps, *pt, *pf;
  CHECK(sc_plan_get(plan, &n, &np, &off, &ps, &pt, &pf) == SC_OK);
  CHECK(n == 4 && np == 4 * 21 && off[4] == np);
  for (int32_t i = 0; i < n; ++i)   // page_frame: the absolute latent frame, chunk * 3 + f
    for (int32_t q = off[i]; q < off[i + 1]; ++q)
      CHECK(ps[q] >= 0 && ps[q] < 30 && pt[q] == 104 && pf[q] >= 0 && pf[q] / 3 <= pack[i].chunk);
  CHECK(sc_cache_free_slot_count(cc.c) == 0);  // the pack's 12 slots are reserved
  // a released history state makes the plan stale for attention
  CHECK(sc_cache_release(cc.c, {0, 0}) == SC_OK);
  CHECK(sc_attention(plan, cc.c, 0, fake(0x40000000), fake(0x50000000), 0.1f, nullptr, 0, nullptr) == SC_ESTALE);
  CHECK(sc_cache_release(cc.c, {0, 0}) == SC_ENOTFOUND);
  sc_plan_free(plan);
  sc_selection_free(sel);

  // clean history of an in-flight chunk is unavailable (Eq. 8)
  sc_policy clean = policy(SC_POLICY_CLEAN, 3, 1);
  sc_node k3[2] = {{0, 2}, {1, 3}};
  Cache c2(1, 12);
  c2.append_all_layers({0, 3});
  CHECK(sc_selection_build(&clean, k3, 2, &sel) == SC_OK);
  CHECK(sc_plan_build(sel, c2.c, &plan) == SC_EUNAVAILABLE && plan == nullptr);
  sc_selection_free(sel);
  sc_policy same = policy(SC_POLICY_SAME, 3, 1);
  CHECK(sc_selection_build(&same, k3, 2, &sel) == SC_OK);
  CHECK(sc_plan_build(sel, c2.c, &plan) == SC_OK);
  sc_plan_free(plan);
  sc_selection_free(sel);

  // a condition plan over one cached state
  sc_node cond[2] = {{0, 3}, {0, 3}};
  CHECK(sc_plan_condition(c2.c, cond, 2, 64, &plan) == SC_OK);
  sc_plan_free(plan);
  sc_node missing = {5, 0};
  CHECK(sc_plan_condition(c2.c, &missing, 1, 64, &plan) == SC_ENOTFOUND);
}

static void test_schedule() {
  const int K = 4, B = 16;
  CHECK(sc_pipeline_rounds(K, B, 1) == K + B && sc_pipeline_rounds(K, B, 0) == K + B - 1);
  int forwards = 0;
  sc_node nodes[K + 1];
  for (int r = 0; r < K + B; ++r) {
    int32_t m = 0;
    CHECK(sc_pipeline_round_nodes(K, B, 1, r, nodes, &m) == SC_OK);
    for (int32_t i = 1; i < m; ++i) CHECK(nodes[i].chunk > nodes[i - 1].chunk);
    forwards += m;
  }
  CHECK(forwards == B * (K + 1));
  CHECK(sc_serial_steps(K, B, 1) == B * (K + 1));
  sc_node nd;
  CHECK(sc_serial_step_node(K, B, 1, K, &nd) == SC_OK && nd.chunk == 0 && nd.level == 0);
  CHECK(sc_serial_step_node(K, B, 1, K + 1, &nd) == SC_OK && nd.chunk == 1 && nd.level == K);
  CHECK(sc_serial_step_node(K, B, 1, B * (K + 1), &nd) == SC_EINVAL);

  // the release rule over a whole progressive schedule: every plan stays available
  Cache cc(1, (6 + 2 * K + 4) * 3);
  sc_policy p = policy(SC_POLICY_PROG, K, 6);
  std::vector<sc_node> all;
  for (int r = 0; r < K + B; ++r) {
    int32_t m = 0;
    sc_pipeline_round_nodes(K, B, 1, r, nodes, &m);
    all.insert(all.end(), nodes, nodes + m);
  }
  size_t done = 0;
  for (int r = 0; r < K + B; ++r) {
    int32_t m = 0;
    sc_pipeline_round_nodes(K, B, 1, r, nodes, &m);
    sc_selection* sel = nullptr;
    sc_plan* plan = nullptr;
    CHECK(sc_selection_build(&p, nodes, m, &sel) == SC_OK);
    CHECK(sc_plan_build(sel, cc.c, &plan) == SC_OK);
    for (int32_t i = 0; i < m; ++i) cc.append_all_layers(nodes[i]);
    done += m;
    CHECK(sc_cache_release_unread(cc.c, &p, all.data() + done, (int32_t)(all.size() - done)) >= 0);
    sc_plan_free(plan);
    sc_selection_free(sel);
  }
  CHECK(sc_cache_free_slot_count(cc.c) == (6 + 2 * K + 4) * 3);
}

static sc_block_weights weights(int mlp) {
  sc_block_weights w;
  std::memset(&w, 0, sizeof w);
  w.hidden = 256;
  w.n_heads = 2;
  w.head_dim = 128;
  w.mlp = mlp;
  w.w_qkv = fake(0x60000000);
  w.w_o = fake(0x61000000);
  w.w_up = fake(0x62000000);
  w.w_down = fake(0x63000000);
  return w;
}

static void test_block_error_paths() {
  sc_policy p = policy(SC_POLICY_PROG, 4, 6);
  sc_node pack[4] = {{6, 1}, {7, 2}, {8, 3}, {9, 4}};
  const int32_t T = 4 * 312;
  sc_block_weights w = weights(512);
  const size_t ws = sc_block_workspace_bytes(&w, T);
  size_t qo = 0, oo = 0;
  CHECK(sc_block_workspace_views(&w, T, &qo, &oo) == SC_OK && qo > 0 && oo > qo && oo + T * 256 * 2 <= ws);

  auto fresh = [&](Cache& cc, sc_plan** plan) {
    for (int ch = 0; ch < 6; ++ch) cc.append_all_layers({ch, 0});
    sc_selection* sel = nullptr;
    CHECK(sc_selection_build(&p, pack, 4, &sel) == SC_OK);
    CHECK(sc_plan_build(sel, cc.c, plan) == SC_OK);
    sc_selection_free(sel);
  };
  // count the launches of one block
  int per_block = 0;
  {
    Cache cc(1, 40);
    sc_plan* plan = nullptr;
    fresh(cc, &plan);
    g_fail_at = -1;
    g_launches = 0;
    CHECK(sc_block_forward(&w, cc.c, 0, plan, fake(0x70000000), nullptr, fake(0x80000000), ws, nullptr) == SC_OK);
    per_block = g_launches;
    for (auto& nd : pack) CHECK(sc_cache_contains(cc.c, nd, 0) == 1);
    CHECK(sc_block_forward(&w, cc.c, 0, plan, fake(0x70000000), nullptr, fake(0x80000000), ws, nullptr) == SC_EEXIST);
    sc_plan_free(plan);
  }
  CHECK(per_block >= 6);
  // a failure at any launch leaves the pack unwritten, and the block runs again
  for (int k = 1; k <= per_block; ++k) {
    Cache cc(1, 40);
    sc_plan* plan = nullptr;
    fresh(cc, &plan);
    g_launches = 0;
    g_fail_at = k;
    CHECK(sc_block_forward(&w, cc.c, 0, plan, fake(0x70000000), nullptr, fake(0x80000000), ws, nullptr) == SC_EDEVICE);
    for (auto& nd : pack) CHECK(sc_cache_contains(cc.c, nd, 0) == 0);
    g_fail_at = -1;
    CHECK(sc_block_forward(&w, cc.c, 0, plan, fake(0x70000000), nullptr, fake(0x80000000), ws, nullptr) == SC_OK);
    for (auto& nd : pack) CHECK(sc_cache_contains(cc.c, nd, 0) == 1);
    sc_plan_free(plan);
  }
  // an unsupported MLP width is refused before any launch
  {
    Cache cc(1, 40);
    sc_plan* plan = nullptr;
    fresh(cc, &plan);
    sc_block_weights bad = weights(320);
    g_launches = 0;
    CHECK(sc_block_forward(&bad, cc.c, 0, plan, fake(0x70000000), nullptr, fake(0x80000000), ws, nullptr) ==
          SC_EUNSUPPORTED);
    CHECK(g_launches == 0);
    sc_plan_free(plan);
  }
  // a two-layer stack failing in its second layer leaves both layers unwritten
  {
    Cache cc(2, 40);
    sc_plan* plan = nullptr;
    fresh(cc, &plan);
    sc_block_weights ws2[2] = {w, w};
    g_launches = 0;
    g_fail_at = per_block + 2;
    CHECK(sc_stack_forward(ws2, 2, cc.c, plan, fake(0x70000000), nullptr, fake(0x80000000), ws, nullptr) == SC_EDEVICE);
    for (auto& nd : pack)
      for (int l = 0; l < 2; ++l) CHECK(sc_cache_contains(cc.c, nd, l) == 0);
    g_fail_at = -1;
    CHECK(sc_stack_forward(ws2, 2, cc.c, plan, fake(0x70000000), nullptr, fake(0x80000000), ws, nullptr) == SC_OK);
    for (auto& nd : pack)
      for (int l = 0; l < 2; ++l) CHECK(sc_cache_contains(cc.c, nd, l) == 1);
    sc_plan_free(plan);
  }
}

// The quotient as the kernels form it: (high 32 bits of n * mul, + n) >> shift.
static uint32_t magic_quotient(uint32_t n, const sc::DivMagic& m) {
  const uint32_t hi = (uint32_t)(((uint64_t)n * m.mul) >> 32);
  return (hi + n) >> m.shift;
}

static void test_magic_div() {
  std::vector<uint32_t> divs;
  for (uint32_t d = 1; d <= 4096; ++d) divs.push_back(d);
  // node sizes, page sizes and grid widths of the workloads, and large ones
  for (uint32_t d : {4680u, 9360u, 14040u, 18720u, 23400u, 1560u, 3120u, 6241u, 65535u, 65536u, 65537u,
                     1000003u, (1u << 30) - 1, 1u << 30, (1u << 30) + 1, (1u << 31) - 1})
    divs.push_back(d);
  uint64_t state = 0x9e3779b97f4a7c15ull;  // xorshift64 numerators
  int bad = 0;
  for (uint32_t d : divs) {
    const sc::DivMagic m = sc::magic_div(d);
    if (m.div != d) ++bad;
    // quotient boundaries k d - 1, k d for small k and near 2^31, then random n < 2^31
    std::vector<uint32_t> ns = {0u, 1u, (1u << 31) - 1, (1u << 31) - 2};
    for (uint32_t k = 1; k <= 64; ++k) {
      const uint64_t kd = (uint64_t)k * d, top = (uint64_t)((((1ull << 31) - 1) / d) - (k - 1)) * d;
      if (kd < (1ull << 31)) ns.insert(ns.end(), {(uint32_t)(kd - 1), (uint32_t)kd});
      if (top > 0 && top < (1ull << 31)) ns.insert(ns.end(), {(uint32_t)(top - 1), (uint32_t)top});
    }
    for (int i = 0; i < 256; ++i) {
      state ^= state << 13;
      state ^= state >> 7;
      state ^= state << 17;
      ns.push_back((uint32_t)(state & 0x7fffffffu));
    }
    for (uint32_t n : ns)
      if (magic_quotient(n, m) != n / d) ++bad;
  }
  CHECK(bad == 0);
}

int main() {
  CHECK(sc_abi_version() == SC_ABI_VERSION);
  test_magic_div();
  test_selection();
  test_cache_and_plan();
  test_schedule();
  test_block_error_paths();
  if (g_failed) {
    std::fprintf(stderr, "%d check(s) failed\n", g_failed);
    return 1;
  }
  std::printf("host core checks passed\n");
  return 0;
}
