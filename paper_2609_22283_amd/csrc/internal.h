// Internal declarations shared by the host core and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <map>
#include <string>
#include <utility>
#include <vector>

#include "../../include/streamctx.h"
#include "../../include/streamctx_measure.h"

namespace sc {

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int hip_fail(hipError_t e, const char* what);

#define SC_HIP(call)                                   \
  do {                                                 \
    hipError_t e_ = (call);                            \
    if (e_ != hipSuccess) return ::sc::hip_fail(e_, #call); \
  } while (0)

using StateKey = std::pair<int32_t, int32_t>;  // (chunk, level)

struct StateEntry {
  std::vector<int32_t> slots;    // pages_per_chunk slot ids, frames ascending
  std::vector<uint8_t> written;  // per layer
};

inline size_t dtype_size(int32_t dtype) { return dtype == SC_DTYPE_F32 ? 4 : 2; }

}  // namespace sc

struct sc_selection {
  std::vector<sc_node> nodes;
  std::vector<int32_t> seg_off, seg_chunk, seg_level, seg_src;
  std::vector<sc_node> states;
  std::vector<uint8_t> vis;
};

struct sc_cache {
  sc_cache_desc d;
  char* pool;
  size_t slot_bytes;    // bytes of one slot in one layer (K and V)
  size_t kv_half;       // offset of V within a slot
  std::vector<uint8_t> used;
  std::vector<uint32_t> gen;
  std::vector<sc::StateKey> owner;  // slot -> state (valid when used)
  std::map<sc::StateKey, sc::StateEntry> states;
  // [layer * n_slots + slot]: the written flag of the slot's state at that
  // layer (a flat copy of StateEntry::written, so that checking a plan's
  // pages costs no map lookups); kept by set_written
  std::vector<uint8_t> slot_written;
};

struct sc_plan {
  std::vector<sc_node> nodes;
  std::vector<int32_t> page_off, page_slot, page_tokens, page_frame;
  std::vector<uint32_t> page_gen;
  std::vector<sc::StateKey> page_state;
  const sc_cache* cache;
  int32_t nq;  // query tokens per node
  // page slots in the bf16 attention's traversal order (built on first use)
  mutable std::vector<int32_t> attn_slot;
};

namespace sc {

// Validates a plan against the cache for reading `layer` (generations and
// written flags).  Returns SC_OK or an error code with the message set.
int plan_check(const sc_plan* plan, const sc_cache* cache, int32_t layer);

// Sets a state's written flag at `layer` and its slots' copies of it.
void set_written(sc_cache* cache, StateEntry& e, int32_t layer, uint8_t v);

// Policy helpers shared by the selection builder and the release rule:
// validation (SC_OK or SC_EINVAL with the message set), whether offset r is
// selected for node (c, j), and the level it reads (Eq. 4-5).
int policy_check(const sc_policy* p);
bool policy_selects(const sc_policy* p, int32_t c, int32_t j, int32_t r);
int32_t policy_level(const sc_policy* p, int32_t c, int32_t j, int32_t r);

// Compute units of the target GPU (MI355X): one launch round of
// one-work-group-per-CU kernels.
constexpr int32_t kCUs = 256;

// Kernel launchers (device code lives in the .hip files).
// Whether launch_attention supports the plan's shape (pack and plan sizes,
// head_dim and page size of the dtype's kernel): SC_OK or SC_EUNSUPPORTED.
int attention_check(const sc_plan* plan, const sc_cache* cache);
int launch_attention(const sc_plan* plan, const sc_cache* cache, int32_t layer,
                     const void* q, void* o, float scale, void* ws, size_t ws_bytes,
                     hipStream_t stream);
// Workspace of the bf16 attention for a plan (0 for fp32 caches and plans
// whose units fill whole rounds of the CUs), and its bound over all plans
// (at most kAttnMaxPieces partial results).
constexpr int32_t kAttnMaxPieces = 1024;
constexpr int32_t kAttnMinSplitTiles = 32;  // mean 64-key tiles per unit below which nothing is cut
size_t attention_workspace_bytes(const sc_plan* plan, const sc_cache* cache);
size_t attention_workspace_bound();
int launch_append(const sc_cache* cache, int32_t layer, const int32_t* slots, int32_t chunk,
                  const void* k, const void* v, const sc_rope* rope, hipStream_t stream);
int launch_rope_table(const sc_rope_desc* d, void* table, hipStream_t stream);

// Kernel timer: launchers bracket their kernel with timer_begin/timer_end.
enum TimerKind {
  TK_ATTENTION = 0, TK_GEMM_QKV, TK_GEMM_OUT, TK_GEMM_UP, TK_GEMM_DOWN, TK_RMSNORM, TK_APPEND,
  TK_SAMPLER, TK_ATTN_COMBINE, TK_QK_NORM, TK_CROSS_ATTENTION, TK_GEMM_CROSS_Q,
  TK_GEMM_CROSS_OUT, TK_GEMM_CONDITION, TK_ROW_SCALE, TK_COUNT
};
void timer_begin(int kind, hipStream_t stream);
void timer_end(int kind, hipStream_t stream);
// While alive, launches recorded under kind `from` are recorded under `to`
// (the cross-attention reuses the attention launcher).
struct TimerAlias {
  TimerAlias(int from, int to);
  ~TimerAlias();
  int from, prev;
};

// Offsets of the three axis tables inside a RoPE table, in float2 units.
struct RopeLayout {
  int32_t pairs_t, pairs_h, pairs_w;
  int64_t off_t, off_h, off_w, total;  // float2 entries
};
RopeLayout rope_layout(const sc_rope_desc* d);

}  // namespace sc
