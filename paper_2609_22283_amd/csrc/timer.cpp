// Kernel timer: HIP events around every library kernel launch while enabled.
#include <cstring>

#include "internal.h"

namespace sc {

namespace {

const char* const kNames[TK_COUNT] = {"attention", "gemm_qkv", "gemm_out", "gemm_up",
                                      "gemm_down", "rmsnorm", "append", "sampler",
                                      "attention_combine", "qk_norm", "cross_attention",
                                      "gemm_cross_q", "gemm_cross_out", "gemm_condition",
                                      "row_scale"};

struct Record {
  int kind;
  hipEvent_t start, stop;
};

struct Timer {
  bool on = false;
  std::vector<Record> records;   // in launch order since enable
  std::vector<hipEvent_t> pool;  // reusable events
  int open_kind = -1;
  hipEvent_t open_start = nullptr;
};

Timer g_timer;
int g_alias[TK_COUNT] = {};  // 0: no alias, else kind + 1 to record under

hipEvent_t take_event() {
  if (!g_timer.pool.empty()) {
    hipEvent_t e = g_timer.pool.back();
    g_timer.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void recycle_all() {
  for (auto& r : g_timer.records) {
    g_timer.pool.push_back(r.start);
    g_timer.pool.push_back(r.stop);
  }
  g_timer.records.clear();
}

}  // namespace

TimerAlias::TimerAlias(int from_, int to) : from(from_), prev(g_alias[from_]) { g_alias[from] = to + 1; }
TimerAlias::~TimerAlias() { g_alias[from] = prev; }

static int aliased(int kind) { return g_alias[kind] ? g_alias[kind] - 1 : kind; }

void timer_begin(int kind, hipStream_t stream) {
  if (!g_timer.on) return;
  kind = aliased(kind);
  hipEvent_t e = take_event();
  if (!e) return;
  if (hipEventRecord(e, stream) != hipSuccess) {  // an unrecorded launch is not timed
    g_timer.pool.push_back(e);
    return;
  }
  g_timer.open_kind = kind;
  g_timer.open_start = e;
}

void timer_end(int kind, hipStream_t stream) {
  kind = aliased(kind);
  if (!g_timer.on || g_timer.open_kind != kind || !g_timer.open_start) return;
  hipEvent_t e = take_event();
  if (!e) return;
  if (hipEventRecord(e, stream) != hipSuccess) {
    g_timer.pool.push_back(e);
    return;
  }
  g_timer.records.push_back(Record{kind, g_timer.open_start, e});
  g_timer.open_kind = -1;
  g_timer.open_start = nullptr;
}

}  // namespace sc

using namespace sc;

extern "C" int sc_timer_enable(int on) {
  recycle_all();
  g_timer.on = on != 0;
  return SC_OK;
}

extern "C" int sc_timer_read(const char* kind, int32_t* launches, double* total_ms) {
  if (!kind || !launches || !total_ms) return fail(SC_EINVAL, "null argument");
  int k = -1;
  for (int i = 0; i < TK_COUNT; ++i)
    if (std::strcmp(kind, kNames[i]) == 0) k = i;
  if (k < 0) return fail(SC_EINVAL, "unknown kernel kind '%s'", kind);
  int32_t n = 0;
  double total = 0.0;
  for (auto& r : g_timer.records) {
    if (r.kind != k) continue;
    SC_HIP(hipEventSynchronize(r.stop));
    float ms = 0.f;
    SC_HIP(hipEventElapsedTime(&ms, r.start, r.stop));
    total += ms;
    ++n;
  }
  *launches = n;
  *total_ms = total;
  return SC_OK;
}
