// Stand-ins for the library's device launchers, for a CPU build of the host
// core (selection, cache, plan, schedule and block orchestration) under
// AddressSanitizer and UndefinedBehaviorSanitizer.  No kernel runs: every
// launcher only counts its call, and fails with SC_EDEVICE on the call
// numbered g_fail_at (1-based), so the driver can force an error at any
// point of a block's launch sequence.
#include "../../paper_2609_22283_amd/csrc/gemm.h"
#include "../../paper_2609_22283_amd/csrc/internal.h"

int g_launches = 0;
int g_fail_at = -1;

namespace sc {

static int launched(const char* what) {
  ++g_launches;
  if (g_launches == g_fail_at) return fail(SC_EDEVICE, "%s: launch %d failed (forced)", what, g_launches);
  return SC_OK;
}

int launch_attention(const sc_plan*, const sc_cache*, int32_t, const void*, void*, float, void*, size_t,
                     hipStream_t) {
  return launched("attention");
}
int attention_check(const sc_plan*, const sc_cache*) { return SC_OK; }
size_t attention_workspace_bytes(const sc_plan*, const sc_cache*) { return 0; }
size_t attention_workspace_bound() { return 4096; }
int launch_append(const sc_cache*, int32_t, const int32_t*, int32_t, const void*, const void*, const sc_rope*,
                  hipStream_t) {
  return launched("append");
}
int launch_rope_table(const sc_rope_desc*, void*, hipStream_t) { return launched("rope table"); }
int launch_gemm(int, int, const uint16_t*, const uint16_t*, int32_t, int32_t, int32_t, const GemmEpilogue&,
                hipStream_t) {
  return launched("gemm");
}
int launch_norm_scale(int32_t, const NormScale&, hipStream_t) { return launched("norm scale"); }
int launch_rmsnorm(const uint16_t*, uint16_t*, int32_t, int32_t, const NormMod&, hipStream_t) {
  return launched("rmsnorm");
}
int launch_row_scale(const float*, int32_t, int32_t, int32_t, float, float*, hipStream_t) {
  return launched("row_scale");
}
int launch_row_rms(const uint16_t*, int32_t, int32_t, float*, hipStream_t) { return launched("row_rms"); }
TimerAlias::TimerAlias(int from_, int to) : from(from_), prev(to) {}
TimerAlias::~TimerAlias() {}

}  // namespace sc

extern "C" const char* hipGetErrorString(hipError_t) { return "HIP runtime absent in the host-core check build"; }
