/*
 * streamctx measurement support -- not part of the hot path.
 *
 * Calls a benchmark uses to time the library's own launches and to probe
 * the matrix cores' sustained rate on the same GPU; the product path never
 * needs them.  Conventions (return codes, streams, ownership) are those of
 * streamctx.h.
 */
#ifndef STREAMCTX_MEASURE_H
#define STREAMCTX_MEASURE_H

#include "streamctx.h"

#ifdef __cplusplus
extern "C" {
#endif

/* ---- Kernel timing (measurement support) ------------------------------
 * While enabled, every kernel the library launches is bracketed by two HIP
 * events recorded on the launch stream.  sc_timer_read synchronises those
 * events and returns, for one kernel kind, the number of launches and the
 * summed elapsed milliseconds since the timer was last enabled.  Kinds:
 * "attention", "gemm_qkv", "gemm_out", "gemm_up", "gemm_down", "rmsnorm",
 * "append", "sampler", "attention_combine" (the merge of split key ranges;
 * "attention" is the main kernel alone), "qk_norm" (the per-token scaling of
 * qk-norm and of the normalised condition queries and keys),
 * "cross_attention", "gemm_cross_q", "gemm_cross_out", "gemm_condition"
 * (the projections of sc_condition_append), "row_scale" (the 1 / rms per
 * token of an RMSNorm folded into the MLP's first GEMM).  Enabling clears earlier records.  Events are created
 * lazily and reused; the cost is two event records per launch. */
int sc_timer_enable(int on);
int sc_timer_read(const char* kind, int32_t* launches, double* total_ms);

/* ---- Matrix-core ceiling probe (measurement support) ------------------
 * Launches one kernel on `stream` that issues only 16x16x32 bf16 MFMAs from
 * registers (two 8-wave work-groups per CU, `iters` rounds of 16 MFMAs per
 * wave) and sets *flops to the work it performs; the caller times it with
 * its own events.  random_operands != 0 fills the operands with random bf16
 * values, else with constants; the two rates show how much the
 * power-limited clock depends on the data.  out: device scratch of at least
 * sc_probe_mfma_out_bytes() bytes (one float per thread, written so the
 * work is not optimised away).  Errors: SC_EINVAL, SC_EDEVICE. */
size_t sc_probe_mfma_out_bytes(void);
int sc_probe_mfma(int32_t random_operands, int32_t iters, void* out, size_t out_bytes,
                  double* flops, sc_stream stream);

/* ---- Streaming-read probe (measurement support) -----------------------
 * Launches one kernel on `stream` that reads the `bytes` bytes of device
 * buffer `buf` once with 16-byte loads (8192 work-groups of 256 lanes,
 * grid-stride, four loads in flight per lane) and stores nothing but, never
 * in practice, one word at `out` (device, 4 bytes).  The caller times it:
 * the plain-read bandwidth a kernel can reach on this GPU, for buffers
 * beyond the last-level cache (HBM) or within it.  buf 16-byte aligned,
 * bytes a positive multiple of 16.  Errors: SC_EINVAL, SC_EDEVICE. */
int sc_probe_read(const void* buf, size_t bytes, void* out, sc_stream stream);

#ifdef __cplusplus
}
#endif
#endif /* STREAMCTX_MEASURE_H */
