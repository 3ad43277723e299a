// GEMM / RMSNorm launch interface used by the block orchestration.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

#include "divmagic.h"

namespace sc {

enum { EPI_STORE = 0, EPI_QKV = 1, EPI_GELU = 2, EPI_RESIDUAL = 3 };

constexpr int kGemmMaxNodes = 64;
constexpr int kGemmMaxNodePages = 256;
constexpr int kSsPartWidth = 64;  // features per sum-of-squares partial (qk-norm)

struct GemmEpilogue {
  // STORE / GELU / RESIDUAL: out[t * ld_out + f]
  uint16_t* out;
  int32_t ld_out;
  // QKV
  uint16_t* q_out;  // [T][hidden]
  char* layer_base;
  uint64_t slot_bytes, kv_half;
  int32_t hidden, head_dim, nq, tpp, ppc, grid_w;
  DivMagic nq_div, tpp_div, gw_div;  // set by the launcher from nq, tpp, grid_w
  const float2* rope_table;  // NULL: no rotation
  int32_t pairs_t, pairs_h, pairs_w;
  int64_t rope_off_h, rope_off_w;
  int32_t node_chunk[kGemmMaxNodes];
  int32_t node_slot[kGemmMaxNodePages];  // [node][frame] page slot of the node's own state
  // RESIDUAL with noise-level conditioning: out += gate[level of t's node] * D,
  // gate rows of a [levels][6][F] fp32 table (gate_row = 2 or 5); NULL: out += D
  const float* mod;
  int32_t gate_row;
  int32_t node_level[kGemmMaxNodes];
  // QKV, GELU and STORE with row_scale: an RMSNorm of the input rows folded
  // into the GEMM.  X holds the raw rows; each token's accumulators are
  // multiplied by row_scale[t] (1 / rms of its row: launch_row_scale or
  // launch_row_rms) before anything else of the epilogue.  NULL: none.
  const float* row_scale;
  // Sums of squares for a later RMSNorm over features (qk-norm), STORE and
  // QKV (q and k sections): ss_part[t * n_part + f / kSsPartWidth] = sum of
  // D[f'][t]^2 over the kSsPartWidth features f' of f's group, before any
  // gain or RoPE.  RESIDUAL: the same over the updated rows as stored (bf16)
  // but part-major, ss_part[(f / kSsPartWidth) * T + t], for an RMSNorm of
  // the result folded into the next GEMM (n_part unused).
  // NULL: none.  QKV with ss_part also multiplies q and k by qk_gain
  // ([2][hidden], the gains of q then k) before RoPE.
  float* ss_part;
  int32_t n_part;
  const float* qk_gain;
};

// Second half of an RMSNorm whose sums of squares came from a GEMM epilogue:
// for each token t, inv = 1 / sqrt(sum_p part[t * n_part + p0 + p] / D + eps)
// over the D / kSsPartWidth partials of one tensor, then
//   rows[t][:] *= inv (* gain[:] when gain != NULL)   (token-major, q)
//   the token's k rows in its node's page slot *= inv  (k of the QKV pass)
struct NormScale {
  const float* part;
  int32_t n_part, D;
  float eps;
  uint16_t* rows;          // token-major [T][ld] rows (part offset 0), or NULL
  int32_t ld;
  const float* gain;       // [D] fp32 for rows, or NULL
  char* layer_base;        // page-slot keys (part offset D / kSsPartWidth), or NULL
  uint64_t slot_bytes;
  int32_t nq, tpp, ppc, head_dim;
  int32_t node_slot[kGemmMaxNodePages];
};

// Per-level shift/scale after RMSNorm (noise-level conditioning): row r of
// x belongs to node r / nq; y = RMSNorm(x) * (1 + scale) + shift with shift,
// scale rows (3 * which, 3 * which + 1) of the [levels][6][D] table.
struct NormMod {
  const float* mod;  // NULL: plain RMSNorm
  int32_t nq, which;
  int32_t node_level[kGemmMaxNodes];
};

int launch_gemm(int epi, int timer_kind, const uint16_t* W, const uint16_t* X, int32_t F, int32_t T,
                int32_t Kd, const GemmEpilogue& ep, hipStream_t stream);
int launch_norm_scale(int32_t T, const NormScale& ns, hipStream_t stream);
int launch_rmsnorm(const uint16_t* x, uint16_t* y, int32_t rows, int32_t D, const NormMod& nm,
                   hipStream_t stream);
// The factor alone of an RMSNorm without modulation or gain, from the rows
// themselves: scale[r] = 1 / sqrt(mean_f x[r][f]^2 + 1e-6) (a read of x,
// no write of the normalised rows).  Feeds GemmEpilogue::row_scale.
int launch_row_rms(const uint16_t* x, int32_t rows, int32_t D, float* scale, hipStream_t stream);
// The second half of an RMSNorm without modulation or gain whose sums of
// squares a RESIDUAL epilogue stored part-major: for t < T,
//   scale[t] = 1 / sqrt(sum_{p < n_part} part[p * T + t] / D + eps),
// summed in increasing p (deterministic).  Feeds GemmEpilogue::row_scale.
int launch_row_scale(const float* part, int32_t n_part, int32_t T, int32_t D, float eps, float* scale,
                     hipStream_t stream);

}  // namespace sc
