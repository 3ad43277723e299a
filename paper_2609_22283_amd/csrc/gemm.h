// GEMM / RMSNorm launch interface used by the block orchestration.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace sc {

enum { EPI_STORE = 0, EPI_QKV = 1, EPI_GELU = 2, EPI_RESIDUAL = 3 };

constexpr int kGemmMaxNodes = 64;
constexpr int kGemmMaxNodePages = 256;

struct GemmEpilogue {
  // STORE / GELU / RESIDUAL: out[t * ld_out + f]
  uint16_t* out;
  int32_t ld_out;
  // QKV
  uint16_t* q_out;  // [T][hidden]
  char* layer_base;
  uint64_t slot_bytes, kv_half;
  int32_t hidden, head_dim, nq, tpp, ppc, grid_w;
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
int launch_rmsnorm(const uint16_t* x, uint16_t* y, int32_t rows, int32_t D, const NormMod& nm,
                   hipStream_t stream);

}  // namespace sc
