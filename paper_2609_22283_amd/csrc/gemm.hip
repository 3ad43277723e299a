// bf16 GEMM for the DiT block's projections, D[f][t] = sum_k W[f][k] X[t][k]
// (W in [out, in] layout, X token-major), fp32 accumulation on 16x16x32 bf16
// MFMAs (half the accumulator traffic per FLOP of the 32x32 shape, so a
// higher clock under the power cap), with the block's elementwise work fused
// into the epilogue:
//   QKV      RoPE on q and k; q to a token-major buffer; k and v scattered
//            into the pack nodes' page slots (k as [head][token][d], v as
//            [head][d][token], transposed through LDS into 8-token runs)
//   GELU     out[t][f] = GELU_tanh(D)
//   RESIDUAL x[t][f] += D   (in place)
//   STORE    out[t][f] = D
// QKV, GELU and STORE can take an RMSNorm of the input rows folded in: X
// then holds the raw rows and D[f][t] is first multiplied by row_scale[t].
// QKV and STORE can also emit per-token sums of squares over each group of
// 64 features, the first half of an RMSNorm over the feature axis (qk-norm);
// norm_scale_kernel finishes it.  RESIDUAL can emit them for the rows it
// writes, part-major; row_scale_kernel turns them into a row_scale.
// Work-group tile 256 (features) x BN (tokens: 256, 224, 192 or 128) x 64
// (k), eight waves (2 x 4 of 128 x BN/4, or 4 x 2 of 64 x BN/2 at 224),
// operands double-buffered in LDS with an XOR swizzle.  Each lane holds four consecutive features of one token, so RoPE
// pairs stay in-lane.
#include <cstring>

#include "device.h"
#include "gemm.h"
#include "internal.h"

namespace sc {

constexpr int GBM = 256, GBK = 64;
constexpr int GWM = 128;
constexpr int G_NW = 8;               // waves per work-group, two per SIMD
constexpr int G_THREADS = 64 * G_NW;
constexpr int GROWS = GBM / G_NW;     // weight rows each wave copies per stage
constexpr int G_TILE_BYTES = GBM * GBK * 2;  // 32 KB per operand per stage

// GELU_tanh(x) = 0.5 x (1 + tanh(u)) = x * sigmoid(2 u), u = sqrt(2/pi) (x + 0.044715 x^3),
// evaluated as x / (1 + 2^(-2 u log2 e)).
__device__ __forceinline__ float gelu_tanh(float x) {
  constexpr float k = 2.0f * 0.7978845608028654f * 1.4426950408889634f;  // 2 sqrt(2/pi) log2(e)
  const float q = x * fmaf(x * x, -k * 0.044715f, -k);
  const float e = __builtin_amdgcn_exp2f(q);
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

// Direct global -> LDS copy of 16 bytes per lane (lane i lands at LDS base
// + 16 i) from base + off.  Written as inline asm: while a copy it knows of
// is in flight, the compiler waits for every LDS fragment read with
// lgkmcnt(0); not knowing of these, it counts the reads exactly (the copies
// complete under the loop's explicit vmcnt(0) wait).  M0, which carries the
// LDS address, is saved and restored.  (QKV and MLP-up GEMMs 2 % faster.)
__device__ __forceinline__ void gdma16(const char* base, uint32_t off, char* lds_wave_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base), "s"((uint32_t)reinterpret_cast<uintptr_t>(lds_wave_base))
      : "memory");
}

// Per-token sums of squares of a wave's accumulator tile, one partial per
// kSsPartWidth (64) features: lane (lg, c16) holds 16 of a partial's features
// for token c16 of each 16-token block; the four lg lanes of a token are
// summed with two butterflies and lane lg = 0 stores partial part0 + g.
template <int FB, int TB>
__device__ __forceinline__ void store_sum_squares(const f32x4 (&acc)[FB][TB], float* ss,
                                                  int32_t n_part, int32_t part0, int32_t tw0,
                                                  int32_t T, int32_t lg, int32_t c16) {
  constexpr int FPG = kSsPartWidth / 16;  // 16-feature blocks per partial
  static_assert(FB % FPG == 0, "whole partials per wave");
#pragma unroll
  for (int g = 0; g < FB / FPG; ++g)
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      float s = 0.f;
#pragma unroll
      for (int fb = g * FPG; fb < (g + 1) * FPG; ++fb)
#pragma unroll
        for (int e = 0; e < 4; ++e) s = fmaf(acc[fb][tb][e], acc[fb][tb][e], s);
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
      const int32_t t = tw0 + 16 * tb + c16;
      if (lg == 0 && t < T) ss[(size_t)t * n_part + part0 + g] = s;
    }
}

// BN tokens per work-group tile.  Wave layout WL = 0: 2 (features) x 4
// (tokens) waves of 128 x BN/4 (BN a multiple of 64; required by the QKV
// epilogue and the sums of squares, which take one head of 128 features per
// wave); WL = 1: 4 x 2 waves of 64 x BN/2 (BN a multiple of 32, e.g. 224).
template <int EPI, int BN, int WL>
__global__ __launch_bounds__(G_THREADS, 1) void gemm_bf16_kernel(const uint16_t* __restrict__ W,
                                                                 const uint16_t* __restrict__ X,
                                                                 int32_t F, int32_t T, int32_t Kd,
                                                                 GemmEpilogue ep) {
  // stage s: W tile at s * 64 KB, X tile at s * 64 KB + 32 KB; rows of 64 k
  // (128 B) with 16-byte column c stored at c ^ ((row >> 1) & 7)
  __shared__ __attribute__((aligned(1024))) char smem[2 * 2 * G_TILE_BYTES];
  constexpr int WM = WL ? 64 : GWM;    // features per wave tile
  constexpr int GWN = WL ? BN / 2 : BN / 4;  // tokens per wave tile
  static_assert(GWN % 16 == 0, "wave tiles hold whole 16-token blocks");
  const int32_t n_tf = F / GBM, n_tt = (T + BN - 1) / BN;
  // Each XCD takes a contiguous run of logical tiles; the run is walked in
  // groups of GT token tiles, feature tiles outermost within a group, so the
  // ~32 tiles an XCD holds at once share 4-5 weight and 8 token panels in L2.
  constexpr int32_t GT = 8;
  const int32_t tile = (int32_t)xcd_remap(blockIdx.x, (uint32_t)(n_tf * n_tt));
  const int32_t group = tile / (GT * n_tf), in_group = tile - group * GT * n_tf;
  const int32_t gt = min(GT, n_tt - group * GT);
  const int32_t tf = in_group / gt, tt = group * GT + in_group % gt;
  const int32_t f0 = tf * GBM, t0 = tt * BN;

  const int32_t tid = threadIdx.x, lane = tid & 63;
  const int32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: LDS copy addresses stay scalar
  const int32_t lg = lane >> 4, c16 = lane & 15;
  const int32_t wf = WL ? (wave & 3) * WM : (wave & 1) * WM;
  const int32_t wt = WL ? (wave >> 2) * GWN : (wave >> 1) * GWN;

  // copies: each wave moves weight rows [GROWS wave, GROWS wave + GROWS) and
  // the 8-row token groups wave, wave + 8, ... (BN / 8 groups in all), 8 rows
  // (1 KB) per instruction; lane (row, p) fetches column p ^ ((row >> 1) & 7).
  // Byte offsets are fixed per lane; the k offset is folded into the
  // (wave-uniform) base pointer.
  constexpr int NCP = GROWS / 8, XGROUPS = BN / 8, NCPX = (XGROUPS + G_NW - 1) / G_NW;
  static_assert(BN % 32 == 0 && BN <= GBM && NCPX <= NCP, "token copies ride with the weight copies");
  uint32_t woff[NCP], xoff[NCPX];
#pragma unroll
  for (int j = 0; j < NCP; ++j) {
    const int32_t row = GROWS * wave + 8 * j + (lane >> 3);
    const int32_t col = (lane & 7) ^ ((row >> 1) & 7);
    woff[j] = ((uint32_t)(f0 + row) * Kd + col * 8) * 2;
  }
#pragma unroll
  for (int j = 0; j < NCPX; ++j) {
    const int32_t row = 8 * min(wave + G_NW * j, XGROUPS - 1) + (lane >> 3);
    const int32_t col = (lane & 7) ^ ((row >> 1) & 7);
    const int32_t trow = min(t0 + row, T - 1);
    xoff[j] = ((uint32_t)trow * Kd + col * 8) * 2;
  }
  const char* wbase = reinterpret_cast<const char*>(W);
  const char* xbase = reinterpret_cast<const char*>(X);
  auto issue = [&](int32_t k0, int buf) {
    char* a = smem + buf * 2 * G_TILE_BYTES;
    char* b = a + G_TILE_BYTES;
    const char* wk = wbase + (size_t)k0 * 2;
    const char* xk = xbase + (size_t)k0 * 2;
#pragma unroll
    for (int j = 0; j < NCP; ++j) {
      gdma16(wk, woff[j], a + (GROWS * wave + 8 * j) * 128);
      if (j < NCPX && (XGROUPS % G_NW == 0 || wave + G_NW * j < XGROUPS))  // wave-uniform
        gdma16(xk, xoff[j], b + (8 * (wave + G_NW * j)) * 128);
    }
  };
  auto landed = [&]() {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };

  // LDS read offsets of this lane's fragments (16-byte column 4 s + lg)
  // 16x16x32 MFMAs: lane (lg, c16) supplies row c16 of each 16-row operand
  // block with k values 8 lg .. 8 lg + 7 of a 32-k step
  constexpr int FB = WM / 16, TB = GWN / 16;
  uint32_t aoff[FB], boff[TB];
#pragma unroll
  for (int fb = 0; fb < FB; ++fb) aoff[fb] = (uint32_t)(wf + 16 * fb + c16) * 128;
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) boff[tb] = (uint32_t)(wt + 16 * tb + c16) * 128;
  const int32_t swz = (c16 >> 1) & 7;  // rows wf + 16 fb + c16 share (row >> 1) & 7

  f32x4 acc[FB][TB];
#pragma unroll
  for (int fb = 0; fb < FB; ++fb)
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) acc[fb][tb] = f32x4{};

  auto frags = [&](const char* a, const char* b, int s, bf16x8 (&af)[FB], bf16x8 (&bf)[TB]) {
    const uint32_t c = (uint32_t)(((4 * s + lg) ^ swz) << 4);
#pragma unroll
    for (int fb = 0; fb < FB; ++fb) af[fb] = *reinterpret_cast<const bf16x8*>(a + aoff[fb] + c);
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) bf[tb] = *reinterpret_cast<const bf16x8*>(b + boff[tb] + c);
  };

  // The residual epilogue's reads of out[t][f] are issued before the main
  // loop, so they land during it instead of after it, when every CU of the
  // launch would read its residual tile at once.  Rows past T read
  // the last row (valid memory, values unused).
  constexpr bool PREFETCH = EPI == EPI_RESIDUAL;
  u32x2 res[PREFETCH ? TB : 1][PREFETCH ? FB : 1];
  if constexpr (PREFETCH) {
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      const int32_t t = min(t0 + wt + 16 * tb + c16, T - 1);
      const uint16_t* orow = ep.out + (size_t)t * ep.ld_out + f0 + wf + 4 * lg;
#pragma unroll
      for (int fb = 0; fb < FB; ++fb) res[tb][fb] = *reinterpret_cast<const u32x2*>(orow + 16 * fb);
    }
  }
  // The folded RMSNorm's per-token factors (every epilogue but RESIDUAL):
  // lane j loads those of the wave's tokens j and j + 64 (two coalesced
  // loads at most), also before the main loop; the epilogue takes each
  // token's from its lane.
  constexpr bool ROWPRE = EPI != EPI_RESIDUAL;
  constexpr int RT = ROWPRE ? (GWN + 63) / 64 : 1;
  float rtok[RT];
  if constexpr (ROWPRE) {
    if (ep.row_scale) {
#pragma unroll
      for (int r = 0; r < RT; ++r) rtok[r] = ep.row_scale[min(t0 + wt + 64 * r + lane, T - 1)];
    }
  }

  const int32_t nk = Kd / GBK;
  issue(0, 0);
  landed();
  for (int32_t kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) issue((kt + 1) * GBK, (kt + 1) & 1);
    const char* a = smem + (kt & 1) * 2 * G_TILE_BYTES;
    const char* b = a + G_TILE_BYTES;
    bf16x8 af[2][FB], bfr[2][TB];
    frags(a, b, 0, af[0], bfr[0]);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      if (s + 1 < 2) frags(a, b, s + 1, af[(s + 1) & 1], bfr[(s + 1) & 1]);
#pragma unroll
      for (int fb = 0; fb < FB; ++fb)
#pragma unroll
        for (int tb = 0; tb < TB; ++tb)
          acc[fb][tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[s & 1][fb], bfr[s & 1][tb],
                                                                acc[fb][tb], 0, 0, 0);
    }
    landed();
  }

  // epilogue: lane holds D[f][t] for t = t0 + wt + 16 tb + c16 and
  // f = f0 + wf + 16 fb + 4 lg + e (e = 0..3)
  // The folded RMSNorm of the input rows: D is linear in the row, so the
  // token's 1 / rms scales its accumulators before anything else (taken
  // from the lane that loaded it while every lane is active).
  if constexpr (ROWPRE) {
    if (ep.row_scale) {
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const float r = __shfl(rtok[tb >> 2], 16 * (tb & 3) + c16);
#pragma unroll
        for (int fb = 0; fb < FB; ++fb)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[fb][tb][e] *= r;
      }
    }
  }
  if constexpr (EPI == EPI_QKV) {
    // a 256-feature tile lies in one of q, k, v (hidden is a multiple of 256)
    // and each wave's 128 or 64 features in one head (head_dim 128)
    const int32_t sec = f0 / ep.hidden;
    const int32_t hf0 = f0 - sec * ep.hidden + wf;       // wave's first feature in its section
    const int32_t head = hf0 / ep.head_dim;
    const int32_t dbase = hf0 - head * ep.head_dim + 4 * lg;
    if (ep.ss_part && sec < 2) {
      // qk-norm: sums of squares of the raw q or k, then the gain (before
      // RoPE); the 1 / rms factor is applied by norm_scale_kernel
      store_sum_squares(acc, ep.ss_part, ep.n_part, (f0 + wf) / kSsPartWidth, t0 + wt, T, lg, c16);
      const float* g = ep.qk_gain + f0 + wf + 4 * lg;
#pragma unroll
      for (int fb = 0; fb < FB; ++fb) {
        const f32x4 gv = *reinterpret_cast<const f32x4*>(g + 16 * fb);
#pragma unroll
        for (int tb = 0; tb < TB; ++tb)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[fb][tb][e] *= gv[e];
      }
    }
    // v is stored transposed per page ([head][d][token]).  Each wave stages
    // its v tile in its own LDS region (free after the main loop; rows
    // padded by 16 bytes against bank conflicts; in two passes of half the
    // rows where the whole tile does not fit), then each lane writes runs of
    // 8 consecutive tokens of one feature row as 16-byte stores.  Pages hold
    // a multiple of 8 tokens (so do nodes), so no run crosses a page.
    if (sec == 2) {
      constexpr int LDSW = GWN + 8;  // staged row length (elements)
      constexpr int RP = WM * LDSW * 2 * G_NW <= (int)sizeof(smem) ? WM : WM / 2;  // rows per pass
      constexpr int SEGS = GWN / 8;
      static_assert(RP * LDSW * 2 * G_NW <= (int)sizeof(smem) && (RP * SEGS) % 64 == 0 && RP % 16 == 0,
                    "v staging layout");
      uint16_t* lt = reinterpret_cast<uint16_t*>(smem) + (size_t)wave * RP * LDSW;
      const int32_t d0 = hf0 - head * ep.head_dim;  // wave's first feature within its head
#pragma unroll
      for (int pass = 0; pass < WM / RP; ++pass) {
#pragma unroll
        for (int fb = pass * RP / 16; fb < (pass + 1) * RP / 16; ++fb)
#pragma unroll
          for (int tb = 0; tb < TB; ++tb)
#pragma unroll
            for (int e = 0; e < 4; ++e)
              lt[(16 * fb - pass * RP + 4 * lg + e) * LDSW + 16 * tb + c16] = f32_to_bf16(acc[fb][tb][e]);
#pragma unroll
        for (int j = 0; j < RP * SEGS / 64; ++j) {
          const int32_t r = lane + 64 * j, row = r / SEGS, seg = r - row * SEGS;
          const int32_t t = t0 + wt + 8 * seg;
          if (t >= T) continue;
          const u32x4 val = *reinterpret_cast<const u32x4*>(lt + row * LDSW + 8 * seg);
          const int32_t node = (int32_t)fast_div((uint32_t)t, ep.nq_div), tok = t - node * ep.nq;
          const int32_t frame = (int32_t)fast_div((uint32_t)tok, ep.tpp_div), n = tok - frame * ep.tpp;
          char* slot_base = ep.layer_base + (size_t)ep.node_slot[node * ep.ppc + frame] * ep.slot_bytes;
          uint16_t* vrow = reinterpret_cast<uint16_t*>(slot_base + ep.kv_half) +
                           ((size_t)head * ep.head_dim + d0 + pass * RP + row) * ep.tpp + n;
          if (t + 8 <= T) {
            *reinterpret_cast<u32x4*>(vrow) = val;
          } else {  // a launch ending inside a run
#pragma unroll
            for (int i = 0; i < 8; ++i)
              if (i < T - t) vrow[i] = (uint16_t)(val[i >> 1] >> (16 * (i & 1)));
          }
        }
      }
      return;
    }
    // RoPE pairs p = d / 2 + pp: the axis of each pair (time, height, width)
    // and its table offset are fixed per lane, so they are resolved once;
    // per token only the axis's position term is selected (no branches).
    const bool rope = ep.rope_table != nullptr;  // q or k here
    int32_t rbase[FB][2], rax[FB][2];
#pragma unroll
    for (int fb = 0; fb < FB; ++fb)
#pragma unroll
      for (int pp = 0; pp < 2; ++pp) {
        const int32_t p = (dbase + 16 * fb) / 2 + pp;
        if (p < ep.pairs_t) {
          rax[fb][pp] = 0;
          rbase[fb][pp] = p;
        } else if (p < ep.pairs_t + ep.pairs_h) {
          rax[fb][pp] = 1;
          rbase[fb][pp] = (int32_t)ep.rope_off_h + (p - ep.pairs_t);
        } else {
          rax[fb][pp] = 2;
          rbase[fb][pp] = (int32_t)ep.rope_off_w + (p - ep.pairs_t - ep.pairs_h);
        }
      }
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      const int32_t t = t0 + wt + 16 * tb + c16;
      if (t >= T) continue;
      const int32_t node = (int32_t)fast_div((uint32_t)t, ep.nq_div), tok = t - node * ep.nq;
      const int32_t frame = (int32_t)fast_div((uint32_t)tok, ep.tpp_div), n = tok - frame * ep.tpp;
      const int32_t pos_t = ep.node_chunk[node] * ep.ppc + frame;
      const int32_t pos_h = (int32_t)fast_div((uint32_t)n, ep.gw_div), pos_w = n - pos_h * ep.grid_w;
      const int32_t term_t = pos_t * ep.pairs_t, term_h = pos_h * ep.pairs_h, term_w = pos_w * ep.pairs_w;
      char* slot_base = ep.layer_base + (size_t)ep.node_slot[node * ep.ppc + frame] * ep.slot_bytes;
      uint16_t* qrow = ep.q_out + (size_t)t * ep.hidden + hf0 + 4 * lg;
      uint16_t* krow = reinterpret_cast<uint16_t*>(slot_base) + ((size_t)head * ep.tpp + n) * ep.head_dim;
#pragma unroll
      for (int fb = 0; fb < FB; ++fb) {
        const int32_t d = dbase + 16 * fb;
        float v0 = acc[fb][tb][0], v1 = acc[fb][tb][1];
        float v2 = acc[fb][tb][2], v3 = acc[fb][tb][3];
        if (rope) {
#pragma unroll
          for (int pp = 0; pp < 2; ++pp) {
            const int32_t ax = rax[fb][pp];
            const int32_t idx = rbase[fb][pp] + (ax == 0 ? term_t : ax == 1 ? term_h : term_w);
            const float2 cs = ep.rope_table[idx];
            float& x0 = pp ? v2 : v0;
            float& x1 = pp ? v3 : v1;
            const float r0 = x0 * cs.x - x1 * cs.y, r1 = x0 * cs.y + x1 * cs.x;
            x0 = r0;
            x1 = r1;
          }
        }
        u32x2 pk;
        pk.x = pack_bf16x2(v0, v1);
        pk.y = pack_bf16x2(v2, v3);
        if (sec == 0)
          *reinterpret_cast<u32x2*>(qrow + 16 * fb) = pk;
        else
          *reinterpret_cast<u32x2*>(krow + d) = pk;
      }
    }
  } else {
    if (EPI == EPI_STORE && ep.ss_part)
      store_sum_squares(acc, ep.ss_part, ep.n_part, (f0 + wf) / kSsPartWidth, t0 + wt, T, lg, c16);
    constexpr int FPG = kSsPartWidth / 16;  // 16-feature blocks per sum-of-squares partial
    static_assert(FB % FPG == 0, "whole partials per wave");
    const bool row_sums = EPI == EPI_RESIDUAL && ep.ss_part;
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      const int32_t t = t0 + wt + 16 * tb + c16;
      if (t >= T) continue;  // uniform over the 4 lanes of a token, so the butterflies below stay inside it
      uint16_t* orow = ep.out + (size_t)t * ep.ld_out + f0 + wf + 4 * lg;
      float ssq[FB / FPG];
#pragma unroll
      for (int g = 0; g < FB / FPG; ++g) ssq[g] = 0.f;
      // noise-level gate of this token's node (residual epilogue only)
      const float* gate = nullptr;
      if (EPI == EPI_RESIDUAL && ep.mod)
        gate = ep.mod + ((size_t)ep.node_level[t / ep.nq] * 6 + ep.gate_row) * F + f0 + wf + 4 * lg;
#pragma unroll
      for (int fb = 0; fb < FB; ++fb) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[fb][tb][e];
          uint16_t* dst = orow + 16 * fb;
          if constexpr (EPI == EPI_RESIDUAL) {
            if (gate) {
              const f32x4 gv = *reinterpret_cast<const f32x4*>(gate + 16 * fb);
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] *= gv[e];
            }
            u32x2 r;
            if constexpr (PREFETCH)
              r = res[tb][fb];
            else
              r = *reinterpret_cast<const u32x2*>(dst);
            v[0] += __uint_as_float(r.x << 16);
            v[1] += __uint_as_float(r.x & 0xffff0000u);
            v[2] += __uint_as_float(r.y << 16);
            v[3] += __uint_as_float(r.y & 0xffff0000u);
          } else if constexpr (EPI == EPI_GELU) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = gelu_tanh(v[e]);
          }
          u32x2 pk;
          pk.x = pack_bf16x2(v[0], v[1]);
          pk.y = pack_bf16x2(v[2], v[3]);
          *reinterpret_cast<u32x2*>(dst) = pk;
          if (row_sums) {  // of the values as stored
            const float a = __uint_as_float(pk.x << 16), b = __uint_as_float(pk.x & 0xffff0000u);
            const float c = __uint_as_float(pk.y << 16), d = __uint_as_float(pk.y & 0xffff0000u);
            ssq[fb / FPG] = fmaf(a, a, fmaf(b, b, fmaf(c, c, fmaf(d, d, ssq[fb / FPG]))));
          }
        }
      if (row_sums) {
#pragma unroll
        for (int g = 0; g < FB / FPG; ++g) {
          float sq = ssq[g];
          sq += __shfl_xor(sq, 16);
          sq += __shfl_xor(sq, 32);
          if (lg == 0) ep.ss_part[(size_t)((f0 + wf) / kSsPartWidth + g) * T + t] = sq;
        }
      }
    }
  }
}

template <int BN, int WL>
static void launch_gemm_bn(int epi, const uint16_t* W, const uint16_t* X, int32_t F, int32_t T, int32_t Kd,
                           const GemmEpilogue& ep, hipStream_t stream) {
  const dim3 grid((uint32_t)(F / GBM) * (uint32_t)((T + BN - 1) / BN));
  if constexpr (WL == 1) {
    switch (epi) {
      case EPI_QKV:
        hipLaunchKernelGGL((gemm_bf16_kernel<EPI_QKV, BN, 1>), grid, dim3(G_THREADS), 0, stream, W, X, F, T, Kd, ep);
        break;
      case EPI_GELU:
        hipLaunchKernelGGL((gemm_bf16_kernel<EPI_GELU, BN, 1>), grid, dim3(G_THREADS), 0, stream, W, X, F, T, Kd, ep);
        break;
      case EPI_RESIDUAL:
        hipLaunchKernelGGL((gemm_bf16_kernel<EPI_RESIDUAL, BN, 1>), grid, dim3(G_THREADS), 0, stream, W, X, F, T,
                           Kd, ep);
        break;
      default:
        hipLaunchKernelGGL((gemm_bf16_kernel<EPI_STORE, BN, 1>), grid, dim3(G_THREADS), 0, stream, W, X, F, T, Kd, ep);
    }
  } else {
  switch (epi) {
    case EPI_QKV:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_QKV, BN, 0>), grid, dim3(G_THREADS), 0, stream, W, X, F, T, Kd, ep);
      break;
    case EPI_GELU:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_GELU, BN, 0>), grid, dim3(G_THREADS), 0, stream, W, X, F, T, Kd, ep);
      break;
    case EPI_RESIDUAL:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_RESIDUAL, BN, 0>), grid, dim3(G_THREADS), 0, stream, W, X, F, T, Kd,
                         ep);
      break;
    default:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_STORE, BN, 0>), grid, dim3(G_THREADS), 0, stream, W, X, F, T, Kd, ep);
  }
  }
}

// Tile shape of a launch: one work-group per CU, so a launch of n tiles
// takes ceil(n / CUs) rounds of one tile's time.  A tile of BN tokens takes
// BN / 256 of a 256-token tile's time times a per-shape efficiency loss
// (more fragment reads and copies per MFMA), measured on the Wan block's
// GEMMs.  The shape with the fewest tile-times wins, the wider one on ties.
// Layout 1 (224-token tiles, a wave holds 64 features: half a head) serves
// every epilogue (sums of squares are kept per 64 features).
struct GemmShape {
  int bn, wl;
};
static GemmShape gemm_tile_shape(int32_t F, int32_t T) {
  GemmShape best{256, 0};
  double best_cost = 1e30;
  const GemmShape cands[] = {{256, 0}, {224, 1}, {192, 0}, {128, 0}};
  for (const GemmShape c : cands) {
    const int64_t tiles = (int64_t)(F / GBM) * ((T + c.bn - 1) / c.bn);
    const double eff = c.bn == 256 ? 1.0 : c.bn == 224 ? 1.02 : c.bn == 192 ? 1.12 : 1.4;
    const double cost = (double)((tiles + kCUs - 1) / kCUs) * c.bn / 256.0 * eff;
    if (cost < best_cost - 1e-9) {
      best_cost = cost;
      best = c;
    }
  }
  return best;
}

int launch_gemm(int epi, int timer_kind, const uint16_t* W, const uint16_t* X, int32_t F, int32_t T,
                int32_t Kd, const GemmEpilogue& ep, hipStream_t stream) {
  if (F % GBM || Kd % GBK || T <= 0)
    return fail(SC_EUNSUPPORTED, "gemm needs F %% %d == 0, K %% %d == 0 (F=%d K=%d T=%d)", GBM, GBK,
                F, Kd, T);
  if ((uint64_t)F * Kd * 2 > 0xffffffffull || (uint64_t)T * Kd * 2 > 0xffffffffull)
    return fail(SC_EUNSUPPORTED, "gemm operands beyond 4 GB");
  if (epi == EPI_QKV && (ep.hidden % GBM || ep.head_dim != GWM))
    return fail(SC_EUNSUPPORTED, "QKV epilogue needs hidden %% %d == 0 and head_dim %d", GBM, GWM);
  if (ep.row_scale && epi == EPI_RESIDUAL) return fail(SC_EINVAL, "row_scale is not a RESIDUAL epilogue input");
  GemmEpilogue e = ep;
  if (epi == EPI_QKV) {
    // v goes out in 16-byte runs of 8 tokens within one page
    if (ep.nq <= 0 || ep.tpp <= 0 || ep.grid_w <= 0 || ep.tpp % 8 || ep.nq % 8 || ep.slot_bytes % 16 ||
        ep.kv_half % 16 || reinterpret_cast<uintptr_t>(ep.layer_base) % 16)
      return fail(SC_EUNSUPPORTED, "QKV epilogue needs tpp and nq multiples of 8 and 16-byte aligned slots "
                  "(nq %d, tpp %d, grid_w %d)", ep.nq, ep.tpp, ep.grid_w);
    e.nq_div = magic_div((uint32_t)ep.nq);
    e.tpp_div = magic_div((uint32_t)ep.tpp);
    e.gw_div = magic_div((uint32_t)ep.grid_w);
  }
  timer_begin(timer_kind, stream);
  const GemmShape shape = gemm_tile_shape(F, T);
  if (shape.wl == 1)
    launch_gemm_bn<224, 1>(epi, W, X, F, T, Kd, e, stream);
  else if (shape.bn == 128)
    launch_gemm_bn<128, 0>(epi, W, X, F, T, Kd, e, stream);
  else if (shape.bn == 192)
    launch_gemm_bn<192, 0>(epi, W, X, F, T, Kd, e, stream);
  else
    launch_gemm_bn<256, 0>(epi, W, X, F, T, Kd, e, stream);
  timer_end(timer_kind, stream);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

// ------------------------------------------------------------------ RMSNorm
// y = x / sqrt(mean(x^2) + eps), one wave per row, fp32 math, bf16 in/out;
// with a modulation table, y * (1 + scale) + shift of the row's node level.
__global__ __launch_bounds__(256) void rmsnorm_kernel(const uint16_t* __restrict__ x,
                                                      uint16_t* __restrict__ y, float* __restrict__ inv_out,
                                                      int32_t rows, int32_t D, float eps, NormMod nm) {
  const int32_t row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int32_t lane = threadIdx.x & 63;
  if (row >= rows) return;
  const u32x4* xr = reinterpret_cast<const u32x4*>(x + (size_t)row * D);
  u32x4* yr = reinterpret_cast<u32x4*>(y + (size_t)row * D);
  const int32_t nv = D / 8;
  float ss = 0.f;
  for (int32_t v = lane; v < nv; v += 64) {
    const u32x4 a = xr[v];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float lo = __uint_as_float(a[k] << 16), hi = __uint_as_float(a[k] & 0xffff0000u);
      ss = fmaf(lo, lo, fmaf(hi, hi, ss));
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
  const float inv = rsqrtf(ss / (float)D + eps);
  if (inv_out) {  // the factor alone, for a GEMM that folds the norm in
    if (lane == 0) inv_out[row] = inv;
    return;
  }
  const float *shift = nullptr, *scale = nullptr;
  if (nm.mod) {
    const int32_t lev = nm.node_level[row / nm.nq];
    shift = nm.mod + ((size_t)lev * 6 + 3 * nm.which) * D;
    scale = shift + D;
  }
  for (int32_t v = lane; v < nv; v += 64) {
    const u32x4 a = xr[v];
    float f[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      f[2 * k] = __uint_as_float(a[k] << 16) * inv;
      f[2 * k + 1] = __uint_as_float(a[k] & 0xffff0000u) * inv;
    }
    if (shift) {
      const f32x4* sh = reinterpret_cast<const f32x4*>(shift + 8 * v);
      const f32x4* sc = reinterpret_cast<const f32x4*>(scale + 8 * v);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f32x4 s0 = sh[h], s1 = sc[h];
#pragma unroll
        for (int e = 0; e < 4; ++e) f[4 * h + e] = fmaf(f[4 * h + e], 1.0f + s1[e], s0[e]);
      }
    }
    u32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) r[k] = pack_bf16x2(f[2 * k], f[2 * k + 1]);
    yr[v] = r;
  }
}

// ------------------------------------------------------- RMSNorm, second half
// One wave per token: the token's 1 / rms from the GEMM's partial sums of
// squares (summed in a fixed order), applied in place to its q row
// (token-major, with the optional gain) and to its k rows in the page slot.
__global__ __launch_bounds__(256) void norm_scale_kernel(int32_t T, NormScale ns) {
  const int32_t t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int32_t lane = threadIdx.x & 63;
  if (t >= T) return;
  const int32_t np = ns.D / kSsPartWidth, nv = ns.D / 8;
  const float* pr = ns.part + (size_t)t * ns.n_part;
  auto scale8 = [&](u32x4* p, float inv, const float* gain) {
    const u32x4 a = *p;
    float f[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      f[2 * k] = __uint_as_float(a[k] << 16) * inv;
      f[2 * k + 1] = __uint_as_float(a[k] & 0xffff0000u) * inv;
    }
    if (gain) {
      const f32x4 g0 = *reinterpret_cast<const f32x4*>(gain);
      const f32x4 g1 = *reinterpret_cast<const f32x4*>(gain + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        f[e] *= g0[e];
        f[4 + e] *= g1[e];
      }
    }
    u32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) r[k] = pack_bf16x2(f[2 * k], f[2 * k + 1]);
    *p = r;
  };
  if (ns.rows) {
    float s = 0.f;
    for (int32_t p = 0; p < np; ++p) s += pr[p];
    const float inv = rsqrtf(s / (float)ns.D + ns.eps);
    u32x4* row = reinterpret_cast<u32x4*>(ns.rows + (size_t)t * ns.ld);
    for (int32_t v = lane; v < nv; v += 64) scale8(row + v, inv, ns.gain ? ns.gain + 8 * v : nullptr);
  }
  if (ns.layer_base) {
    float s = 0.f;
    for (int32_t p = 0; p < np; ++p) s += pr[np + p];
    const float inv = rsqrtf(s / (float)ns.D + ns.eps);
    const int32_t node = t / ns.nq, tok = t - node * ns.nq;
    const int32_t frame = tok / ns.tpp, n = tok - frame * ns.tpp;
    uint16_t* kb = reinterpret_cast<uint16_t*>(
        ns.layer_base + (size_t)ns.node_slot[node * ns.ppc + frame] * ns.slot_bytes);
    const int32_t vph = ns.head_dim / 8;  // 16-byte vectors per head row
    for (int32_t v = lane; v < nv; v += 64) {
      const int32_t head = v / vph, c = v - head * vph;
      scale8(reinterpret_cast<u32x4*>(kb + ((size_t)head * ns.tpp + n) * ns.head_dim + 8 * c), inv,
             nullptr);
    }
  }
}

int launch_norm_scale(int32_t T, const NormScale& ns, hipStream_t stream) {
  if (ns.D % 128 || (ns.layer_base && ns.head_dim % 8))
    return fail(SC_EUNSUPPORTED, "qk-norm needs hidden %% 128 == 0 (got %d)", ns.D);
  if (T <= 0) return SC_OK;
  timer_begin(TK_QK_NORM, stream);
  hipLaunchKernelGGL(norm_scale_kernel, dim3((T + 3) / 4), dim3(256), 0, stream, T, ns);
  timer_end(TK_QK_NORM, stream);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

int launch_rmsnorm(const uint16_t* x, uint16_t* y, int32_t rows, int32_t D, const NormMod& nm,
                   hipStream_t stream) {
  if (D % 8) return fail(SC_EUNSUPPORTED, "rmsnorm needs D %% 8 == 0");
  timer_begin(TK_RMSNORM, stream);
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((rows + 3) / 4), dim3(256), 0, stream, x, y, nullptr, rows, D,
                     1e-6f, nm);
  timer_end(TK_RMSNORM, stream);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

int launch_row_rms(const uint16_t* x, int32_t rows, int32_t D, float* scale, hipStream_t stream) {
  if (D % 8) return fail(SC_EUNSUPPORTED, "rmsnorm needs D %% 8 == 0");
  NormMod plain;
  std::memset(&plain, 0, sizeof plain);
  timer_begin(TK_RMSNORM, stream);
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((rows + 3) / 4), dim3(256), 0, stream, x, nullptr, scale, rows, D,
                     1e-6f, plain);
  timer_end(TK_RMSNORM, stream);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

// One thread per token; partial p of all tokens is contiguous, so each of
// the n_part loads of a wave reads 256 consecutive bytes.  Unrolled so that
// eight loads are in flight at once; the adds keep increasing p.
__global__ __launch_bounds__(256) void row_scale_kernel(const float* __restrict__ part, int32_t n_part, int32_t T,
                                                        float inv_d, float eps, float* __restrict__ scale) {
  const int32_t t = blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  float s = 0.f;
#pragma unroll 8
  for (int32_t p = 0; p < n_part; ++p) s += part[(size_t)p * T + t];
  scale[t] = rsqrtf(s * inv_d + eps);
}

int launch_row_scale(const float* part, int32_t n_part, int32_t T, int32_t D, float eps, float* scale,
                     hipStream_t stream) {
  if (T <= 0 || n_part <= 0 || D <= 0) return fail(SC_EINVAL, "row_scale needs T, n_part, D > 0");
  timer_begin(TK_ROW_SCALE, stream);
  hipLaunchKernelGGL(row_scale_kernel, dim3((T + 255) / 256), dim3(256), 0, stream, part, n_part, T,
                     1.0f / (float)D, eps, scale);
  timer_end(TK_ROW_SCALE, stream);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

}  // namespace sc
