// bf16 GEMM for the DiT block's projections, D[f][t] = sum_k W[f][k] X[t][k]
// (W in [out, in] layout, X token-major), fp32 accumulation on 32x32x16 bf16
// MFMAs, with the block's elementwise work fused into the epilogue:
//   QKV      RoPE on q and k; q to a token-major buffer; k and v scattered
//            into the pack nodes' page slots (k as [head][token][d], v as
//            [head][d][token])
//   GELU     out[t][f] = GELU_tanh(D)
//   RESIDUAL x[t][f] += D   (in place)
// Work-group tile 256 (features) x 256 (tokens) x 64 (k), eight waves of
// 128 x 64, operands double-buffered in LDS with an XOR swizzle.  Each lane
// holds four consecutive features of one token, so RoPE pairs stay in-lane.
#include "device.h"
#include "gemm.h"
#include "internal.h"

namespace sc {

constexpr int GBM = 256, GBN = 256, GBK = 64;
constexpr int GWM = 128, GWN = 64;
constexpr int G_THREADS = 512;
constexpr int G_TILE_BYTES = GBM * GBK * 2;  // 32 KB per operand per stage

__device__ __forceinline__ float gelu_tanh(float x) {
  const float u = 0.7978845608028654f * fmaf(0.044715f * x, x * x, x);
  // tanh(u) = 1 - 2 / (exp(2u) + 1), saturating correctly at +-inf
  const float e = __expf(2.f * u);
  const float th = 1.f - 2.f / (e + 1.f);
  return 0.5f * x * (1.f + th);
}

template <int EPI>
__global__ __launch_bounds__(G_THREADS, 1) void gemm_bf16_kernel(const uint16_t* __restrict__ W,
                                                                 const uint16_t* __restrict__ X,
                                                                 int32_t F, int32_t T, int32_t Kd,
                                                                 GemmEpilogue ep) {
  __shared__ __attribute__((aligned(16))) char smem[2 * 2 * G_TILE_BYTES];
  const int32_t n_tf = F / GBM, n_tt = (T + GBN - 1) / GBN;
  const uint32_t tile = xcd_remap(blockIdx.x, (uint32_t)(n_tf * n_tt));
  const int32_t tf = tile % n_tf, tt = tile / n_tf;
  const int32_t f0 = tf * GBM, t0 = tt * GBN;

  const int32_t tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int32_t hl = lane >> 5, r32 = lane & 31;
  const int32_t wf = (wave & 1) * GWM, wt = (wave >> 1) * GWN;

  // loader: 4 chunks of 16 B for W and for X per thread per stage
  u32x4 wpre[4], xpre[4];
  const uint16_t* wsrc[4];
  const uint16_t* xsrc[4];
  int32_t lds_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int32_t c = tid + G_THREADS * i;  // 0..2047
    const int32_t row = c >> 3, col = c & 7;
    wsrc[i] = W + (size_t)(f0 + row) * Kd + col * 8;
    const int32_t trow = min(t0 + row, T - 1);
    xsrc[i] = X + (size_t)trow * Kd + col * 8;
    lds_off[i] = row * 128 + ((col ^ ((row >> 1) & 7)) << 4);
  }
  auto issue = [&](int32_t k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      wpre[i] = *reinterpret_cast<const u32x4*>(wsrc[i] + k0);
      xpre[i] = *reinterpret_cast<const u32x4*>(xsrc[i] + k0);
    }
  };
  auto stash = [&](int buf) {
    char* a = smem + buf * 2 * G_TILE_BYTES;
    char* b = a + G_TILE_BYTES;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<u32x4*>(a + lds_off[i]) = wpre[i];
      *reinterpret_cast<u32x4*>(b + lds_off[i]) = xpre[i];
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = f32x16{};

  const int32_t nk = Kd / GBK;
  issue(0);
  stash(0);
  __syncthreads();
  for (int32_t kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) issue((kt + 1) * GBK);
    const char* a = smem + (kt & 1) * 2 * G_TILE_BYTES;
    const char* b = a + G_TILE_BYTES;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int32_t col = 2 * s + hl;
      bf16x8 af[4], bfr[2];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const int32_t row = wf + 32 * mb + r32;
        af[mb] = *reinterpret_cast<const bf16x8*>(a + row * 128 + ((col ^ ((row >> 1) & 7)) << 4));
      }
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int32_t row = wt + 32 * nb + r32;
        bfr[nb] = *reinterpret_cast<const bf16x8*>(b + row * 128 + ((col ^ ((row >> 1) & 7)) << 4));
      }
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bfr[nb], acc[mb][nb], 0, 0, 0);
    }
    if (kt + 1 < nk) stash((kt + 1) & 1);
    __syncthreads();
  }

  // epilogue: lane holds D[f][t] for t = t0 + wt + 32 nb + r32 and
  // f = f0 + wf + 32 mb + 8 g + 4 hl + e (e = 0..3)
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int32_t t = t0 + wt + 32 * nb + r32;
    if (t >= T) continue;
    if constexpr (EPI == EPI_QKV) {
      const int32_t node = t / ep.nq, tok = t - node * ep.nq;
      const int32_t frame = tok / ep.tpp, n = tok - frame * ep.tpp;
      const int32_t pos_t = ep.node_chunk[node] * ep.ppc + frame;
      const int32_t pos_h = n / ep.grid_w, pos_w = n - pos_h * ep.grid_w;
      char* slot_base = ep.layer_base + (size_t)ep.node_slot[node * ep.ppc + frame] * ep.slot_bytes;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int32_t f = f0 + wf + 32 * mb + 8 * g + 4 * hl;
          const int32_t sec = f / ep.hidden, hf = f - sec * ep.hidden;
          const int32_t head = hf / ep.head_dim, d = hf - head * ep.head_dim;
          float v0 = acc[mb][nb][4 * g + 0], v1 = acc[mb][nb][4 * g + 1];
          float v2 = acc[mb][nb][4 * g + 2], v3 = acc[mb][nb][4 * g + 3];
          if (sec < 2 && ep.rope_table) {
#pragma unroll
            for (int pp = 0; pp < 2; ++pp) {
              int32_t p = d / 2 + pp;
              float2 cs;
              if (p < ep.pairs_t) cs = ep.rope_table[(int64_t)pos_t * ep.pairs_t + p];
              else if ((p -= ep.pairs_t) < ep.pairs_h) cs = ep.rope_table[ep.rope_off_h + (int64_t)pos_h * ep.pairs_h + p];
              else cs = ep.rope_table[ep.rope_off_w + (int64_t)pos_w * ep.pairs_w + (p - ep.pairs_h)];
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
          if (sec == 0) {
            *reinterpret_cast<u32x2*>(ep.q_out + (size_t)t * ep.hidden + hf) = pk;
          } else if (sec == 1) {
            uint16_t* kd = reinterpret_cast<uint16_t*>(slot_base) + ((size_t)head * ep.tpp + n) * ep.head_dim + d;
            *reinterpret_cast<u32x2*>(kd) = pk;
          } else {
            uint16_t* vd = reinterpret_cast<uint16_t*>(slot_base + ep.kv_half) +
                           ((size_t)head * ep.head_dim + d) * ep.tpp + n;
            vd[0] = (uint16_t)(pk.x & 0xffff);
            vd[ep.tpp] = (uint16_t)(pk.x >> 16);
            vd[2 * ep.tpp] = (uint16_t)(pk.y & 0xffff);
            vd[3 * ep.tpp] = (uint16_t)(pk.y >> 16);
          }
        }
    } else {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int32_t f = f0 + wf + 32 * mb + 8 * g + 4 * hl;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[mb][nb][4 * g + e];
          uint16_t* dst = ep.out + (size_t)t * ep.ld_out + f;
          if constexpr (EPI == EPI_RESIDUAL) {
            const u32x2 r = *reinterpret_cast<const u32x2*>(dst);
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
        }
    }
  }
}

int launch_gemm(int epi, int timer_kind, const uint16_t* W, const uint16_t* X, int32_t F, int32_t T,
                int32_t Kd, const GemmEpilogue& ep, hipStream_t stream) {
  if (F % GBM || Kd % GBK || T <= 0)
    return fail(SC_EUNSUPPORTED, "gemm needs F %% %d == 0, K %% %d == 0 (F=%d K=%d T=%d)", GBM, GBK,
                F, Kd, T);
  const uint32_t tiles = (uint32_t)(F / GBM) * (uint32_t)((T + GBN - 1) / GBN);
  timer_begin(timer_kind, stream);
  switch (epi) {
    case EPI_QKV:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_QKV>, dim3(tiles), dim3(G_THREADS), 0, stream, W, X, F,
                         T, Kd, ep);
      break;
    case EPI_GELU:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_GELU>, dim3(tiles), dim3(G_THREADS), 0, stream, W, X,
                         F, T, Kd, ep);
      break;
    case EPI_RESIDUAL:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_RESIDUAL>, dim3(tiles), dim3(G_THREADS), 0, stream, W,
                         X, F, T, Kd, ep);
      break;
    default:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_STORE>, dim3(tiles), dim3(G_THREADS), 0, stream, W, X,
                         F, T, Kd, ep);
  }
  timer_end(timer_kind, stream);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

// ------------------------------------------------------------------ RMSNorm
// y = x / sqrt(mean(x^2) + eps), one wave per row, fp32 math, bf16 in/out.
__global__ __launch_bounds__(256) void rmsnorm_kernel(const uint16_t* __restrict__ x,
                                                      uint16_t* __restrict__ y, int32_t rows,
                                                      int32_t D, float eps) {
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
  for (int32_t v = lane; v < nv; v += 64) {
    const u32x4 a = xr[v];
    u32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float lo = __uint_as_float(a[k] << 16), hi = __uint_as_float(a[k] & 0xffff0000u);
      r[k] = pack_bf16x2(lo * inv, hi * inv);
    }
    yr[v] = r;
  }
}

int launch_rmsnorm(const uint16_t* x, uint16_t* y, int32_t rows, int32_t D, hipStream_t stream) {
  if (D % 8) return fail(SC_EUNSUPPORTED, "rmsnorm needs D %% 8 == 0");
  timer_begin(TK_RMSNORM, stream);
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((rows + 3) / 4), dim3(256), 0, stream, x, y, rows, D, 1e-6f);
  timer_end(TK_RMSNORM, stream);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

}  // namespace sc
