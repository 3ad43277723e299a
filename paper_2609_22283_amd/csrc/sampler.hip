// Sampler step of Eq. 1 for a pack of nodes (the re-noising reading):
//   x^{j-1} = (1 - t_{j-1}) * y + t_{j-1} * xi     for nodes with j >= 1.
#include "device.h"
#include "internal.h"

namespace sc {

constexpr int kMaxSamplerNodes = 64;

struct SamplerCoef {
  float a[kMaxSamplerNodes];  // weight of y   (negative: node left untouched)
  float b[kMaxSamplerNodes];  // weight of noise
};

// 8 bf16 per thread; elems_per_node is a multiple of 8.
__global__ __launch_bounds__(256) void sampler_kernel(uint16_t* __restrict__ out,
                                                      const uint16_t* __restrict__ y,
                                                      const uint16_t* __restrict__ noise,
                                                      int64_t elems_per_node, int32_t n_nodes,
                                                      SamplerCoef coef) {
  const int64_t vec_per_node = elems_per_node / 8;
  const int64_t total = vec_per_node * n_nodes;
  for (int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; v < total;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t node = (int32_t)(v / vec_per_node);
    const float a = coef.a[node], b = coef.b[node];
    if (a < 0.f) continue;
    const u32x4 yv = reinterpret_cast<const u32x4*>(y)[v];
    const u32x4 nv = reinterpret_cast<const u32x4*>(noise)[v];
    u32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float y0 = __uint_as_float(yv[k] << 16), y1 = __uint_as_float(yv[k] & 0xffff0000u);
      const float n0 = __uint_as_float(nv[k] << 16), n1 = __uint_as_float(nv[k] & 0xffff0000u);
      r[k] = pack_bf16x2(fmaf(a, y0, b * n0), fmaf(a, y1, b * n1));
    }
    reinterpret_cast<u32x4*>(out)[v] = r;
  }
}

}  // namespace sc

using namespace sc;

extern "C" int sc_sampler_step(const sc_node* nodes, int32_t n, const float* t, int32_t K, void* out,
                               const void* y, const void* noise, int64_t elems_per_node,
                               sc_stream stream) {
  if (!nodes || !t || !out || !y || !noise || n < 0 || K < 1 || elems_per_node <= 0)
    return fail(SC_EINVAL, "bad sampler arguments");
  if (n > kMaxSamplerNodes) return fail(SC_EUNSUPPORTED, "more than %d nodes", kMaxSamplerNodes);
  if (elems_per_node % 8) return fail(SC_EINVAL, "elems_per_node must be a multiple of 8");
  if ((reinterpret_cast<uintptr_t>(out) | reinterpret_cast<uintptr_t>(y) |
       reinterpret_cast<uintptr_t>(noise)) & 15)
    return fail(SC_EINVAL, "buffers must be 16-byte aligned");
  SamplerCoef coef;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t j = nodes[i].level;
    if (j < 0 || j > K) return fail(SC_EINVAL, "node level %d outside [0, K]", j);
    if (j == 0) {
      coef.a[i] = -1.f;
      coef.b[i] = 0.f;
    } else {
      coef.a[i] = 1.f - t[j - 1];
      coef.b[i] = t[j - 1];
    }
  }
  if (n == 0) return SC_OK;
  const int64_t total = elems_per_node / 8 * n;
  const int threads = 256;
  const int64_t blocks = std::min<int64_t>((total + threads - 1) / threads, 4096);
  timer_begin(TK_SAMPLER, static_cast<hipStream_t>(stream));
  hipLaunchKernelGGL(sampler_kernel, dim3((unsigned)blocks), dim3(threads), 0,
                     static_cast<hipStream_t>(stream), static_cast<uint16_t*>(out),
                     static_cast<const uint16_t*>(y), static_cast<const uint16_t*>(noise),
                     elems_per_node, n, coef);
  timer_end(TK_SAMPLER, static_cast<hipStream_t>(stream));
  SC_HIP(hipGetLastError());
  return SC_OK;
}
