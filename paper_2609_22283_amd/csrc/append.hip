// KV append into the paged cache (+ 3D RoPE on keys) and the RoPE table.
//
// One page slot holds one latent frame of one state: K[head][token][d] then
// V[head][d][token].  Keys are rotated at their absolute positions (time =
// chunk * pages_per_chunk + frame, height = n / grid_w, width = n % grid_w)
// with interleaved channel pairs split over the three axes.
#include "device.h"
#include "internal.h"

namespace sc {

// cos/sin of pos * theta^(-2 i / dim_a) for every (position, pair) of the
// three axes, computed in double and stored as fp32 (cos, sin).
__global__ void rope_table_kernel(float2* table, int32_t pt, int32_t ph, int32_t pw, int64_t off_h,
                                  int64_t off_w, int64_t total, float theta) {
  int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= total) return;
  int32_t pos, i, dim;
  if (e < off_h) {
    pos = (int32_t)(e / pt); i = (int32_t)(e % pt); dim = 2 * pt;
  } else if (e < off_w) {
    pos = (int32_t)((e - off_h) / ph); i = (int32_t)((e - off_h) % ph); dim = 2 * ph;
  } else {
    pos = (int32_t)((e - off_w) / pw); i = (int32_t)((e - off_w) % pw); dim = 2 * pw;
  }
  const double freq = pow((double)theta, -2.0 * (double)i / (double)dim);
  const double ang = (double)pos * freq;
  table[e] = make_float2((float)cos(ang), (float)sin(ang));
}

int launch_rope_table(const sc_rope_desc* d, void* table, hipStream_t stream) {
  RopeLayout L = rope_layout(d);
  if (L.total == 0) return SC_OK;
  const int threads = 256;
  const int64_t blocks = (L.total + threads - 1) / threads;
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)blocks), dim3(threads), 0, stream,
                     static_cast<float2*>(table), L.pairs_t, L.pairs_h, L.pairs_w, L.off_h, L.off_w,
                     L.total, d->theta);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

struct RopeArgs {
  const float2* table;
  int32_t grid_w, pairs_t, pairs_h, pairs_w;
  int64_t off_h, off_w;
  int32_t frame0;  // absolute latent frame of the state's first page
};

// Rotation of channel pair p of a token at (t, hh, ww).
__device__ __forceinline__ float2 rope_cs(const RopeArgs& r, int32_t p, int32_t t, int32_t hh,
                                          int32_t ww) {
  if (p < r.pairs_t) return r.table[(int64_t)t * r.pairs_t + p];
  p -= r.pairs_t;
  if (p < r.pairs_h) return r.table[r.off_h + (int64_t)hh * r.pairs_h + p];
  p -= r.pairs_h;
  return r.table[r.off_w + (int64_t)ww * r.pairs_w + p];
}

struct SlotList {
  int32_t slot[32];
};

// Element type traits: bf16 is stored as uint16 bit patterns.
template <typename T> struct Elt;
template <> struct Elt<uint16_t> {
  static __device__ __forceinline__ float ld(uint16_t v) { return bf16_to_f32(v); }
  static __device__ __forceinline__ uint16_t st(float f) { return f32_to_bf16(f); }
};
template <> struct Elt<float> {
  static __device__ __forceinline__ float ld(float v) { return v; }
  static __device__ __forceinline__ float st(float f) { return f; }
};

// Grid: x = page (frame) * token blocks of 64, y = head.  256 threads.
// Tokens of the source: [frame * tpp + t][head][d].
template <typename T, int HD>
__global__ __launch_bounds__(256) void append_kernel(const T* __restrict__ k, const T* __restrict__ v,
                                                     char* __restrict__ layer_base, size_t slot_bytes,
                                                     size_t kv_half, SlotList slots, int32_t n_heads,
                                                     int32_t tpp, int32_t use_rope, RopeArgs rope) {
  constexpr int TB = 64;
  __shared__ T vt[TB][HD + 1];
  const int32_t blocks_per_page = (tpp + TB - 1) / TB;
  const int32_t page = blockIdx.x / blocks_per_page;
  const int32_t t0 = (blockIdx.x % blocks_per_page) * TB;
  const int32_t h = blockIdx.y;
  const int32_t ntok = min(TB, tpp - t0);
  char* slot_base = layer_base + (size_t)slots.slot[page] * slot_bytes;
  T* kdst = reinterpret_cast<T*>(slot_base) + ((size_t)h * tpp) * HD;
  T* vdst = reinterpret_cast<T*>(slot_base + kv_half) + (size_t)h * HD * tpp;
  const size_t row_stride = (size_t)n_heads * HD;
  // keys (with rotation) and values into LDS, one channel pair per thread step
  for (int32_t e = threadIdx.x; e < ntok * (HD / 2); e += blockDim.x) {
    const int32_t tt = e / (HD / 2), p = e % (HD / 2);
    const int32_t tok = t0 + tt;
    const size_t src = ((size_t)page * tpp + tok) * row_stride + (size_t)h * HD + 2 * p;
    float k0 = Elt<T>::ld(k[src]), k1 = Elt<T>::ld(k[src + 1]);
    if (use_rope) {
      const float2 cs = rope_cs(rope, p, rope.frame0 + page, tok / rope.grid_w, tok % rope.grid_w);
      const float r0 = k0 * cs.x - k1 * cs.y;
      const float r1 = k0 * cs.y + k1 * cs.x;
      k0 = r0;
      k1 = r1;
    }
    kdst[(size_t)tok * HD + 2 * p] = Elt<T>::st(k0);
    kdst[(size_t)tok * HD + 2 * p + 1] = Elt<T>::st(k1);
    vt[tt][2 * p] = v[src];
    vt[tt][2 * p + 1] = v[src + 1];
  }
  __syncthreads();
  // values transposed: V[head][d][token]
  for (int32_t e = threadIdx.x; e < ntok * HD; e += blockDim.x) {
    const int32_t d = e / ntok, tt = e % ntok;
    vdst[(size_t)d * tpp + t0 + tt] = vt[tt][d];
  }
}

int launch_append(const sc_cache* c, int32_t layer, const int32_t* slots, int32_t chunk,
                  const void* k, const void* v, const sc_rope* rope, hipStream_t stream) {
  const sc_cache_desc& d = c->d;
  if (d.pages_per_chunk > 32) return fail(SC_EUNSUPPORTED, "pages_per_chunk > 32");
  SlotList sl;
  for (int i = 0; i < d.pages_per_chunk; ++i) sl.slot[i] = slots[i];
  RopeArgs ra{};
  if (rope) {
    RopeLayout L = rope_layout(&rope->desc);
    ra.table = static_cast<const float2*>(rope->dev_table);
    ra.grid_w = rope->desc.grid_w;
    ra.pairs_t = L.pairs_t;
    ra.pairs_h = L.pairs_h;
    ra.pairs_w = L.pairs_w;
    ra.off_h = L.off_h;
    ra.off_w = L.off_w;
    ra.frame0 = chunk * d.pages_per_chunk;
  }
  char* layer_base = c->pool + (size_t)layer * d.n_slots * c->slot_bytes;
  dim3 grid(d.pages_per_chunk * ((d.tokens_per_page + 63) / 64), d.n_heads);
  const int use_rope = rope ? 1 : 0;
  timer_begin(TK_APPEND, stream);
  if (d.dtype == SC_DTYPE_BF16) {
    if (d.head_dim == 128)
      hipLaunchKernelGGL((append_kernel<uint16_t, 128>), grid, dim3(256), 0, stream,
                         static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), layer_base,
                         c->slot_bytes, c->kv_half, sl, d.n_heads, d.tokens_per_page, use_rope, ra);
    else
      hipLaunchKernelGGL((append_kernel<uint16_t, 64>), grid, dim3(256), 0, stream,
                         static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), layer_base,
                         c->slot_bytes, c->kv_half, sl, d.n_heads, d.tokens_per_page, use_rope, ra);
  } else {
    if (d.head_dim == 128)
      hipLaunchKernelGGL((append_kernel<float, 128>), grid, dim3(256), 0, stream,
                         static_cast<const float*>(k), static_cast<const float*>(v), layer_base,
                         c->slot_bytes, c->kv_half, sl, d.n_heads, d.tokens_per_page, use_rope, ra);
    else
      hipLaunchKernelGGL((append_kernel<float, 64>), grid, dim3(256), 0, stream,
                         static_cast<const float*>(k), static_cast<const float*>(v), layer_base,
                         c->slot_bytes, c->kv_half, sl, d.n_heads, d.tokens_per_page, use_rope, ra);
  }
  timer_end(TK_APPEND, stream);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

}  // namespace sc
