// Packed paged block-causal attention (Eq. 6 over the plan's page lists).
//
// For every pack node i and head h: O = softmax(Q K^T * scale) V over the
// keys of node i's pages only.  The visibility mask is never formed: the page
// list is the mask.  Keys are concatenated page after page; every page holds
// a multiple of 8 tokens, so any 8 consecutive keys of the concatenation that
// start at a multiple of 8 lie in one page.
//
// bf16 kernel (head_dim 128), per work-group: 128 queries of one (node, head),
// four waves of 32 queries.  Key tiles of 64 are staged through LDS (double
// buffered, XOR-swizzled against bank conflicts); each wave computes
// S^T = K Q^T and O^T += V^T P^T with 32x32x16 bf16 MFMAs and keeps an online
// softmax in fp32.  The K rows feeding the S^T MFMA are permuted so that each
// lane's probabilities are exactly the B operand of the PV MFMA, and V is
// stored transposed in the cache so its A operand is one 16-byte LDS read.
#include "device.h"
#include "internal.h"

namespace sc {

constexpr int kMaxNodes = 64;
constexpr int kMaxPages = 800;

struct AttnPlan {
  int32_t page_off[kMaxNodes + 1];
  int32_t page_slot[kMaxPages];
};

struct AttnGeom {
  const char* layer_base;
  uint64_t slot_bytes, kv_half;
  int32_t n_nodes, n_heads, tpp, nq, n_qtiles;
  DivMagic tpp_div;
  float scale_log2;  // scale * log2(e): softmax evaluated with exp2
  float scale;
};

static DivMagic magic_div(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  uint64_t m = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
  return DivMagic{(uint32_t)m, l, d};
}

// ------------------------------------------------------------- fp32 kernel
// One thread per query row, keys streamed from the cache; used for the fp32
// path (small parity shapes), not tuned.
template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ q, float* __restrict__ o,
                                                      AttnGeom g, AttnPlan plan) {
  const uint32_t qt_n = (g.nq + 63) / 64;
  const uint32_t w = blockIdx.x;
  const int32_t qt = w % qt_n;
  const int32_t node = (w / qt_n) % g.n_nodes;
  const int32_t head = w / (qt_n * g.n_nodes);
  const int32_t row = qt * 64 + threadIdx.x;
  if (row >= g.nq) return;
  const size_t qoff = (((size_t)node * g.nq + row) * g.n_heads + head) * HD;
  float qr[HD], acc[HD];
  for (int d = 0; d < HD; ++d) {
    qr[d] = q[qoff + d] * g.scale;
    acc[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int32_t p = plan.page_off[node]; p < plan.page_off[node + 1]; ++p) {
    const char* base = g.layer_base + (size_t)plan.page_slot[p] * g.slot_bytes;
    const float* kb = reinterpret_cast<const float*>(base) + (size_t)head * g.tpp * HD;
    const float* vb = reinterpret_cast<const float*>(base + g.kv_half) + (size_t)head * HD * g.tpp;
    for (int32_t t = 0; t < g.tpp; ++t) {
      float s = 0.f;
      for (int d = 0; d < HD; ++d) s = fmaf(qr[d], kb[(size_t)t * HD + d], s);
      const float mn = fmaxf(m, s);
      const float alpha = expf(m - mn);
      const float pr = expf(s - mn);
      l = l * alpha + pr;
      for (int d = 0; d < HD; ++d) acc[d] = fmaf(pr, vb[(size_t)d * g.tpp + t], acc[d] * alpha);
      m = mn;
    }
  }
  const float inv = 1.f / l;
  for (int d = 0; d < HD; ++d) o[qoff + d] = acc[d] * inv;
}

// ------------------------------------------------------------- bf16 kernel
constexpr int BQ = 128;       // queries per work-group
constexpr int BK = 64;        // keys per tile
constexpr int HDB = 128;      // head dim of the bf16 kernel
constexpr int KT_BYTES = BK * HDB * 2;   // 16 KB
constexpr int VT_BYTES = HDB * BK * 2;   // 16 KB

__device__ __forceinline__ void load16_global(u32x4& r, const char* p) {
  r = *reinterpret_cast<const u32x4*>(p);
}

__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(const uint16_t* __restrict__ q,
                                                           uint16_t* __restrict__ o, AttnGeom g,
                                                           AttnPlan plan) {
  __shared__ __attribute__((aligned(16))) char smem[2 * (KT_BYTES + VT_BYTES)];
  const uint32_t nwg = (uint32_t)g.n_nodes * g.n_heads * g.n_qtiles;
  const uint32_t w = xcd_remap(blockIdx.x, nwg);
  const int32_t qt = w % g.n_qtiles;
  const int32_t node = (w / g.n_qtiles) % g.n_nodes;
  const int32_t head = w / (g.n_qtiles * g.n_nodes);

  const int32_t tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int32_t hl = lane >> 5, r32 = lane & 31;
  const int32_t p0 = plan.page_off[node];
  const int32_t nk = (plan.page_off[node + 1] - p0) * g.tpp;
  const int32_t ntiles = (nk + BK - 1) / BK;

  // Q^T operand: lane holds Q[row][16 s + 8 hl .. +7] for s = 0..7.
  const int32_t qrow = qt * BQ + wave * 32 + r32;
  const int32_t qrow_c = qrow < g.nq ? qrow : g.nq - 1;
  const uint16_t* qp = q + (((size_t)node * g.nq + qrow_c) * g.n_heads + head) * HDB + 8 * hl;
  bf16x8 qreg[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) qreg[s] = *reinterpret_cast<const bf16x8*>(qp + 16 * s);

  // Row of the S^T MFMA that holds key sigma(r): lane-local probabilities then
  // come out as keys 8*hl .. 8*hl+7 (+16) of each 32-key block.
  const int32_t sa = r32 >> 3, sh = (r32 >> 2) & 1, sb = r32 & 3;
  const int32_t sigma = 16 * (sa >> 1) + 8 * sh + 4 * (sa & 1) + sb;

  // Tile loaders: 4 K chunks and 4 V^T chunks of 16 bytes per thread.
  const char* kbase = g.layer_base + (size_t)head * g.tpp * HDB * 2;
  const char* vbase = g.layer_base + g.kv_half + (size_t)head * HDB * g.tpp * 2;
  u32x4 kpre[4], vpre[4];
  auto issue_loads = [&](int32_t t0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int32_t c = tid + 256 * i;
      const int32_t row = c >> 4, col = c & 15;
      int32_t key = t0 + row;
      key = key < nk ? key : nk - 1;
      const int32_t pg = fast_div(key, g.tpp_div);
      const int32_t off = key - pg * g.tpp;
      const size_t slot = plan.page_slot[p0 + pg];
      load16_global(kpre[i], kbase + slot * g.slot_bytes + ((size_t)off * HDB + col * 8) * 2);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int32_t c = tid + 256 * i;
      const int32_t d = c >> 3, col = c & 7;
      int32_t key = t0 + col * 8;
      key = key < nk ? key : nk - 8;
      const int32_t pg = fast_div(key, g.tpp_div);
      const int32_t off = key - pg * g.tpp;
      const size_t slot = plan.page_slot[p0 + pg];
      load16_global(vpre[i], vbase + slot * g.slot_bytes + ((size_t)d * g.tpp + off) * 2);
    }
  };
  auto store_lds = [&](int buf) {
    char* kl = smem + buf * (KT_BYTES + VT_BYTES);
    char* vl = kl + KT_BYTES;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int32_t c = tid + 256 * i;
      const int32_t row = c >> 4, col = c & 15;
      *reinterpret_cast<u32x4*>(kl + row * 256 + ((col ^ (row & 15)) << 4)) = kpre[i];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int32_t c = tid + 256 * i;
      const int32_t d = c >> 3, col = c & 7;
      *reinterpret_cast<u32x4*>(vl + d * 128 + ((col ^ ((d >> 1) & 7)) << 4)) = vpre[i];
    }
  };

  f32x16 oacc[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) oacc[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const float c2 = g.scale_log2;

  issue_loads(0);
  store_lds(0);
  __syncthreads();

  for (int32_t t = 0; t < ntiles; ++t) {
    const int32_t t0 = t * BK;
    if (t + 1 < ntiles) issue_loads(t0 + BK);
    const char* kl = smem + (t & 1) * (KT_BYTES + VT_BYTES);
    const char* vl = kl + KT_BYTES;

    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x16{};
      const int32_t krow = 32 * kb + sigma;
#pragma unroll
      for (int si = 0; si < 8; ++si) {
        const int32_t col = 2 * si + hl;
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(kl + krow * 256 + ((col ^ (krow & 15)) << 4));
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[si], s[kb], 0, 0, 0);
      }
    }
    if (t0 + BK > nk) {  // ragged last tile: keys beyond nk get no weight
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int32_t key = t0 + 32 * kb + 16 * (i >> 3) + 8 * hl + (i & 7);
          if (key >= nk) s[kb][i] = -INFINITY;
        }
    }
    float mx = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kb][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx * c2);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[db][i] *= alpha;

    bf16x8 pb[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int mm = 0; mm < 2; ++mm)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float p = exp2f(fmaf(s[kb][8 * mm + e], c2, -m_new));
          l_run += p;
          pb[kb][mm][e] = static_cast<__bf16>(p);
        }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int mm = 0; mm < 2; ++mm) {
        const int32_t col = 4 * kb + 2 * mm + hl;
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const int32_t drow = 32 * db + r32;
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(vl + drow * 128 + ((col ^ ((drow >> 1) & 7)) << 4));
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[kb][mm], oacc[db], 0, 0, 0);
        }
      }
    if (t + 1 < ntiles) store_lds((t + 1) & 1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.f / l_tot;
  if (qrow < g.nq) {
    uint16_t* op = o + (((size_t)node * g.nq + qrow) * g.n_heads + head) * HDB;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int gi = 0; gi < 4; ++gi) {
        const int32_t d = 32 * db + 8 * gi + 4 * hl;
        u32x2 v;
        v.x = pack_bf16x2(oacc[db][4 * gi + 0] * inv, oacc[db][4 * gi + 1] * inv);
        v.y = pack_bf16x2(oacc[db][4 * gi + 2] * inv, oacc[db][4 * gi + 3] * inv);
        *reinterpret_cast<u32x2*>(op + d) = v;
      }
  }
}

int launch_attention(const sc_plan* p, const sc_cache* c, int32_t layer, const void* q, void* o,
                     float scale, hipStream_t stream) {
  const sc_cache_desc& d = c->d;
  const int32_t n = (int32_t)p->nodes.size();
  if (n > kMaxNodes) return fail(SC_EUNSUPPORTED, "pack of %d nodes exceeds %d", n, kMaxNodes);
  if ((int32_t)p->page_slot.size() > kMaxPages)
    return fail(SC_EUNSUPPORTED, "plan of %zu pages exceeds %d", p->page_slot.size(), kMaxPages);
  AttnPlan plan;
  for (int32_t i = 0; i <= n; ++i) plan.page_off[i] = p->page_off[i];
  for (size_t i = 0; i < p->page_slot.size(); ++i) plan.page_slot[i] = p->page_slot[i];
  AttnGeom g;
  g.layer_base = c->pool + (size_t)layer * d.n_slots * c->slot_bytes;
  g.slot_bytes = c->slot_bytes;
  g.kv_half = c->kv_half;
  g.n_nodes = n;
  g.n_heads = d.n_heads;
  g.tpp = d.tokens_per_page;
  g.nq = p->nq;
  g.tpp_div = magic_div((uint32_t)d.tokens_per_page);
  g.scale = scale;
  g.scale_log2 = scale * 1.4426950408889634f;
  timer_begin(TK_ATTENTION, stream);
  if (d.dtype == SC_DTYPE_F32) {
    g.n_qtiles = (p->nq + 63) / 64;
    const uint32_t nwg = (uint32_t)n * d.n_heads * g.n_qtiles;
    if (d.head_dim == 64)
      hipLaunchKernelGGL((attn_f32_kernel<64>), dim3(nwg), dim3(64), 0, stream,
                         static_cast<const float*>(q), static_cast<float*>(o), g, plan);
    else
      hipLaunchKernelGGL((attn_f32_kernel<128>), dim3(nwg), dim3(64), 0, stream,
                         static_cast<const float*>(q), static_cast<float*>(o), g, plan);
  } else {
    if (d.head_dim != HDB) return fail(SC_EUNSUPPORTED, "bf16 attention needs head_dim 128");
    g.n_qtiles = (p->nq + BQ - 1) / BQ;
    const uint32_t nwg = (uint32_t)n * d.n_heads * g.n_qtiles;
    hipLaunchKernelGGL(attn_bf16_kernel, dim3(nwg), dim3(256), 0, stream,
                       static_cast<const uint16_t*>(q), static_cast<uint16_t*>(o), g, plan);
  }
  timer_end(TK_ATTENTION, stream);
  SC_HIP(hipGetLastError());
  return SC_OK;
}

}  // namespace sc
