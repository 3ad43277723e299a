// Packed paged block-causal attention (Eq. 6 over the plan's page lists).
//
// For every pack node i and head h: O = softmax(Q K^T * scale) V over the
// keys of node i's pages only.  The visibility mask is never formed: the page
// list is the mask.  Keys are concatenated page after page; every page holds
// a multiple of 8 tokens, so any 8 consecutive keys of the concatenation that
// start at a multiple of 8 lie in one page.
//
// bf16 kernel (head_dim 128), per work-group: 256 queries of one (node, head),
// eight waves of two 16-query blocks.  Key tiles of 64 are copied into LDS
// (double buffered, XOR-swizzled against bank conflicts); each wave computes
// S^T = K Q^T and O^T += V^T P^T with 16x16x32 bf16 MFMAs and keeps an online
// softmax in fp32.  The K rows feeding the S^T MFMA are permuted so that each
// lane's probabilities are exactly the B operand of the PV MFMA, and V is
// stored transposed in the cache so its A operand is one 16-byte LDS read.
#include <algorithm>
#include <climits>
#include <cstring>
#include <map>
#include <mutex>
#include <type_traits>

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
  // schedule of the bf16 kernel: whole units, then tail units cut in pieces
  int32_t whole_units, tail_units, tail_split;
  float* part_o;          // [tail_units * tail_split][BQ][128] unnormalised partial outputs
  float* part_ml;         // [tail_units * tail_split][2][BQ] partial max (log2 units) and sum
                          // (BQ: queries per work-group of the instantiation launched)
};

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
// Three work-group shapes: 8 waves x 32 queries (256 per work-group, one
// work-group per CU) and 4 waves x 32 queries (128, two per CU, for nodes of
// at most 128 queries), both with two waves per SIMD and 64-key tiles; and
// 2 waves x 32 queries (64, for nodes of at most 64) on 32-key tiles, whose
// deeper K/V rings (3 or 4 tiles of 16 KB) keep two or three tiles in flight
// per work-group, three or two work-groups per CU.  Such nodes are short and
// their attention streams K/V from HBM: in-flight copies, bounded by LDS,
// set its rate.  A wave's 32 queries are two 16-query blocks of the
// 16x16x32 MFMA; key tiles hold KH halves of 32 keys.
constexpr int HDB = 128;  // head dim of the bf16 kernels
template <int KH>
struct Tile {
  static constexpr int BK = 32 * KH;                  // keys per LDS tile
  static constexpr int KT_BYTES = BK * HDB * 2;       // K tile: BK rows of 256 bytes
  static constexpr int VT_BYTES = HDB * BK * 2;       // V^T tile: 128 rows of 2 BK bytes
};
constexpr int BQ_TINY = 64, BQ_SMALL = 128, BQ_MAX = 256;  // queries per work-group of the three shapes
// Softmax bookkeeping.  Q is pre-scaled by scale*log2(e), so S is in log2
// units, and each S tile starts its accumulation at -m: p = exp2(S)
// directly.  m is the exact maximum of the work item's first tile and is
// never raised inside the loop: later probabilities may exceed 1, which fp32
// sums and bf16 products represent with the same relative precision, up to
// a guard of 2^64 on each lane's tile sum.  A work-group in which any wave
// reaches the guard (logits more than 64 log2 units above the first tile's
// maximum) redoes its item exactly in two passes (attn_exact).  Rescaling in
// place would keep the accumulators and the recomputation live in the loop.
// The row sums come from the matrix cores: one more 16-row block of V^T whose
// first row is all ones turns O^T += V^T P^T into l += sum_k p as well, so
// the sum sees the same bf16 p as the numerator.  Since p >= 0 the final sum
// bounds every partial one, and the guard is checked once, on it.
constexpr float P_GUARD = 18446744073709551616.0f;  // 2^64

// Matrix-core shape: v_mfma_f32_16x16x32_bf16.  Lane l (g = l / 16,
// c = l % 16) supplies row c of A and column c of B with 8 consecutive k
// values 8 g .. 8 g + 7, and receives D[4 g + r][c], r = 0..3.  (The 16x16
// shape sustains more FLOP/s than 32x32x16 under the power cap: half the
// accumulator traffic per FLOP.)
__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// XOR swizzle of a K tile row: 16-byte column c of row r is stored at
// c ^ kswz(r).  Bit 4 of the row enters so that the 16 rows one 16-lane
// group reads for an S^T MFMA (see attn_lane) fall on distinct banks.
__device__ __forceinline__ uint32_t kswz(int32_t row) { return (uint32_t)((row & 15) ^ ((row >> 2) & 4)); }

struct AttnLane {
  // per-lane LDS read offsets (bytes) inside one buffer
  uint32_t koff[2][4];  // K row of block b, 16-byte column 4 ds + g (second 32 rows add 8192)
  uint32_t voff[2];     // V^T row c, 16-byte column 4 h + g (16-row block db adds 32 BK)
};

// XOR swizzle of a V^T tile row d (16-byte columns): 64-key rows (128 bytes)
// take (d / 2) mod 8, 32-key rows (64 bytes) (d / 4) mod 4, so the 16 rows
// of a PV operand read fall on distinct banks.
template <int KH>
__device__ __forceinline__ uint32_t vswz(int32_t d) {
  return KH == 2 ? (uint32_t)((d >> 1) & 7) : (uint32_t)((d >> 2) & 3);
}

// A row i of the S^T MFMA for 16-key block b of a 32-key half holds key
// 8 (i / 4) + 4 b + i % 4: each lane's four results of blocks 0 and 1 are
// then keys 8 g .. 8 g + 7 of the half -- exactly the B operand of the PV
// MFMA, which therefore needs no shuffle.
template <int KH>
__device__ __forceinline__ AttnLane attn_lane(int32_t c, int32_t g) {
  AttnLane L;
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int32_t row = 8 * (c >> 2) + 4 * b + (c & 3);
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) L.koff[b][ds] = row * 256 + (((4 * ds + g) ^ kswz(row)) << 4);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h)
    L.voff[h] = c * (64 * KH) + (((4 * h + g) ^ vswz<KH>(c)) << 4);  // h < KH only is used
  return L;
}

// Q^T operand of a 16-query block: lane holds Q[row][32 ds + 8 g .. +7].
// Rows past the node's end repeat its last row.  The loads are issued with
// the first tile copies (their latencies overlap); scale_q then pre-scales
// the values to log2 units once they have landed.
__device__ __forceinline__ void load_q(const uint16_t* q, const AttnGeom& g, int32_t node, int32_t head,
                                       int32_t qrow, int32_t lg, bf16x8 (&qreg)[4]) {
  const int32_t qrow_c = qrow < g.nq ? qrow : g.nq - 1;
  const uint16_t* qp = q + (((size_t)node * g.nq + qrow_c) * g.n_heads + head) * HDB + 8 * lg;
#pragma unroll
  for (int ds = 0; ds < 4; ++ds) qreg[ds] = *reinterpret_cast<const bf16x8*>(qp + 32 * ds);
}

__device__ __forceinline__ void scale_q(const AttnGeom& g, bf16x8 (&qreg)[4]) {
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
#pragma unroll
    for (int e = 0; e < 8; ++e) qreg[ds][e] = static_cast<__bf16>(static_cast<float>(qreg[ds][e]) * g.scale_log2);
}

// Logits of one 64-key tile for a wave's two 16-query blocks:
// s[h][b][qb] holds, in lane (g, c) value r, key 32 h + 8 g + 4 b + r of the
// tile for query c of block qb.
template <int KH>
using STile = f32x4[KH][2][2];

// Sum / maximum of one query's values over the four lane groups.
__device__ __forceinline__ float group_sum(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}
__device__ __forceinline__ float group_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}

// A operand of the row-sum MFMA: row 0 all ones, rows 1..15 zero (lane c
// supplies row c).  D[0][query] = sum over the 32 keys of p.
__device__ __forceinline__ bf16x8 ones_row(int32_t c) {
  bf16x8 a;
  const __bf16 v = static_cast<__bf16>(c == 0 ? 1.0f : 0.0f);
#pragma unroll
  for (int e = 0; e < 8; ++e) a[e] = v;
  return a;
}

// Column maxima of a tile, per query block.
template <int KH>
__device__ __forceinline__ void tile_max(const STile<KH>& s, float (&mx)[2]) {
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    float m = s[0][0][qb][0];
#pragma unroll
    for (int h = 0; h < KH; ++h)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) m = fmaxf(m, s[h][b][qb][r]);
    mx[qb] = group_max(m);
  }
}

// Keys at or past the node's end get no weight (t0: the tile's first key).
template <int KH>
__device__ __forceinline__ void mask_tile(STile<KH>& s, int32_t t0, int32_t nk, int32_t lg) {
#pragma unroll
  for (int h = 0; h < KH; ++h)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (t0 + 32 * h + 8 * lg + 4 * b + r >= nk) s[h][b][qb][r] = -INFINITY;
}

// p = exp2(s) rounded to bf16: pb[h][qb] is the B operand of the PV MFMA for
// the 32-key half h.
template <int KH>
__device__ __forceinline__ void probs(const STile<KH>& s, bf16x8 (&pb)[KH][2]) {
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int h = 0; h < KH; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pb[h][qb][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(s[h][e >> 2][qb][e & 3]));
}

// The same, also returning this lane's sums of the rounded values per block
// (the exact redo path).
template <int KH>
__device__ __forceinline__ void probs_tile(const STile<KH>& s, bf16x8 (&pb)[KH][2], float (&lt)[2]) {
  const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    float l0 = 0.f, l1 = 0.f;
#pragma unroll
    for (int h = 0; h < KH; ++h) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pb[h][qb][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(s[h][e >> 2][qb][e & 3]));
#pragma unroll
      for (int e = 0; e < 8; e += 4) {
        l0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[h][qb][e], pb[h][qb][e + 1]}, ones, l0, false);
        l1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[h][qb][e + 2], pb[h][qb][e + 3]}, ones, l1, false);
      }
    }
    lt[qb] = l0 + l1;
  }
}

// Direct global -> LDS copy of 16 bytes per lane (gfx950 LDS DMA): lane i
// of the wave writes bytes [16 i, 16 i + 16) after the wave-uniform LDS
// address, so the XOR swizzle is applied by choosing each lane's source
// (base + off).  Written as inline asm: while a copy it knows of is in
// flight, the compiler waits for every LDS read with lgkmcnt(0), so no
// fragment read could overlap another; the copies themselves complete
// under this wave's explicit vmcnt waits (landed, landed_but).  M0, which
// carries the LDS address, is saved and restored.
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return (uint32_t)reinterpret_cast<uintptr_t>(p);
}
__device__ __forceinline__ void dma16(const char* base, uint32_t off, char* lds_wave_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base), "s"(lds_addr(lds_wave_base))
      : "memory");
}

// Copies of BK-key K and V^T tiles of one (node, head) from the paged cache
// into LDS, split over the NW waves of a work-group.  A tile spans at most
// two pages (pages hold >= BK tokens), so the page of a key is chosen against
// one wave-uniform boundary.
// Offsets are 32-bit, relative to the layer's slots (the host checks that a
// layer fits in 4 GB); the per-page parts are wave-uniform.  A copy
// instruction moves 1 KB: 4 K rows, or RPI = 512 / BK V^T rows of BK / 8
// 16-byte columns.  Each wave issues KCP of the first and VCP of the second
// per tile; lane (row, physical column p) fetches logical column
// p ^ swizzle(row).  K rows of keys past the node's end fetch its last key,
// V^T columns the tile's first key (valid memory; their probabilities are
// zero).
template <int NW, int KH>
struct KvTiles {
  static constexpr int BK = Tile<KH>::BK;
  static constexpr int KCP = BK / (4 * NW), VCP = BK / (4 * NW);
  static constexpr int LPR = BK / 8, RPI = 64 / LPR;  // V^T: lanes per row, rows per copy instruction
  static_assert(LPR == 1 << (KH + 1), "V^T lanes per row");
  static_assert(KCP >= 1 && KCP * 4 * NW == BK, "K copy split");
  struct Slots {
    uint32_t lo, hi;  // byte offsets of the slots of the tile's first page and the next one
    int32_t plo;      // index of the tile's first page within the node
  };
  const char* lbase;
  const int32_t* page_slot;  // the node's page slots
  int32_t npages, nk, tpp, wave;
  uint32_t slot_bytes, khead, vhead, kbad;
  DivMagic tpp_div;
  uint32_t klane[KCP], vlane[VCP];
  int32_t vkey[VCP], krow0;

  __device__ __forceinline__ KvTiles(const AttnPlan& plan, const AttnGeom& g, int32_t node, int32_t head,
                                     int32_t wave_, int32_t lane) {
    const int32_t p0 = plan.page_off[node];
    lbase = g.layer_base;
    page_slot = plan.page_slot + p0;
    npages = plan.page_off[node + 1] - p0;
    tpp = g.tpp;
    nk = npages * tpp;
    wave = wave_;
    slot_bytes = (uint32_t)g.slot_bytes;
    tpp_div = g.tpp_div;
    khead = (uint32_t)head * tpp * HDB * 2;
    vhead = (uint32_t)g.kv_half + (uint32_t)head * HDB * tpp * 2;
    kbad = (uint32_t)page_slot[npages - 1] * slot_bytes + khead + (uint32_t)(tpp - 1) * 256;
    krow0 = 4 * KCP * wave + (lane >> 4);
    const int32_t kp = lane & 15;
    const int32_t vrow0 = RPI * VCP * wave + (lane >> (KH + 1)), vp = lane & (LPR - 1);  // LPR = 2^(KH+1)
#pragma unroll
    for (int j = 0; j < KCP; ++j) {
      const int32_t row = krow0 + 4 * j;
      klane[j] = (uint32_t)row * 256 + ((kp ^ kswz(row)) << 4);  // plus key t0 * 256
    }
#pragma unroll
    for (int j = 0; j < VCP; ++j) {
      const int32_t d = vrow0 + RPI * j;
      vkey[j] = 8 * (vp ^ (int32_t)vswz<KH>(d));                     // key offset in tile
      vlane[j] = (uint32_t)d * tpp * 2 + (uint32_t)vkey[j] * 2;      // plus key t0 * 2
    }
  }
  // Page slots of the tile starting at key t0 >= 0 (two scalar loads),
  // fetched ahead of the copy that uses them so their latency overlaps other
  // work (a step, or the barrier wait before the copy).  Clamped to the
  // node's pages: a tile past the end is never read.
  __device__ __forceinline__ Slots slots(int32_t t0) const {
    Slots sl;
    sl.plo = min((int32_t)fast_div((uint32_t)t0, tpp_div), npages - 1);
    const int32_t phi = sl.plo + 1 < npages ? sl.plo + 1 : sl.plo;
    sl.lo = (uint32_t)page_slot[sl.plo] * slot_bytes;
    sl.hi = (uint32_t)page_slot[phi] * slot_bytes;
    return sl;
  }
  // The 4 K rows of one copy instruction are tile rows 4 (KCP wave + j) ..
  // +3; page boundaries and the node's end are multiples of 8 keys, so the
  // page (or the out-of-range fallback) is one wave-uniform choice per
  // instruction.
  __device__ __forceinline__ void copy_k(int32_t t0, char* kl, const Slots& sl) const {
    const int32_t bkey = (sl.plo + 1) * tpp;
    const uint32_t lo = sl.lo + khead + (uint32_t)(t0 - sl.plo * tpp) * 256;
    const uint32_t hi = sl.hi + khead + (uint32_t)(t0 - bkey) * 256;
    const int32_t lim = nk - t0, split = bkey - t0;
#pragma unroll
    for (int j = 0; j < KCP; ++j) {
      const int32_t rg = 4 * KCP * wave + 4 * j;  // first tile row of this copy (wave-uniform)
      const uint32_t src = rg >= lim ? kbad + (klane[j] & 255u) : (rg >= split ? hi : lo) + klane[j];
      dma16(lbase, src, kl + rg * 256);
    }
  }
  // A V^T row holds the tile's BK keys; a page boundary or the node's end
  // falls inside the tile for about one tile in a page, so the per-lane
  // choice is taken only then (wave-uniform branch).
  __device__ __forceinline__ void copy_v(int32_t t0, char* vl, const Slots& sl) const {
    const int32_t bkey = (sl.plo + 1) * tpp;
    const uint32_t lo = sl.lo + vhead + (uint32_t)(t0 - sl.plo * tpp) * 2;
    const int32_t lim = nk - t0, split = bkey - t0;
    if (split >= BK && lim >= BK) {
#pragma unroll
      for (int j = 0; j < VCP; ++j) {
        // opaque, so the offset stays one add of the scalar base (the
        // compiler otherwise re-derives it with a per-lane multiply)
        uint32_t off = vlane[j];
        asm volatile("" : "+v"(off));
        dma16(lbase, lo + off, vl + (RPI * VCP * wave + RPI * j) * 2 * BK);
      }
      return;
    }
    const uint32_t hi = sl.hi + vhead + (uint32_t)(t0 - bkey) * 2;
#pragma unroll
    for (int j = 0; j < VCP; ++j) {
      const int32_t rk = vkey[j];
      const bool in = rk < lim;
      const uint32_t off = in ? vlane[j] : vlane[j] - (uint32_t)rk * 2;
      const uint32_t base = (in && rk >= split) ? hi : lo;
      dma16(lbase, base + off, vl + (RPI * VCP * wave + RPI * j) * 2 * BK);
    }
  }
};

__device__ __forceinline__ void landed() {  // this wave's copies are in LDS, then everyone's
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
}

// The same for all but this wave's n most recent vector-memory operations (a
// wave's loads complete in issue order for this counter), n even, at most
// 16 (wave-uniform).  The barrier is issued without __syncthreads' release
// fence, which would wait for every outstanding copy; the memory clobber
// keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void landed_but(int32_t n) {
#define SC_LANDED_BUT(k) \
  case k:                \
    asm volatile("s_waitcnt vmcnt(" #k ")\n\ts_barrier" ::: "memory"); \
    break;
  switch (n) {
    SC_LANDED_BUT(2) SC_LANDED_BUT(4) SC_LANDED_BUT(6) SC_LANDED_BUT(8) SC_LANDED_BUT(10)
    SC_LANDED_BUT(12) SC_LANDED_BUT(14) SC_LANDED_BUT(16)
    default: asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory"); break;
  }
#undef SC_LANDED_BUT
}

// Schedule.  A unit is a (head, node, query tile) triple, numbered head-major
// then node then query tile; a unit's key tiles are processed in order by one
// work-group.  The work-groups an XCD runs side by side are then the query
// tiles of one or two nodes of one head, which read the same K/V tiles at
// about the same time and share them in its L2; every node's page list
// starts at the state most nodes of the pack read (see shared_order), so
// two nodes there read their shared states together too.  (With the node
// fastest, four nodes' streams shared an XCD's L2 and it fetched 11 % more.)
// Equal units fill the resident work-groups in whole rounds but the
// last U mod R; those "tail" units are each cut into S pieces of their key
// range, numbered piece-major (piece p of every tail unit before piece p+1),
// so the last round is S times shorter.  Pieces leave unnormalised partials
// that attn_combine_kernel merges in piece order.
struct AttnItem {
  int32_t head, node, qt;
  int32_t ta, tb;   // key tiles [ta, tb) of the unit
  int32_t ntiles;   // key tiles of the whole unit
  int32_t slot;     // partial slot, or -1 for a whole unit
};

template <int KH>
__device__ __forceinline__ int32_t node_tiles(const AttnPlan& plan, const AttnGeom& g, int32_t node) {
  constexpr int BK = Tile<KH>::BK;
  return ((plan.page_off[node + 1] - plan.page_off[node]) * g.tpp + BK - 1) / BK;
}

template <int KH>
__device__ __forceinline__ AttnItem decode_item(const AttnPlan& plan, const AttnGeom& g, uint32_t b) {
  AttnItem it;
  int32_t unit;
  if (b < (uint32_t)g.whole_units) {
    unit = (int32_t)xcd_remap(b, (uint32_t)g.whole_units);
    it.slot = -1;
  } else {
    const int32_t j = (int32_t)xcd_remap(b - (uint32_t)g.whole_units,
                                         (uint32_t)(g.tail_units * g.tail_split));
    unit = g.whole_units + j % g.tail_units;
    it.slot = j;
  }
  it.qt = unit % g.n_qtiles;
  it.node = (unit / g.n_qtiles) % g.n_nodes;
  it.head = unit / (g.n_qtiles * g.n_nodes);
  it.ntiles = node_tiles<KH>(plan, g, it.node);
  if (it.slot < 0) {
    it.ta = 0;
    it.tb = it.ntiles;
  } else {
    const int32_t piece = it.slot / g.tail_units;
    it.ta = piece * it.ntiles / g.tail_split;
    it.tb = (piece + 1) * it.ntiles / g.tail_split;
  }
  return it;
}

// The result of a work item for one 16-query block: the normalised output
// of a whole unit, or a piece's unnormalised partial with its max and sum.
// oacc[db] holds, in lane (g, c) value r, O[query c][16 db + 4 g + r].
template <int BQ>
__device__ __forceinline__ void store_rows(const AttnItem& it, const AttnGeom& g, uint16_t* o,
                                           const f32x4 (&oacc)[8], float m_run, float l_run,
                                           int32_t lrow, int32_t lg) {
  const float l_tot = group_sum(l_run);
  if (it.slot < 0) {
    const float inv = 1.f / l_tot;
    const int32_t qrow = it.qt * BQ + lrow;
    if (qrow < g.nq) {
      uint16_t* op = o + (((size_t)it.node * g.nq + qrow) * g.n_heads + it.head) * HDB + 4 * lg;
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        u32x2 v;
        v.x = pack_bf16x2(oacc[db][0] * inv, oacc[db][1] * inv);
        v.y = pack_bf16x2(oacc[db][2] * inv, oacc[db][3] * inv);
        *reinterpret_cast<u32x2*>(op + 16 * db) = v;
      }
    }
  } else {
    float* po = g.part_o + ((size_t)it.slot * BQ + lrow) * HDB + 4 * lg;
#pragma unroll
    for (int db = 0; db < 8; ++db) *reinterpret_cast<f32x4*>(po + 16 * db) = oacc[db];
    if (lg == 0) {
      g.part_ml[((size_t)it.slot * 2 + 0) * BQ + lrow] = m_run;
      g.part_ml[((size_t)it.slot * 2 + 1) * BQ + lrow] = l_tot;
    }
  }
}

// S^T of one tile, s[h][b][qb] = K_(h,b) Q_qb^T - m_qb: all 4 KH
// accumulators advance together.
template <int KH>
__device__ __forceinline__ void qk_tile(const char* kl, const AttnLane& L, const bf16x8 (&qreg)[2][4],
                                        STile<KH>& s, const float (&m)[2]) {
  f32x4 acc[KH][2][2];
#pragma unroll
  for (int h = 0; h < KH; ++h)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[h][b][qb][r] = -m[qb];
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
#pragma unroll
    for (int h = 0; h < KH; ++h)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(kl + L.koff[b][ds] + h * 8192);
        acc[h][b][0] = mfma16(a, qreg[0][ds], acc[h][b][0]);
        acc[h][b][1] = mfma16(a, qreg[1][ds], acc[h][b][1]);
      }
#pragma unroll
  for (int h = 0; h < KH; ++h)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) s[h][b][qb] = acc[h][b][qb];
}

// O^T += V^T P^T for a tile whose V^T sits at vl.
template <int KH>
__device__ __forceinline__ void pv_tile(const char* vl, const AttnLane& L, const bf16x8 (&pb)[KH][2],
                                        f32x4 (&oacc)[2][8]) {
#pragma unroll
  for (int h = 0; h < KH; ++h)
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(vl + L.voff[h] + db * (16 * 2 * Tile<KH>::BK));
      oacc[0][db] = mfma16(a, pb[h][0], oacc[0][db]);
      oacc[1][db] = mfma16(a, pb[h][1], oacc[1][db]);
    }
}

// One step of the software-pipelined loop, for tile t: probabilities of
// S(t) (held in s), the next tile's S(t+1) = K(t+1) Q^T - m on the matrix
// cores while the exponentials of tile t run on the vector ALUs, then
// O^T += V(t)^T P(t) and the row sums lsum += 1^T P(t).  K runs one tile
// ahead of V: K(t+1) sits in K buffer KN, V(t) in V buffer VC.
template <int KH, int KN, int VC, bool NEXT, bool MASK>
__device__ __forceinline__ void attn_step(const char* smem, const AttnLane& L, const bf16x8 (&qreg)[2][4],
                                          f32x4 (&oacc)[2][8], STile<KH>& s, const float (&m)[2],
                                          f32x4 (&lsum)[2], const bf16x8& ones, int32_t t0, int32_t nk,
                                          int32_t lg) {
  using T = Tile<KH>;
  if constexpr (NEXT && !MASK && KH == 2) {
    // One stream of 32 fragment reads (the 16 K fragments of S(t+1), then
    // the 16 V^T fragments of tile t), each issued PF fragments ahead of the
    // two MFMAs it feeds; the 32 exponentials of P(t) ride two to a K group.
    // The fences keep that order: left to itself the compiler reads each
    // fragment just before its MFMAs, which then wait out the LDS latency.
    constexpr int PF = 4, NKF = 16, NF = 32;
    const char* kl = smem + KN * T::KT_BYTES;
    const char* vl = smem + 2 * T::KT_BYTES + VC * T::VT_BYTES;
    auto frag = [&](int i) -> bf16x8 {
      if (i < NKF) return *reinterpret_cast<const bf16x8*>(kl + L.koff[i & 1][i >> 2] + ((i >> 1) & 1) * 8192);
      const int j = i - NKF;
      return *reinterpret_cast<const bf16x8*>(vl + L.voff[j >> 3] + (j & 7) * (16 * 2 * T::BK));
    };
    STile<2> sn;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int r = 0; r < 4; ++r) sn[h][b][qb][r] = -m[qb];
    bf16x8 pb[2][2];
    bf16x8 ring[PF];
#pragma unroll
    for (int i = 0; i < PF; ++i) ring[i] = frag(i);
#pragma unroll
    for (int i = 0; i < NF; ++i) {
      const bf16x8 f = ring[i % PF];
      if (i + PF < NF) ring[i % PF] = frag(i + PF);
      if (i < NKF) {  // K fragment (ds, h, b) = (i / 4, i / 2 mod 2, i mod 2), as in qk_tile
        const int ds = i >> 2, h = (i >> 1) & 1, b = i & 1;
        sn[h][b][0] = mfma16(f, qreg[0][ds], sn[h][b][0]);
        sn[h][b][1] = mfma16(f, qreg[1][ds], sn[h][b][1]);
        const int ph = i >> 3, pq = (i >> 2) & 1, pe = 2 * (i & 3);  // pb[ph][pq] elements pe, pe + 1
        pb[ph][pq][pe] = static_cast<__bf16>(__builtin_amdgcn_exp2f(s[ph][pe >> 2][pq][pe & 3]));
        pb[ph][pq][pe + 1] = static_cast<__bf16>(__builtin_amdgcn_exp2f(s[ph][(pe + 1) >> 2][pq][(pe + 1) & 3]));
      } else {  // V^T fragment (h, db) = (j / 8, j mod 8), as in pv_tile
        const int j = i - NKF, h = j >> 3, db = j & 7;
        oacc[0][db] = mfma16(f, pb[h][0], oacc[0][db]);
        oacc[1][db] = mfma16(f, pb[h][1], oacc[1][db]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      lsum[0] = mfma16(ones, pb[h][0], lsum[0]);
      lsum[1] = mfma16(ones, pb[h][1], lsum[1]);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) s[h][b][qb] = sn[h][b][qb];
    return;
  }
  if constexpr (MASK) mask_tile<KH>(s, t0, nk, lg);
  bf16x8 pb[KH][2];
  probs<KH>(s, pb);
  STile<KH> sn;
  if constexpr (NEXT) qk_tile<KH>(smem + KN * T::KT_BYTES, L, qreg, sn, m);
  pv_tile<KH>(smem + 2 * T::KT_BYTES + VC * T::VT_BYTES, L, pb, oacc);
#pragma unroll
  for (int h = 0; h < KH; ++h) {
    lsum[0] = mfma16(ones, pb[h][0], lsum[0]);
    lsum[1] = mfma16(ones, pb[h][1], lsum[1]);
  }
  if constexpr (NEXT) {
#pragma unroll
    for (int h = 0; h < KH; ++h)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) s[h][b][qb] = sn[h][b][qb];
  }
}

// Exact two-pass redo of a work item in which a wave reached the 2^64 guard:
// each query's maximum logit over the item's keys, then the softmax from
// that maximum (every p <= 1).  Single-buffered K and V tiles; slow, and
// taken only for logits far above the first tile's maximum.
template <int NW, int KH>
__device__ __forceinline__ void attn_exact(char* smem, const KvTiles<NW, KH>& kv, const AttnLane& L,
                                           const bf16x8 (&qreg)[2][4], f32x4 (&oacc)[2][8], float (&m)[2],
                                           float (&l)[2], int32_t ta, int32_t ntiles, int32_t lg) {
  constexpr int BK = Tile<KH>::BK;
  char* const kl = smem;
  char* const vl = smem + 2 * Tile<KH>::KT_BYTES;
  const int32_t nk = kv.nk;
  const float zero[2] = {0.f, 0.f};
  float mx[2] = {-INFINITY, -INFINITY};
  for (int32_t t = ta; t < ntiles; ++t) {
    kv.copy_k(t * BK, kl, kv.slots(t * BK));
    landed();
    STile<KH> s;
    qk_tile<KH>(kl, L, qreg, s, zero);
    mask_tile<KH>(s, t * BK, nk, lg);
    float tm[2];
    tile_max<KH>(s, tm);
    mx[0] = fmaxf(mx[0], tm[0]);
    mx[1] = fmaxf(mx[1], tm[1]);
    __syncthreads();
  }
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    m[qb] = mx[qb];
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < 8; ++db) oacc[qb][db] = f32x4{};
  }
  for (int32_t t = ta; t < ntiles; ++t) {
    const typename KvTiles<NW, KH>::Slots sl = kv.slots(t * BK);
    kv.copy_k(t * BK, kl, sl);
    kv.copy_v(t * BK, vl, sl);
    landed();
    STile<KH> s;
    qk_tile<KH>(kl, L, qreg, s, m);
    mask_tile<KH>(s, t * BK, nk, lg);
    bf16x8 pb[KH][2];
    float lt[2];
    probs_tile<KH>(s, pb, lt);
    l[0] += lt[0];
    l[1] += lt[1];
    pv_tile<KH>(vl, L, pb, oacc);
    __syncthreads();
  }
}

// NW = 8: 256 queries per work-group, one work-group per CU; NW = 4: 128
// queries, two per CU; NW = 2: 64 queries, three or two per CU.  Each wave
// owns two 16-query blocks.  KH: 32-key halves per key tile; D: tiles of the
// K and of the V^T ring.  The long-context form (KH = 2, D = 2; NW = 8, 4)
// keeps one tile in flight, its buffer parity unrolled, two waves per SIMD.
// The streaming form (KH = 1, D = 3 or 4: runtime ring slots, D - 1 tiles in
// flight; NW = 2) serves nodes of at most 64 queries, whose attention
// streams K/V from HBM: it trades resident waves for copies in flight.
template <int NW, int KH, int D>
__global__ __launch_bounds__(64 * NW, NW == 8 || D == 4 ? 1 : 2) void attn_bf16_kernel(const uint16_t* __restrict__ q,
                                                                    uint16_t* __restrict__ o, AttnGeom g,
                                                                    AttnPlan plan) {
  constexpr int BQ = 32 * NW;
  using T = Tile<KH>;
  constexpr int BK = T::BK, KT_BYTES = T::KT_BYTES, VT_BYTES = T::VT_BYTES;
  static_assert((D == 2 && KH == 2) || (KH == 1 && (D == 3 || D == 4)), "ring depth");
  // K buffers 0 .. D-1 then V^T buffers 0 .. D-1 (KT_BYTES, VT_BYTES each)
  __shared__ __attribute__((aligned(1024))) char smem[D * (KT_BYTES + VT_BYTES)];
  __shared__ int32_t any_bad;
  const AttnItem it = decode_item<KH>(plan, g, blockIdx.x);
  if (it.ta == it.tb) return;  // empty piece of a unit shorter than the split
  const int32_t ta = it.ta, ntiles = it.tb;  // this item's key tiles: [ta, ntiles)
  const int32_t tid = threadIdx.x, lane = tid & 63;
  const int32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: LDS copy addresses stay scalar
  const int32_t lg = lane >> 4, c = lane & 15;
  if (tid == 0) any_bad = 0;
  const KvTiles<NW, KH> kv(plan, g, it.node, it.head, wave, lane);
  const int32_t nk = kv.nk;
  const bool ragged = it.tb == it.ntiles && (nk % BK) != 0;
  bf16x8 qreg[2][4];
  const AttnLane L = attn_lane<KH>(c, lg);

  f32x4 oacc[2][8];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int db = 0; db < 8; ++db) oacc[qb][db] = f32x4{};
  float m[2] = {0.f, 0.f}, l[2];
  f32x4 lsum[2] = {f32x4{}, f32x4{}};  // value 0 of lanes 0..15: row sums of the two blocks
  const bf16x8 ones = ones_row(c);
  // A wave whose 32 queries all lie past the node's end (in a node's last
  // query tile) still copies its share of every tile and meets every
  // barrier, but skips the matrix and softmax work.
  const bool active = it.qt * BQ + wave * 32 < g.nq;
  STile<KH> s;
  auto run = [&](auto act) __attribute__((always_inline)) {
    constexpr bool ACT = decltype(act)::value;
    // prologue: K(ta), V(ta), K(ta+1) in flight; S(ta) = K(ta) Q^T; m = its exact column maxima
    {
      const typename KvTiles<NW, KH>::Slots s0 = kv.slots(ta * BK);
      kv.copy_k(ta * BK, smem, s0);
      kv.copy_v(ta * BK, smem + 2 * KT_BYTES, s0);
      if (ta + 1 < ntiles) kv.copy_k((ta + 1) * BK, smem + KT_BYTES, kv.slots((ta + 1) * BK));
    }
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
      load_q(q, g, it.node, it.head, it.qt * BQ + wave * 32 + 16 * qb + c, lg, qreg[qb]);
    landed();
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) scale_q(g, qreg[qb]);
    if constexpr (ACT) {
      qk_tile<KH>(smem, L, qreg, s, m);
      if (ta + 1 == ntiles && ragged) mask_tile<KH>(s, ta * BK, nk, lg);
      tile_max<KH>(s, m);
#pragma unroll
      for (int h = 0; h < KH; ++h)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int r = 0; r < 4; ++r) s[h][b][qb][r] -= m[qb];
    }
    __syncthreads();  // every wave has read K(ta) before K(ta+2) is copied over it

    // iteration t (buffer parity counted from ta): copy K(t+2) over K(t) and
    // V(t+1) over V(t-1), then step t
    int32_t t = ta;
    typename KvTiles<NW, KH>::Slots sk = kv.slots(min(ta + 2, it.ntiles - 1) * BK);
    typename KvTiles<NW, KH>::Slots sv = kv.slots(min(ta + 1, it.ntiles - 1) * BK);
    for (; t + 2 < ntiles; t += 2) {
      kv.copy_k((t + 2) * BK, smem, sk);
      kv.copy_v((t + 1) * BK, smem + 2 * KT_BYTES + VT_BYTES, sv);
      if constexpr (ACT) attn_step<KH, 1, 0, true, false>(smem, L, qreg, oacc, s, m, lsum, ones, t * BK, nk, lg);
      // the next copies' page slots: their scalar loads share the LDS wait
      // counter, so they are issued after the step's fragment reads (a wait
      // for one fragment would otherwise wait for them too)
      __builtin_amdgcn_sched_barrier(0);
      sk = kv.slots(min(t + 3, it.ntiles - 1) * BK);
      sv = kv.slots(min(t + 2, it.ntiles - 1) * BK);
      landed();
      if (t + 3 < ntiles) kv.copy_k((t + 3) * BK, smem + KT_BYTES, sk);
      kv.copy_v((t + 2) * BK, smem + 2 * KT_BYTES, sv);
      if constexpr (ACT)
        attn_step<KH, 0, 1, true, false>(smem, L, qreg, oacc, s, m, lsum, ones, (t + 1) * BK, nk, lg);
      __builtin_amdgcn_sched_barrier(0);
      sk = kv.slots(min(t + 4, it.ntiles - 1) * BK);
      sv = kv.slots(min(t + 3, it.ntiles - 1) * BK);
      landed();
    }
    if (t + 1 < ntiles) {  // two tiles left, parity 0
      kv.copy_v((t + 1) * BK, smem + 2 * KT_BYTES + VT_BYTES, sv);
      if constexpr (ACT) attn_step<KH, 1, 0, true, false>(smem, L, qreg, oacc, s, m, lsum, ones, t * BK, nk, lg);
      landed();
      ++t;
      if constexpr (ACT) {
        if (ragged)
          attn_step<KH, 0, 1, false, true>(smem, L, qreg, oacc, s, m, lsum, ones, t * BK, nk, lg);
        else
          attn_step<KH, 0, 1, false, false>(smem, L, qreg, oacc, s, m, lsum, ones, t * BK, nk, lg);
      }
    } else if constexpr (ACT) {  // one tile left, parity 0 (masking twice is harmless)
      if (ragged)
        attn_step<KH, 1, 0, false, true>(smem, L, qreg, oacc, s, m, lsum, ones, t * BK, nk, lg);
      else
        attn_step<KH, 1, 0, false, false>(smem, L, qreg, oacc, s, m, lsum, ones, t * BK, nk, lg);
    }
  };
  // The ring form: tile r of the item (key tile ta + r) sits in K slot and
  // V^T slot r mod D.  Copies are issued in pairs (V(j), K(j + 1)), j = 1,
  // 2, ...: pairs up to D - 2 in the prologue, pair r + D - 1 at step r into
  // the slots steps r - 1 (V) and r - 1 (K, read by the QK of step r - 1)
  // have finished with.  After step r, tiles K(r + 2) and V(r + 1) (pair
  // r + 1) must have landed: the wait leaves the copies of the later pairs
  // in flight, counted exactly (a pair past the item's end issues nothing).
  auto run_ring = [&](auto act) __attribute__((always_inline)) {
    constexpr bool ACT = decltype(act)::value;
    using KV = KvTiles<NW, KH>;
    constexpr int32_t KC = KV::KCP, VC = KV::VCP;
    static_assert(KC % 2 == 0 && VC % 2 == 0 && (D - 2) * (KC + VC) <= 16, "wait counts of landed_but");
    const int32_t n = ntiles - ta;
    auto kbuf = [&](int32_t r) { return smem + (r % D) * KT_BYTES; };
    auto vbuf = [&](int32_t r) { return smem + D * KT_BYTES + (r % D) * VT_BYTES; };
    // copies of pair j (relative tiles); returns nothing, issues V(j) if it
    // exists, then K(j + 1) if it exists
    auto issue_pair = [&](int32_t j) __attribute__((always_inline)) {
      if (j < n) kv.copy_v((ta + j) * BK, vbuf(j), kv.slots((ta + j) * BK));
      if (j + 1 < n) kv.copy_k((ta + j + 1) * BK, kbuf(j + 1), kv.slots((ta + j + 1) * BK));
    };
    // copy instructions of pairs a .. b issued by this wave: V(j) for j < n,
    // K(j + 1) for j < n - 1
    auto copies = [&](int32_t a, int32_t b) {
      return VC * max(0, min(b, n - 1) - a + 1) + KC * max(0, min(b, n - 2) - a + 1);
    };
    {
      const typename KV::Slots s0 = kv.slots(ta * BK);
      kv.copy_k(ta * BK, kbuf(0), s0);
      kv.copy_v(ta * BK, vbuf(0), s0);
      if (n > 1) kv.copy_k((ta + 1) * BK, kbuf(1), kv.slots((ta + 1) * BK));
    }
    if constexpr (ACT) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
        load_q(q, g, it.node, it.head, it.qt * BQ + wave * 32 + 16 * qb + c, lg, qreg[qb]);
    }
    landed();
    for (int32_t j = 1; j <= D - 2; ++j) issue_pair(j);
    if constexpr (ACT) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) scale_q(g, qreg[qb]);
      qk_tile<KH>(kbuf(0), L, qreg, s, m);
      if (n == 1 && ragged) mask_tile<KH>(s, ta * BK, nk, lg);
      tile_max<KH>(s, m);
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int r = 0; r < 4; ++r) s[0][b][qb][r] -= m[qb];
    } else {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) qreg[qb][ds] = bf16x8{};  // defined values for the exact redo
    }
    landed_but(copies(1, D - 2));  // K(ta) read by every wave before pair D - 1 overwrites its slot
    for (int32_t r = 0; r + 1 < n; ++r) {
      issue_pair(r + D - 1);
      if constexpr (ACT) {
        // step r with runtime slots: the same arithmetic as attn_step
        bf16x8 pb[KH][2];
        probs<KH>(s, pb);
        STile<KH> sn;
        qk_tile<KH>(kbuf(r + 1), L, qreg, sn, m);
        if (r + 2 == n && ragged) mask_tile<KH>(sn, (ta + r + 1) * BK, nk, lg);
        pv_tile<KH>(vbuf(r), L, pb, oacc);
#pragma unroll
        for (int h = 0; h < KH; ++h) {
          lsum[0] = mfma16(ones, pb[h][0], lsum[0]);
          lsum[1] = mfma16(ones, pb[h][1], lsum[1]);
        }
#pragma unroll
        for (int h = 0; h < KH; ++h)
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) s[h][b][qb] = sn[h][b][qb];
      }
      landed_but(copies(r + 2, r + D - 1));
    }
    if constexpr (ACT) {  // the last tile (already masked if ragged)
      bf16x8 pb[KH][2];
      probs<KH>(s, pb);
      pv_tile<KH>(vbuf(n - 1), L, pb, oacc);
#pragma unroll
      for (int h = 0; h < KH; ++h) {
        lsum[0] = mfma16(ones, pb[h][0], lsum[0]);
        lsum[1] = mfma16(ones, pb[h][1], lsum[1]);
      }
    }
  };
  if constexpr (D == 2) {
    if (active)
      run(std::true_type{});
    else
      run(std::false_type{});
  } else {
    if (active)
      run_ring(std::true_type{});
    else
      run_ring(std::false_type{});
  }
  // the guard, on the final sums (also NaN / inf)
  const bool bad = __builtin_amdgcn_ballot_w64(!(lsum[0][0] < P_GUARD && lsum[1][0] < P_GUARD)) != 0;
  l[0] = lsum[0][0];  // zero outside lanes 0..15, so the group sum is the row sum
  l[1] = lsum[1][0];
  if (bad && lane == 0) atomicOr(&any_bad, 1);
  __syncthreads();  // every wave is done with the ring; any_bad is final
  if (any_bad) attn_exact(smem, kv, L, qreg, oacc, m, l, ta, ntiles, lg);
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) store_rows<BQ>(it, g, o, oacc[qb], m[qb], l[qb], wave * 32 + 16 * qb + c, lg);
}

// Merges the pieces of each tail unit, in piece order.  A work-group takes 8
// query rows of one tail unit; 32 lanes share a row, each holding 4 of its
// 128 outputs, so every partial row is read as one contiguous 512-byte run.
// With m = max m_p:
//   O = sum_p 2^(m_p - m) O_p / sum_p 2^(m_p - m) l_p.
template <int BQ, int KH>
__global__ __launch_bounds__(256) void attn_combine_kernel(uint16_t* __restrict__ o, AttnGeom g, AttnPlan plan) {
  const int32_t tu = blockIdx.x;
  const int32_t unit = g.whole_units + tu;
  const int32_t qt = unit % g.n_qtiles;
  const int32_t node = (unit / g.n_qtiles) % g.n_nodes;
  const int32_t head = unit / (g.n_qtiles * g.n_nodes);
  const int32_t lrow = blockIdx.y * 8 + (threadIdx.x >> 5);
  const int32_t dl = threadIdx.x & 31;
  const int32_t qrow = qt * BQ + lrow;
  if (qrow >= g.nq) return;
  const int32_t nt = node_tiles<KH>(plan, g, node);
  auto nonempty = [&](int32_t p) { return p * nt / g.tail_split < (p + 1) * nt / g.tail_split; };
  float m = -INFINITY;
  for (int32_t p = 0; p < g.tail_split; ++p)
    if (nonempty(p)) m = fmaxf(m, g.part_ml[((size_t)(p * g.tail_units + tu) * 2 + 0) * BQ + lrow]);
  f32x4 acc = {};
  float l = 0.f;
  for (int32_t p = 0; p < g.tail_split; ++p) {
    if (!nonempty(p)) continue;
    const size_t slot = (size_t)p * g.tail_units + tu;
    const float a = __builtin_amdgcn_exp2f(g.part_ml[(slot * 2 + 0) * BQ + lrow] - m);
    l += a * g.part_ml[(slot * 2 + 1) * BQ + lrow];
    const f32x4 v = *reinterpret_cast<const f32x4*>(g.part_o + (slot * BQ + lrow) * HDB + 4 * dl);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] += a * v[e];
  }
  const float inv = 1.f / l;
  u32x2 r;
  r.x = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  r.y = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  *reinterpret_cast<u32x2*>(o + (((size_t)node * g.nq + qrow) * g.n_heads + head) * HDB + 4 * dl) = r;
}

// Tail split for a plan: units = heads x nodes x query tiles; the last
// (units mod resident work-groups) are cut into S pieces, S chosen to
// minimise the tail's rounds (in units of one whole unit) plus a per-piece
// cost of about two key tiles (prologue and partial write), with at most
// max_pieces pieces and no more pieces than the shortest node has key
// tiles.
// The kernel form for a plan: queries per work-group (the smallest of 64,
// 128, 256 that holds a node), 32-key halves per key tile and ring depth.
// Nodes of at most 64 queries take the streaming form (ring 4 when the units
// fit the 512 work-groups resident with it, else ring 3 with 768); larger
// ones the long-context form.  (The streaming form with 128 queries per
// work-group measured 2-8 % slower than the long-context one on the
// short-context sweep: its 32-key steps cost more than the deeper ring
// gains.)
struct AttnShape {
  int32_t bq, kh, ring;
};
static int32_t shape_queries(int32_t nq) { return nq <= BQ_TINY ? BQ_TINY : nq <= BQ_SMALL ? BQ_SMALL : BQ_MAX; }
// Work-groups resident per CU: at most 8 waves (256 VGPRs each, 2 per SIMD)
// and 160 KB of LDS, 2 x ring x 8 KB per streaming work-group.
static int32_t per_cu(const AttnShape& s) {
  const int32_t by_vgpr = 8 / (s.bq / 32);
  return s.kh == 2 ? by_vgpr : std::min(by_vgpr, (160 * 1024) / (s.ring * 16 * 1024 + 4));
}
static AttnShape attn_shape(const sc_plan* p, const sc_cache* c) {
  AttnShape s;
  s.bq = shape_queries(p->nq);
  s.kh = s.bq == BQ_TINY ? 1 : 2;
  s.ring = 2;
  if (s.kh == 1) {
    const int32_t units = (int32_t)p->nodes.size() * c->d.n_heads * ((p->nq + s.bq - 1) / s.bq);
    s.ring = 4;
    if (units > kCUs * per_cu(s)) s.ring = 3;
  }
  return s;
}

struct TailSplit {
  AttnShape sh;
  int32_t whole, tail, split;
};
static TailSplit tail_split(const sc_plan* p, const sc_cache* c, int32_t max_pieces = kAttnMaxPieces) {
  const int32_t n = (int32_t)p->nodes.size();
  TailSplit ts;
  ts.sh = attn_shape(p, c);
  const int32_t bq = ts.sh.bq, bk = 32 * ts.sh.kh;
  const int32_t n_qtiles = (p->nq + bq - 1) / bq;
  const int32_t units = n * c->d.n_heads * n_qtiles;
  int64_t tiles = 0;
  int32_t min_tiles = INT32_MAX;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t nt = (int32_t)(((int64_t)(p->page_off[i + 1] - p->page_off[i]) * c->d.tokens_per_page +
                                  bk - 1) / bk);
    tiles += nt;
    min_tiles = std::min(min_tiles, nt);
  }
  const double mean_tiles = (double)tiles / std::max(n, 1);
  const int32_t slots = kCUs * per_cu(ts.sh);  // work-groups resident at once
  ts.tail = units % slots;
  ts.whole = units - ts.tail;
  ts.split = 1;
  // Short units are not cut: the combine launch and the partial traffic are
  // fixed costs that a few-tile unit cannot repay (measured on the short
  // K/V streaming sweep).  The threshold is in 64-key tiles.
  if (ts.tail == 0 || mean_tiles * bk < kAttnMinSplitTiles * 64) return ts;
  double best = 1e30;
  const int32_t smax = std::max(1, std::min({16, max_pieces / ts.tail, min_tiles}));
  for (int32_t sp = 1; sp <= smax; ++sp) {
    const double rounds = (double)((ts.tail * sp + slots - 1) / slots);
    const double cost = rounds * (1.0 / sp + 2.0 / mean_tiles);
    if (cost < best - 1e-9) {
      best = cost;
      ts.split = sp;
    }
  }
  return ts;
}

size_t attention_workspace_bytes(const sc_plan* p, const sc_cache* c) {
  if (c->d.dtype != SC_DTYPE_BF16 || p->nodes.empty()) return 0;
  const TailSplit ts = tail_split(p, c);
  if (ts.split == 1) return 0;
  return (size_t)ts.tail * ts.split * ts.sh.bq * (HDB + 2) * sizeof(float);
}

size_t attention_workspace_bound() { return (size_t)kAttnMaxPieces * BQ_MAX * (HDB + 2) * sizeof(float); }

int attention_check(const sc_plan* p, const sc_cache* c) {
  const sc_cache_desc& d = c->d;
  const int32_t n = (int32_t)p->nodes.size();
  if (n > kMaxNodes) return fail(SC_EUNSUPPORTED, "pack of %d nodes exceeds %d", n, kMaxNodes);
  if ((int32_t)p->page_slot.size() > kMaxPages)
    return fail(SC_EUNSUPPORTED, "plan of %zu pages exceeds %d", p->page_slot.size(), kMaxPages);
  if (d.dtype == SC_DTYPE_F32) return SC_OK;
  if (d.head_dim != HDB) return fail(SC_EUNSUPPORTED, "bf16 attention needs head_dim 128");
  const int32_t bk = 32 * attn_shape(p, c).kh;  // a key tile spans at most two pages
  if (d.tokens_per_page < bk)
    return fail(SC_EUNSUPPORTED, "bf16 attention of %d-query nodes needs pages of >= %d tokens (got %d)",
                p->nq, bk, d.tokens_per_page);
  if ((uint64_t)d.n_slots * c->slot_bytes > 0xffffffffull)
    return fail(SC_EUNSUPPORTED, "bf16 attention needs one layer of the pool within 4 GB");
  return SC_OK;
}

// Page lists in a traversal order shared by the pack's nodes.  The softmax
// sum does not depend on the order of a node's keys, so each node's list (its
// states' pages, oldest state first) is rotated to start at the anchor: the
// state read by the most nodes, the oldest of those.  Nodes of a progressive
// or same-level pack read overlapping windows of consecutive chunks; rotated
// this way, their work-groups read the shared states at the same time
// instead of one chunk apart.
// The order is a property of the plan alone: computed on its first launch
// and kept in it (a plan is immutable once built).
static void shared_order(const sc_plan* p, AttnPlan& plan) {
  const int32_t n = (int32_t)p->nodes.size();
  if (p->attn_slot.size() != p->page_slot.size()) {
    std::map<StateKey, int32_t> readers;
    for (int32_t i = 0; i < n; ++i)
      for (int32_t q = p->page_off[i]; q < p->page_off[i + 1]; ++q)
        if (q == p->page_off[i] || p->page_state[q] != p->page_state[q - 1]) ++readers[p->page_state[q]];
    StateKey anchor(INT32_MIN, INT32_MIN);
    int32_t most = 0;
    for (const auto& kv : readers)  // ascending (chunk, level): the oldest wins ties
      if (kv.second > most) {
        most = kv.second;
        anchor = kv.first;
      }
    std::vector<int32_t> order(p->page_slot.size());
    for (int32_t i = 0; i < n; ++i) {
      const int32_t a = p->page_off[i], b = p->page_off[i + 1];
      int32_t r = a;
      while (r < b && p->page_state[r] < anchor) ++r;
      if (r == b) r = a;
      int32_t o = a;
      for (int32_t q = r; q < b; ++q) order[o++] = p->page_slot[q];
      for (int32_t q = a; q < r; ++q) order[o++] = p->page_slot[q];
    }
    p->attn_slot.swap(order);
  }
  for (int32_t i = 0; i <= n; ++i) plan.page_off[i] = p->page_off[i];
  std::copy(p->attn_slot.begin(), p->attn_slot.end(), plan.page_slot);
}

// The launch of a plan whose split uses at most max_pieces pieces.
static int launch_attention_pieces(const sc_plan* p, const sc_cache* c, int32_t layer, const void* q,
                                   void* o, float scale, void* ws, size_t ws_bytes, int32_t max_pieces,
                                   hipStream_t stream);

int launch_attention(const sc_plan* p, const sc_cache* c, int32_t layer, const void* q, void* o,
                     float scale, void* ws, size_t ws_bytes, hipStream_t stream) {
  return launch_attention_pieces(p, c, layer, q, o, scale, ws, ws_bytes, kAttnMaxPieces, stream);
}

static int launch_attention_pieces(const sc_plan* p, const sc_cache* c, int32_t layer, const void* q,
                                   void* o, float scale, void* ws, size_t ws_bytes, int32_t max_pieces,
                                   hipStream_t stream) {
  const sc_cache_desc& d = c->d;
  const int32_t n = (int32_t)p->nodes.size();
  const int rc = attention_check(p, c);
  if (rc != SC_OK) return rc;
  AttnPlan plan;
  shared_order(p, plan);
  AttnGeom g;
  std::memset(&g, 0, sizeof g);
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
  if (d.dtype == SC_DTYPE_F32) {
    g.n_qtiles = (p->nq + 63) / 64;
    const uint32_t nwg = (uint32_t)n * d.n_heads * g.n_qtiles;
    timer_begin(TK_ATTENTION, stream);
    if (d.head_dim == 64)
      hipLaunchKernelGGL((attn_f32_kernel<64>), dim3(nwg), dim3(64), 0, stream,
                         static_cast<const float*>(q), static_cast<float*>(o), g, plan);
    else
      hipLaunchKernelGGL((attn_f32_kernel<128>), dim3(nwg), dim3(64), 0, stream,
                         static_cast<const float*>(q), static_cast<float*>(o), g, plan);
    timer_end(TK_ATTENTION, stream);
    SC_HIP(hipGetLastError());
    return SC_OK;
  }
  const TailSplit ts = tail_split(p, c, max_pieces);
  const size_t need = ts.split == 1 ? 0 : (size_t)ts.tail * ts.split * ts.sh.bq * (HDB + 2) * sizeof(float);
  if (ws_bytes < need || (need && !ws))
    return fail(SC_EINVAL, "attention workspace of %zu bytes, need %zu", ws_bytes, need);
  if (reinterpret_cast<uintptr_t>(ws) & 15) return fail(SC_EINVAL, "workspace must be 16-byte aligned");
  const int32_t bq = ts.sh.bq;
  g.n_qtiles = (p->nq + bq - 1) / bq;
  g.whole_units = ts.whole;
  g.tail_units = ts.tail;
  g.tail_split = ts.split;
  if (ts.split == 1) {  // no pieces: the tail units run whole
    g.whole_units += ts.tail;
    g.tail_units = 0;
  }
  g.part_o = static_cast<float*>(ws);
  g.part_ml = g.part_o + (size_t)g.tail_units * g.tail_split * bq * HDB;
  const uint32_t items = (uint32_t)(g.whole_units + g.tail_units * g.tail_split);
  const uint16_t* qb = static_cast<const uint16_t*>(q);
  uint16_t* ob = static_cast<uint16_t*>(o);
  timer_begin(TK_ATTENTION, stream);
  const int32_t ring = ts.sh.ring;
  if (bq == BQ_TINY && ring == 4)
    hipLaunchKernelGGL((attn_bf16_kernel<2, 1, 4>), dim3(items), dim3(128), 0, stream, qb, ob, g, plan);
  else if (bq == BQ_TINY)
    hipLaunchKernelGGL((attn_bf16_kernel<2, 1, 3>), dim3(items), dim3(128), 0, stream, qb, ob, g, plan);
  else if (bq == BQ_SMALL)
    hipLaunchKernelGGL((attn_bf16_kernel<4, 2, 2>), dim3(items), dim3(256), 0, stream, qb, ob, g, plan);
  else
    hipLaunchKernelGGL((attn_bf16_kernel<8, 2, 2>), dim3(items), dim3(512), 0, stream, qb, ob, g, plan);
  timer_end(TK_ATTENTION, stream);
  if (g.tail_units) {
    timer_begin(TK_ATTN_COMBINE, stream);
    const dim3 grid((uint32_t)g.tail_units, (uint32_t)bq / 8);
    if (bq == BQ_TINY)
      hipLaunchKernelGGL((attn_combine_kernel<BQ_TINY, 1>), grid, dim3(256), 0, stream, ob, g, plan);
    else if (bq == BQ_SMALL)
      hipLaunchKernelGGL((attn_combine_kernel<BQ_SMALL, 2>), grid, dim3(256), 0, stream, ob, g, plan);
    else
      hipLaunchKernelGGL((attn_combine_kernel<BQ_MAX, 2>), grid, dim3(256), 0, stream, ob, g, plan);
    timer_end(TK_ATTN_COMBINE, stream);
  }
  SC_HIP(hipGetLastError());
  return SC_OK;
}

// ------------------------------------------------ attention without allocation
// The split-key partials of sc_attention_noalloc live in this library-owned
// array; every GPU the library runs on holds its own copy until the process
// ends.  Host code never passes the array's name to a kernel (on the host it
// is a stand-in, not a device address): the device address comes from
// hipGetSymbolAddress, once per device, with that device current.
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

static std::mutex g_scratch_mu;
static std::map<int, void*> g_scratch_ptr;  // device ordinal -> address of its scratch

static int scratch_address(void** out) {
  int dev = -1;
  SC_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it == g_scratch_ptr.end()) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!ptr || (reinterpret_cast<uintptr_t>(ptr) & 255))
      return fail(SC_EDEVICE, "scratch of device %d at unusable address %p", dev, ptr);
    it = g_scratch_ptr.emplace(dev, ptr).first;
  }
  *out = it->second;
  return SC_OK;
}

}  // namespace sc

extern "C" size_t sc_attention_noalloc_scratch_bytes(void) { return sc::kNoAllocScratchBytes; }

extern "C" int sc_attention_noalloc(const sc_plan* p, const sc_cache* c, int32_t layer, const void* q,
                                    void* o, float scale, sc_stream stream) {
  using namespace sc;
  if (!p || !c || !q || !o) return fail(SC_EINVAL, "null argument");
  int rc = plan_check(p, c, layer);
  if (rc != SC_OK) return rc;
  if (p->nodes.empty()) return SC_OK;
  if ((rc = attention_check(p, c)) != SC_OK) return rc;
  void* ptr = nullptr;
  if (c->d.dtype == SC_DTYPE_BF16 && (rc = scratch_address(&ptr)) != SC_OK) return rc;
  // as many key-range pieces as the scratch holds partials for
  const int32_t bq = attn_shape(p, c).bq;
  const size_t piece_bytes = (size_t)bq * (HDB + 2) * sizeof(float);
  const int32_t max_pieces = (int32_t)std::min<size_t>(kAttnMaxPieces, kNoAllocScratchBytes / piece_bytes);
  const TailSplit ts = tail_split(p, c, max_pieces);
  const size_t need = ts.split == 1 ? 0 : (size_t)ts.tail * ts.split * piece_bytes;
  if (need > kNoAllocScratchBytes)
    return fail(SC_ECAPACITY, "attention partials of %zu bytes exceed the %zu-byte scratch", need,
                kNoAllocScratchBytes);
  return launch_attention_pieces(p, c, layer, q, o, scale, ptr, ptr ? kNoAllocScratchBytes : 0, max_pieces,
                                 static_cast<hipStream_t>(stream));
}
