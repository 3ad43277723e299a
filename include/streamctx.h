/*
 * streamctx -- packed causal-context DiT step on MI355X (gfx950).
 *
 * C ABI of the hot path of progressive-history pipelining from "Rethinking
 * Streaming Video Diffusion Model: Context, Execution, and Training":
 * several in-flight denoising nodes (chunk, level) run as one forward, and
 * every node attends over the cached keys/values of the historical states its
 * context policy selects.
 *
 * Conventions shared by every call
 *  - Return codes: SC_OK (0) or a negative SC_E* code.  The message of the
 *    last failing call on the calling thread is returned by sc_last_error().
 *    No C++ exception crosses this boundary.
 *  - Nodes: chunk c is 0-based (the paper's b = c + 1); level 0 is the clean
 *    endpoint x^0 and level K the initial noise x^K (Sec. 3.1).
 *  - Device pointers are plain HIP device addresses owned by the caller; the
 *    library never allocates device memory.  Device work is enqueued on the
 *    given stream (sc_stream is a hipStream_t; NULL is the null stream) and
 *    runs asynchronously.  Host-side table work completes before the call
 *    returns.
 *  - Handles are not thread-safe; one handle is used by one thread at a time.
 *  - bf16 tensors are raw bfloat16 bit patterns (uint16), fp32 tensors IEEE
 *    binary32.
 */
#ifndef STREAMCTX_H
#define STREAMCTX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SC_ABI_VERSION 7

enum {
  SC_OK = 0,
  SC_EINVAL = -1,        /* bad argument, policy or node set            */
  SC_EUNAVAILABLE = -2,  /* a selected state is neither cached nor produced in the pack */
  SC_ECAPACITY = -3,     /* not enough free page slots                  */
  SC_EEXIST = -4,        /* state's K/V for this layer already written  */
  SC_ENOTFOUND = -5,     /* state not in the cache                      */
  SC_ESTALE = -6,        /* plan refers to a slot released since it was built */
  SC_EDEVICE = -7,       /* HIP runtime error                           */
  SC_EUNSUPPORTED = -8   /* shape or dtype this build has no kernel for */
};

enum { SC_POLICY_CLEAN = 0, SC_POLICY_SAME = 1, SC_POLICY_PROG = 2, SC_POLICY_TABLE = 3 };
enum { SC_DTYPE_BF16 = 0, SC_DTYPE_F32 = 1 };

typedef void* sc_stream; /* hipStream_t */

typedef struct {
  int32_t chunk; /* 0-based chunk index c              */
  int32_t level; /* noise level j, 0 (clean) .. K      */
} sc_node;

/* History selection policy, Sec. 3.2 Eq. 4-5.  For a node (c, j) the offsets
 * r = min(W, c) .. 1 with r_mask[j*W + r-1] != 0 (all of them when r_mask is
 * NULL) select the state of chunk c - r at level phi(j, r):
 *   SC_POLICY_CLEAN  phi = 0
 *   SC_POLICY_SAME   phi = j
 *   SC_POLICY_PROG   phi = max(j - r, 0)
 *   SC_POLICY_TABLE  phi = phi_table[j*W + r-1]   (entries in [0, K])
 * Position-dependent policies (Eq. 4's Phi_b and R_b,j may depend on the
 * chunk): with n_chunks > 0 the tables gain a leading chunk index --
 * phi_table[(c*(K+1) + j)*W + r-1] and r_mask[(c*(K+1) + j)*W + r-1] -- and
 * every node must have c < n_chunks.  The arrays are read during the call
 * only (sc_selection_build, sc_cache_release_unread). */
typedef struct {
  int32_t kind;
  int32_t K;                 /* number of noise levels above clean, >= 1 */
  int32_t W;                 /* history window in chunks, >= 0           */
  const int8_t* phi_table;   /* [n_chunks x] (K+1) x W, kind TABLE only, else NULL */
  const uint8_t* r_mask;     /* [n_chunks x] (K+1) x W, or NULL (dense offsets)    */
  int32_t n_chunks;          /* 0: tables independent of the chunk          */
} sc_policy;

typedef struct sc_selection sc_selection;
typedef struct sc_cache sc_cache;
typedef struct sc_plan sc_plan;

int sc_abi_version(void);
const char* sc_last_error(void);
const char* sc_status_name(int status);

/* ---- Selection table (Sec. 3.2, Eq. 4-5) -------------------------------
 * Builds the canonical table of a pack of n distinct nodes (pack order is the
 * caller's).  Node i's segments are its selected history states from the
 * oldest chunk to the newest, then its own state (c, j): a query chunk sees
 * its own tokens (Eq. 6 text: within-chunk attention is bidirectional).
 * seg_src[s] is the index of the pack node that produces state s in this
 * pack (in-pack history, or the node itself), else -1 (must be cached).
 * Errors: SC_EINVAL for K < 1, W < 0, n_chunks < 0, an unknown kind, a phi
 * entry outside [0, K], a node with chunk < 0 (or >= n_chunks when
 * n_chunks > 0) or level outside [0, K], or a duplicate node.
 * The returned handle owns every array; free it with sc_selection_free. */
int sc_selection_build(const sc_policy* policy, const sc_node* nodes, int32_t n,
                       sc_selection** out);
int sc_selection_get(const sc_selection* sel, int32_t* n_nodes, int32_t* n_segments,
                     const int32_t** seg_off, const int32_t** seg_chunk,
                     const int32_t** seg_level, const int32_t** seg_src);
/* Node-level visibility (the chunk-level form of Eq. 6's mask M): the
 * distinct states read by the pack, sorted by (chunk, level), and a row-major
 * n_nodes x n_states 0/1 matrix. */
int sc_visibility_get(const sc_selection* sel, int32_t* n_states, const sc_node** states,
                      const uint8_t** vis);
void sc_selection_free(sc_selection* sel);

/* ---- Paged history KV cache (Sec. 3.2, "Effective context") ------------
 * The representations of selected states are cached keys/values.  One page
 * slot holds one latent frame (tokens_per_page tokens) of one state, for
 * every layer; a state occupies pages_per_chunk slots, the same slot ids in
 * every layer.  The pool is caller device memory of sc_cache_pool_bytes():
 *   pool[layer][slot] = { K[head][token][d], V[head][d][token] }
 * (V is stored transposed: the attention kernel reads it as the A operand of
 * O^T = V^T P^T).  Slots are handed out lowest-free-first.  Requirements:
 * tokens_per_page a positive multiple of 8, head_dim 64 or 128 (bf16: 128).
 * The pool must outlive the cache handle. */
typedef struct {
  int32_t n_layers, n_heads, head_dim, tokens_per_page, pages_per_chunk, n_slots, dtype;
} sc_cache_desc;

size_t sc_cache_pool_bytes(const sc_cache_desc* desc);
int sc_cache_create(const sc_cache_desc* desc, void* dev_pool, sc_cache** out);
void sc_cache_free(sc_cache* cache);
/* 1 when the state holds slots (appended or reserved by a plan), 0 if not;
 * with layer >= 0, 1 only when that layer has been written. */
int sc_cache_contains(const sc_cache* cache, sc_node state, int32_t layer);
/* Copies the state's pages_per_chunk slot ids to slots[]. SC_ENOTFOUND. */
int sc_cache_slots(const sc_cache* cache, sc_node state, int32_t* slots);
int sc_cache_free_slot_count(const sc_cache* cache);
/* Frees the state's slots in every layer and bumps their generation, so a
 * plan that still names them fails with SC_ESTALE.  SC_ENOTFOUND. */
int sc_cache_release(sc_cache* cache, sc_node state);

/* ---- 3D RoPE table ------------------------------------------------------
 * The paper does not define the positional encoding; this follows the
 * Wan-shaped workload: head_dim split into dim_t + dim_h + dim_w channels
 * (44/42/42 for 128), interleaved pairs, pair i of axis a rotated by
 * pos_a * theta^(-2 i / dim_a); token n of frame f of chunk c sits at
 * (t, h, w) = (c * pages_per_chunk + f, n / grid_w, n % grid_w).
 * The table holds cos/sin per (position, pair) for each axis, in fp32,
 * computed on the device in double precision; build it once. */
typedef struct {
  int32_t grid_h, grid_w, dim_t, dim_h, dim_w, max_frames;
  float theta;
} sc_rope_desc;
typedef struct {
  sc_rope_desc desc;
  const void* dev_table; /* built by sc_rope_table_build */
} sc_rope;
size_t sc_rope_table_bytes(const sc_rope_desc* desc);
int sc_rope_table_build(const sc_rope_desc* desc, void* dev_table, sc_stream stream);

/* Writes the K/V of one state for one layer into its page slots (allocating
 * them, lowest free first, unless a plan reserved them).  k, v: device
 * [pages_per_chunk * tokens_per_page, n_heads, head_dim] in the cache dtype,
 * read asynchronously on the stream.  With rope != NULL the keys are rotated
 * at the state's absolute positions first (grid_h * grid_w must equal
 * tokens_per_page).  Errors: SC_EEXIST (layer already written),
 * SC_ECAPACITY, SC_EINVAL, SC_EDEVICE. */
int sc_cache_append(sc_cache* cache, int32_t layer, sc_node state, const void* k,
                    const void* v, const sc_rope* rope, sc_stream stream);

/* ---- Plan: availability and page lists (Eq. 6, Eq. 8) ------------------
 * Resolves every segment of the selection to page slots and checks
 * availability: a state read by a node must be in the cache or produced by
 * the pack (Sec. 3.3, "Restrictions on context selection"; for Eq. 7 packs
 * this is Eq. 8).  Pack states not yet cached get slots reserved now, in pack
 * order.  Node i's pages are its segments' frames, in segment order.
 * Errors: SC_EUNAVAILABLE, SC_ECAPACITY (the cache is unchanged on error).
 * The plan stays valid for every layer until one of its slots is released. */
int sc_plan_build(const sc_selection* sel, sc_cache* cache, sc_plan** out);
int sc_plan_get(const sc_plan* plan, int32_t* n_nodes, int32_t* n_pages,
                const int32_t** page_off, const int32_t** page_slot,
                const int32_t** page_tokens, const int32_t** page_frame);
void sc_plan_free(sc_plan* plan);

/* Plan over a condition cache: the condition c of Eq. 1 (e.g. text tokens)
 * is read by every query of a node, with no visibility mask and no position.
 * Node i of a pack reads all pages of the cached state conditions[i]
 * (several nodes may name one state), with nq query rows per node -- the
 * nq of the pack's own plan.  Each state must hold slots in the cache
 * (written by sc_condition_append or sc_cache_append); whether a layer has
 * been written is checked when the plan is used.  Errors: SC_EINVAL (null
 * argument, n < 1 or nq < 1), SC_ENOTFOUND (a state not in the cache). */
int sc_plan_condition(sc_cache* cache, const sc_node* conditions, int32_t n, int32_t nq,
                      sc_plan** out);

/* ---- Packed block-causal attention (Eq. 6 over the plan) ---------------
 * For every pack node i and head h:
 *   O_i = softmax(Q_i K_i^T * scale) V_i
 * where K_i, V_i are the keys/values of node i's pages at this layer -- the
 * tokens Eq. 6's mask leaves visible; no dense mask is formed.
 * q, o: device [n_nodes * Nq, n_heads, head_dim] in the cache dtype, node i
 * at rows [i*Nq, (i+1)*Nq) with Nq = pages_per_chunk * tokens_per_page.
 * Every page must have been written at this layer by calls enqueued earlier
 * on the same stream.  Limits of this build: at most 64 pack nodes and 800
 * pages per plan (the page lists travel by value in the kernel arguments, so
 * no per-round host-to-device copy is needed); larger plans fail with
 * SC_EUNSUPPORTED before anything is launched.  bf16 caches need head_dim
 * 128 and pages of at least one key tile: 32 tokens when Nq <= 64, 64
 * otherwise (else SC_EUNSUPPORTED).  ws: device scratch, 16-byte aligned, of at least
 * sc_attention_workspace_bytes(plan, cache) bytes (may be NULL when that is
 * 0, as for fp32 caches); the bf16 kernel splits long key ranges across
 * work-groups and merges their partial softmax sums there.  Its contents are
 * undefined on return; calls sharing one workspace must be ordered on one
 * stream.  Errors: SC_ESTALE, SC_EUNAVAILABLE (a page's state not written at
 * this layer), SC_EINVAL (workspace too small or misaligned), SC_EUNSUPPORTED,
 * SC_EDEVICE. */
size_t sc_attention_workspace_bytes(const sc_plan* plan, const sc_cache* cache);
int sc_attention(const sc_plan* plan, const sc_cache* cache, int32_t layer, const void* q,
                 void* o, float scale, void* ws, size_t ws_bytes, sc_stream stream);

/* ---- Attention that allocates nothing -----------------------------------
 * For callers that cannot allocate device memory or hand over a workspace:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  sc_attention with its split-key partials kept in a
 * library-owned device array of sc_attention_noalloc_scratch_bytes() bytes
 * (64 MiB) on each GPU, held from the first call on that GPU until the
 * process ends; the call itself allocates nothing.  Key ranges are cut into
 * no more pieces than that array holds partials for, so the output equals
 * sc_attention's up to the summation order.  Every call on a GPU shares that
 * GPU's array (its contents are undefined between calls): calls that overlap
 * on one GPU -- other streams, other threads -- race, and the caller must
 * order them.  Arguments and errors as sc_attention, plus SC_ECAPACITY if a
 * plan needed more partials than the array holds and SC_EDEVICE if the
 * array's address cannot be resolved on the current device. */
size_t sc_attention_noalloc_scratch_bytes(void);
int sc_attention_noalloc(const sc_plan* plan, const sc_cache* cache, int32_t layer, const void* q,
                         void* o, float scale, sc_stream stream);

/* ---- Condition K/V (the condition c of Eq. 1) ---------------------------
 * Projects a condition sequence once per layer and caches it:
 *   K_c = ctx Wk^T (then RMSNorm over the hidden width times k_norm, when
 *         k_norm != NULL), V_c = ctx Wv^T, no RoPE,
 * written into the pages of `state` in a condition cache whose geometry
 * holds one condition per state (n_tokens = tokens_per_page *
 * pages_per_chunk; hidden = n_heads * head_dim, a multiple of 256, head_dim
 * 128, bf16).  ctx: device bf16 [n_tokens, hidden]; w_k, w_v: device bf16
 * [hidden, hidden] in [out, in] layout; k_norm: device fp32 [hidden],
 * 16-byte aligned, or NULL.  ws: device workspace of at least
 * sc_condition_workspace_bytes(cache) bytes, 16-byte aligned.  Slots are
 * allocated as by sc_cache_append.  Errors: SC_EEXIST (layer already
 * written), SC_ECAPACITY, SC_EINVAL, SC_EUNSUPPORTED, SC_EDEVICE. */
size_t sc_condition_workspace_bytes(const sc_cache* cache);
int sc_condition_append(sc_cache* cache, int32_t layer, sc_node state, const void* ctx,
                        const void* w_k, const void* w_v, const float* k_norm, void* ws,
                        size_t ws_bytes, sc_stream stream);

/* ---- One DiT block over the pack ----------------------------------------
 * The network F_theta of Eq. 1 for the packed nodes, one block (bf16 only):
 *   h = RMSNorm(x); [q k v] = h Wqkv^T; q, k = RoPE(q), RoPE(k)
 *   (k, v of each pack node are appended to its reserved slots, this layer)
 *   o = sc_attention(q); x' = x + o Wo^T
 *   x = x' + GELU_tanh(RMSNorm(x') Wup^T) Wdown^T
 * RMSNorm: eps 1e-6, unit gain.  Weights: device bf16 in [out, in] layout
 * (Wqkv is [3*hidden, hidden] = Wq;Wk;Wv).  x: device bf16
 * [n_nodes * Nq, hidden], updated in place.  ws: device workspace of at least
 * sc_block_workspace_bytes() bytes.  The block form is the Wan-shaped
 * reading of the workload (the paper does not define the network).
 * Limits: hidden and mlp multiples of 256, head_dim 128, at most 64 pack
 * nodes owning at most 256 page slots (the QKV epilogue's node table), and
 * the attention limits above; all are checked before the first launch.
 * The pack's states are marked written at this layer only once every launch
 * has been enqueued: after an error they are still unwritten (their pages
 * and x hold partial results) and the block can be run again.
 *
 * Noise-level conditioning (optional, mod != NULL): the denoiser of Eq. 1
 * depends on the node's level j.  mod is a device fp32 table
 * [mod_levels][6][hidden] of per-level vectors (shift_a, scale_a, gate_a,
 * shift_m, scale_m, gate_m), e.g. a timestep embedding projected per layer
 * (computed by the caller); every pack node needs j < mod_levels.  With it:
 *   h  = RMSNorm(x)  * (1 + scale_a[j]) + shift_a[j]
 *   x' = x + gate_a[j] * (o Wo^T)
 *   h2 = RMSNorm(x') * (1 + scale_m[j]) + shift_m[j]
 *   x  = x' + gate_m[j] * (GELU_tanh(h2 Wup^T) Wdown^T)
 * (elementwise over hidden).  mod == NULL is the unconditioned form above.
 *
 * qk-norm (optional, qk_norm != NULL): q and k are RMS-normalised over the
 * whole hidden width and multiplied by the gains before RoPE:
 *   q = RMSNorm(h Wq^T) * qk_norm[0:hidden], k = RMSNorm(h Wk^T) * qk_norm[hidden:2*hidden]
 * (device fp32 [2][hidden], 16-byte aligned; the cached keys are the
 * normalised ones).
 *
 * Cross-attention to the condition (optional, cross != NULL), after the
 * self-attention residual and before the MLP, which then reads its result:
 *   qc = RMSNorm(x') Wcq^T  [then RMSNorm(qc) * q_norm when q_norm != NULL]
 *   x' = x' + Attn(qc, K_c, V_c) Wco^T       (scale 1/sqrt(head_dim))
 * K_c, V_c are read through cross->plan (sc_plan_condition over
 * cross->cache, one node per pack node, the pack plan's nq) at this layer;
 * the condition cache has the block's head geometry.  The block forms are
 * the Wan-shaped reading of F_theta (the paper does not define the network;
 * c of Eq. 1 is read by cross-attention). */
typedef struct {
  const void* w_q;        /* [hidden, hidden] bf16 */
  const void* w_o;        /* [hidden, hidden] bf16 */
  const float* q_norm;    /* [hidden] fp32 gain, 16-byte aligned, or NULL */
  const sc_cache* cache;  /* condition cache (bf16)                       */
  const sc_plan* plan;    /* sc_plan_condition over that cache            */
} sc_cross_attn;

typedef struct {
  int32_t hidden, n_heads, head_dim, mlp;
  const void* w_qkv;  /* [3*hidden, hidden] */
  const void* w_o;    /* [hidden, hidden]   */
  const void* w_up;   /* [mlp, hidden]      */
  const void* w_down; /* [hidden, mlp]      */
  const float* mod;   /* [mod_levels][6][hidden] fp32, or NULL */
  int32_t mod_levels;
  const float* qk_norm;        /* [2][hidden] fp32 gains, or NULL */
  const sc_cross_attn* cross;  /* or NULL */
} sc_block_weights;
size_t sc_block_workspace_bytes(const sc_block_weights* w, int32_t n_tokens);
/* For inspection of a block's intermediates: byte offsets inside the
 * workspace of the rotated queries q and the self-attention output o of the
 * last sc_block_forward that used it, both bf16 [n_tokens][hidden]
 * token-major (node i at rows [i*Nq, (i+1)*Nq)).  They hold those values
 * once the block's work on the stream has completed, until the workspace
 * is used again; with cross-attention they hold its query and output
 * instead.  Errors: SC_EINVAL (null pointer, n_tokens < 1). */
int sc_block_workspace_views(const sc_block_weights* w, int32_t n_tokens, size_t* q_offset,
                             size_t* o_offset);
int sc_block_forward(const sc_block_weights* w, sc_cache* cache, int32_t layer,
                     const sc_plan* plan, void* x, const sc_rope* rope, void* ws,
                     size_t ws_bytes, sc_stream stream);

/* ---- Sampler step (Eq. 1) ----------------------------------------------
 * For each node i with level j >= 1:
 *   out_i = (1 - t[j-1]) * y_i + t[j-1] * noise_i
 * (the network output is read as a clean-state prediction and re-noised to
 * the next input time; a reading, the paper leaves S_j open).  Nodes at
 * level 0 are left untouched.  y, noise, out: device bf16
 * [n_nodes, elems_per_node]; out may alias y.  t: host, K+1 input times. */
int sc_sampler_step(const sc_node* nodes, int32_t n_nodes, const float* t, int32_t K,
                    void* out, const void* y, const void* noise, int64_t elems_per_node,
                    sc_stream stream);

/* ---- Execution schedule (Sec. 3.3) --------------------------------------
 * Pipelined execution, Eq. 7: round n advances every active chunk by one
 * level -- chunk n - K + j sits at level j -- for chunks 0..B-1.  Without
 * the refresh node the levels are 1..K (K + B - 1 rounds, B*K updates); with
 * it the clean-state refresh (c, 0) of one chunk per round joins the round
 * as its oldest node (K + B rounds, B*(K+1) forwards; the paper refreshes
 * each chunk's clean KV once but does not say where, this is the reading).
 * Nodes are written oldest chunk first; out needs room for K + 1 nodes.
 * Errors: SC_EINVAL (K < 1, B < 1, n outside the schedule). */
int sc_pipeline_rounds(int32_t K, int32_t B, int32_t refresh);
int sc_pipeline_round_nodes(int32_t K, int32_t B, int32_t refresh, int32_t n, sc_node* out,
                            int32_t* n_out);

/* Fully serial execution, Eq. 2: one node per forward, all updates of chunk
 * c (levels K, K-1, .., 1, then the refresh (c, 0) when refresh != 0)
 * before chunk c + 1.  sc_serial_steps returns the number of forwards
 * (B*K, or B*(K+1) with the refresh); sc_serial_step_node writes the node of
 * forward n.  Errors: SC_EINVAL (K < 1, B < 1, n outside the schedule). */
int sc_serial_steps(int32_t K, int32_t B, int32_t refresh);
int sc_serial_step_node(int32_t K, int32_t B, int32_t refresh, int32_t n, sc_node* out);

/* Releases every cached state that none of the given future nodes reads
 * under the policy (Eq. 4-5 offsets and levels), keeping only what the rest
 * of the schedule needs ("earlier states are retained", Sec. 3.3).  Returns
 * the number of states released, or a negative SC_E* code. */
int sc_cache_release_unread(sc_cache* cache, const sc_policy* policy, const sc_node* future,
                            int32_t n_future);

/* The network F_theta of Eq. 1 as a stack of n_layers blocks over one pack:
 * sc_block_forward for layer 0 .. n_layers-1 in order (layers[l] holds the
 * weights of layer l), x updated in place, one plan for every layer.  On an
 * error in layer l, the pack's states are left unwritten in every layer
 * (x holds a partial result): the caller restores x and runs it again. */
int sc_stack_forward(const sc_block_weights* layers, int32_t n_layers, sc_cache* cache,
                     const sc_plan* plan, void* x, const sc_rope* rope, void* ws, size_t ws_bytes,
                     sc_stream stream);

/* Measurement support (kernel timer, matrix-core probe): streamctx_measure.h */

#ifdef __cplusplus
}
#endif
#endif /* STREAMCTX_H */
