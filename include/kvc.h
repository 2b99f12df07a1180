/*
 * kvc.h -- C ABI of libkvc: online low-rank KV-cache correction for shared context across agents (KVCMAS).
 *
 * Three operations on a paged K/V cache, all asynchronous on the caller's HIP stream:
 *
 *   kvc_fit_state  Eq. 12 then Eq. 7.  For each (layer, K/V, KV head) unit of an item, Z = C_dst - Align(C_src)
 *                  over the first T_s rows (the observed transition after a dense prefill), or Z = C_dst (a base
 *                  cache, Section 3.3), and its rank-r truncated SVD Z ~ A B with A = U_r Sigma_r (T_s x r, "coef")
 *                  and B = R_r^T (r x d, "basis", orthonormal rows), plus sigma.  Align is the identity, except for
 *                  the keys of a rotary cache, which are fitted in canonical coordinates (see kvc_rope_style).
 *   kvc_apply      Eq. 4 with the source agent's materialised cache as the reference (Section 3.2, Eq. 6) and one
 *                  state (Eq. 8 with a single anchor, w = 1): C_dst[t] = C_src[t] + A[t] B for t < T_s and
 *                  C_dst[t] = C_src[t] (bit copy) for T_s <= t < T (Appendix A.3, "Variable Segment Lengths");
 *                  the keys of a rotary cache are corrected in canonical coordinates and rotated to the target
 *                  positions in the same pass (Appendix A.3, "Positional Alignment").
 *   kvc_chain      Eq. 6 composed in low rank: from S1 = Delta_{j<-i} and S2 = Delta_{k<-j}, the rank-r_out truncated
 *                  SVD of A1 B1 + A2 B2 (rows past a state's coverage are zero), without forming any T x d matrix.
 *
 * With an anchor pool (Section 3.3, Appendix A.3) the correction of a transfer is estimated from V anchors:
 *
 *   kvc_anchor_weights  token-wise interpolation weights from the mean absolute distance of the source cache to
 *                       each anchor's reconstructed base, softmax over the anchors (Appendix A.3).
 *   kvc_apply_anchored  Eq. 8 with those weights: C_dst[t] = C_src[t] + sum_v w_v[t] A_v[t] B_v.
 *   kvc_gate_distances  Eq. 9: value-state distances of the source prefix to each anchor's base; kvc_gate_decide
 *                       turns them into the gate weights, normalised entropy and accept/reject of Eq. 10-11, and
 *                       kvc_pool_* keep the pool's insertion and eviction bookkeeping (host only).
 *
 * Layout.  One pool per layer for K and one for V.  Token slot s of physical block b of KV head h starts at element
 *   b * block_stride + s * token_stride + h * head_stride
 * of the layer's pool, and its head_dim elements are contiguous.  An item's token t sits at position p = offset + t of
 * its block sequence: block = table[p / block_size] (or p / block_size when the table pointer is NULL, i.e.
 * contiguous rows), slot = p % block_size.  A state's unit u = (layer, kv, head) with kv = 0 for K and 1 for V keeps
 *   coef  [L][2][H][T_s][r]  (coef_dtype)      basis [L][2][H][r][d] (float32)      sigma [L][2][H][r] (float32)
 *
 * Ownership.  The caller allocates every buffer (pools, tables, states, workspaces, the item scratch); the library
 * allocates no device memory, keeps no pointer after a call returns, holds no global state (except the static
 * scratch of kvc_gate_distances_noalloc) and may be called from several threads.  Source rows are only read.  The one host-side object is the anchor-pool bookkeeping
 * of kvc_pool_create, owned by the caller until kvc_pool_destroy (not thread-safe per pool).
 *
 * Errors.  Every argument check runs on the host before anything is enqueued; on an error nothing is enqueued and
 * the status says why.  A failed launch returns KVC_ERR_HIP (kvc_last_hip_error() gives the hipError_t of the
 * calling thread).  Faults inside a kernel surface at the caller's next synchronisation.  A row whose source or
 * destination block-table entry lies outside [0, num_blocks) is neither read nor written (its destination keeps its
 * bytes).  NaN and Inf of the cache rows propagate through the corrections; a non-finite state entry gives NaN in the
 * rows it touches.
 */
#ifndef KVC_H
#define KVC_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVC_VERSION 1
#define KVC_MAX_RANK 128   /* largest r of a state */
#define KVC_MAX_ANCHORS 16 /* largest V of an anchor set in one call */
/* Bytes of the static device scratch of kvc_gate_distances_noalloc (one copy per GPU the library runs on). */
#define KVC_NOALLOC_SCRATCH_BYTES (2u << 20)

typedef enum kvc_status {
  KVC_OK = 0,
  KVC_ERR_NULL_ARG = 1,    /* a required pointer is NULL */
  KVC_ERR_SHAPE = 2,       /* sizes inconsistent or out of range */
  KVC_ERR_DTYPE = 3,       /* unknown dtype, or dtypes that do not go together */
  KVC_ERR_ALIGN = 4,       /* a row or a coefficient array is not 16-byte aligned */
  KVC_ERR_ALIAS = 5,       /* destination rows may overlap source rows or another item's destination rows */
  KVC_ERR_WORKSPACE = 6,   /* workspace missing, misaligned or smaller than the query says */
  KVC_ERR_UNSUPPORTED = 7, /* head_dim other than 64 or 128, or a state grouping or rotary setting the entry point
                              does not take (stated at each entry point) */
  KVC_ERR_HIP = 8,         /* the HIP runtime refused a launch */
  KVC_ERR_TOO_LARGE = 9    /* the call needs more than the static scratch of an allocation-free entry point */
} kvc_status;

typedef enum kvc_dtype { KVC_F32 = 0, KVC_BF16 = 1 } kvc_dtype;

/* Rotary position encoding of the key rows (the models the method serves use RoPE).  The key of a token at context
 * position p carries every feature pair i rotated by the angle p * inv_freq[i].  Sharing a segment across agents
 * moves its tokens to other positions, so keys are compared, fitted and corrected in canonical coordinates
 * (segment token t at position t) and the corrected keys are rotated to their target positions (Section 2.2,
 * Appendix A.3 "Positional Alignment"); values are never rotated. */
typedef enum kvc_rope_style {
  KVC_ROPE_NONE = 0,  /* the keys carry no rotary encoding (no re-alignment anywhere) */
  KVC_ROPE_HALF = 1,  /* pair i = features (i, i + head_dim / 2): the rotate-half layout of Llama and Qwen models */
  KVC_ROPE_PAIRS = 2  /* pair i = features (2 i, 2 i + 1) */
} kvc_rope_style;

typedef enum kvc_fit_mode {
  KVC_FIT_DELTA = 0, /* Z = C_dst - C_src: the observed transition of Eq. 12 */
  KVC_FIT_BASE = 1   /* Z = C_dst: a base cache (Z in {C, Delta}, Section 3.3); the src side is not read */
} kvc_fit_mode;

/* A paged K/V pool set.  k_layers / v_layers are HOST arrays of num_layers DEVICE pointers.  Strides are in
 * elements; block_stride, token_stride and head_stride times the element size must be multiples of 16 bytes and
 * every layer pointer 16-byte aligned.  head_dim is 64 or 128.  rope_style says how the key rows are rotary-encoded
 * (KVC_ROPE_NONE when they are not; a zero-initialised struct is that); with another style rope_inv_freq is a HOST
 * array of head_dim / 2 finite angles per position step, read during the call only. */
typedef struct kvc_cache {
  kvc_dtype dtype;
  int32_t num_layers;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t block_size;
  int32_t num_blocks;
  int64_t block_stride;
  int64_t token_stride;
  int64_t head_stride;
  void* const* k_layers;
  void* const* v_layers;
  int32_t rope_style;          /* kvc_rope_style */
  int32_t rope_reserved;       /* must be 0 */
  const double* rope_inv_freq; /* HOST [head_dim / 2], or NULL with KVC_ROPE_NONE */
} kvc_cache;

/* Factorisation unit of a state.  The paper factorises each layer's keys (values) with the KV feature dimension D
 * of the layer (Section 3.3); per KV head D = head_dim, per layer D = num_kv_heads * head_dim. */
typedef enum kvc_grouping {
  KVC_GROUP_HEAD = 0, /* unit (layer, K/V, head): coef [L][2][H][T_s][r], basis [L][2][H][r][d], sigma [L][2][H][r] */
  KVC_GROUP_LAYER = 1 /* unit (layer, K/V): coef [L][2][T_s][r], basis [L][2][r][H d] (head h's features are the
                         columns h d .. h d + d - 1 of a row), sigma [L][2][r] */
} kvc_grouping;

/* Low-rank state of one sequence (Eq. 7): coef = A, basis = B per unit.  DEVICE pointers.  coef_dtype is the cache
 * dtype for fit/apply (bf16 coefficients for bf16 caches, float32 for float32 caches).  0 <= rank <= min(D,
 * KVC_MAX_RANK) with D the unit's feature dimension; rank 0 makes apply a copy.  coef must be 16-byte aligned.
 * sigma may be NULL.  Per-layer states (KVC_GROUP_LAYER) are fitted by kvc_fit_state and read by kvc_apply; the
 * chain and anchor calls take per-head states. */
typedef struct kvc_state {
  int32_t num_layers;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t num_tokens; /* T_s: coefficient rows per unit */
  int32_t rank;
  kvc_dtype coef_dtype;
  int32_t grouping;   /* kvc_grouping */
  int32_t reserved;   /* must be 0 */
  void* coef;
  float* basis;
  float* sigma;
} kvc_state;

/* One shared segment of an agent edge.  apply reads `state`; fit writes it (its rank, num_tokens and pointers say
 * what to produce: rows t < state.num_tokens are fitted).  state.num_tokens <= num_tokens.  src_position and
 * dst_position place the segment in the source and target agents' contexts (token t at position + t); they matter
 * only for the keys of a rotary cache, whose states are kept in canonical coordinates. */
typedef struct kvc_item {
  int32_t num_tokens;   /* T: rows of the segment */
  int32_t src_offset;   /* position of row 0 within the src block sequence */
  int32_t dst_offset;   /* position of row 0 within the dst block sequence */
  int32_t src_position; /* context position of row 0 in the source agent, >= 0 */
  int32_t dst_position; /* context position of row 0 in the target agent, >= 0 */
  int32_t reserved;     /* must be 0 */
  kvc_state state;
} kvc_item;

/* A batch of independent items handled by one launch per kernel.  `items` is a HOST array: the library checks it and
 * then copies it (hipMemcpyAsync on the call's stream, before its first launch) into `item_scratch`, a DEVICE buffer
 * of at least kvc_item_scratch_bytes(num_items) bytes, 16-byte aligned, from which the kernels read the items; the
 * kernels therefore see exactly the bytes that were checked.  Like every other buffer of an asynchronous call, the
 * host items (when they are in pinned memory) and the scratch belong to the call until its work on the stream is done:
 * calls that overlap in time need scratch buffers of their own.  kvc_apply and kvc_fit_state use the scratch; the
 * anchor calls take their one item by value and ignore it.  Tables are DEVICE int32 arrays [num_items][max_blocks] of
 * physical block ids; NULL means the identity mapping (contiguous rows). */
typedef struct kvc_batch {
  int32_t num_items;
  int32_t max_blocks;
  const kvc_item* items;
  void* item_scratch;
  const int32_t* src_tables;
  const int32_t* dst_tables;
} kvc_batch;

int32_t kvc_version(void);
const char* kvc_status_str(kvc_status status);
/* hipError_t of the last failed HIP call made by this thread inside the library (0 if none). */
int32_t kvc_last_hip_error(void);

/* Bytes of the device item scratch of a batch of num_items items (0 for a negative count). */
size_t kvc_item_scratch_bytes(int32_t num_items);
/* Bytes of one low-rank state (coef + basis + sigma), the O(N r (L + D)) term of Section 3.3. */
size_t kvc_state_bytes(int32_t num_layers, int32_t num_kv_heads, int32_t head_dim, int32_t num_tokens, int32_t rank,
                       kvc_dtype coef_dtype);
/* Bytes of a per-layer state (KVC_GROUP_LAYER): L x {K,V} x (T r coefficients + r H d basis + r sigma). */
size_t kvc_layer_state_bytes(int32_t num_layers, int32_t num_kv_heads, int32_t head_dim, int32_t num_tokens,
                             int32_t rank, kvc_dtype coef_dtype);
/* Bytes of the same segment kept full-dimensional (L x {K,V} x T x H d), the O(N L D) term of Section 3.1. */
size_t kvc_dense_bytes(int32_t num_layers, int32_t num_kv_heads, int32_t head_dim, int32_t num_tokens,
                       kvc_dtype dtype);

/* Materialise each item's destination rows from its source rows and state, for layers [layer_begin, layer_end).
 * One launch covers every item, layer, K/V and head of the call (a serving batch corrects a whole layer at once).
 * Destination rows must not overlap any source row of the call, nor another item's destination rows.  With both
 * tables NULL the host checks this on the row ranges of all items (KVC_ERR_ALIAS); with tables the block ids live in
 * device memory, so the host only rejects src_tables == dst_tables and the caller guarantees the rest.
 * Keys of a rotary cache (rope_style != KVC_ROPE_NONE), with R(p) the rotation to position p, ps = src_position and
 * pd = dst_position: C_dst[t] = R(pd) (R(-ps) C_src[t] + A[t] B) for t < T_s (the state is canonical) and
 * C_dst[t] = R(pd - ps) C_src[t] for T_s <= t < T (the re-aligned source; a bit copy when pd = ps), one rounding. */
kvc_status kvc_apply(const kvc_cache* cache, const kvc_batch* batch, int32_t layer_begin, int32_t layer_end,
                     hipStream_t stream);

/* Workspace kvc_fit_state needs for this call (bytes, 256-byte aligned start required). */
size_t kvc_fit_workspace_bytes(const kvc_cache* cache, const kvc_batch* batch, int32_t layer_begin,
                               int32_t layer_end);
/* Fit each item's state for layers [layer_begin, layer_end); other layers of the state are left as they are.
 * Sigma descending; each basis row has its largest-magnitude entry positive.  Keys of a rotary cache:
 * Z = R(-dst_position) C_dst - R(-src_position) C_src (KVC_FIT_BASE: Z = R(-dst_position) C_dst), so the state is in
 * canonical coordinates.  Per-layer states (KVC_GROUP_LAYER, every item of the call): Z = [Z_0 ... Z_{H-1}] with the
 * heads side by side (each head's key rows in canonical coordinates for a rotary cache), D = H d <= 1024, rank <= 112
 * (KVC_ERR_UNSUPPORTED otherwise; float32 caches also need rank * D * 4 + 1024 <= 160 KiB, and rotary keys in a
 * bf16 cache a power-of-two block size of at least 8 with every head of a row within 2 GiB); the SVD is reached by subspace iteration on Z^T Z (k = 64 columns for
 * rank <= 48, else 128) with a Rayleigh-Ritz step after 4 iterations and every 4 more, stopping per layer unit once
 * every top-r Ritz pair (theta, y) has ||Z^T Z y - theta y|| <= 1e-6 theta_1, or after 48 iterations (a spectrum with
 * no gap between sigma_r and sigma_{k+1}); the kernels of a stopped unit return at once. */
kvc_status kvc_fit_state(const kvc_cache* cache, const kvc_batch* batch, int32_t layer_begin, int32_t layer_end,
                         kvc_fit_mode mode, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace kvc_chain needs (bytes, 256-byte aligned start required). */
size_t kvc_chain_workspace_bytes(const kvc_state* first, const kvc_state* second, const kvc_state* out,
                                 int32_t layer_begin, int32_t layer_end);
/* out = truncated SVD of first + second (Eq. 6), rank out->rank <= min(first->rank + second->rank, head_dim), for
 * layers [layer_begin, layer_end).  out->num_tokens must equal max(first->num_tokens, second->num_tokens); all three
 * share num_layers, num_kv_heads, head_dim and coef_dtype.  With out->rank = first->rank + second->rank <= head_dim
 * the composition is lossless. */
kvc_status kvc_chain(const kvc_state* first, const kvc_state* second, kvc_state* out, int32_t layer_begin,
                     int32_t layer_end, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ---- anchor pool (Section 3.3 low-rank anchors, Appendix A.3) --------------------------------------------------- */

/* The anchors of one shared segment, for one call.  `states` is a HOST array of num_anchors states -- each anchor's
 * base cache (kvc_anchor_weights, kvc_gate_distances) or its delta correction for the consuming agent
 * (kvc_apply_anchored) -- sharing the cache's num_layers, num_kv_heads, head_dim and dtype, rank >= 1, each covering
 * at least num_tokens rows.  `weights` is a DEVICE float32 array [layer_end - layer_begin][2][num_tokens]
 * [num_anchors] (layer relative to layer_begin, then K = 0 / V = 1, token, anchor): written by kvc_anchor_weights,
 * read by kvc_apply_anchored. */
typedef struct kvc_anchors {
  int32_t num_anchors; /* V, 1 .. KVC_MAX_ANCHORS */
  int32_t num_tokens;  /* T_s: rows weighted and corrected */
  const kvc_state* states;
  float* weights;
} kvc_anchors;

/* Token-wise interpolation weights (Appendix A.3, correction weighting), for layers [layer_begin, layer_end), K and
 * V separately, and t < T_s: d_v[t] = mean over the layer's K (or V) row -- every KV head and feature, the paper's
 * D = H d -- of |C_src[t] - (A_v B_v)[t]|, with A_v B_v anchor v's reconstructed base, and
 * w_v[t] = exp(-d_v[t] / temperature) / sum_u exp(-d_u[t] / temperature) (temperature 1 in the paper).  `batch`
 * holds exactly one item whose source rows are compared (its state, dst side and item_scratch are not used);
 * T_s <= item.num_tokens.  Keys of a rotary cache are compared in canonical coordinates, R(-src_position) C_src[t]
 * (the anchors' bases are canonical). */
kvc_status kvc_anchor_weights(const kvc_cache* cache, const kvc_batch* batch, const kvc_anchors* anchors,
                              int32_t layer_begin, int32_t layer_end, float temperature, hipStream_t stream);

/* Eq. 8 with token-wise weights: for layers [layer_begin, layer_end), every K/V unit and t < T_s,
 * C_dst[t] = C_src[t] + sum_v w_v[t] A_v[t] B_v (A_v B_v anchor v's delta correction, w from `anchors->weights`),
 * one rounding to the storage dtype; rows T_s <= t < item.num_tokens are bit copies.  One item (its state and
 * item_scratch are not used); destination rows must not overlap source rows (as for kvc_apply).  Keys of a rotary
 * cache as in kvc_apply: R(pd) (R(-ps) C_src[t] + sum_v w_v[t] A_v[t] B_v), re-aligned source past T_s. */
kvc_status kvc_apply_anchored(const kvc_cache* cache, const kvc_batch* batch, const kvc_anchors* anchors,
                              int32_t layer_begin, int32_t layer_end, hipStream_t stream);

/* Workspace kvc_gate_distances needs (bytes, 256-byte aligned start required). */
size_t kvc_gate_workspace_bytes(const kvc_cache* cache, const kvc_anchors* anchors, int32_t prefix,
                                int32_t layer_begin, int32_t layer_end);
/* Eq. 9: d_v = (sum over layers [layer_begin, layer_end) of ||V_src[:k] - V_v[:k]||_F^2)^(1/2) with k = prefix,
 * V_src the value rows of the item's source cache (every KV head) and V_v anchor v's reconstructed base values.
 * `distances` is a DEVICE float32 array [num_anchors]; the partial sums are added in a fixed order (the result does
 * not depend on scheduling).  anchors->weights is not used; 1 <= prefix <= anchors->num_tokens.  Values carry no
 * rotary encoding, so positions play no part here. */
kvc_status kvc_gate_distances(const kvc_cache* cache, const kvc_batch* batch, const kvc_anchors* anchors,
                              int32_t prefix, int32_t layer_begin, int32_t layer_end, float* distances,
                              void* workspace, size_t workspace_bytes, hipStream_t stream);
/* For callers that cannot allocate device memory (code under HIP graph capture, serving loops that forbid
 * hipMalloc): kvc_gate_distances without a workspace argument.  The partial sums live in a static device array of
 * KVC_NOALLOC_SCRATCH_BYTES bytes that the library holds on every GPU it runs on until the process ends; a call that
 * needs more than that (kvc_gate_workspace_bytes) returns KVC_ERR_TOO_LARGE before anything is enqueued.  Nothing is
 * allocated and no allocating routine is called.  Every call on one GPU shares that GPU's array: the kernels write
 * each partial before it is read, so no contents carry over between calls, but calls that overlap in time on one GPU
 * (other streams, other threads) race and must be serialised by the caller.  Arguments, results and errors otherwise
 * as kvc_gate_distances. */
kvc_status kvc_gate_distances_noalloc(const kvc_cache* cache, const kvc_batch* batch, const kvc_anchors* anchors,
                                      int32_t prefix, int32_t layer_begin, int32_t layer_end, float* distances,
                                      hipStream_t stream);
/* Eq. 10-11 on the host: g_v = softmax(-d_v / temperature) over the n compatible anchors (HOST arrays), normalised
 * entropy H = -sum g log2 g / log2 n; returns 1 (accept the correction) when n >= 2 and H <= tau, else 0 (dense
 * prefill).  gate_weights may be NULL; with n < 2 *entropy is set to 1. */
int32_t kvc_gate_decide(const float* distances, int32_t n, float tau, float temperature, float* gate_weights,
                        float* entropy);

/* Anchor-pool bookkeeping of one shared-context slot (Appendix A.3, pool updates), host only: up to `capacity`
 * anchors with a stored length and a use count.  A new anchor takes the first free slot; in a full pool it replaces
 * the least frequently used of the five oldest anchors (the oldest of them on equal counts).  The caller keeps the
 * anchors' states; the pool only says which slot to overwrite. */
typedef struct kvc_pool kvc_pool;
kvc_pool* kvc_pool_create(int32_t capacity);
void kvc_pool_destroy(kvc_pool* pool);
/* Slot for a new anchor (id, stored length); *evicted_id gets the replaced anchor's id, or -1 for a free slot.
 * Returns the slot, or -1 on a bad argument. */
int32_t kvc_pool_insert(kvc_pool* pool, int64_t anchor_id, int32_t length, int64_t* evicted_id);
/* Count one use of each listed slot (the anchors of an accepted correction). */
kvc_status kvc_pool_record_use(kvc_pool* pool, const int32_t* slots, int32_t n);
/* Occupied slots whose stored length is at least `prefix`, ascending; returns their number (at most capacity). */
int32_t kvc_pool_eligible(const kvc_pool* pool, int32_t prefix, int32_t* slots);
/* Id, length and use count of a slot (returns KVC_ERR_SHAPE for a free or invalid slot). */
kvc_status kvc_pool_slot(const kvc_pool* pool, int32_t slot, int64_t* anchor_id, int32_t* length, int64_t* uses);

#ifdef __cplusplus
}
#endif

#endif /* KVC_H */
