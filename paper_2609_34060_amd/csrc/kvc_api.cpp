// Host entry points of libkvc: argument checks, launch sizing and dispatch.  Every check runs before anything is
// enqueued; on an error nothing is enqueued.
#include <algorithm>
#include <cstdint>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "kvc.h"
#include "kvc_launch.h"

namespace {

thread_local int32_t g_last_hip_error = 0;

kvc_status hip_status(hipError_t e) {
  if (e == hipSuccess) return KVC_OK;
  g_last_hip_error = static_cast<int32_t>(e);
  return KVC_ERR_HIP;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t dtype_size(kvc_dtype t) { return t == KVC_BF16 ? 2 : 4; }

bool valid_dtype(kvc_dtype t) { return t == KVC_F32 || t == KVC_BF16; }

kvc_status check_cache(const kvc_cache* c, int32_t lb, int32_t le) {
  if (!c) return KVC_ERR_NULL_ARG;
  if (!valid_dtype(c->dtype)) return KVC_ERR_DTYPE;
  if (c->head_dim != 64 && c->head_dim != 128) return KVC_ERR_UNSUPPORTED;
  if (c->num_layers < 1 || c->num_kv_heads < 1 || c->block_size < 1 || c->num_blocks < 1) return KVC_ERR_SHAPE;
  if (lb < 0 || le < lb || le > c->num_layers) return KVC_ERR_SHAPE;
  if (c->block_stride < 1 || c->token_stride < 1 || c->head_stride < 1) return KVC_ERR_SHAPE;
  const int64_t es = static_cast<int64_t>(dtype_size(c->dtype));
  if ((c->block_stride * es) % 16 || (c->token_stride * es) % 16 || (c->head_stride * es) % 16) return KVC_ERR_ALIGN;
  // a row must fit between two token slots and two heads (head_dim contiguous elements)
  if (c->head_stride < c->head_dim && c->num_kv_heads > 1) return KVC_ERR_SHAPE;
  if (c->rope_reserved != 0) return KVC_ERR_SHAPE;
  if (c->rope_style != KVC_ROPE_NONE && c->rope_style != KVC_ROPE_HALF && c->rope_style != KVC_ROPE_PAIRS)
    return KVC_ERR_SHAPE;
  if (c->rope_style != KVC_ROPE_NONE) {
    if (!c->rope_inv_freq) return KVC_ERR_NULL_ARG;
    for (int32_t i = 0; i < c->head_dim / 2; ++i)
      if (!std::isfinite(c->rope_inv_freq[i])) return KVC_ERR_SHAPE;
  }
  if (le > lb && (!c->k_layers || !c->v_layers)) return KVC_ERR_NULL_ARG;
  for (int32_t l = lb; l < le; ++l) {
    if (!c->k_layers[l] || !c->v_layers[l]) return KVC_ERR_NULL_ARG;
    if (!aligned16(c->k_layers[l]) || !aligned16(c->v_layers[l])) return KVC_ERR_ALIGN;
  }
  return KVC_OK;
}

kvc_status check_state_shape(const kvc_state& s, int32_t L, int32_t H, int32_t d) {
  if (s.num_layers != L || s.num_kv_heads != H || s.head_dim != d) return KVC_ERR_SHAPE;
  if (!valid_dtype(s.coef_dtype)) return KVC_ERR_DTYPE;
  if (s.reserved != 0 || (s.grouping != KVC_GROUP_HEAD && s.grouping != KVC_GROUP_LAYER)) return KVC_ERR_SHAPE;
  const int32_t D = s.grouping == KVC_GROUP_LAYER ? H * d : d;
  if (s.rank < 0 || s.rank > std::min<int32_t>(D, KVC_MAX_RANK) || s.num_tokens < 0) return KVC_ERR_SHAPE;
  if (s.rank > 0 && s.num_tokens > 0) {
    if (!s.coef || !s.basis) return KVC_ERR_NULL_ARG;
    if (!aligned16(s.coef) || !aligned16(s.basis)) return KVC_ERR_ALIGN;
  }
  return KVC_OK;
}

// Rows [off, off + T) of a block sequence must stay inside its table row (or the pool for the identity mapping).
bool positions_fit(int64_t off, int64_t T, bool has_table, const kvc_batch* b, const kvc_cache* c) {
  if (off < 0) return false;
  const int64_t end = off + T;
  if (end > INT32_MAX) return false;
  const int64_t cap = has_table ? static_cast<int64_t>(b->max_blocks) * c->block_size
                                : static_cast<int64_t>(c->num_blocks) * c->block_size;
  return T == 0 || end <= cap;
}

kvc_status check_batch(const kvc_cache* c, const kvc_batch* b, bool needs_src) {
  if (!b) return KVC_ERR_NULL_ARG;
  if (b->num_items < 0 || b->max_blocks < 0) return KVC_ERR_SHAPE;
  if (b->num_items == 0) return KVC_OK;
  if (!b->items || !b->item_scratch) return KVC_ERR_NULL_ARG;
  if (!aligned16(b->item_scratch)) return KVC_ERR_ALIGN;
  if ((b->src_tables || b->dst_tables) && b->max_blocks < 1) return KVC_ERR_SHAPE;
  for (int32_t i = 0; i < b->num_items; ++i) {
    const kvc_item& it = b->items[i];
    if (it.reserved != 0 || it.num_tokens < 0 || it.src_position < 0 || it.dst_position < 0) return KVC_ERR_SHAPE;
    if (!positions_fit(it.dst_offset, it.num_tokens, b->dst_tables != nullptr, b, c)) return KVC_ERR_SHAPE;
    if (needs_src && !positions_fit(it.src_offset, it.num_tokens, b->src_tables != nullptr, b, c))
      return KVC_ERR_SHAPE;
    kvc_status s = check_state_shape(it.state, c->num_layers, c->num_kv_heads, c->head_dim);
    if (s != KVC_OK) return s;
    if (it.state.coef_dtype != c->dtype) return KVC_ERR_DTYPE;
    if (it.state.num_tokens > it.num_tokens) return KVC_ERR_SHAPE;
  }
  return KVC_OK;
}

// The kernels read the items from the caller's device scratch; the library writes the checked host items there on
// the call's stream before its first launch, so no unchecked item reaches a kernel.
kvc_status upload_items(const kvc_batch* b, hipStream_t stream) {
  const size_t bytes = static_cast<size_t>(b->num_items) * sizeof(kvc_item);
  return hip_status(hipMemcpyAsync(b->item_scratch, b->items, bytes, hipMemcpyHostToDevice, stream));
}

const kvc_item* device_items(const kvc_batch* b) { return static_cast<const kvc_item*>(b->item_scratch); }

// With both tables NULL all items address the same identity-mapped rows: no destination range of the call may overlap
// a source range or another destination range.  Sorted sweep over the row ranges of every item.
bool contiguous_ranges_overlap(const kvc_batch* b) {
  struct Range {
    int64_t begin, end;
    bool dst;
  };
  std::vector<Range> rs;
  rs.reserve(2 * static_cast<size_t>(b->num_items));
  for (int32_t i = 0; i < b->num_items; ++i) {
    const kvc_item& it = b->items[i];
    if (it.num_tokens <= 0) continue;
    rs.push_back({it.src_offset, static_cast<int64_t>(it.src_offset) + it.num_tokens, false});
    rs.push_back({it.dst_offset, static_cast<int64_t>(it.dst_offset) + it.num_tokens, true});
  }
  std::sort(rs.begin(), rs.end(), [](const Range& x, const Range& y) { return x.begin < y.begin; });
  // every range is compared with the open ranges before it: the furthest-reaching source and destination so far
  int64_t src_end = INT64_MIN, dst_end = INT64_MIN;
  for (const Range& r : rs) {
    if (r.dst && (src_end > r.begin || dst_end > r.begin)) return true;
    if (!r.dst && dst_end > r.begin) return true;
    (r.dst ? dst_end : src_end) = std::max(r.dst ? dst_end : src_end, r.end);
  }
  return false;
}

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Workspace layout and launch grouping of a fit call.  Units are processed in groups of at most 128 layers and as
// many items as keep items x layers below 65536; the workspace holds one group.  A unit's Gram is split into
// max_parts partials of part_tokens rows (one Gram wave each).
struct FitPlan {
  int32_t layers_per_group = 1, items_per_group = 1, part_tokens = 256, max_parts = 1;
  size_t units = 0, off_partials = 0, off_reflect = 0, off_beta = 0, off_vecs = 0, total = 0;
};

constexpr int64_t kGramWaveTarget = 2048;  // Gram waves per fit launch

FitPlan plan_fit(const kvc_cache* c, const kvc_batch* b, int32_t lb, int32_t le) {
  FitPlan p;
  const int32_t nl = le - lb;
  if (nl <= 0 || b->num_items <= 0) return p;
  p.layers_per_group = std::min<int32_t>(nl, kvc::kMaxLayersPerLaunch);
  p.items_per_group = std::max<int32_t>(1, std::min<int32_t>(b->num_items, 65535 / p.layers_per_group));
  int32_t tmax = 0;
  int64_t tsum = 0;
  for (int32_t i = 0; i < b->num_items; ++i)
    if (b->items[i].state.rank > 0) {
      tmax = std::max(tmax, b->items[i].state.num_tokens);
      tsum += b->items[i].state.num_tokens;
    }
  const int64_t d = c->head_dim;
  p.units = static_cast<size_t>(p.items_per_group) * p.layers_per_group * 2 * c->num_kv_heads;
  // one partial per Gram wave: the rows a launch group holds (on average over the groups) cut into about
  // kGramWaveTarget equal ranges, so ragged batches fill the chip as well as uniform ones; a multiple of 4 partials
  // per unit
  const int64_t group_rows =
      tsum * p.items_per_group / b->num_items * p.layers_per_group * 2 * c->num_kv_heads;
  int64_t part = (std::max<int64_t>(group_rows, 1) + kGramWaveTarget - 1) / kGramWaveTarget;
  part = std::max<int64_t>(256, (part + 31) / 32 * 32);
  p.part_tokens = static_cast<int32_t>(part);
  p.max_parts = static_cast<int32_t>(std::max<int64_t>(1, (tmax + part - 1) / part));
  p.max_parts = (p.max_parts + 3) / 4 * 4;
  size_t off = 0;
  p.off_partials = off;
  off = align256(off + p.units * p.max_parts * d * d * sizeof(float));
  p.off_reflect = off;
  off = align256(off + p.units * d * d * sizeof(double));
  p.off_beta = off;
  off = align256(off + p.units * d * sizeof(double));
  p.off_vecs = off;
  off = align256(off + p.units * KVC_MAX_RANK * d * sizeof(double));
  p.total = off;
  return p;
}

// Per-layer fit (KVC_GROUP_LAYER): items one at a time, all layers of the call (up to the launch limit) together;
// at most 8 token partials per layer unit (a partial of D = H d is up to 4 MB).
struct LayerPlan {
  int32_t layers_per_group = 1, part_tokens = 256, max_parts = 1, k = 64;
  size_t units = 0, off_partials = 0, off_gram = 0, off_x = 0, off_y = 0, off_h = 0, off_spart = 0, off_eps = 0,
         off_vrows = 0, off_vsigma = 0, off_reflect = 0, off_beta = 0, off_vecs = 0, off_resid = 0, off_conv = 0,
         off_iters = 0, total = 0;
};

// Which calls the per-layer path takes (every item per layer, D = H d <= 1024, rank + 16 <= k; rotary keys with bf16
// caches need the LDS Gram: a power-of-two block size of at least 8 and every head of a row within 2 GiB).
kvc_status check_layer_fit(const kvc_cache* c, const kvc_batch* b) {
  const int32_t DL = c->num_kv_heads * c->head_dim;
  if (DL > 1024) return KVC_ERR_UNSUPPORTED;
  if (c->rope_style != KVC_ROPE_NONE && c->dtype == KVC_BF16) {
    bool pow2 = false;
    for (int32_t sh = 3; sh < 31; ++sh) pow2 = pow2 || (int32_t{1} << sh) == c->block_size;
    const bool small_rows = 2 * (static_cast<int64_t>(c->num_kv_heads - 1) * c->head_stride + c->head_dim) <
                            (int64_t{1} << 31);
    if (!pow2 || !small_rows) return KVC_ERR_UNSUPPORTED;
  }
  for (int32_t i = 0; i < b->num_items; ++i) {
    const kvc_state& st = b->items[i].state;
    if (st.grouping != KVC_GROUP_LAYER) return KVC_ERR_UNSUPPORTED;
    const int32_t k = st.rank + 16 <= 64 ? 64 : 128;
    if (st.rank + 16 > 128 || k > DL) return KVC_ERR_UNSUPPORTED;
    // float32: the projection holds the basis and the rotary angle tables (1 KiB) in LDS
    if (c->dtype == KVC_F32 && static_cast<size_t>(st.rank) * DL * 4 + 1024 > 160 * 1024) return KVC_ERR_UNSUPPORTED;
  }
  return KVC_OK;
}

LayerPlan plan_layer_fit(const kvc_cache* c, const kvc_batch* b, int32_t lb, int32_t le) {
  LayerPlan p;
  const int32_t nl = le - lb;
  if (nl <= 0 || b->num_items <= 0) return p;
  p.layers_per_group = std::min<int32_t>(nl, kvc::kMaxLayersPerLaunch);
  int32_t tmax = 0, rmax = 0;
  for (int32_t i = 0; i < b->num_items; ++i) {
    tmax = std::max(tmax, b->items[i].state.num_tokens);
    rmax = std::max(rmax, b->items[i].state.rank);
  }
  p.k = rmax + 16 <= 64 ? 64 : 128;
  const size_t DL = static_cast<size_t>(c->num_kv_heads) * c->head_dim, k = p.k;
  p.units = static_cast<size_t>(p.layers_per_group) * 2;
  // token ranges per unit: enough for about 1024 workgroups of the LDS Gram (one per unit, token range and pair of
  // 256-feature groups), at least two and at least 256 tokens each; more ranges than that only add fp32 partials to
  // write and to reduce (8B/32K, 64 units: two 16384-token ranges, 1280 workgroups)
  const int64_t ng = static_cast<int64_t>((DL + 255) / 256);
  const int64_t per_range = static_cast<int64_t>(p.units) * ng * (ng + 1) / 2;
  const int64_t nranges = std::max<int64_t>(2, (1024 + per_range - 1) / per_range);
  int64_t part = (std::max<int32_t>(tmax, 1) + nranges - 1) / nranges;
  part = std::max<int64_t>(256, (part + 31) / 32 * 32);
  p.part_tokens = static_cast<int32_t>(part);
  p.max_parts = static_cast<int32_t>(std::max<int64_t>(1, (tmax + part - 1) / part));
  p.max_parts = (p.max_parts + 1) / 2 * 2;  // two token ranges per Gram workgroup
  const size_t U = p.units;
  size_t off = 0;
  p.off_partials = off;
  off = align256(off + U * p.max_parts * DL * DL * sizeof(float));
  p.off_gram = off;
  off = align256(off + U * DL * DL * sizeof(double));
  p.off_x = off;
  off = align256(off + U * k * DL * sizeof(double));
  p.off_y = off;
  off = align256(off + U * k * DL * sizeof(double));
  p.off_h = off;
  off = align256(off + U * k * k * sizeof(double));
  p.off_spart = off;
  off = align256(off + U * ((DL + 255) / 256) * k * k * sizeof(double));
  p.off_eps = off;
  off = align256(off + 2 * U * sizeof(double));
  p.off_vrows = off;
  off = align256(off + U * KVC_MAX_RANK * k * sizeof(float));
  p.off_vsigma = off;
  off = align256(off + U * KVC_MAX_RANK * sizeof(float));
  p.off_reflect = off;
  off = align256(off + U * k * k * sizeof(double));
  p.off_beta = off;
  off = align256(off + U * k * sizeof(double));
  p.off_vecs = off;
  off = align256(off + U * KVC_MAX_RANK * k * sizeof(double));
  p.off_resid = off;
  off = align256(off + U * KVC_MAX_RANK * sizeof(double));
  p.off_conv = off;
  off = align256(off + U * sizeof(int32_t));
  p.off_iters = off;
  off = align256(off + U * sizeof(int32_t));
  p.total = off;
  return p;
}

bool batch_is_per_layer(const kvc_batch* b) {
  for (int32_t i = 0; i < b->num_items; ++i)
    if (b->items[i].state.grouping == KVC_GROUP_LAYER) return true;
  return false;
}

kvc_status check_chain(const kvc_state* a, const kvc_state* b, const kvc_state* o, int32_t lb, int32_t le) {
  if (!a || !b || !o) return KVC_ERR_NULL_ARG;
  const int32_t L = a->num_layers, H = a->num_kv_heads, d = a->head_dim;
  if (d != 64 && d != 128) return KVC_ERR_UNSUPPORTED;
  if (L < 1 || H < 1) return KVC_ERR_SHAPE;
  for (const kvc_state* s : {a, b, o}) {
    kvc_status st = check_state_shape(*s, L, H, d);
    if (st != KVC_OK) return st;
    if (s->grouping != KVC_GROUP_HEAD) return KVC_ERR_UNSUPPORTED;
  }
  if (b->coef_dtype != a->coef_dtype || o->coef_dtype != a->coef_dtype) return KVC_ERR_DTYPE;
  if (lb < 0 || le < lb || le > L) return KVC_ERR_SHAPE;
  if (o->num_tokens != std::max(a->num_tokens, b->num_tokens)) return KVC_ERR_SHAPE;
  if (o->rank > std::min<int32_t>({a->rank + b->rank, d, o->num_tokens})) return KVC_ERR_SHAPE;
  // the output must not overwrite an input
  if (o->rank > 0 && o->num_tokens > 0) {
    for (const kvc_state* s : {a, b}) {
      if (s->rank > 0 && (o->coef == s->coef || o->basis == s->basis)) return KVC_ERR_ALIAS;
    }
  }
  return KVC_OK;
}

// Chain workspace: H partials (chunks sized as in the fit), the fp64 intermediates of G = K H K^T, the eigensolver
// scratch and Y.
struct ChainPlan {
  int32_t mp = 16, part_tokens = 256, max_parts = 1, gram_wave_ft = 0;
  size_t units = 0, off_partials = 0, off_hsum = 0, off_pmat = 0, off_gram = 0, off_reflect = 0, off_beta = 0,
         off_vecs = 0, off_ymat = 0, total = 0;
};

ChainPlan plan_chain(const kvc_state* a, const kvc_state* b, const kvc_state* o, int32_t lb, int32_t le) {
  ChainPlan p;
  const size_t d = a->head_dim;
  const size_t m = static_cast<size_t>(a->rank) + b->rank;
  p.mp = static_cast<int32_t>(std::max<size_t>(16, (m + 15) / 16 * 16));
  // bf16 coefficients whose ranks split into whole FT-wide segments use the LDS-free wave Gram
  if (a->coef_dtype == KVC_BF16) {
    for (int32_t ft : {2, 4, 8}) {
      if (m <= static_cast<size_t>(16 * ft) && a->rank % ft == 0 && b->rank % ft == 0) {
        p.gram_wave_ft = ft;
        p.mp = 16 * ft;
        break;
      }
    }
  }
  p.units = static_cast<size_t>(le - lb) * 2 * a->num_kv_heads;
  const int64_t T = std::max<int32_t>(o->num_tokens, 1);
  // the wave Gram has one partial per wave (about 2048 per call, a multiple of 4 per unit); the LDS Gram one per
  // workgroup (about 4096 per call)
  const int64_t target = p.gram_wave_ft ? 2048 : 4096;
  const int64_t want_parts = std::max<int64_t>(1, (target + static_cast<int64_t>(p.units) - 1) /
                                                      std::max<int64_t>(1, static_cast<int64_t>(p.units)));
  int64_t part = (T + want_parts - 1) / want_parts;
  part = std::max<int64_t>(256, (part + 31) / 32 * 32);
  p.part_tokens = static_cast<int32_t>(part);
  p.max_parts = static_cast<int32_t>((T + part - 1) / part);
  if (p.gram_wave_ft) p.max_parts = (p.max_parts + 3) / 4 * 4;
  const size_t U = p.units, mp = p.mp;
  size_t off = 0;
  p.off_partials = off;
  off = align256(off + U * p.max_parts * mp * mp * sizeof(float));
  p.off_hsum = off;
  off = align256(off + U * m * m * sizeof(double));
  p.off_pmat = off;
  off = align256(off + U * m * d * sizeof(double));
  p.off_gram = off;
  off = align256(off + U * d * d * sizeof(double));
  p.off_reflect = off;
  off = align256(off + U * d * d * sizeof(double));
  p.off_beta = off;
  off = align256(off + U * d * sizeof(double));
  p.off_vecs = off;
  off = align256(off + U * KVC_MAX_RANK * d * sizeof(double));
  p.off_ymat = off;
  off = align256(off + U * m * static_cast<size_t>(o->rank) * sizeof(float));
  p.total = off;
  return p;
}

void fill_pool_view(const kvc_cache* c, kvc::PoolView& pv) {
  pv.block_stride = c->block_stride;
  pv.token_stride = c->token_stride;
  pv.head_stride = c->head_stride;
  pv.block_size = c->block_size;
  pv.num_blocks = c->num_blocks;
  pv.num_kv_heads = c->num_kv_heads;
  pv.head_dim = c->head_dim;
  pv.block_shift = -1;
  for (int32_t sh = 0; sh < 31; ++sh)
    if ((int32_t{1} << sh) == c->block_size) pv.block_shift = sh;
  std::memset(&pv.rope, 0, sizeof(pv.rope));
  pv.rope.style = c->rope_style;
  if (c->rope_style != KVC_ROPE_NONE)
    for (int32_t i = 0; i < c->head_dim / 2; ++i) pv.rope.inv_freq[i] = c->rope_inv_freq[i];
}


// Checks shared by the anchor entry points: one item, the anchor states, the weighted rows.
kvc_status check_anchor_call(const kvc_cache* c, const kvc_batch* b, const kvc_anchors* an, int32_t lb, int32_t le,
                             bool needs_dst, bool needs_weights) {
  kvc_status s = check_cache(c, lb, le);
  if (s != KVC_OK) return s;
  if (!b || !an) return KVC_ERR_NULL_ARG;
  if (b->num_items != 1 || b->max_blocks < 0) return KVC_ERR_SHAPE;
  if (!b->items) return KVC_ERR_NULL_ARG;
  if ((b->src_tables || b->dst_tables) && b->max_blocks < 1) return KVC_ERR_SHAPE;
  const kvc_item& it = b->items[0];
  if (it.reserved != 0 || it.num_tokens < 0 || it.src_position < 0 || it.dst_position < 0) return KVC_ERR_SHAPE;
  if (!positions_fit(it.src_offset, it.num_tokens, b->src_tables != nullptr, b, c)) return KVC_ERR_SHAPE;
  if (needs_dst && !positions_fit(it.dst_offset, it.num_tokens, b->dst_tables != nullptr, b, c)) return KVC_ERR_SHAPE;
  if (an->num_anchors < 1 || an->num_anchors > KVC_MAX_ANCHORS) return KVC_ERR_SHAPE;
  if (!an->states) return KVC_ERR_NULL_ARG;
  if (an->num_tokens < 0 || an->num_tokens > it.num_tokens) return KVC_ERR_SHAPE;
  if (needs_weights && !an->weights) return KVC_ERR_NULL_ARG;
  for (int32_t v = 0; v < an->num_anchors; ++v) {
    const kvc_state& st = an->states[v];
    s = check_state_shape(st, c->num_layers, c->num_kv_heads, c->head_dim);
    if (s != KVC_OK) return s;
    if (st.grouping != KVC_GROUP_HEAD) return KVC_ERR_UNSUPPORTED;
    if (st.coef_dtype != c->dtype) return KVC_ERR_DTYPE;
    if (st.rank < 1 || st.num_tokens < an->num_tokens) return KVC_ERR_SHAPE;
    if (!st.coef || !st.basis) return KVC_ERR_NULL_ARG;
  }
  return KVC_OK;
}

void fill_anchor_args(const kvc_cache* c, const kvc_batch* b, const kvc_anchors* an, int32_t lb, int32_t le,
                      kvc::AnchorArgs& a) {
  std::memset(&a, 0, sizeof(a));
  fill_pool_view(c, a.pv);
  const kvc_item& it = b->items[0];
  a.src_table = b->src_tables;
  a.dst_table = b->dst_tables;
  a.src_offset = it.src_offset;
  a.dst_offset = it.dst_offset;
  a.src_position = it.src_position;
  a.dst_position = it.dst_position;
  a.num_tokens = it.num_tokens;
  a.num_weighted = an->num_tokens;
  a.layer_begin = lb;
  a.num_layers = le - lb;
  for (int32_t l = lb; l < le; ++l) {
    a.layers.k[l - lb] = c->k_layers[l];
    a.layers.v[l - lb] = c->v_layers[l];
  }
  a.num_anchors = an->num_anchors;
  for (int32_t v = 0; v < an->num_anchors; ++v) {
    a.rank[v] = an->states[v].rank;
    a.tokens[v] = an->states[v].num_tokens;
    a.coef[v] = an->states[v].coef;
    a.basis[v] = an->states[v].basis;
    a.max_rank = std::max(a.max_rank, an->states[v].rank);
  }
  a.weights = an->weights;
  a.inv_temperature = 1.0f;
}

// Anchor-pool bookkeeping (Appendix A.3): slots with id, stored length, use count and insertion order.
struct PoolSlot {
  bool used = false;
  int64_t id = -1, uses = 0, order = 0;
  int32_t length = 0;
};

}  // namespace

// Allocation-free gate: the partial sums live in this static array instead of a caller workspace.  Host code never
// passes the array's name to a kernel (in host code it is only a stand-in for the symbol); it uses the device address
// that hipGetSymbolAddress returns, taken once per device with that device current.
static __device__ __align__(256) float scratch[KVC_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of `scratch` on the device of `stream` (the null stream: the current device).
kvc_status scratch_address(hipStream_t stream, float** out) {
  int dev = -1;
  kvc_status s = hip_status(hipStreamGetDevice(stream, &dev));
  if (s != KVC_OK) return s;
  if (dev < 0 || dev >= kMaxScratchDevices) return KVC_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = -1;
    s = hip_status(hipGetDevice(&cur));
    if (s != KVC_OK) return s;
    if (cur != dev && (s = hip_status(hipSetDevice(dev))) != KVC_OK) return s;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if ((s = hip_status(e)) != KVC_OK) return s;
    if (!p) return KVC_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = static_cast<float*>(g_scratch_ptr[dev]);
  return KVC_OK;
}

}  // namespace

struct kvc_pool {
  std::vector<PoolSlot> slots;
  int64_t clock = 0;
};

namespace {
}  // namespace

extern "C" {

int32_t kvc_version(void) { return KVC_VERSION; }

const char* kvc_status_str(kvc_status s) {
  switch (s) {
    case KVC_OK: return "ok";
    case KVC_ERR_NULL_ARG: return "null argument";
    case KVC_ERR_SHAPE: return "inconsistent or out-of-range sizes";
    case KVC_ERR_DTYPE: return "unsupported or mismatched dtype";
    case KVC_ERR_ALIGN: return "pointer or stride not 16-byte aligned";
    case KVC_ERR_ALIAS: return "destination rows may overlap source rows";
    case KVC_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case KVC_ERR_UNSUPPORTED: return "head_dim other than 64 or 128, or a grouping or rotary setting the call does not take";
    case KVC_ERR_HIP: return "HIP runtime error";
    case KVC_ERR_TOO_LARGE: return "the call needs more than the static scratch of the allocation-free entry point";
  }
  return "unknown status";
}

int32_t kvc_last_hip_error(void) { return g_last_hip_error; }

size_t kvc_item_scratch_bytes(int32_t num_items) {
  return num_items > 0 ? static_cast<size_t>(num_items) * sizeof(kvc_item) : 0;
}

size_t kvc_state_bytes(int32_t L, int32_t H, int32_t d, int32_t T, int32_t r, kvc_dtype coef_dtype) {
  if (L < 0 || H < 0 || d < 0 || T < 0 || r < 0 || !valid_dtype(coef_dtype)) return 0;
  const size_t units = static_cast<size_t>(L) * 2 * H;
  return units * (static_cast<size_t>(T) * r * dtype_size(coef_dtype) + static_cast<size_t>(r) * d * 4 +
                  static_cast<size_t>(r) * 4);
}

size_t kvc_layer_state_bytes(int32_t L, int32_t H, int32_t d, int32_t T, int32_t r, kvc_dtype coef_dtype) {
  if (L < 0 || H < 0 || d < 0 || T < 0 || r < 0 || !valid_dtype(coef_dtype)) return 0;
  const size_t units = static_cast<size_t>(L) * 2;
  return units * (static_cast<size_t>(T) * r * dtype_size(coef_dtype) + static_cast<size_t>(r) * H * d * 4 +
                  static_cast<size_t>(r) * 4);
}

size_t kvc_dense_bytes(int32_t L, int32_t H, int32_t d, int32_t T, kvc_dtype dtype) {
  if (L < 0 || H < 0 || d < 0 || T < 0 || !valid_dtype(dtype)) return 0;
  return static_cast<size_t>(L) * 2 * H * static_cast<size_t>(T) * d * dtype_size(dtype);
}

kvc_status kvc_apply(const kvc_cache* cache, const kvc_batch* batch, int32_t layer_begin, int32_t layer_end,
                     hipStream_t stream) {
  kvc_status s = check_cache(cache, layer_begin, layer_end);
  if (s != KVC_OK) return s;
  s = check_batch(cache, batch, true);
  if (s != KVC_OK) return s;
  if (batch->src_tables && batch->src_tables == batch->dst_tables) return KVC_ERR_ALIAS;
  int max_tokens = 0, max_rank = 0;
  for (int32_t i = 0; i < batch->num_items; ++i) {
    const kvc_item& it = batch->items[i];
    max_tokens = std::max(max_tokens, it.num_tokens);
    max_rank = std::max(max_rank, it.state.rank);
  }
  if (!batch->src_tables && !batch->dst_tables && contiguous_ranges_overlap(batch)) return KVC_ERR_ALIAS;
  if (batch->num_items == 0 || layer_end == layer_begin || max_tokens == 0) return KVC_OK;
  s = upload_items(batch, stream);
  if (s != KVC_OK) return s;
  kvc::ApplyArgs a;
  std::memset(&a, 0, sizeof(a));
  fill_pool_view(cache, a.pv);
  a.items = device_items(batch);
  a.src_tables = batch->src_tables;
  a.dst_tables = batch->dst_tables;
  a.max_blocks = batch->max_blocks;
  for (int32_t l0 = layer_begin; l0 < layer_end; l0 += kvc::kMaxLayersPerLaunch) {
    const int32_t l1 = std::min(layer_end, l0 + kvc::kMaxLayersPerLaunch);
    a.layer_begin = l0;
    a.num_layers = l1 - l0;
    for (int32_t l = l0; l < l1; ++l) {
      a.layers.k[l - l0] = cache->k_layers[l];
      a.layers.v[l - l0] = cache->v_layers[l];
    }
    // grid.z = items x layers must stay below 65536
    const int32_t per_launch_items = std::max<int32_t>(1, 65535 / a.num_layers);
    for (int32_t i0 = 0; i0 < batch->num_items; i0 += per_launch_items) {
      const int32_t n = std::min(per_launch_items, batch->num_items - i0);
      kvc::ApplyArgs ai = a;
      ai.items = device_items(batch) + i0;
      ai.src_tables = batch->src_tables ? batch->src_tables + static_cast<int64_t>(i0) * batch->max_blocks : nullptr;
      ai.dst_tables = batch->dst_tables ? batch->dst_tables + static_cast<int64_t>(i0) * batch->max_blocks : nullptr;
      s = hip_status(kvc::launch_apply(ai, cache->dtype, max_rank, max_tokens, n, stream));
      if (s != KVC_OK) return s;
    }
  }
  return KVC_OK;
}

size_t kvc_fit_workspace_bytes(const kvc_cache* cache, const kvc_batch* batch, int32_t layer_begin,
                               int32_t layer_end) {
  if (check_cache(cache, layer_begin, layer_end) != KVC_OK || !batch || batch->num_items < 0) return 0;
  if (batch->num_items > 0 && !batch->items) return 0;
  if (batch_is_per_layer(batch)) {
    if (check_layer_fit(cache, batch) != KVC_OK) return 0;
    return plan_layer_fit(cache, batch, layer_begin, layer_end).total;
  }
  return plan_fit(cache, batch, layer_begin, layer_end).total;
}

// Per-layer fit: for each item and group of layers, the head-pair Gram, the subspace iteration with its
// Rayleigh-Ritz eigenproblem, the basis rows and the multi-head projection.
kvc_status fit_per_layer(const kvc_cache* cache, const kvc_batch* batch, int32_t layer_begin, int32_t layer_end,
                         kvc_fit_mode mode, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  const LayerPlan p = plan_layer_fit(cache, batch, layer_begin, layer_end);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) || workspace_bytes < p.total)
    return KVC_ERR_WORKSPACE;
  kvc_status s = upload_items(batch, stream);
  if (s != KVC_OK) return s;
  char* ws = static_cast<char*>(workspace);
  kvc::LayerFitArgs la;
  std::memset(&la, 0, sizeof(la));
  fill_pool_view(cache, la.pv);
  la.max_blocks = batch->max_blocks;
  la.mode = mode;
  la.k = p.k;
  la.max_parts = p.max_parts;
  la.part_tokens = p.part_tokens;
  la.partials = reinterpret_cast<float*>(ws + p.off_partials);
  la.gram = reinterpret_cast<double*>(ws + p.off_gram);
  la.x = reinterpret_cast<double*>(ws + p.off_x);
  la.y = reinterpret_cast<double*>(ws + p.off_y);
  la.hmat = reinterpret_cast<double*>(ws + p.off_h);
  la.spart = reinterpret_cast<double*>(ws + p.off_spart);
  la.eps = reinterpret_cast<double*>(ws + p.off_eps);
  la.vrows = reinterpret_cast<float*>(ws + p.off_vrows);
  la.vsigma = reinterpret_cast<float*>(ws + p.off_vsigma);
  la.resid = reinterpret_cast<double*>(ws + p.off_resid);
  la.conv = reinterpret_cast<int32_t*>(ws + p.off_conv);
  la.iters = reinterpret_cast<int32_t*>(ws + p.off_iters);
  for (int32_t i = 0; i < batch->num_items; ++i) {
    const kvc_state& st = batch->items[i].state;
    if (st.rank == 0 || st.num_tokens == 0) continue;
    la.rank = st.rank;
    la.items = device_items(batch) + i;
    la.src_tables = batch->src_tables ? batch->src_tables + static_cast<int64_t>(i) * batch->max_blocks : nullptr;
    la.dst_tables = batch->dst_tables ? batch->dst_tables + static_cast<int64_t>(i) * batch->max_blocks : nullptr;
    for (int32_t l0 = layer_begin; l0 < layer_end; l0 += p.layers_per_group) {
      const int32_t l1 = std::min(layer_end, l0 + p.layers_per_group);
      la.layer_begin = l0;
      la.num_layers = l1 - l0;
      la.num_units = 2 * la.num_layers;
      for (int32_t l = l0; l < l1; ++l) {
        la.layers.k[l - l0] = cache->k_layers[l];
        la.layers.v[l - l0] = cache->v_layers[l];
      }
      // the Rayleigh-Ritz eigenproblem of each layer unit, through the dense-input eigensolver into scratch rows
      kvc::EigArgs ea;
      std::memset(&ea, 0, sizeof(ea));
      ea.n = p.k;
      ea.num_units = la.num_units;
      ea.dense = la.hmat;
      ea.items = nullptr;
      ea.state.num_layers = la.num_layers;
      ea.state.num_kv_heads = 1;
      ea.state.head_dim = p.k;
      ea.state.num_tokens = st.num_tokens;
      ea.state.rank = st.rank;
      ea.state.coef_dtype = cache->dtype;
      ea.state.basis = la.vrows;
      ea.state.sigma = la.vsigma;
      ea.layer_begin = 0;
      ea.num_layers = la.num_layers;
      ea.num_kv_heads = 1;
      ea.reflect = reinterpret_cast<double*>(ws + p.off_reflect);
      ea.reflect_beta = reinterpret_cast<double*>(ws + p.off_beta);
      ea.vecs = reinterpret_cast<double*>(ws + p.off_vecs);
      ea.seed = 0x1A7Eu;
      s = hip_status(kvc::launch_layer_gram(la, cache->dtype, stream));
      if (s != KVC_OK) return s;
      s = hip_status(kvc::launch_layer_subspace(la, ea, stream));
      if (s != KVC_OK) return s;
      s = hip_status(kvc::launch_layer_proj(la, cache->dtype, st.num_tokens, stream));
      if (s != KVC_OK) return s;
    }
  }
  return KVC_OK;
}

kvc_status kvc_fit_state(const kvc_cache* cache, const kvc_batch* batch, int32_t layer_begin, int32_t layer_end,
                         kvc_fit_mode mode, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  kvc_status s = check_cache(cache, layer_begin, layer_end);
  if (s != KVC_OK) return s;
  if (mode != KVC_FIT_DELTA && mode != KVC_FIT_BASE) return KVC_ERR_SHAPE;
  s = check_batch(cache, batch, mode == KVC_FIT_DELTA);
  if (s != KVC_OK) return s;
  int max_rank = 0, max_tokens = 0;
  for (int32_t i = 0; i < batch->num_items; ++i) {
    const kvc_state& st = batch->items[i].state;
    // Eq. 7 keeps at most min(T_s, d) singular triplets
    if (st.rank > st.num_tokens) return KVC_ERR_SHAPE;
    max_rank = std::max(max_rank, st.rank);
    if (st.rank > 0) max_tokens = std::max(max_tokens, st.num_tokens);
  }
  if (batch_is_per_layer(batch)) {
    s = check_layer_fit(cache, batch);
    if (s != KVC_OK) return s;
  }
  if (batch->num_items == 0 || layer_end == layer_begin || max_rank == 0) return KVC_OK;
  if (batch_is_per_layer(batch))
    return fit_per_layer(cache, batch, layer_begin, layer_end, mode, workspace, workspace_bytes, stream);
  const FitPlan p = plan_fit(cache, batch, layer_begin, layer_end);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) || workspace_bytes < p.total)
    return KVC_ERR_WORKSPACE;
  s = upload_items(batch, stream);
  if (s != KVC_OK) return s;
  char* ws = static_cast<char*>(workspace);

  kvc::FitArgs fa;
  std::memset(&fa, 0, sizeof(fa));
  fill_pool_view(cache, fa.pv);
  fa.max_blocks = batch->max_blocks;
  fa.mode = mode;
  fa.partials = reinterpret_cast<float*>(ws + p.off_partials);
  fa.max_parts = p.max_parts;
  fa.part_tokens = p.part_tokens;
  kvc::EigArgs ea;
  std::memset(&ea, 0, sizeof(ea));
  ea.n = cache->head_dim;
  ea.partials = fa.partials;
  ea.max_parts = p.max_parts;
  ea.part_tokens = p.part_tokens;
  ea.num_kv_heads = cache->num_kv_heads;
  ea.reflect = reinterpret_cast<double*>(ws + p.off_reflect);
  ea.reflect_beta = reinterpret_cast<double*>(ws + p.off_beta);
  ea.vecs = reinterpret_cast<double*>(ws + p.off_vecs);
  ea.seed = 0x5EEDu;
  for (int32_t l0 = layer_begin; l0 < layer_end; l0 += p.layers_per_group) {
    const int32_t l1 = std::min(layer_end, l0 + p.layers_per_group);
    fa.layer_begin = ea.layer_begin = l0;
    fa.num_layers = ea.num_layers = l1 - l0;
    for (int32_t l = l0; l < l1; ++l) {
      fa.layers.k[l - l0] = cache->k_layers[l];
      fa.layers.v[l - l0] = cache->v_layers[l];
    }
    for (int32_t i0 = 0; i0 < batch->num_items; i0 += p.items_per_group) {
      const int32_t n = std::min(p.items_per_group, batch->num_items - i0);
      fa.items = ea.items = device_items(batch) + i0;
      fa.src_tables = batch->src_tables ? batch->src_tables + static_cast<int64_t>(i0) * batch->max_blocks : nullptr;
      fa.dst_tables = batch->dst_tables ? batch->dst_tables + static_cast<int64_t>(i0) * batch->max_blocks : nullptr;
      ea.num_units = n * fa.num_layers * 2 * cache->num_kv_heads;
      s = hip_status(kvc::launch_fit_gram(fa, cache->dtype, n, stream));
      if (s != KVC_OK) return s;
      s = hip_status(kvc::launch_eig(ea, stream));
      if (s != KVC_OK) return s;
      s = hip_status(kvc::launch_fit_proj(fa, cache->dtype, n, max_tokens, max_rank, stream));
      if (s != KVC_OK) return s;
    }
  }
  return KVC_OK;
}
size_t kvc_chain_workspace_bytes(const kvc_state* first, const kvc_state* second, const kvc_state* out,
                                 int32_t layer_begin, int32_t layer_end) {
  if (check_chain(first, second, out, layer_begin, layer_end) != KVC_OK) return 0;
  return plan_chain(first, second, out, layer_begin, layer_end).total;
}

kvc_status kvc_chain(const kvc_state* first, const kvc_state* second, kvc_state* out, int32_t layer_begin,
                     int32_t layer_end, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  kvc_status s = check_chain(first, second, out, layer_begin, layer_end);
  if (s != KVC_OK) return s;
  if (layer_end == layer_begin || out->rank == 0 || out->num_tokens == 0) return KVC_OK;
  const ChainPlan p = plan_chain(first, second, out, layer_begin, layer_end);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) || workspace_bytes < p.total)
    return KVC_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  kvc::ChainArgs ca;
  std::memset(&ca, 0, sizeof(ca));
  ca.first = *first;
  ca.second = *second;
  ca.out = *out;
  ca.layer_begin = layer_begin;
  ca.num_layers = layer_end - layer_begin;
  ca.num_units = static_cast<int32_t>(p.units);
  ca.mp = p.mp;
  ca.gram_wave_ft = p.gram_wave_ft;
  ca.partials = reinterpret_cast<float*>(ws + p.off_partials);
  ca.max_parts = p.max_parts;
  ca.part_tokens = p.part_tokens;
  ca.hsum = reinterpret_cast<double*>(ws + p.off_hsum);
  ca.pmat = reinterpret_cast<double*>(ws + p.off_pmat);
  ca.gram = reinterpret_cast<double*>(ws + p.off_gram);
  ca.ymat = reinterpret_cast<float*>(ws + p.off_ymat);
  kvc::EigArgs ea;
  std::memset(&ea, 0, sizeof(ea));
  ea.n = first->head_dim;
  ea.num_units = ca.num_units;
  ea.dense = ca.gram;
  ea.state = *out;
  ea.layer_begin = layer_begin;
  ea.num_layers = ca.num_layers;
  ea.num_kv_heads = first->num_kv_heads;
  ea.reflect = reinterpret_cast<double*>(ws + p.off_reflect);
  ea.reflect_beta = reinterpret_cast<double*>(ws + p.off_beta);
  ea.vecs = reinterpret_cast<double*>(ws + p.off_vecs);
  ea.seed = 0xC4A1u;
  return hip_status(kvc::launch_chain(ca, ea, stream));
}

kvc_status kvc_anchor_weights(const kvc_cache* cache, const kvc_batch* batch, const kvc_anchors* anchors,
                              int32_t layer_begin, int32_t layer_end, float temperature, hipStream_t stream) {
  kvc_status s = check_anchor_call(cache, batch, anchors, layer_begin, layer_end, false, true);
  if (s != KVC_OK) return s;
  if (!(temperature > 0.0f) || !std::isfinite(temperature)) return KVC_ERR_SHAPE;
  if (layer_end - layer_begin > kvc::kMaxLayersPerLaunch) return KVC_ERR_SHAPE;
  if (anchors->num_tokens == 0 || layer_end == layer_begin) return KVC_OK;
  kvc::AnchorArgs a;
  fill_anchor_args(cache, batch, anchors, layer_begin, layer_end, a);
  a.inv_temperature = 1.0f / temperature;
  return hip_status(kvc::launch_anchor_weights(a, cache->dtype, stream));
}

kvc_status kvc_apply_anchored(const kvc_cache* cache, const kvc_batch* batch, const kvc_anchors* anchors,
                              int32_t layer_begin, int32_t layer_end, hipStream_t stream) {
  kvc_status s = check_anchor_call(cache, batch, anchors, layer_begin, layer_end, true, anchors && anchors->num_tokens > 0);
  if (s != KVC_OK) return s;
  if (layer_end - layer_begin > kvc::kMaxLayersPerLaunch) return KVC_ERR_SHAPE;
  if (batch->src_tables && batch->src_tables == batch->dst_tables) return KVC_ERR_ALIAS;
  const kvc_item& it = batch->items[0];
  if (!batch->src_tables && !batch->dst_tables && it.num_tokens > 0) {
    const int64_t a0 = it.src_offset, a1 = a0 + it.num_tokens, b0 = it.dst_offset, b1 = b0 + it.num_tokens;
    if (a0 < b1 && b0 < a1) return KVC_ERR_ALIAS;
  }
  if (it.num_tokens == 0 || layer_end == layer_begin) return KVC_OK;
  kvc::AnchorArgs a;
  fill_anchor_args(cache, batch, anchors, layer_begin, layer_end, a);
  return hip_status(kvc::launch_apply_anchored(a, cache->dtype, stream));
}

size_t kvc_gate_workspace_bytes(const kvc_cache* cache, const kvc_anchors* anchors, int32_t prefix,
                                int32_t layer_begin, int32_t layer_end) {
  if (check_cache(cache, layer_begin, layer_end) != KVC_OK || !anchors || prefix < 1) return 0;
  if (anchors->num_anchors < 1 || anchors->num_anchors > KVC_MAX_ANCHORS) return 0;
  const int chunk = cache->dtype == KVC_BF16 ? kvc::anchor_chunk_tokens() : 64;
  size_t chunks = static_cast<size_t>((prefix + chunk - 1) / chunk);
  if (cache->dtype == KVC_BF16) {  // bf16 kernels keep one partial per chunk and KV head (512 tokens and up)
    const int res = kvc::anchor_resident_chunk_tokens();
    chunks = std::max(chunks, static_cast<size_t>((prefix + res - 1) / res)) * static_cast<size_t>(cache->num_kv_heads);
  }
  return align256(static_cast<size_t>(layer_end - layer_begin) * chunks * anchors->num_anchors * sizeof(float));
}

kvc_status kvc_gate_distances(const kvc_cache* cache, const kvc_batch* batch, const kvc_anchors* anchors,
                              int32_t prefix, int32_t layer_begin, int32_t layer_end, float* distances,
                              void* workspace, size_t workspace_bytes, hipStream_t stream) {
  kvc_status s = check_anchor_call(cache, batch, anchors, layer_begin, layer_end, false, false);
  if (s != KVC_OK) return s;
  if (!distances) return KVC_ERR_NULL_ARG;
  if (prefix < 1 || prefix > anchors->num_tokens) return KVC_ERR_SHAPE;
  if (layer_end - layer_begin > kvc::kMaxLayersPerLaunch || layer_end == layer_begin) return KVC_ERR_SHAPE;
  const size_t need = kvc_gate_workspace_bytes(cache, anchors, prefix, layer_begin, layer_end);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) || workspace_bytes < need)
    return KVC_ERR_WORKSPACE;
  kvc::AnchorArgs a;
  fill_anchor_args(cache, batch, anchors, layer_begin, layer_end, a);
  a.num_weighted = prefix;
  const int chunk = cache->dtype == KVC_BF16 ? kvc::anchor_chunk_tokens() : 64;
  a.gate_chunks = (prefix + chunk - 1) / chunk;
  a.gate_partials = static_cast<float*>(workspace);
  a.distances = distances;
  return hip_status(kvc::launch_gate_distances(a, cache->dtype, stream));
}

kvc_status kvc_gate_distances_noalloc(const kvc_cache* cache, const kvc_batch* batch, const kvc_anchors* anchors,
                                      int32_t prefix, int32_t layer_begin, int32_t layer_end, float* distances,
                                      hipStream_t stream) {
  kvc_status s = check_anchor_call(cache, batch, anchors, layer_begin, layer_end, false, false);
  if (s != KVC_OK) return s;
  if (!distances) return KVC_ERR_NULL_ARG;
  if (prefix < 1 || prefix > anchors->num_tokens) return KVC_ERR_SHAPE;
  if (layer_end - layer_begin > kvc::kMaxLayersPerLaunch || layer_end == layer_begin) return KVC_ERR_SHAPE;
  if (kvc_gate_workspace_bytes(cache, anchors, prefix, layer_begin, layer_end) > KVC_NOALLOC_SCRATCH_BYTES)
    return KVC_ERR_TOO_LARGE;
  float* partials = nullptr;
  s = scratch_address(stream, &partials);
  if (s != KVC_OK) return s;
  kvc::AnchorArgs a;
  fill_anchor_args(cache, batch, anchors, layer_begin, layer_end, a);
  a.num_weighted = prefix;
  const int chunk = cache->dtype == KVC_BF16 ? kvc::anchor_chunk_tokens() : 64;
  a.gate_chunks = (prefix + chunk - 1) / chunk;
  a.gate_partials = partials;
  a.distances = distances;
  return hip_status(kvc::launch_gate_distances(a, cache->dtype, stream));
}

int32_t kvc_gate_decide(const float* distances, int32_t n, float tau, float temperature, float* gate_weights,
                        float* entropy) {
  if (n < 2 || !distances || !(temperature > 0.0f)) {
    if (entropy) *entropy = 1.0f;
    if (gate_weights && distances)
      for (int32_t v = 0; v < n; ++v) gate_weights[v] = 1.0f;
    return 0;
  }
  double dmin = distances[0];
  for (int32_t v = 1; v < n; ++v) dmin = std::min<double>(dmin, distances[v]);
  std::vector<double> g(static_cast<size_t>(n));
  double sum = 0.0;
  for (int32_t v = 0; v < n; ++v) sum += (g[v] = std::exp(-(distances[v] - dmin) / temperature));
  double h = 0.0;
  for (int32_t v = 0; v < n; ++v) {
    g[v] /= sum;
    if (g[v] > 0.0) h -= g[v] * std::log2(g[v]);
    if (gate_weights) gate_weights[v] = static_cast<float>(g[v]);
  }
  h /= std::log2(static_cast<double>(n));
  if (entropy) *entropy = static_cast<float>(h);
  return h <= tau ? 1 : 0;
}

kvc_pool* kvc_pool_create(int32_t capacity) {
  if (capacity < 1) return nullptr;
  kvc_pool* p = new (std::nothrow) kvc_pool;
  if (p) p->slots.resize(static_cast<size_t>(capacity));
  return p;
}

void kvc_pool_destroy(kvc_pool* pool) { delete pool; }

int32_t kvc_pool_insert(kvc_pool* pool, int64_t anchor_id, int32_t length, int64_t* evicted_id) {
  if (!pool || length < 0) return -1;
  const int32_t cap = static_cast<int32_t>(pool->slots.size());
  int32_t slot = -1;
  int64_t evicted = -1;
  for (int32_t i = 0; i < cap && slot < 0; ++i)
    if (!pool->slots[i].used) slot = i;
  if (slot < 0) {
    // the five oldest slots, then the least used among them (the older one on equal counts)
    std::vector<int32_t> order(static_cast<size_t>(cap));
    for (int32_t i = 0; i < cap; ++i) order[i] = i;
    std::sort(order.begin(), order.end(),
              [&](int32_t x, int32_t y) { return pool->slots[x].order < pool->slots[y].order; });
    const int32_t m = std::min<int32_t>(5, cap);
    slot = order[0];
    for (int32_t i = 1; i < m; ++i) {
      const PoolSlot& c = pool->slots[order[i]];
      const PoolSlot& b = pool->slots[slot];
      if (c.uses < b.uses || (c.uses == b.uses && c.order < b.order)) slot = order[i];
    }
    evicted = pool->slots[slot].id;
  }
  PoolSlot& e = pool->slots[slot];
  e.used = true;
  e.id = anchor_id;
  e.length = length;
  e.uses = 0;
  e.order = pool->clock++;
  if (evicted_id) *evicted_id = evicted;
  return slot;
}

kvc_status kvc_pool_record_use(kvc_pool* pool, const int32_t* slots, int32_t n) {
  if (!pool || (n > 0 && !slots)) return KVC_ERR_NULL_ARG;
  const int32_t cap = static_cast<int32_t>(pool->slots.size());
  for (int32_t i = 0; i < n; ++i)
    if (slots[i] < 0 || slots[i] >= cap || !pool->slots[slots[i]].used) return KVC_ERR_SHAPE;
  for (int32_t i = 0; i < n; ++i) ++pool->slots[slots[i]].uses;
  return KVC_OK;
}

int32_t kvc_pool_eligible(const kvc_pool* pool, int32_t prefix, int32_t* slots) {
  if (!pool) return 0;
  int32_t n = 0;
  for (int32_t i = 0; i < static_cast<int32_t>(pool->slots.size()); ++i)
    if (pool->slots[i].used && pool->slots[i].length >= prefix) {
      if (slots) slots[n] = i;
      ++n;
    }
  return n;
}

kvc_status kvc_pool_slot(const kvc_pool* pool, int32_t slot, int64_t* anchor_id, int32_t* length, int64_t* uses) {
  if (!pool) return KVC_ERR_NULL_ARG;
  if (slot < 0 || slot >= static_cast<int32_t>(pool->slots.size()) || !pool->slots[slot].used) return KVC_ERR_SHAPE;
  const PoolSlot& e = pool->slots[slot];
  if (anchor_id) *anchor_id = e.id;
  if (length) *length = e.length;
  if (uses) *uses = e.uses;
  return KVC_OK;
}

}  // extern "C"
