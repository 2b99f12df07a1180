// Internal interface between the host entry points (kvc_api.cpp) and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include "kvc.h"
#include "kvc_device.h"

namespace kvc {

struct ApplyArgs {
  PoolView pv;
  LayerPtrs layers;            // pools of layers [layer_begin, layer_begin + num_layers)
  const kvc_item* items;       // device
  const int32_t* src_tables;   // device or null
  const int32_t* dst_tables;   // device or null
  int32_t max_blocks;
  int32_t layer_begin;
  int32_t num_layers;
  int32_t kv_begin;            // the launch covers K/V sides kv_begin .. (grid y: one or both sides' heads)
  int32_t chunk_order;         // set by the launcher: kChunksFast, kChunksRotated or kItemsFast (chunk_grid)
};

// Grids of the kernels over (token chunk, unit, item x layer).  Consecutive workgroups are dealt round-robin to the
// eight XCDs, so with the chunks fastest an XCD receives the same chunk indices in every row (unit, item x layer)
// when the row length is a multiple of 8; in a launch over items of different lengths the XCDs that own the late
// chunks then idle while the others work.  Launches over several items therefore either rotate each row's chunk
// order by the row index (kernels whose workgroups in a row share the unit's basis and tables, which then stay
// next to one another), or put the items fastest (the Gram, whose few long partials per row gain most from
// running every item's first partial first).  Measured on 64 requests of 1K-16K tokens at rank 64: projection
// 2.07 -> 1.35 ms and apply 1.22 -> 1.19 ms rotated (1.93 and 1.70 ms with the items fastest); ring Gram 1.97 ->
// 1.86 ms with the items fastest (2.0 ms rotated), and 2.15 -> 1.16 ms when the 64 lengths are equal.
constexpr int32_t kChunksFast = 0, kChunksRotated = 1, kItemsFast = 2;
// The order a launch over num_items items with `chunks` chunks per row takes (the items-fast layout needs the
// chunks within the z limit).
inline int32_t multi_item_order(int num_items, int chunks, int32_t wanted) {
  if (num_items <= 1) return kChunksFast;
  return wanted == kItemsFast && chunks > 65535 ? kChunksRotated : wanted;
}
inline dim3 chunk_grid(int chunks, int units, int item_layers, int32_t order) {
  return order == kItemsFast ? dim3(item_layers, units, chunks) : dim3(chunks, units, item_layers);
}

int apply_chunk_tokens();
hipError_t launch_apply(const ApplyArgs& a, kvc_dtype dtype, int max_rank, int max_tokens, int num_items,
                        hipStream_t stream);

// Fit (kvc_fit.hip): Gram partials, then projection after the eigensolver.
struct FitArgs {
  PoolView pv;
  LayerPtrs layers;
  const kvc_item* items;       // device; each item's state receives the fit
  const int32_t* src_tables;
  const int32_t* dst_tables;
  int32_t max_blocks;
  int32_t layer_begin;
  int32_t num_layers;
  int32_t mode;                // kvc_fit_mode
  float* partials;             // workspace [unit][max_parts][d][d]
  int32_t max_parts;
  int32_t part_tokens;
  int32_t kv_begin;            // the launch covers K/V sides kv_begin .. (grid y: one or both sides' heads)
  int32_t chunk_order;         // set by the launcher (chunk_grid)
};
hipError_t launch_fit_gram(const FitArgs& a, kvc_dtype dtype, int num_items, hipStream_t stream);
hipError_t launch_fit_proj(const FitArgs& a, kvc_dtype dtype, int num_items, int max_tokens, int max_rank,
                           hipStream_t stream);

// Per-layer factorisation (kvc_layer.hip).  A layer unit u = (item * num_layers + layer - layer_begin) * 2 + kv
// covers every KV head of one layer's K (or V) rows: Z is T x D with D = H d.
struct LayerFitArgs {
  PoolView pv;
  LayerPtrs layers;
  const kvc_item* items;       // device; each item's (per-layer) state receives the fit
  const int32_t* src_tables;
  const int32_t* dst_tables;
  int32_t max_blocks;
  int32_t layer_begin, num_layers;
  int32_t mode;                // kvc_fit_mode
  int32_t num_units;
  int32_t k;                   // subspace columns (64 or 128)
  int32_t rank;                // the items' rank (one rank per call group)
  int32_t max_parts, part_tokens;
  float* partials;             // [unit][max_parts][D][D]
  double* gram;                // [unit][D][D]
  double* x;                   // [unit][k][D] orthonormal columns (stored as rows)
  double* y;                   // [unit][k][D]
  double* hmat;                // [unit][k][k]; during the iteration R^{-1} of the Cholesky QR
  double* spart;               // [unit][ceil(D / 256)][k][k] partial Y^T Y of the Cholesky QR
  double* eps;                 // [2][unit] perturbation size of the Cholesky QR, by round parity
  float* vrows;                // [unit][rank][k] eigenvectors of hmat (rows)
  float* vsigma;               // [unit][rank]
  double* resid;               // [unit][KVC_MAX_RANK] residual norms of the Ritz pairs of the last check
  int32_t* conv;               // [unit] 0 while iterating, 1 once the top-r Ritz pairs met the tolerance, 2 at the cap
  int32_t* iters;              // [unit] subspace iterations done when the unit stopped
};
// Subspace iteration with Rayleigh-Ritz checks: the first check after kLayerFirstIters iterations, then every
// kLayerCheckEvery, until every top-r Ritz pair (theta, y) has ||G y - theta y|| <= kLayerTol * theta_1 or
// kLayerMaxIters iterations are done.  A unit that has stopped skips the remaining launches.
constexpr int kLayerFirstIters = 4, kLayerCheckEvery = 4, kLayerMaxIters = 48;
constexpr double kLayerTol = 1e-6;
struct EigArgs;
hipError_t launch_layer_gram(const LayerFitArgs& a, kvc_dtype dtype, hipStream_t stream);
hipError_t launch_layer_subspace(const LayerFitArgs& a, const EigArgs& ea, hipStream_t stream);
hipError_t launch_layer_proj(const LayerFitArgs& a, kvc_dtype dtype, int max_tokens, hipStream_t stream);

// Top-r eigenpairs of per-unit Gram matrices (kvc_eig.hip).  Unit u enumerates (item, layer, K/V, head) with the
// head fastest: u = ((item * num_layers + layer - layer_begin) * 2 + kv) * num_kv_heads + head.
struct EigArgs {
  int32_t n;                  // head_dim
  int32_t num_units;
  const float* partials;      // fp32 partial Grams [unit][max_parts][n][n], or null
  int32_t max_parts;
  int32_t part_tokens;        // tokens per partial: a unit with T_s rows has ceil(T_s / part_tokens) partials
  const double* dense;        // fp64 Grams [unit][n][n] when partials is null
  const kvc_item* items;      // device items whose states receive basis/sigma, or null
  kvc_state state;            // the receiving state when items is null
  int32_t layer_begin;
  int32_t num_layers;
  int32_t num_kv_heads;
  double* reflect;            // workspace [unit][n][n]
  double* reflect_beta;       // workspace [unit][n]
  double* vecs;               // workspace [unit][KVC_MAX_RANK][n]
  uint32_t seed;
  const int32_t* skip;        // [unit] nonzero: leave the unit's outputs as they are (null: every unit)
};
size_t eig_lds_bytes(int n);
hipError_t launch_eig(const EigArgs& a, hipStream_t stream);

// Chain (kvc_chain.hip).  Unit u = (layer - layer_begin) * 2 H + kv * H + head.
struct ChainArgs {
  kvc_state first, second, out;
  int32_t layer_begin;
  int32_t num_layers;
  int32_t num_units;
  int32_t mp;                  // row stride of the H partials (r1 + r2 rounded up to a multiple of 16)
  int32_t gram_wave_ft;        // 2, 4 or 8: the LDS-free wave Gram with mp = 16 * gram_wave_ft; 0: LDS Gram
  float* partials;             // workspace [unit][max_parts][mp][mp]
  int32_t max_parts;
  int32_t part_tokens;
  double* hsum;                // [unit][m][m]
  double* pmat;                // [unit][m][d]
  double* gram;                // [unit][d][d]
  float* ymat;                 // [unit][m][r_out]
};
hipError_t launch_chain(const ChainArgs& a, const EigArgs& ea, hipStream_t stream);

// Anchors (kvc_anchor.hip): distances / weights, anchored apply, gate distances.  One item per call.
constexpr int kResMaxChunks = 10;  // 32-rank chunks of all anchors of one unit held in LDS at once

struct AnchorArgs {
  PoolView pv;
  LayerPtrs layers;
  const int32_t* src_table;    // device row of the item's src table, or null
  const int32_t* dst_table;
  int32_t src_offset, dst_offset;
  int32_t src_position, dst_position;  // context positions of row 0 (keys of a rotary cache)
  int32_t num_tokens;          // T: rows of the item (apply copies rows T_s <= t < T)
  int32_t num_weighted;        // T_s (weights, apply) or the gate prefix k
  int32_t layer_begin, num_layers;
  int32_t num_anchors;
  int32_t max_rank;            // largest anchor rank (LDS staging width)
  int32_t rank[KVC_MAX_ANCHORS];
  int32_t tokens[KVC_MAX_ANCHORS];  // coefficient rows per unit of each anchor's state
  const void* coef[KVC_MAX_ANCHORS];
  const float* basis[KVC_MAX_ANCHORS];
  float* weights;              // [num_layers][2][num_weighted][num_anchors]
  float inv_temperature;
  float* gate_partials;        // [num_layers][chunks][num_anchors] sums of squares (gate)
  int32_t gate_chunks;
  float* distances;            // [num_anchors] (gate)
  // resident-basis kernels: the anchors' ranks cut into 32-rank chunks (an anchor of rank 0 keeps one zero chunk)
  int32_t num_chunks;
  int32_t chunk_anchor[kResMaxChunks];
  int32_t chunk_k0[kResMaxChunks];
  int32_t chunk_last[kResMaxChunks];  // 1 on an anchor's last chunk
};
int anchor_chunk_tokens();
int anchor_resident_chunk_tokens();
size_t anchor_lds_bytes(int head_dim, int max_rank, kvc_dtype dtype, int which);
hipError_t launch_anchor_weights(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream);
hipError_t launch_apply_anchored(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream);
hipError_t launch_gate_distances(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream);

}  // namespace kvc
