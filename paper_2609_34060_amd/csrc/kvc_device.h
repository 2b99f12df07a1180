// Device helpers shared by the libkvc kernels (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvc.h"

namespace kvc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Rotary encoding of the key rows (device-side view of kvc_cache's rope fields): pair i of a key at position p is
// rotated by the angle p * inv_freq[i].
struct RopeView {
  int32_t style;        // kvc_rope_style
  int32_t pad;
  double inv_freq[64];  // [head_dim / 2]
};

// Per-launch description of the pools of one cache (device-side view of kvc_cache).
struct PoolView {
  int64_t block_stride, token_stride, head_stride;  // elements
  int32_t block_size, num_blocks, num_kv_heads, head_dim;
  int32_t block_shift;                               // log2(block_size) when it is a power of two, else -1
  RopeView rope;
};

// Layer pointer tables travel in the kernel arguments (up to this many layers per launch).
constexpr int kMaxLayersPerLaunch = 128;
struct LayerPtrs {
  const void* k[kMaxLayersPerLaunch];
  const void* v[kMaxLayersPerLaunch];
};

// ---- bf16 <-> f32 ----------------------------------------------------------------------------------------------

__device__ __forceinline__ float bf16_lo_to_f32(uint32_t packed) { return __uint_as_float(packed << 16); }
__device__ __forceinline__ float bf16_hi_to_f32(uint32_t packed) { return __uint_as_float(packed & 0xffff0000u); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two floats -> packed bf16 pair, round to nearest even (one v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float x) { return pack_bf16x2(x, 0.0f) & 0xffffu; }

// x = hi + lo + O(2^-17 |x|) with hi = bf16(x) and lo = bf16(x - hi): the two-term split that lets bf16 MFMA carry
// about 16 significant bits of an fp32 operand.  Pairs of values, packed.
__device__ __forceinline__ void split_bf16x2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  hi = pack_bf16x2(x0, x1);
  lo = pack_bf16x2(x0 - __uint_as_float(hi << 16), x1 - __uint_as_float(hi & 0xffff0000u));
}
__device__ __forceinline__ void split_bf16(float x, uint32_t& hi_bits, uint32_t& lo_bits) {
  uint32_t h, l;
  split_bf16x2(x, 0.0f, h, l);
  hi_bits = h & 0xffffu;
  lo_bits = l & 0xffffu;
}

// ---- paged row addressing --------------------------------------------------------------------------------------
// Token t of a block sequence with row offset `off`: position p = off + t, block = table[p / bs] (identity when
// table is null), slot = p % bs.  Returns the element offset of the row, or -1 when the block id is out of range.
__device__ __forceinline__ int64_t row_offset(const PoolView& pv, const int32_t* __restrict__ table, int32_t off,
                                              int32_t t, int32_t head) {
  const int32_t p = off + t;
  const int32_t lb = pv.block_shift >= 0 ? p >> pv.block_shift : p / pv.block_size;
  const int32_t slot = p - lb * pv.block_size;
  const int32_t blk = table ? table[lb] : lb;
  if (blk < 0 || blk >= pv.num_blocks) return -1;
  return (int64_t)blk * pv.block_stride + (int64_t)slot * pv.token_stride + (int64_t)head * pv.head_stride;
}

__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& v) { return __builtin_bit_cast(bf16x8, v); }

// Row-correction layout shared by the apply-type kernels: a 16-token tile is the MFMA product D^T = B^T A^T with M =
// feature (16 per M-tile), N = token, K = rank.  Feature held by MFMA row m of M-tile mt: the lanes of token-group
// g = m / 4 own features 32 q + 8 g + [0, 8) of 16-byte row load q = mt / 2, the first four in M-tile 2q and the
// last four in 2q + 1.
__device__ __forceinline__ int mfma_row_feature(int mt, int m) {
  return 32 * (mt >> 1) + 8 * (m >> 2) + 4 * (mt & 1) + (m & 3);
}

// ---- rotary re-alignment of key rows (Appendix A.3, positional alignment) ----------------------------------------
// Pair i of a row is features (i, i + D/2) (KVC_ROPE_HALF) or (2i, 2i + 1) (KVC_ROPE_PAIRS); rotating it by the angle
// th maps (a, b) to (a cos th - b sin th, a sin th + b cos th).

// cos / sin of the angles p * inv_freq[i] of the D/2 pairs, evaluated in fp64 and rounded to fp32, by the threads
// of the calling workgroup (the caller synchronises before reading c and s).
__device__ __forceinline__ void rope_table(const RopeView& rp, int D, double p, float* c, float* s) {
  for (int i = threadIdx.x; i < D / 2; i += blockDim.x) {
    double sn, cs;
    sincos(p * rp.inv_freq[i], &sn, &cs);
    c[i] = (float)cs;
    s[i] = (float)sn;
  }
}
__device__ __forceinline__ int rope_partner(int style, int D, int f) {
  return style == KVC_ROPE_HALF ? (f < D / 2 ? f + D / 2 : f - D / 2) : (f ^ 1);
}
__device__ __forceinline__ int rope_pair(int style, int D, int f) {
  return style == KVC_ROPE_HALF ? (f < D / 2 ? f : f - D / 2) : (f >> 1);
}
__device__ __forceinline__ bool rope_first(int style, int D, int f) {
  return style == KVC_ROPE_HALF ? f < D / 2 : (f & 1) == 0;
}
// Feature value after the rotation, from its own value x and its partner's y (angle given by c, s).
__device__ __forceinline__ float rope_rotated(bool first, float x, float y, float c, float s) {
  return first ? x * c - y * s : y * s + x * c;
}
// Rotate a row held in the row layout of the MFMA kernels (the lane of token-group g holds features 32 q + 8 g + e,
// e < 8, in v[2 q + (e >> 2)][e & 3]) by the angles of a table; the pairs of both styles stay inside the lane.
template <int D>
__device__ __forceinline__ void rope_rotate_rows(f32x4* v, int style, int g, const float* c, const float* s) {
  constexpr int NQ = D / 32;
  if (style == KVC_ROPE_HALF) {
#pragma unroll
    for (int q = 0; q < NQ / 2; ++q)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int i = 32 * q + 8 * g + e, ja = 2 * q + (e >> 2), jb = 2 * (q + NQ / 2) + (e >> 2);
        const float a = v[ja][e & 3], b = v[jb][e & 3], cc = c[i], ss = s[i];
        v[ja][e & 3] = a * cc - b * ss;
        v[jb][e & 3] = a * ss + b * cc;
      }
  } else {
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const int i = 16 * q + 4 * g + (e >> 1), j = 2 * q + (e >> 2);
        const float a = v[j][e & 3], b = v[j][(e & 3) + 1], cc = c[i], ss = s[i];
        v[j][e & 3] = a * cc - b * ss;
        v[j][(e & 3) + 1] = a * ss + b * cc;
      }
  }
}

// Rotary angle table of one wave: lane L holds cos / sin of pair rope_wave_pair(L) at angle p * inv_freq[pair]; the
// lanes of token group g (the MFMA row layout: features 32 q + 8 g + e) need D / 8 pairs, lanes g D / 8 .. of the
// table, in the order rope_rotate_rows visits them.
template <int D>
__device__ __forceinline__ int rope_wave_pair(int style, int lane) {
  constexpr int NP = D / 8;
  const int gg = (lane / NP) & 3, k = lane % NP;
  return style == KVC_ROPE_HALF ? 32 * (k / 8) + 8 * gg + k % 8 : 16 * (k / 4) + 4 * gg + k % 4;
}
template <int D>
__device__ __forceinline__ void rope_wave_table(const RopeView& rp, double p, int lane, float& c, float& s) {
  double sn, cs;
  sincos(p * rp.inv_freq[rope_wave_pair<D>(rp.style, lane)], &sn, &cs);
  c = (float)cs;
  s = (float)sn;
}
// rope_rotate_rows with the angles of a wave table (converged control flow: lane shuffles).
template <int D>
__device__ __forceinline__ void rope_rotate_rows_wave(f32x4* v, int style, int g, float tc, float ts) {
  constexpr int NQ = D / 32, NP = D / 8;
  if (style == KVC_ROPE_HALF) {
#pragma unroll
    for (int q = 0; q < NQ / 2; ++q)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int src = g * NP + 8 * q + e, ja = 2 * q + (e >> 2), jb = 2 * (q + NQ / 2) + (e >> 2);
        const float cc = __shfl(tc, src, kWave), ss = __shfl(ts, src, kWave);
        const float a = v[ja][e & 3], b = v[jb][e & 3];
        v[ja][e & 3] = a * cc - b * ss;
        v[jb][e & 3] = a * ss + b * cc;
      }
  } else {
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const int src = g * NP + 4 * q + (e >> 1), j = 2 * q + (e >> 2);
        const float cc = __shfl(tc, src, kWave), ss = __shfl(ts, src, kWave);
        const float a = v[j][e & 3], b = v[j][(e & 3) + 1];
        v[j][e & 3] = a * cc - b * ss;
        v[j][(e & 3) + 1] = a * ss + b * cc;
      }
  }
}

// Offset of unit (layer, kv, head) in a state's per-unit arrays.
// Position of a workgroup in a grid over (chunk, unit, item x layer) laid out by chunk_grid: order 0 has the chunks
// fastest, 1 shifts each row's (y, z) chunks by the row index modulo the row length, 2 has the items fastest (x and
// z trade places).
__device__ __forceinline__ int grid_chunk(int order) {
  if (order == 2) return (int)blockIdx.z;
  if (order == 1) {
    const unsigned row = blockIdx.y + gridDim.y * blockIdx.z;
    return (int)((blockIdx.x + row % gridDim.x) % gridDim.x);
  }
  return (int)blockIdx.x;
}
__device__ __forceinline__ int grid_item_layer(int order) { return (int)(order == 2 ? blockIdx.x : blockIdx.z); }

__device__ __forceinline__ int64_t unit_index(int32_t layer, int32_t kv, int32_t head, int32_t num_kv_heads) {
  return ((int64_t)layer * 2 + kv) * num_kv_heads + head;
}

// ---- Gram fragments (shared by the fit and chain Gram kernels) ----------------------------------------------

// Tile idx of the upper triangle (row-major over fi <= fj) of an FT x FT grid of 16 x 16 tiles.
constexpr int tile_fi(int idx, int FT) {
  int fi = 0;
  while (idx >= FT - fi) {
    idx -= FT - fi;
    ++fi;
  }
  return fi;
}
constexpr int tile_fj(int idx, int FT) {
  int fi = 0;
  while (idx >= FT - fi) {
    idx -= FT - fi;
    ++fi;
  }
  return fi + idx;
}

// The Gram is computed in a permuted feature order: output tile (fi, fj) holds G[FT m + fi][FT n + fj] for
// m, n in [0, 16).  Lane (g, m) of a wave then needs, for its 8 tokens 8 g + j, the FT contiguous features
// FT m .. FT m + FT - 1 of each row (one 2 FT-byte read per token), and the MFMA fragment of tile row fi is
// element fi of those 8 segments, gathered with byte permutes.
template <int FT>
struct GramSeg;
template <>
struct GramSeg<8> {
  using T = u32x4;
};
template <>
struct GramSeg<4> {
  using T = uint2;
};
template <>
struct GramSeg<2> {
  using T = uint32_t;
};

template <int FT>
__device__ __forceinline__ uint32_t seg_dword(const typename GramSeg<FT>::T& s, int w) {
  if constexpr (FT == 8) return s[w];
  else if constexpr (FT == 4) return w == 0 ? s.x : s.y;
  else return s;
}

// Fragment of tile row fi: bf16 element fi of each of the 8 token segments (tokens 8 g + 0 .. 7).
template <int FT, int FI>
__device__ __forceinline__ bf16x8 gram_fragment(const typename GramSeg<FT>::T* seg) {
  constexpr uint32_t sel = (FI & 1) ? 0x07060302u : 0x05040100u;
  u32x4 f;
#pragma unroll
  for (int w = 0; w < 4; ++w)
    f[w] = __builtin_amdgcn_perm(seg_dword<FT>(seg[2 * w + 1], FI >> 1), seg_dword<FT>(seg[2 * w], FI >> 1), sel);
  return as_bf16x8(f);
}

// Row offsets of the 8 consecutive tokens t .. t + 7 of a block sequence (entries past t_end are -1); with a
// power-of-two block size of at least 8 the 8 tokens touch at most two blocks, so two table reads suffice.
__device__ __forceinline__ void row_offsets8(const PoolView& pv, const int32_t* __restrict__ table, int32_t off,
                                             int t, int t_end, int head, int64_t* o) {
  if (pv.block_shift >= 3) {
    const int32_t p = off + t;
    const int32_t lb0 = p >> pv.block_shift, lb1 = (p + 7) >> pv.block_shift;
    // a table entry is read only if a token before t_end lies in its block (the host checked those are in range)
    const int32_t b0 = t < t_end ? (table ? table[lb0] : lb0) : -1;
    const int first_in_lb1 = (lb1 << pv.block_shift) - off;
    const int32_t b1 = lb1 == lb0 ? b0 : (first_in_lb1 < t_end ? (table ? table[lb1] : lb1) : -1);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int32_t pj = p + j;
      const int32_t lb = pj >> pv.block_shift;
      const int32_t blk = lb == lb0 ? b0 : b1;
      const bool ok = (t + j < t_end) && blk >= 0 && blk < pv.num_blocks;
      o[j] = ok ? (int64_t)blk * pv.block_stride + (int64_t)(pj - (lb << pv.block_shift)) * pv.token_stride +
                      (int64_t)head * pv.head_stride
                : -1;
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = (t + j < t_end) ? row_offset(pv, table, off, t + j, head) : -1;
  }
}

}  // namespace kvc
