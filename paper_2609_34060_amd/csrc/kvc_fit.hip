// kvc_fit_state kernels: the observed transition Z = C_dst - C_src of Eq. 12 (or Z = C_dst for a base cache) and
// its rank-r truncated SVD (Eq. 7) through the Gram matrix G = Z^T Z:
//   gram   one wave per (unit, token range) writes that range's partial Gram (fp32, d x d); the eigensolver sums
//          the partials of a unit in a fixed order in fp64, so the result does not depend on scheduling.
//   proj   coef = Z R_r (= U_r Sigma_r), re-reading Z from the cache after the basis is known.
//
// bf16 caches: Z is formed in fp32 (the difference of two bf16 values is exact in fp32) and split into a bf16
// hi/lo pair; every product is hi*hi + hi*lo + lo*hi on v_mfma_f32_16x16x32_bf16 with fp32 accumulation, about
// 16 significant bits per operand.  The Gram keeps the token index in the MFMA K slot by a permuted feature order
// (see GramSeg) so that its operands come straight from coalesced row loads; only tiles on or above the diagonal
// are computed and each is stored with its mirror.  In the projection the rows are read straight into the MFMA
// B-operand layout (16 contiguous bytes per lane), the basis hi/lo is staged in LDS.
// float32 caches use plain fp32 VALU kernels.
#include <utility>

#include "kvc_device.h"
#include "kvc_launch.h"

namespace kvc {

constexpr int kFitThreads = 256;
constexpr int kFitWaves = kFitThreads / kWave;

struct FitUnit {
  int item, lrel, layer, kv, head;
  int64_t unit;  // index within the item's state
};

__device__ __forceinline__ FitUnit fit_unit(const FitArgs& a) {
  FitUnit f;
  const int H = a.pv.num_kv_heads;
  const int il = grid_item_layer(a.chunk_order);
  f.item = il / a.num_layers;
  f.lrel = il - f.item * a.num_layers;
  f.layer = a.layer_begin + f.lrel;
  const int y = blockIdx.y;
  f.kv = a.kv_begin + y / H;
  f.head = y % H;
  f.unit = unit_index(f.layer, f.kv, f.head, H);
  return f;
}

// Linear unit id shared with the eigensolver: ((item * num_layers + lrel) * 2 + kv) * H + head.
__device__ __forceinline__ int64_t fit_linear_unit(const FitArgs& a, const FitUnit& f) {
  return (((int64_t)f.item * a.num_layers + f.lrel) * 2 + f.kv) * a.pv.num_kv_heads + f.head;
}

// ---------------------------------------------------------------------------------------------------------------
// Gram, bf16 caches
// ---------------------------------------------------------------------------------------------------------------

template <int D>
struct GramShape {
  static constexpr int FT = D / 16;                 // 16 x 16 output tiles per side
  static constexpr int NTILES = FT * (FT + 1) / 2;  // tiles on or above the diagonal
};

// Tile Q of wave W (tile index W + 4 Q): acc += Z_fi^T Z_fj with the hi/lo products.
template <int D, int W, int Q>
__device__ __forceinline__ void gram_tile(f32x4* acc, const typename GramSeg<D / 16>::T* sh,
                                          const typename GramSeg<D / 16>::T* sl) {
  constexpr int FT = D / 16;
  constexpr int idx = W + Q * kFitWaves;
  if constexpr (idx < GramShape<D>::NTILES) {
    constexpr int fi = tile_fi(idx, FT), fj = tile_fj(idx, FT);
    const bf16x8 ah = gram_fragment<FT, fi>(sh), al = gram_fragment<FT, fi>(sl);
    const bf16x8 bh = gram_fragment<FT, fj>(sh), bl = gram_fragment<FT, fj>(sl);
    acc[Q] = mfma16x16x32(al, bh, acc[Q]);
    acc[Q] = mfma16x16x32(ah, bl, acc[Q]);
    acc[Q] = mfma16x16x32(ah, bh, acc[Q]);
  }
}
template <int D, int W, int Q>
__device__ __forceinline__ void gram_store(float* P, const f32x4* acc, int g, int n) {
  constexpr int FT = D / 16;
  constexpr int idx = W + Q * kFitWaves;
  if constexpr (idx < GramShape<D>::NTILES) {
    constexpr int fi = tile_fi(idx, FT), fj = tile_fj(idx, FT);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = FT * (4 * g + i) + fi, col = FT * n + fj;
      P[row * D + col] = acc[Q][i];
      P[col * D + row] = acc[Q][i];
    }
  }
}
// All tiles of the upper triangle for one wave: acc[idx] += Z_fi^T Z_fj (hi/lo products).
template <int D, int... Is>
__device__ __forceinline__ void gram_all_tiles(f32x4* acc, const typename GramSeg<D / 16>::T* sh,
                                               const typename GramSeg<D / 16>::T* sl, std::integer_sequence<int, Is...>) {
  (gram_tile<D, Is, 0>(acc + Is, sh, sl), ...);
}
template <int D, int... Is>
__device__ __forceinline__ void gram_all_stores(float* P, const f32x4* acc, int g, int n,
                                                std::integer_sequence<int, Is...>) {
  (gram_store<D, Is, 0>(P, acc + Is, g, n), ...);
}

// bf16 Gram, one wave per partial: the wave streams its own token range 32 tokens at a time.  Lane (g, m) loads,
// for tokens t0 + 8 g + j (j = 0..7), the 2 FT bytes of features FT m .. FT m + FT - 1 of the dst (and src) row:
// sixteen lanes cover one row with one coalesced load.  Z = dst - src is split into bf16 hi/lo in registers and
// the MFMA fragments of every tile row are gathered from those segments with byte permutes, so the Gram needs no
// LDS and no barrier; all upper tiles accumulate in the wave's registers.  The next step's rows are loaded while
// the current step is multiplied.
// ROPE: keys of a rotary cache are fitted in canonical coordinates, Z = R(-pd) C_dst - R(-ps) C_src.  The partner of
// a rotate-half pair sits in lane n ^ 8 of the same row (features FT n + e and FT (n + 8) + e) and is fetched with a
// row rotation by 8; an adjacent pair sits in the same dword.
template <int D, bool ROPE>
__global__ __launch_bounds__(kFitThreads) void gram_bf16_mfma(FitArgs a) {
  constexpr int FT = D / 16;
  constexpr int NT = FT * (FT + 1) / 2;
  constexpr int STEP = 32;
  using Seg = typename GramSeg<FT>::T;
  const FitUnit f = fit_unit(a);
  const kvc_item* itp = a.items + f.item;
  const int r = itp->state.rank;
  const int Ts = itp->state.num_tokens;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // angle tables of -pd (dst rows) and -ps (src rows), before any wave leaves (the barrier needs every wave)
  __shared__ float s_rope[4][ROPE ? D / 2 : 1];
  const bool rope = ROPE && f.kv == 0;  // uniform over the workgroup
  const int style = a.pv.rope.style;
  if (rope) {
    rope_table(a.pv.rope, D, -(double)itp->dst_position, s_rope[0], s_rope[1]);
    rope_table(a.pv.rope, D, -(double)itp->src_position, s_rope[2], s_rope[3]);
    __syncthreads();
  }
  const int part = grid_chunk(a.chunk_order) * kFitWaves + wave;
  const int t_begin = part * a.part_tokens;
  if (r == 0 || t_begin >= Ts) return;  // per wave: the kernel has no barrier
  const int t_end = min(Ts, t_begin + a.part_tokens);
  const int g = lane >> 4, n = lane & 15;
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)f.item * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)f.item * a.max_blocks : nullptr;
  const uint16_t* pool = static_cast<const uint16_t*>(f.kv ? a.layers.v[f.lrel] : a.layers.k[f.lrel]);
  const bool delta = a.mode == KVC_FIT_DELTA;

  f32x4 acc[NT];
#pragma unroll
  for (int q = 0; q < NT; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load = [&](int t0, Seg* rd, Seg* rs) {
    int64_t od[8], os[8];
    const int t = t0 + 8 * g;
    row_offsets8(a.pv, dst_tab, itp->dst_offset, t, t_end, f.head, od);
    if (delta) row_offsets8(a.pv, src_tab, itp->src_offset, t, t_end, f.head, os);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      rd[j] = od[j] >= 0 ? *reinterpret_cast<const Seg*>(pool + od[j] + FT * n) : Seg{};
      rs[j] = (delta && os[j] >= 0) ? *reinterpret_cast<const Seg*>(pool + os[j] + FT * n) : Seg{};
    }
  };
  // Z of the loaded step into bf16 hi/lo segments
  auto form_z = [&](const Seg* rd, const Seg* rs, Seg* zh, Seg* zl) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
#pragma unroll
      for (int w = 0; w < FT / 2; ++w) {
        const uint32_t dw = seg_dword<FT>(rd[j], w), sw = seg_dword<FT>(rs[j], w);
        uint32_t h, l;
        split_bf16x2(bf16_lo_to_f32(dw) - bf16_lo_to_f32(sw), bf16_hi_to_f32(dw) - bf16_hi_to_f32(sw), h, l);
        if constexpr (FT == 8) {
          zh[j][w] = h;
          zl[j][w] = l;
        } else {
          if (w == 0) {
            zh[j].x = h;
            zl[j].x = l;
          } else {
            zh[j].y = h;
            zl[j].y = l;
          }
        }
      }
    }
  };

  // canonical Z of the loaded step (rotary keys): per element its own and its partner's value, both sides rotated
  float rc[2][FT], rsn[2][FT];  // cos / sin of -pd and -ps for the lane's FT features
  if (ROPE && rope) {
#pragma unroll
    for (int e = 0; e < FT; ++e) {
      const int i = rope_pair(style, D, FT * n + e);
      rc[0][e] = s_rope[0][i];
      rsn[0][e] = s_rope[1][i];
      rc[1][e] = s_rope[2][i];
      rsn[1][e] = s_rope[3][i];
    }
  }
  auto form_z_rope = [&](const Seg* rd, const Seg* rs, Seg* zh, Seg* zl) {
    const bool half = style == KVC_ROPE_HALF;
    const bool first_half = FT * n < D / 2;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
#pragma unroll
      for (int w = 0; w < FT / 2; ++w) {
        const uint32_t dw = seg_dword<FT>(rd[j], w), sw = seg_dword<FT>(rs[j], w);
        // partner dword: the same dword of lane n ^ 8 (rotate-half) or this dword with its halves swapped
        const uint32_t dpw = half ? (uint32_t)__builtin_amdgcn_mov_dpp((int)dw, 0x128, 0xF, 0xF, false)
                                  : ((dw >> 16) | (dw << 16));
        const uint32_t spw = half ? (uint32_t)__builtin_amdgcn_mov_dpp((int)sw, 0x128, 0xF, 0xF, false)
                                  : ((sw >> 16) | (sw << 16));
        float z[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int e = 2 * w + h;
          const bool first = half ? first_half : h == 0;
          const float xd = h ? bf16_hi_to_f32(dw) : bf16_lo_to_f32(dw);
          const float yd = h ? bf16_hi_to_f32(dpw) : bf16_lo_to_f32(dpw);
          const float xs = h ? bf16_hi_to_f32(sw) : bf16_lo_to_f32(sw);
          const float ys = h ? bf16_hi_to_f32(spw) : bf16_lo_to_f32(spw);
          z[h] = rope_rotated(first, xd, yd, rc[0][e], rsn[0][e]) - rope_rotated(first, xs, ys, rc[1][e], rsn[1][e]);
        }
        uint32_t hh, ll;
        split_bf16x2(z[0], z[1], hh, ll);
        if constexpr (FT == 8) {
          zh[j][w] = hh;
          zl[j][w] = ll;
        } else {
          if (w == 0) {
            zh[j].x = hh;
            zl[j].x = ll;
          } else {
            zh[j].y = hh;
            zl[j].y = ll;
          }
        }
      }
    }
  };

  // one register stage: the next step's rows are loaded into the same registers once Z of this step is formed,
  // so they are in flight while this step's 3 x NT MFMAs run
  Seg rd[8], rs[8];
  load(t_begin, rd, rs);
  for (int t0 = t_begin; t0 < t_end; t0 += STEP) {
    Seg zh[8], zl[8];
    if (ROPE && rope) form_z_rope(rd, rs, zh, zl);
    else form_z(rd, rs, zh, zl);
    if (t0 + STEP < t_end) load(t0 + STEP, rd, rs);
    gram_all_tiles<D>(acc, zh, zl, std::make_integer_sequence<int, NT>{});
  }
  const int64_t lu = fit_linear_unit(a, f);
  float* P = a.partials + ((size_t)lu * a.max_parts + part) * D * D;
  gram_all_stores<D>(P, acc, g, n, std::make_integer_sequence<int, NT>{});
}

// bf16 Gram, head_dim 128, rows staged through LDS: the same wave-per-partial Gram, but the rows of the next two
// 32-token steps are loaded straight into a per-wave LDS ring (global_load_lds, 16 bytes per lane), so that twice
// the bytes of the register pipeline are in flight while only the step being multiplied occupies registers.
// Each lane reads back exactly the bytes its own loads wrote, so the ring needs no barrier, only vmcnt waits; the
// read-back is inline assembly because the compiler would otherwise wait for every outstanding LDS load before
// each LDS read.  Table entries are read with scalar loads (a 32-token step touches at most three blocks of at
// least 16 tokens), so that using them does not wait on the row loads either.
constexpr int kGramRing = 2;                          // steps in flight per wave

// The bf16 pair (-1, 0) or (0, -1) in a scalar register: dot2 with it subtracts the low or the high element.  The
// move is opaque to the compiler, which would otherwise fold the low-element constant into an inline constant that
// the hardware reads as the 32-bit float -1.0, i.e. the pair (0, -1).
// A 32-bit word as a bf16 pair.  (Through memcpy: a bit_cast of a vector element to bf16x2 inside an unrolled loop
// has been seen to lose the element index in code generation.)
__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t w) {
  bf16x2 v;
  __builtin_memcpy(&v, &w, sizeof(v));
  return v;
}
__device__ __forceinline__ bf16x2 bf16_pair_const(uint32_t bits) {
  uint32_t v;
  asm volatile("s_mov_b32 %0, %1" : "=s"(v) : "i"(bits));
  return __builtin_bit_cast(bf16x2, v);
}
constexpr int kGramSlotBytes = 16 * kWave * 16;       // 8 dst + 8 src loads of 16 bytes per lane
constexpr int kGramTabMax = 768;                      // table entries per partial (dst and src)
constexpr size_t kGramLdsBytes = (size_t)kFitWaves * (kGramRing * kGramSlotBytes + 2 * kGramTabMax * 4);

// The 16 row segments of one ring slot (8 dst, then 8 src), each 16 bytes at lane * 16 of a 1 KB block.
__device__ __forceinline__ void gram_ring_read(uint32_t addr, u32x4* d, u32x4* s) {
  asm volatile(
      "ds_read_b128 %0, %16\n\tds_read_b128 %1, %16 offset:1024\n\t"
      "ds_read_b128 %2, %16 offset:2048\n\tds_read_b128 %3, %16 offset:3072\n\t"
      "ds_read_b128 %4, %16 offset:4096\n\tds_read_b128 %5, %16 offset:5120\n\t"
      "ds_read_b128 %6, %16 offset:6144\n\tds_read_b128 %7, %16 offset:7168\n\t"
      "ds_read_b128 %8, %16 offset:8192\n\tds_read_b128 %9, %16 offset:9216\n\t"
      "ds_read_b128 %10, %16 offset:10240\n\tds_read_b128 %11, %16 offset:11264\n\t"
      "ds_read_b128 %12, %16 offset:12288\n\tds_read_b128 %13, %16 offset:13312\n\t"
      "ds_read_b128 %14, %16 offset:14336\n\tds_read_b128 %15, %16 offset:15360\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(d[0]), "=&v"(d[1]), "=&v"(d[2]), "=&v"(d[3]), "=&v"(d[4]), "=&v"(d[5]), "=&v"(d[6]), "=&v"(d[7]),
        "=&v"(s[0]), "=&v"(s[1]), "=&v"(s[2]), "=&v"(s[3]), "=&v"(s[4]), "=&v"(s[5]), "=&v"(s[6]), "=&v"(s[7])
      : "v"(addr)
      : "memory");
}

template <bool DELTA>
__global__ __launch_bounds__(kFitThreads) void gram_bf16_ring(FitArgs a) {
  constexpr int D = 128, FT = 8, NT = FT * (FT + 1) / 2, STEP = 32;
  constexpr int LPS = DELTA ? 16 : 8;  // loads per step and lane
  extern __shared__ __attribute__((aligned(16))) unsigned char gram_lds[];
  // block (part, kv x head group, item x layer): the four waves take four heads of the same token range, so that a
  // workgroup reads 4 x 256 contiguous bytes of each token row
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int H = a.pv.num_kv_heads;
  const int HG = (H + kFitWaves - 1) / kFitWaves;
  FitUnit f;
  const int il = grid_item_layer(a.chunk_order);
  f.item = il / a.num_layers;
  f.lrel = il - f.item * a.num_layers;
  f.layer = a.layer_begin + f.lrel;
  f.kv = a.kv_begin + (int)blockIdx.y / HG;
  f.head = ((int)blockIdx.y % HG) * kFitWaves + wave;
  if (f.head >= H) return;
  f.unit = unit_index(f.layer, f.kv, f.head, H);
  const kvc_item* itp = a.items + f.item;
  const int r = itp->state.rank;
  const int Ts = itp->state.num_tokens;
  const int part = grid_chunk(a.chunk_order);
  const int t_begin = part * a.part_tokens;
  if (r == 0 || t_begin >= Ts) return;  // per wave: the kernel has no barrier
  const int t_end = min(Ts, t_begin + a.part_tokens);
  const int g = lane >> 4, n = lane & 15;
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)f.item * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)f.item * a.max_blocks : nullptr;
  const uint16_t* pool = static_cast<const uint16_t*>(f.kv ? a.layers.v[f.lrel] : a.layers.k[f.lrel]);
  const int shift = a.pv.block_shift;
  const int bmask = (1 << shift) - 1;
  unsigned char* ring = gram_lds + wave * (kGramRing * kGramSlotBytes);

  f32x4 acc[NT];
#pragma unroll
  for (int q = 0; q < NT; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};

  // The block-table entries of the wave's whole token range are copied once, before the first row load, into the
  // wave's LDS table (lane-parallel); a step reads its (at most three) entries back with scalar-addressed LDS reads,
  // so the loop issues no global memory operation besides the row loads.
  struct Tab {
    int32_t lbs, lbe, off;
    uint32_t lds;  // LDS byte address of the wave's copy
  };
  int32_t* tab_lds = reinterpret_cast<int32_t*>(gram_lds + kFitWaves * kGramRing * kGramSlotBytes) +
                     wave * 2 * kGramTabMax;
  auto load_tab = [&](const int32_t* tab, int32_t off, int which) {
    Tab tb;
    tb.off = __builtin_amdgcn_readfirstlane(off);
    tb.lbs = (tb.off + t_begin) >> shift;
    tb.lbe = (tb.off + t_end - 1) >> shift;
    int32_t* dstp = tab_lds + which * kGramTabMax;
    for (int i = lane; i < kGramTabMax; i += kWave) {
      const int32_t lb = tb.lbs + i;
      dstp[i] = lb <= tb.lbe ? (tab ? tab[lb] : lb) : -1;
    }
    tb.lds = (uint32_t)(uintptr_t)dstp;
    return tb;
  };
  const Tab tdst = load_tab(dst_tab, itp->dst_offset, 0);
  Tab tsrc;
  if (DELTA) tsrc = load_tab(src_tab, itp->src_offset, 1);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the tables are in LDS before any read-back
  // entries lb0, lb0 + 1, lb0 + 2 (lb0 uniform); entries past the range read as -1
  auto entries = [&](const Tab& tb, int32_t lb0, int32_t& e0, int32_t& e1, int32_t& e2) {
    const int32_t i0 = min(lb0 - tb.lbs, kGramTabMax - 3);
    const uint32_t addr = tb.lds + 4u * (uint32_t)i0;
    asm volatile(
        "ds_read_b32 %0, %3\n\tds_read_b32 %1, %3 offset:4\n\tds_read_b32 %2, %3 offset:8\n\ts_waitcnt lgkmcnt(0)"
        : "=&v"(e0), "=&v"(e1), "=&v"(e2)
        : "v"(addr)
        : "memory");
    e0 = lb0 <= tb.lbe ? e0 : -1;
    e1 = lb0 + 1 <= tb.lbe ? e1 : -1;
    e2 = lb0 + 2 <= tb.lbe ? e2 : -1;
  };

  // Loads of one step's rows into an LDS slot; returns the validity mask (bit j: token t0 + 8 g + j).  A lane's
  // eight tokens touch at most two blocks; the row address of token j is the address of the lane's first token
  // plus j token strides, or, past the block boundary, the start of the next block plus the remaining strides.
  const int64_t head_off = (int64_t)f.head * a.pv.head_stride + FT * n;
  auto issue_rows = [&](const Tab& tb, int t0, unsigned char* dst_lds) -> uint32_t {
    const int32_t p0 = tb.off + t0;
    const int32_t lb0 = p0 >> shift;
    int32_t e0, e1, e2;
    entries(tb, lb0, e0, e1, e2);
    const int32_t pl = p0 + 8 * g;                    // position of the lane's first token
    const int bi = (pl >> shift) - lb0;               // its block among the step's three
    const int32_t blk_a = bi == 0 ? e0 : (bi == 1 ? e1 : e2);
    const int32_t blk_b = bi == 0 ? e1 : e2;          // the next block
    const int32_t slot_a = pl & bmask;
    const int ja = (int)min(8, (1 << shift) - slot_a);  // tokens of the lane left in block a
    const bool ok_a = blk_a >= 0 && blk_a < a.pv.num_blocks, ok_b = blk_b >= 0 && blk_b < a.pv.num_blocks;
    const uint16_t* base_a = pool + (int64_t)(ok_a ? blk_a : 0) * a.pv.block_stride +
                             (int64_t)slot_a * a.pv.token_stride + head_off;
    const uint16_t* base_b = pool + (int64_t)(ok_b ? blk_b : 0) * a.pv.block_stride + head_off;
    const int tl = t_end - (t0 + 8 * g);              // tokens of the lane before t_end
    uint32_t m = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool in_a = j < ja;
      const uint16_t* src = in_a ? base_a + (int64_t)j * a.pv.token_stride
                                 : base_b + (int64_t)(j - ja) * a.pv.token_stride;
      const bool ok = j < tl && (in_a ? ok_a : ok_b);
      __builtin_amdgcn_global_load_lds(ok ? src : pool, dst_lds + j * (kWave * 16), 16, 0, 0);
      m |= ok ? 1u << j : 0u;
    }
    return m;
  };
  auto issue = [&](int sl, int t0) -> uint32_t {
    unsigned char* base = ring + sl * kGramSlotBytes;
    uint32_t m = issue_rows(tdst, t0, base);
    if (DELTA) m |= issue_rows(tsrc, t0, base + 8 * kWave * 16) << 8;
    return m;
  };

  // Z of a step into bf16 hi/lo segments (rows outside the range read as zero).  With dot2 (two bf16 products and
  // an fp32 addend, rounded once): z = d - s and the residual z - hi are one instruction per element; both are the
  // same single roundings as fp32 subtractions (the residual is exact).
  const bf16x2 kBf16NegLo = bf16_pair_const(0x0000BF80u), kBf16NegHi = bf16_pair_const(0xBF800000u);
  auto form = [&](const u32x4* rd, const u32x4* rs, uint32_t m, u32x4* zh, u32x4* zl) {
    const bool full = __builtin_amdgcn_ballot_w64(m != (DELTA ? 0xFFFFu : 0xFFu)) == 0;  // uniform
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      u32x4 dv = rd[j], sv = rs[j];
      if (!full) {
        dv = (m >> j) & 1 ? dv : u32x4{0u, 0u, 0u, 0u};
        sv = (DELTA && ((m >> (8 + j)) & 1)) ? sv : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        float z0 = __uint_as_float(dv[w] << 16), z1 = __uint_as_float(dv[w] & 0xffff0000u);
        if (DELTA) {
          const bf16x2 s2 = as_bf16x2(sv[w]);
          z0 = __builtin_amdgcn_fdot2_f32_bf16(s2, kBf16NegLo, z0, false);  // d0 - s0
          z1 = __builtin_amdgcn_fdot2_f32_bf16(s2, kBf16NegHi, z1, false);  // d1 - s1
        }
        const uint32_t h = pack_bf16x2(z0, z1);
        const bf16x2 h2 = as_bf16x2(h);
        const float r0 = __builtin_amdgcn_fdot2_f32_bf16(h2, kBf16NegLo, z0, false);  // z0 - hi0 (exact)
        const float r1 = __builtin_amdgcn_fdot2_f32_bf16(h2, kBf16NegHi, z1, false);  // z1 - hi1 (exact)
        zh[j][w] = h;
        zl[j][w] = pack_bf16x2(r0, r1);
      }
    }
  };
  auto read_slot = [&](int sl, u32x4* rd, u32x4* rs) {
    gram_ring_read((uint32_t)(uintptr_t)(ring + sl * kGramSlotBytes) + lane * 16, rd, rs);
  };

  // Software pipeline: slot sl holds the next step, the other slot the one after; Z of the current step is in
  // registers.  Each iteration reads the next step, refills its slot three steps ahead, and forms the next Z while
  // the current one is multiplied (scheduling groups interleave the MFMAs with the VALU work).  Loads past the
  // range are issued too (all rows invalid; they read the pool's first row) so that the loop body has no branch.
  constexpr int kWaitLps = LPS == 16 ? 0x4F70 : 0x0F78;  // s_waitcnt vmcnt(LPS)
  uint32_t mask[kGramRing];
  mask[0] = issue(0, t_begin);
  mask[1] = issue(1, t_begin + STEP);
  u32x4 zc_h[8], zc_l[8];
  {
    __builtin_amdgcn_s_waitcnt(kWaitLps);
    u32x4 rd[8], rs[8];
    read_slot(0, rd, rs);
    form(rd, rs, mask[0], zc_h, zc_l);
  }
  mask[0] = issue(0, t_begin + 2 * STEP);
  int sl = 1;
  for (int t0 = t_begin; t0 + STEP < t_end; t0 += STEP) {
    __builtin_amdgcn_s_waitcnt(kWaitLps);
    const uint32_t m = sl ? mask[1] : mask[0];
    u32x4 rd[8], rs[8];
    read_slot(sl, rd, rs);
    const uint32_t mn = issue(sl, t0 + 3 * STEP);
    if (sl) mask[1] = mn;
    else mask[0] = mn;
    u32x4 zn_h[8], zn_l[8];
    form(rd, rs, m, zn_h, zn_l);
    gram_all_tiles<D>(acc, zc_h, zc_l, std::make_integer_sequence<int, NT>{});
    // 3 NT = 108 MFMAs, each followed by a share of the VALU work of the next Z
#pragma unroll
    for (int q = 0; q < 3 * NT; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);  // VALU
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      zc_h[j] = zn_h[j];
      zc_l[j] = zn_l[j];
    }
    sl ^= 1;
  }
  gram_all_tiles<D>(acc, zc_h, zc_l, std::make_integer_sequence<int, NT>{});
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): no LDS load outstanding when the wave ends
  const int64_t lu = fit_linear_unit(a, f);
  float* P = a.partials + ((size_t)lu * a.max_parts + part) * D * D;
  gram_all_stores<D>(P, acc, g, n, std::make_integer_sequence<int, NT>{});
}

// ---------------------------------------------------------------------------------------------------------------
// Gram, fp32 caches (VALU, fp32 accumulation)
// ---------------------------------------------------------------------------------------------------------------

template <int D, bool ROPE>
__global__ __launch_bounds__(kFitThreads) void gram_f32_valu(FitArgs a) {
  constexpr int STEP = 32;
  constexpr int NE = D * (D + 1) / 2;
  constexpr int EPT = (NE + kFitThreads - 1) / kFitThreads;
  __shared__ float s_z[STEP][D + 1];

  const FitUnit f = fit_unit(a);
  const kvc_item* itp = a.items + f.item;
  const int r = itp->state.rank;
  const int Ts = itp->state.num_tokens;
  const int c = grid_chunk(a.chunk_order);
  const int t_begin = c * a.part_tokens;
  if (r == 0 || t_begin >= Ts) return;
  const int t_end = min(Ts, t_begin + a.part_tokens);
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)f.item * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)f.item * a.max_blocks : nullptr;
  const float* pool = static_cast<const float*>(f.kv ? a.layers.v[f.lrel] : a.layers.k[f.lrel]);
  const bool delta = a.mode == KVC_FIT_DELTA;
  const int tid = threadIdx.x;
  __shared__ float s_rope[4][ROPE ? D / 2 : 1];  // cos / sin of -pd and -ps (rotary keys)
  const bool rope = ROPE && f.kv == 0;
  const int style = a.pv.rope.style;
  if (rope) {
    rope_table(a.pv.rope, D, -(double)itp->dst_position, s_rope[0], s_rope[1]);
    rope_table(a.pv.rope, D, -(double)itp->src_position, s_rope[2], s_rope[3]);
    __syncthreads();
  }

  int ei[EPT], ej[EPT];
  float acc[EPT];
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    int e = tid + q * kFitThreads;
    acc[q] = 0.f;
    ei[q] = -1;
    ej[q] = 0;
    if (e < NE) {
      int i = 0;
      while (e >= D - i) {
        e -= D - i;
        ++i;
      }
      ei[q] = i;
      ej[q] = i + e;
    }
  }
  for (int t0 = t_begin; t0 < t_end; t0 += STEP) {
    for (int e = tid; e < STEP * D; e += kFitThreads) {
      const int tk = e / D, fe = e - tk * D;
      const int t = t0 + tk;
      float z = 0.f;
      if (t < t_end) {
        const int64_t od = row_offset(a.pv, dst_tab, itp->dst_offset, t, f.head);
        const int64_t os = delta ? row_offset(a.pv, src_tab, itp->src_offset, t, f.head) : -1;
        if (rope) {  // Z = R(-pd) C_dst - R(-ps) C_src
          const int pf = rope_partner(style, D, fe), i = rope_pair(style, D, fe);
          const bool first = rope_first(style, D, fe);
          if (od >= 0) z = rope_rotated(first, pool[od + fe], pool[od + pf], s_rope[0][i], s_rope[1][i]);
          if (os >= 0) z -= rope_rotated(first, pool[os + fe], pool[os + pf], s_rope[2][i], s_rope[3][i]);
        } else {
          if (od >= 0) z = pool[od + fe];
          if (os >= 0) z -= pool[os + fe];
        }
      }
      s_z[tk][fe] = z;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      if (ei[q] < 0) continue;
      float s = acc[q];
      for (int tk = 0; tk < STEP; ++tk) s = fmaf(s_z[tk][ei[q]], s_z[tk][ej[q]], s);
      acc[q] = s;
    }
    __syncthreads();
  }
  float* P = a.partials + ((size_t)fit_linear_unit(a, f) * a.max_parts + c) * D * D;
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    if (ei[q] < 0) continue;
    P[ei[q] * D + ej[q]] = acc[q];
    P[ej[q] * D + ei[q]] = acc[q];
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Projection coef = Z R_r, bf16 caches
// ---------------------------------------------------------------------------------------------------------------

// Workgroups of kProjWaves waves take kProjChunkTokens tokens of one (item, layer, K/V, head) unit (ranks above 32:
// kProjLongChunkTokens, which amortises staging the larger basis); rotary keys take kProjRopeWaves waves and
// kProjRopeChunkTokens tokens (every workgroup forms fp64 angle tables, which the longer chunk amortises, and the
// rotation's registers leave room for fewer waves).  Each wave takes 16-token
// tiles; the loads of its next tile are issued before this tile's products and coefficient stores (loads and
// stores leave a wave in order), and row addresses come from the chunk's block-table slices in LDS, so no table
// read sits between two row loads.
constexpr int kProjWaves = 8, kProjChunkTokens = 512, kProjLongChunkTokens = 1024;
constexpr int kProjRopeWaves = 4, kProjRopeChunkTokens = 1024;
constexpr int kProjChunk = 1024;  // tokens per workgroup of the float32 kernel

__host__ __device__ constexpr size_t proj_lds_bytes(int D, int RP, int nblk) {
  return (size_t)2 * RP * D * 2 + (size_t)2 * nblk * 4;
}

template <int D, int MTR, int W, bool ROPE>
__global__ __launch_bounds__(W * kWave) void proj_bf16_mfma(FitArgs a, int tpw, int nblk) {
  constexpr int KS = D / 32;          // K-steps over features
  constexpr int RP = MTR * 16;        // padded rank
  extern __shared__ __attribute__((aligned(16))) uint16_t s_dyn[];
  uint16_t* s_hi = s_dyn;
  uint16_t* s_lo = s_dyn + RP * D;
  int32_t* s_tab = reinterpret_cast<int32_t*>(s_dyn + 2 * RP * D);  // [2][nblk]: source, destination

  const FitUnit f = fit_unit(a);
  const kvc_item* itp = a.items + f.item;
  const int r = itp->state.rank;
  const int Ts = itp->state.num_tokens;
  const int chunk = W * 16 * tpw;
  const int t_begin = grid_chunk(a.chunk_order) * chunk;
  if (r == 0 || t_begin >= Ts) return;  // whole workgroup
  const int t_end = min(Ts, t_begin + chunk);
  const uint16_t* pool = static_cast<const uint16_t*>(f.kv ? a.layers.v[f.lrel] : a.layers.k[f.lrel]);
  const bool delta = a.mode == KVC_FIT_DELTA;
  const float* basis = itp->state.basis + f.unit * (int64_t)r * D;
  uint16_t* coef = static_cast<uint16_t*>(itp->state.coef) + f.unit * (int64_t)Ts * r;
  const int src_off = itp->src_offset, dst_off = itp->dst_offset;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, n = lane & 15;

  // block ids of the chunk's logical blocks (the host checked that they lie inside the item's table row)
  const int bs = a.pv.block_size, bsh = a.pv.block_shift;
  auto lblock = [&](int p) { return bsh >= 0 ? p >> bsh : p / bs; };
  const int lb0s = lblock(src_off + t_begin), lb0d = lblock(dst_off + t_begin);
  {
    const int ns = delta ? lblock(src_off + t_end - 1) - lb0s + 1 : 0;
    const int nd = lblock(dst_off + t_end - 1) - lb0d + 1;
    const int32_t* st = a.src_tables ? a.src_tables + (int64_t)f.item * a.max_blocks : nullptr;
    const int32_t* dt = a.dst_tables ? a.dst_tables + (int64_t)f.item * a.max_blocks : nullptr;
    for (int i = tid; i < ns; i += W * kWave) s_tab[i] = st ? st[lb0s + i] : lb0s + i;
    for (int i = tid; i < nd; i += W * kWave) s_tab[nblk + i] = dt ? dt[lb0d + i] : lb0d + i;
  }
  // rotary keys: Z = R(-pd) C_dst - R(-ps) C_src (angle tables ready at the staging barrier below)
  __shared__ float s_rope[4][ROPE ? D / 2 : 1];
  const bool rope = ROPE && f.kv == 0;  // uniform over the workgroup
  const int style = a.pv.rope.style;
  if (rope) {
    rope_table(a.pv.rope, D, -(double)itp->dst_position, s_rope[0], s_rope[1]);
    rope_table(a.pv.rope, D, -(double)itp->src_position, s_rope[2], s_rope[3]);
  }
  for (int e = tid; e < RP * D; e += W * kWave) {
    const int k = e / D;
    const float x = k < r ? basis[e] : 0.f;
    uint32_t hb, lb;
    split_bf16(x, hb, lb);
    s_hi[e] = (uint16_t)hb;
    s_lo[e] = (uint16_t)lb;
  }
  __syncthreads();

  // Row offset of token t through a staged table slice (-1 when the block id is out of range: the row reads as 0).
  auto row_off = [&](int off, int lb0, const int32_t* tab, int t) -> int64_t {
    const int p = off + t, lb = lblock(p), slot = p - lb * bs;
    const int32_t blk = tab[lb - lb0];
    if (blk < 0 || blk >= a.pv.num_blocks) return -1;
    return (int64_t)blk * a.pv.block_stride + (int64_t)slot * a.pv.token_stride + (int64_t)f.head * a.pv.head_stride;
  };
  // Rows of tile j: the dst (and src) row of token t0 + n, features 32 ks + 8 g .. + 7; lanes past the chunk load
  // nothing.
  struct Rows {
    u32x4 d[KS], s[KS];
  };
  auto tile_t0 = [&](int j) { return t_begin + (j * W + wave) * 16; };
  auto load_rows = [&](int j, Rows& R) __attribute__((always_inline)) {
    const int t = tile_t0(j) + n;
    const bool valid = t < t_end;
    const int64_t od = valid ? row_off(dst_off, lb0d, s_tab + nblk, t) : -1;
    const int64_t os = (valid && delta) ? row_off(src_off, lb0s, s_tab, t) : -1;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      R.d[ks] = od >= 0 ? *reinterpret_cast<const u32x4*>(pool + od + 32 * ks + 8 * g) : u32x4{0, 0, 0, 0};
      R.s[ks] = os >= 0 ? *reinterpret_cast<const u32x4*>(pool + os + 32 * ks + 8 * g) : u32x4{0, 0, 0, 0};
    }
  };
  // Z hi/lo of tile j, its products with the basis, the coefficient rows.
  auto finish = [&](int j, const Rows& R) __attribute__((always_inline)) {
    const int t = tile_t0(j) + n;
    const bool valid = t < t_end;
    bf16x8 zh[KS], zl[KS];
    if (ROPE && rope) {
      f32x4 dv[2 * KS], sv[2 * KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const u32x4 d = R.d[ks], s = R.s[ks];
        dv[2 * ks] = f32x4{bf16_lo_to_f32(d[0]), bf16_hi_to_f32(d[0]), bf16_lo_to_f32(d[1]), bf16_hi_to_f32(d[1])};
        dv[2 * ks + 1] = f32x4{bf16_lo_to_f32(d[2]), bf16_hi_to_f32(d[2]), bf16_lo_to_f32(d[3]), bf16_hi_to_f32(d[3])};
        sv[2 * ks] = f32x4{bf16_lo_to_f32(s[0]), bf16_hi_to_f32(s[0]), bf16_lo_to_f32(s[1]), bf16_hi_to_f32(s[1])};
        sv[2 * ks + 1] = f32x4{bf16_lo_to_f32(s[2]), bf16_hi_to_f32(s[2]), bf16_lo_to_f32(s[3]), bf16_hi_to_f32(s[3])};
      }
      rope_rotate_rows<D>(dv, style, g, s_rope[0], s_rope[1]);
      rope_rotate_rows<D>(sv, style, g, s_rope[2], s_rope[3]);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        u32x4 hw, lw;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const int jj = 2 * ks + (w >> 1), e = 2 * (w & 1);
          uint32_t hh, ll;
          split_bf16x2(dv[jj][e] - sv[jj][e], dv[jj][e + 1] - sv[jj][e + 1], hh, ll);
          hw[w] = hh;
          lw[w] = ll;
        }
        zh[ks] = as_bf16x8(hw);
        zl[ks] = as_bf16x8(lw);
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const u32x4 d = R.d[ks], s = R.s[ks];
        u32x4 hw, lw;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          // both features of the word split at once (two packed conversions)
          uint32_t hh, ll;
          split_bf16x2(bf16_lo_to_f32(d[w]) - bf16_lo_to_f32(s[w]), bf16_hi_to_f32(d[w]) - bf16_hi_to_f32(s[w]), hh,
                       ll);
          hw[w] = hh;
          lw[w] = ll;
        }
        zh[ks] = as_bf16x8(hw);
        zl[ks] = as_bf16x8(lw);
      }
    }
#pragma unroll
    for (int mt = 0; mt < MTR; ++mt) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int o = (16 * mt + n) * D + 32 * ks + 8 * g;
        const bf16x8 fh = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[o]));
        const bf16x8 fl = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[o]));
        acc = mfma16x16x32(fl, zh[ks], acc);
        acc = mfma16x16x32(fh, zl[ks], acc);
        acc = mfma16x16x32(fh, zh[ks], acc);
      }
      // lane holds coef[t][16 mt + 4 g + i], i = 0..3
      if (valid) {
        const int k0 = 16 * mt + 4 * g;
        uint16_t* cp = coef + (int64_t)t * r + k0;
        if ((r & 3) == 0 && k0 + 4 <= r) {
          uint2 w;
          w.x = pack_bf16x2(acc[0], acc[1]);
          w.y = pack_bf16x2(acc[2], acc[3]);
          *reinterpret_cast<uint2*>(cp) = w;
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (k0 + i < r) cp[i] = (uint16_t)f32_to_bf16_bits(acc[i]);
        }
      }
    }
  };

  // tiles of this wave in pairs: the loads of the next tile are in flight while this one is finished
  Rows ra, rb;
  if (tile_t0(0) >= t_end) return;  // whole wave
  load_rows(0, ra);
  for (int j = 0;; j += 2) {
    const bool m1 = j + 1 < tpw && tile_t0(j + 1) < t_end;
    if (m1) load_rows(j + 1, rb);
    finish(j, ra);
    if (!m1) break;
    const bool m2 = j + 2 < tpw && tile_t0(j + 2) < t_end;
    if (m2) load_rows(j + 2, ra);
    finish(j + 1, rb);
    if (!m2) break;
  }
}

// Projection, fp32 caches: one thread per (token, rank), fp32 FMAs over the features.
template <int D, bool ROPE>
__global__ __launch_bounds__(kFitThreads) void proj_f32_valu(FitArgs a) {
  extern __shared__ __attribute__((aligned(16))) float s_b[];  // [r][D]
  const FitUnit f = fit_unit(a);
  const kvc_item* itp = a.items + f.item;
  const int r = itp->state.rank;
  const int Ts = itp->state.num_tokens;
  const int t_begin = grid_chunk(a.chunk_order) * kProjChunk;
  if (r == 0 || t_begin >= Ts) return;
  const int t_end = min(Ts, t_begin + kProjChunk);
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)f.item * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)f.item * a.max_blocks : nullptr;
  const float* pool = static_cast<const float*>(f.kv ? a.layers.v[f.lrel] : a.layers.k[f.lrel]);
  const bool delta = a.mode == KVC_FIT_DELTA;
  const float* basis = itp->state.basis + f.unit * (int64_t)r * D;
  float* coef = static_cast<float*>(itp->state.coef) + f.unit * (int64_t)Ts * r;
  __shared__ float s_rope[4][ROPE ? D / 2 : 1];  // cos / sin of -pd and -ps (rotary keys)
  const bool rope = ROPE && f.kv == 0;
  const int style = a.pv.rope.style;
  if (rope) {
    rope_table(a.pv.rope, D, -(double)itp->dst_position, s_rope[0], s_rope[1]);
    rope_table(a.pv.rope, D, -(double)itp->src_position, s_rope[2], s_rope[3]);
  }
  for (int e = threadIdx.x; e < r * D; e += kFitThreads) s_b[e] = basis[e];
  __syncthreads();
  const int64_t total = (int64_t)(t_end - t_begin) * r;
  for (int64_t e = threadIdx.x; e < total; e += kFitThreads) {
    const int t = t_begin + (int)(e / r), k = (int)(e % r);
    const int64_t od = row_offset(a.pv, dst_tab, itp->dst_offset, t, f.head);
    const int64_t os = delta ? row_offset(a.pv, src_tab, itp->src_offset, t, f.head) : -1;
    float s = 0.f;
    for (int fe = 0; fe < D; ++fe) {
      float z;
      if (rope) {  // Z = R(-pd) C_dst - R(-ps) C_src
        const int pf = rope_partner(style, D, fe), i = rope_pair(style, D, fe);
        const bool first = rope_first(style, D, fe);
        z = od >= 0 ? rope_rotated(first, pool[od + fe], pool[od + pf], s_rope[0][i], s_rope[1][i]) : 0.f;
        if (os >= 0) z -= rope_rotated(first, pool[os + fe], pool[os + pf], s_rope[2][i], s_rope[3][i]);
      } else {
        z = od >= 0 ? pool[od + fe] : 0.f;
        if (os >= 0) z -= pool[os + fe];
      }
      s = fmaf(z, s_b[k * D + fe], s);
    }
    coef[(int64_t)t * r + k] = s;
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------------------------------------------


// Gram launches of K/V sides kv_begin .. kv_begin + nkv - 1.
template <bool ROPE>
static hipError_t launch_gram_variants(const FitArgs& a0, kvc_dtype dtype, int num_items, int kv_begin, int nkv,
                                       hipStream_t stream) {
  FitArgs a = a0;
  a.kv_begin = kv_begin;
  const int D = a.pv.head_dim;
  const int il = num_items * a.num_layers;
  if (dtype == KVC_BF16) {
    const int pchunks = (a.max_parts + kFitWaves - 1) / kFitWaves;
    a.chunk_order = multi_item_order(num_items, pchunks, kItemsFast);
    dim3 grid = chunk_grid(pchunks, nkv * a.pv.num_kv_heads, il, a.chunk_order);
    if (!ROPE && D == 128 && a.pv.block_shift >= 4 && a.part_tokens / a.pv.block_size + 3 <= kGramTabMax) {
      // LDS-staged rows (block sizes of at least 16 tokens, a partial's table fits the wave's LDS copy)
      const bool delta = a.mode == KVC_FIT_DELTA;
      a.chunk_order = multi_item_order(num_items, a.max_parts, kItemsFast);
      grid = chunk_grid(a.max_parts, nkv * ((a.pv.num_kv_heads + kFitWaves - 1) / kFitWaves), il, a.chunk_order);
      const void* fn = delta ? (const void*)gram_bf16_ring<true> : (const void*)gram_bf16_ring<false>;
      hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kGramLdsBytes);
      if (e != hipSuccess) return e;
      if (delta) hipLaunchKernelGGL(gram_bf16_ring<true>, grid, dim3(kFitThreads), kGramLdsBytes, stream, a);
      else hipLaunchKernelGGL(gram_bf16_ring<false>, grid, dim3(kFitThreads), kGramLdsBytes, stream, a);
    } else if (D == 64) {
      hipLaunchKernelGGL((gram_bf16_mfma<64, ROPE>), grid, dim3(kFitThreads), 0, stream, a);
    } else {
      hipLaunchKernelGGL((gram_bf16_mfma<128, ROPE>), grid, dim3(kFitThreads), 0, stream, a);
    }
  } else {
    a.chunk_order = multi_item_order(num_items, a.max_parts, kItemsFast);
    const dim3 grid = chunk_grid(a.max_parts, nkv * a.pv.num_kv_heads, il, a.chunk_order);
    if (D == 64) hipLaunchKernelGGL((gram_f32_valu<64, ROPE>), grid, dim3(kFitThreads), 0, stream, a);
    else hipLaunchKernelGGL((gram_f32_valu<128, ROPE>), grid, dim3(kFitThreads), 0, stream, a);
  }
  return hipGetLastError();
}

// The keys of a rotary cache take the register-pipelined Gram (the rotation needs each feature's partner, which that
// layout reaches with one row rotation); its values, which carry no rotation, take the plain kernels.
hipError_t launch_fit_gram(const FitArgs& a, kvc_dtype dtype, int num_items, hipStream_t stream) {
  if (a.pv.rope.style == KVC_ROPE_NONE) return launch_gram_variants<false>(a, dtype, num_items, 0, 2, stream);
  const hipError_t e = launch_gram_variants<true>(a, dtype, num_items, 0, 1, stream);
  return e != hipSuccess ? e : launch_gram_variants<false>(a, dtype, num_items, 1, 1, stream);
}

template <int D, int MTR, bool ROPE>
static hipError_t launch_proj_bf16_m(const FitArgs& a0, int nkv, int max_tokens, int num_items, hipStream_t stream) {
  constexpr int W = ROPE ? kProjRopeWaves : kProjWaves;
  const int chunk = ROPE ? kProjRopeChunkTokens : (MTR > 2 ? kProjLongChunkTokens : kProjChunkTokens);
  FitArgs a = a0;
  const int chunks = (max_tokens + chunk - 1) / chunk;
  a.chunk_order = multi_item_order(num_items, chunks, kChunksRotated);
  const dim3 grid = chunk_grid(chunks, nkv * a.pv.num_kv_heads, num_items * a.num_layers, a.chunk_order);
  const int nblk = (chunk + a.pv.block_size - 1) / a.pv.block_size + 1;
  const size_t lds = proj_lds_bytes(D, MTR * 16, nblk);
  hipError_t e = hipFuncSetAttribute((const void*)proj_bf16_mfma<D, MTR, W, ROPE>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((proj_bf16_mfma<D, MTR, W, ROPE>), grid, dim3(W * kWave), lds, stream, a, chunk / (16 * W),
                     nblk);
  return hipGetLastError();
}

template <int D, bool ROPE>
static hipError_t launch_proj_bf16(const FitArgs& a, int mtr, int nkv, int max_tokens, int num_items,
                                   hipStream_t stream) {
  switch (mtr) {
    case 1: return launch_proj_bf16_m<D, 1, ROPE>(a, nkv, max_tokens, num_items, stream);
    case 2: return launch_proj_bf16_m<D, 2, ROPE>(a, nkv, max_tokens, num_items, stream);
    case 3:
    case 4: return launch_proj_bf16_m<D, 4, ROPE>(a, nkv, max_tokens, num_items, stream);
    default: return launch_proj_bf16_m<D, 8, ROPE>(a, nkv, max_tokens, num_items, stream);
  }
}

// Projection launches of K/V sides kv_begin .. kv_begin + nkv - 1.
template <bool ROPE>
static hipError_t launch_proj_variants(const FitArgs& a0, kvc_dtype dtype, int num_items, int max_tokens,
                                       int max_rank, int kv_begin, int nkv, hipStream_t stream) {
  FitArgs a = a0;
  a.kv_begin = kv_begin;
  const int D = a.pv.head_dim;
  if (dtype == KVC_BF16) {
    const int mtr = (max_rank + 15) / 16;
    return D == 64 ? launch_proj_bf16<64, ROPE>(a, mtr, nkv, max_tokens, num_items, stream)
                   : launch_proj_bf16<128, ROPE>(a, mtr, nkv, max_tokens, num_items, stream);
  }
  const int chunks = (max_tokens + kProjChunk - 1) / kProjChunk;
  a.chunk_order = multi_item_order(num_items, chunks, kChunksRotated);
  const dim3 grid = chunk_grid(chunks, nkv * a.pv.num_kv_heads, num_items * a.num_layers, a.chunk_order);
  const size_t lds = (size_t)max_rank * D * sizeof(float);
  if (D == 64) hipLaunchKernelGGL((proj_f32_valu<64, ROPE>), grid, dim3(kFitThreads), lds, stream, a);
  else hipLaunchKernelGGL((proj_f32_valu<128, ROPE>), grid, dim3(kFitThreads), lds, stream, a);
  return hipGetLastError();
}

hipError_t launch_fit_proj(const FitArgs& a, kvc_dtype dtype, int num_items, int max_tokens, int max_rank,
                           hipStream_t stream) {
  if (max_rank == 0 || max_tokens == 0) return hipSuccess;
  // a rotary cache's values carry no rotation: they take the plain kernels
  if (a.pv.rope.style == KVC_ROPE_NONE)
    return launch_proj_variants<false>(a, dtype, num_items, max_tokens, max_rank, 0, 2, stream);
  const hipError_t e = launch_proj_variants<true>(a, dtype, num_items, max_tokens, max_rank, 0, 1, stream);
  return e != hipSuccess ? e : launch_proj_variants<false>(a, dtype, num_items, max_tokens, max_rank, 1, 1, stream);
}

}  // namespace kvc
