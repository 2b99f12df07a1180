// Per-layer factorisation (Section 3.3 with the layer's whole KV feature dimension D = H d).  The K (or V) rows of one
// layer, every KV head side by side, form one T x D matrix Z per (item, layer, K/V) "layer unit"; its rank-r
// truncated SVD (Eq. 7) is reached through the Gram G = Z^T Z (D x D, D up to 1024):
//   gram_layer   the 128 x 128 blocks on and above the diagonal of G over one token range, a 256 x 256 pair of
//                feature groups per workgroup (Z hi/lo staged once per step in LDS as MFMA fragments, bf16 hi/lo MFMA).
//                Block sizes below 8 or not a power of two: gram_pair, the d x d block Z_h1^T Z_h2 of a head pair with
//                its mirror, rows read straight into registers.  float32 caches: 64 x 64 blocks on VALU.
//   gram_reduce  the partials of a unit summed in a fixed order in fp64.
//   subspace     k = 64 or 128 columns: X <- orth(G X) (fp64 GEMM, shifted Cholesky QR; a second, exact pass
//                before each Rayleigh-Ritz step), then the
//                Rayleigh-Ritz matrix X^T G X goes to the per-head eigensolver as a dense k x k input; its top r
//                eigenvectors V give the basis rows (X V^T)^T and sigma = sqrt(Ritz value).  The top-r subspace
//                converges like (lambda_{k+1} / lambda_r)^iterations.
//   proj_layer   coef = Z B^T summed over the heads (bf16 MFMA; each head's d columns of B staged hi/lo in LDS).
#include <algorithm>
#include <type_traits>

#include "kvc_device.h"
#include "kvc_launch.h"

namespace kvc {

constexpr int kLayerThreads = 256;
constexpr int kLayerWaves = kLayerThreads / kWave;

struct LayerUnit {
  int item, lrel, layer, kv;
};
__device__ __forceinline__ LayerUnit layer_unit(const LayerFitArgs& a, int u) {
  LayerUnit lu;
  lu.item = u / (a.num_layers * 2);
  const int rem = u - lu.item * a.num_layers * 2;
  lu.lrel = rem >> 1;
  lu.kv = rem & 1;
  lu.layer = a.layer_begin + lu.lrel;
  return lu;
}

// ---------------------------------------------------------------------------------------------------------------
// Gram of head pairs, bf16
// ---------------------------------------------------------------------------------------------------------------

// Z = dst - src of 8 tokens' segments as bf16 hi/lo (the difference of two bf16 values is exact in fp32).
template <int FT>
__device__ __forceinline__ void pair_form_z(const typename GramSeg<FT>::T* rd, const typename GramSeg<FT>::T* rs,
                                            typename GramSeg<FT>::T* zh, typename GramSeg<FT>::T* zl) {
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
}

// Tile IDX of half HALF: rows fi = HALF FT/2 + IDX / FT of head 1, columns fj = IDX % FT of head 2.
template <int D, int HALF, int IDX>
__device__ __forceinline__ void pair_tile(f32x4* acc, const typename GramSeg<D / 16>::T* ah_,
                                          const typename GramSeg<D / 16>::T* al_,
                                          const typename GramSeg<D / 16>::T* bh_,
                                          const typename GramSeg<D / 16>::T* bl_) {
  constexpr int FT = D / 16, fi = HALF * (FT / 2) + IDX / FT, fj = IDX % FT;
  const bf16x8 ah = gram_fragment<FT, fi>(ah_), al = gram_fragment<FT, fi>(al_);
  const bf16x8 bh = gram_fragment<FT, fj>(bh_), bl = gram_fragment<FT, fj>(bl_);
  acc[IDX] = mfma16x16x32(al, bh, acc[IDX]);
  acc[IDX] = mfma16x16x32(ah, bl, acc[IDX]);
  acc[IDX] = mfma16x16x32(ah, bh, acc[IDX]);
}
template <int D, int HALF, int... Is>
__device__ __forceinline__ void pair_tiles(f32x4* acc, const typename GramSeg<D / 16>::T* ah,
                                           const typename GramSeg<D / 16>::T* al,
                                           const typename GramSeg<D / 16>::T* bh,
                                           const typename GramSeg<D / 16>::T* bl, std::integer_sequence<int, Is...>) {
  (pair_tile<D, HALF, Is>(acc, ah, al, bh, bl), ...);
}

// One wave per (token range, half of the block's tiles); the two waves of a range read the same rows.
template <int D>
__global__ __launch_bounds__(kLayerThreads) void gram_pair_bf16(LayerFitArgs a) {
  constexpr int FT = D / 16, NTW = FT * FT / 2, STEP = 32;
  using Seg = typename GramSeg<FT>::T;
  const int H = a.pv.num_kv_heads, DL = H * D;
  const int u = blockIdx.z;
  const LayerUnit lu = layer_unit(a, u);
  const kvc_item* itp = a.items + lu.item;
  const int r = itp->state.rank, Ts = itp->state.num_tokens;
  int p = blockIdx.y, h1 = 0;
  while (p >= H - h1) {
    p -= H - h1;
    ++h1;
  }
  const int h2 = h1 + p;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 4, n = lane & 15;
  const int part = blockIdx.x * (kLayerWaves / 2) + (wave >> 1), half = wave & 1;
  const int t_begin = part * a.part_tokens;
  if (r == 0 || t_begin >= Ts) return;  // per wave: no barrier in this kernel
  const int t_end = min(Ts, t_begin + a.part_tokens);
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const uint16_t* pool = static_cast<const uint16_t*>(lu.kv ? a.layers.v[lu.lrel] : a.layers.k[lu.lrel]);
  const bool delta = a.mode == KVC_FIT_DELTA;

  f32x4 acc[NTW];
#pragma unroll
  for (int q = 0; q < NTW; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int t0 = t_begin; t0 < t_end; t0 += STEP) {
    const int t = t0 + 8 * g;
    Seg z1h[8], z1l[8], z2h[8], z2l[8];
    {
      int64_t od[8], os[8];
      Seg rd[8], rs[8];
      row_offsets8(a.pv, dst_tab, itp->dst_offset, t, t_end, h1, od);
      if (delta) row_offsets8(a.pv, src_tab, itp->src_offset, t, t_end, h1, os);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        rd[j] = od[j] >= 0 ? *reinterpret_cast<const Seg*>(pool + od[j] + FT * n) : Seg{};
        rs[j] = (delta && os[j] >= 0) ? *reinterpret_cast<const Seg*>(pool + os[j] + FT * n) : Seg{};
      }
      pair_form_z<FT>(rd, rs, z1h, z1l);
      row_offsets8(a.pv, dst_tab, itp->dst_offset, t, t_end, h2, od);
      if (delta) row_offsets8(a.pv, src_tab, itp->src_offset, t, t_end, h2, os);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        rd[j] = od[j] >= 0 ? *reinterpret_cast<const Seg*>(pool + od[j] + FT * n) : Seg{};
        rs[j] = (delta && os[j] >= 0) ? *reinterpret_cast<const Seg*>(pool + os[j] + FT * n) : Seg{};
      }
      pair_form_z<FT>(rd, rs, z2h, z2l);
    }
    if (half == 0) pair_tiles<D, 0>(acc, z1h, z1l, z2h, z2l, std::make_integer_sequence<int, NTW>{});
    else pair_tiles<D, 1>(acc, z1h, z1l, z2h, z2l, std::make_integer_sequence<int, NTW>{});
  }
  float* P = a.partials + ((size_t)u * a.max_parts + part) * DL * DL;
#pragma unroll
  for (int q = 0; q < NTW; ++q) {
    const int fi = half * (FT / 2) + q / FT, fj = q % FT;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = h1 * D + FT * (4 * g + i) + fi, col = h2 * D + FT * n + fj;
      P[(size_t)row * DL + col] = acc[q][i];
      if (h1 != h2) P[(size_t)col * DL + row] = acc[q][i];
    }
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Gram of the layer, bf16, through LDS (power-of-two block size of at least 8)
// ---------------------------------------------------------------------------------------------------------------
// The layer's features fall into 128-feature blocks b and 256-feature groups g = {blocks 2g, 2g + 1}.  One 512-thread
// workgroup per (unit, token range, group pair g1 <= g2).  Each 32-token step every thread forms Z = dst - src for 4
// features x 8 tokens of the pair's features, splits it into bf16 hi/lo and writes it transposed into LDS, 16 bytes
// per (feature, 8 tokens): exactly one MFMA operand lane.  Each wave then accumulates half of one 128 x 128 block
// b1 <= b2 (4 x 8 tiles, 3 products each) from those fragments.  The next step's rows are in flight during the
// products and the table entries one step further ahead; the LDS holds two steps (128 KB) and a step costs one
// barrier.  Only blocks b1 <= b2 are written; the reduction reads the blocks below the diagonal transposed.
constexpr int kGLThreads = 512, kGLStep = 32, kGLSlots = 512;
constexpr size_t kGLBufChunks = (size_t)2 * 4 * kGLSlots;                     // hi/lo x 4 token groups x slots
constexpr size_t kGLLdsBytes = 2 * kGLBufChunks * sizeof(u32x4);              // two steps: 128 KB

// Slot of a feature chunk within its (hi/lo, token group) row: a XOR swizzle inside aligned groups of 8 slots keeps
// both the producers' stores (slots 4q + j) and the fragment reads (16 consecutive slots) free of bank conflicts.
__device__ __forceinline__ int gl_swz(int c) { return c ^ ((c >> 3) & 7); }

// Paging of one pool as the Gram reads it (power-of-two block size of at least 8).
struct GLPaging {
  int64_t block_stride, token_stride;
  int32_t shift, num_blocks;
};

// Table entries of the (at most two) blocks that hold tokens t .. t + 7.  An entry no token before t_end needs is
// read at index 0 instead (every read stays inside the table row) and is never used: gl_row drops tokens past t_end.
// The loaded values are not touched here, so the loads stay in flight until the rows are addressed.
__device__ __forceinline__ int2 gl_blocks(const GLPaging& pg, const int32_t* __restrict__ table, int32_t off, int t,
                                          int t_end) {
  const int32_t p = off + t;
  const int32_t lb0 = p >> pg.shift, lb1 = (p + 7) >> pg.shift;
  const bool ok0 = t < t_end, ok1 = (lb1 != lb0) & ((lb1 << pg.shift) - off < t_end);
  if (!table) return make_int2(lb0, lb1);
  return make_int2(table[ok0 ? lb0 : 0], table[ok1 ? lb1 : 0]);
}

// Rows of the 8 tokens t .. t + 7 of a sequence (head 0): the first n0 lie in block entry b.x from slot k0 on, the
// rest in b.y from slot 0, so row j starts at base0 + j * token_stride (j < n0) or base1 + j * token_stride.  Bit j
// of valid: token t + j lies before t_end in a block inside the pool.
struct GLRows {
  int64_t base0, base1;
  int32_t n0;
  uint32_t valid;
};
__device__ __forceinline__ GLRows gl_rows(const GLPaging& pg, int2 b, int32_t off, int t, int t_end) {
  GLRows r;
  const int32_t p = off + t, k0 = p & ((1 << pg.shift) - 1);
  r.n0 = min(8, (1 << pg.shift) - k0);
  const bool ok0 = (b.x >= 0) & (b.x < pg.num_blocks), ok1 = (b.y >= 0) & (b.y < pg.num_blocks);
  r.base0 = ok0 ? (int64_t)b.x * pg.block_stride + (int64_t)k0 * pg.token_stride : 0;
  r.base1 = ok1 ? (int64_t)b.y * pg.block_stride - (int64_t)r.n0 * pg.token_stride : 0;
  const int in_seq = min(8, max(0, t_end - t));
  const uint32_t seq = (1u << in_seq) - 1u, first = (1u << r.n0) - 1u;
  r.valid = seq & ((ok0 ? first : 0u) | (ok1 ? ~first & 0xffu : 0u));
  return r;
}

// Zero page the LDS Gram reads in place of a missing row (never written): covers a row's lane offsets up to this size.
constexpr int kGLZeroBytes = 65536;
__device__ __attribute__((aligned(256))) uint32_t gl_zero_page[kGLZeroBytes / 4];

// ROPE: the key rows of a rotary cache enter Z in canonical coordinates, Z = R(-pd) C_dst - R(-ps) C_src (Eq. 12 with
// Align): a producer lane holds 4 consecutive features of one head, the partner of a rotate-half pair lies in the lane
// D / 8 away (one xor shuffle per row dword) and the partner of an adjacent pair inside the lane; the lane's 4 angles
// per side are formed once.
template <int D, bool DELTA, bool FULL, bool ROPE>
__global__ __launch_bounds__(kGLThreads) void gram_layer_bf16(LayerFitArgs a, int num_pairs, int num_groups) {
  extern __shared__ __attribute__((aligned(16))) u32x4 gl_lds[];
  const int H = a.pv.num_kv_heads, DL = H * D, NB = (DL + 127) / 128;
  // XCD-aware order: the workgroups one XCD receives (every 8th) take consecutive work items, so the group pairs of
  // one (unit, token range) share that XCD's L2
  const int nwork = gridDim.x, L = blockIdx.x, xcd = L & 7, pos = L >> 3, per = nwork >> 3, rem = nwork & 7;
  const int w = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + pos;
  int pr = w % num_pairs, g1 = 0;
  const int up = w / num_pairs, part = up % a.max_parts, u = up / a.max_parts;
  while (pr >= num_groups - g1) {
    pr -= num_groups - g1;
    ++g1;
  }
  const int g2 = g1 + pr;
  const bool diag = g1 == g2;
  const LayerUnit lu = layer_unit(a, u);
  const kvc_item* itp = a.items + lu.item;
  const int r = itp->state.rank, Ts = itp->state.num_tokens;
  const int t_begin = part * a.part_tokens;
  if (r == 0 || t_begin >= Ts) return;  // whole workgroup
  const int t_end = min(Ts, t_begin + a.part_tokens);
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const uint16_t* pool = static_cast<const uint16_t*>(lu.kv ? a.layers.v[lu.lrel] : a.layers.k[lu.lrel]);
  const int32_t doff = itp->dst_offset, soff = itp->src_offset;
  GLPaging pg;
  pg.block_stride = a.pv.block_stride;
  pg.token_stride = a.pv.token_stride;
  pg.shift = a.pv.block_shift;
  pg.num_blocks = a.pv.num_blocks;
  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index (and every value derived from it alone) is uniform: row addressing runs on the scalar unit
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // producer: slots 4q .. 4q + 3 (group g1 below slot 256, g2 above; a diagonal pair uses g1's only), tokens
  // 8 tg .. 8 tg + 7 of the step; a wave's lanes share tg and cover 256 consecutive slots
  const int q = tid & 127, tg = wave >> 1, slot = 4 * q;
  const int fglob = slot < 256 ? g1 * 256 + slot : g2 * 256 + slot - 256;
  const bool pact = !diag || (wave & 1) == 0;
  const bool inrange = pact && fglob < DL;
  // byte offset of the lane's 4 features within a token's row (the launcher checks it fits 32 bits)
  const uint32_t fbytes = inrange ? 2u * (uint32_t)((fglob / D) * a.pv.head_stride + fglob % D) : 0u;
  // rotary keys: cos / sin of the lane's 4 features' pairs at -pd (dst) and -ps (src), and whether each feature is
  // the first of its pair
  const bool rot = ROPE && lu.kv == 0;  // uniform over the workgroup
  const int style = a.pv.rope.style;
  float rcd[ROPE ? 4 : 1], rsd[ROPE ? 4 : 1], rcs[ROPE ? 4 : 1], rss[ROPE ? 4 : 1];
  bool rfirst = true;
  if constexpr (ROPE) {
    const int f0 = fglob % D;
    rfirst = rope_first(style, D, f0);  // the same for the lane's 4 features (pairs never straddle a lane's quad)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      rcd[e] = 1.0f, rsd[e] = 0.0f, rcs[e] = 1.0f, rss[e] = 0.0f;
      if (rot) {
        const double th = a.pv.rope.inv_freq[rope_pair(style, D, f0 + e)];
        double sn, cs;
        sincos(-(double)itp->dst_position * th, &sn, &cs);
        rcd[e] = (float)cs;
        rsd[e] = (float)sn;
        sincos(-(double)itp->src_position * th, &sn, &cs);
        rcs[e] = (float)cs;
        rss[e] = (float)sn;
      }
    }
  }

  // consumer: wave = 2 x block pair (i1, i2) + row half
  const int bp = wave >> 1, half = wave & 1, i1 = bp >> 1, i2 = bp & 1;
  const int b1 = 2 * g1 + i1, b2 = 2 * g2 + i2;
  const bool job = b1 < NB && b2 < NB && !(diag && i1 > i2);
  const int sA = i1 * 128 + half * 64, sB = (diag ? 0 : 256) + i2 * 128;
  const int lrow = lane & 15, ltg = lane >> 4;

  f32x4 acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  uint2 rd[8], rs[8];
  uint32_t present = 0;  // (uniform) bit j: dst row j of the step exists, bit 8 + j: src row j
  // row loads of one step: a uniform row pointer plus the lane's byte offset.  A missing row (or a lane past D) loads
  // from the pool's first row and is zeroed when used, so no register with a load in flight is written.
  auto issue = [&](int t0, int2 bd, int2 bs) {
    const int t = t0 + 8 * tg;
    const uint32_t fb = fbytes;
    // every row address stays inside the pool (a block holds at least 8 token rows); rows that do not exist are
    // dropped through `present` when used
    auto rows = [&](const GLRows& x, uint2* dstv) {
      if (x.n0 == 8) {  // the 8 tokens share one block
#pragma unroll
        for (int j = 0; j < 8; ++j)
          dstv[j] = *reinterpret_cast<const uint2*>(reinterpret_cast<const char*>(pool + x.base0 + j * pg.token_stride) + fb);
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int64_t o = (j < x.n0 ? x.base0 : x.base1) + j * pg.token_stride;
          dstv[j] = *reinterpret_cast<const uint2*>(reinterpret_cast<const char*>(pool + o) + fb);
        }
      }
    };
    const GLRows xd = gl_rows(pg, bd, doff, t, t_end);
    rows(xd, rd);
    uint32_t m = xd.valid;
    if constexpr (DELTA) {
      const GLRows xs = gl_rows(pg, bs, soff, t, t_end);
      rows(xs, rs);
      m |= xs.valid << 8;
    }
    present = m;
  };
  // Z hi/lo of the loaded rows, transposed into one step's LDS buffer.  MASKED drops rows that do not exist and lanes
  // past D; a step whose 8 (16) rows all exist in a wave wholly inside D skips it.
  const bool wave_inside = pact && ((wave & 1) ? g2 : g1) * 256 + 256 <= DL;
  const uint32_t all_rows = DELTA ? 0xffffu : 0xffu;
  auto produce = [&](u32x4* buf, auto masked) {
    constexpr bool MASKED = decltype(masked)::value;
    uint32_t hi[8][2], lo[8][2];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      uint32_t dx = rd[j].x, dy = rd[j].y, sx = 0u, sy = 0u;
      if constexpr (DELTA) {
        sx = rs[j].x;
        sy = rs[j].y;
      }
      if constexpr (MASKED) {
        const bool pd = inrange && ((present >> j) & 1u), ps = DELTA && inrange && ((present >> (8 + j)) & 1u);
        dx = pd ? dx : 0u;
        dy = pd ? dy : 0u;
        sx = ps ? sx : 0u;
        sy = ps ? sy : 0u;
      }
      float d4[4] = {bf16_lo_to_f32(dx), bf16_hi_to_f32(dx), bf16_lo_to_f32(dy), bf16_hi_to_f32(dy)};
      float s4[4] = {bf16_lo_to_f32(sx), bf16_hi_to_f32(sx), bf16_lo_to_f32(sy), bf16_hi_to_f32(sy)};
      if constexpr (ROPE) {
        if (rot) {  // uniform: every lane of the wave takes part in the shuffles
          float pd4[4], ps4[4];
          if (style == KVC_ROPE_HALF) {
            const uint32_t qdx = __shfl_xor(dx, D / 8, kWave), qdy = __shfl_xor(dy, D / 8, kWave);
            const uint32_t qsx = __shfl_xor(sx, D / 8, kWave), qsy = __shfl_xor(sy, D / 8, kWave);
            pd4[0] = bf16_lo_to_f32(qdx), pd4[1] = bf16_hi_to_f32(qdx);
            pd4[2] = bf16_lo_to_f32(qdy), pd4[3] = bf16_hi_to_f32(qdy);
            ps4[0] = bf16_lo_to_f32(qsx), ps4[1] = bf16_hi_to_f32(qsx);
            ps4[2] = bf16_lo_to_f32(qsy), ps4[3] = bf16_hi_to_f32(qsy);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              pd4[e] = d4[e ^ 1];
              ps4[e] = s4[e ^ 1];
            }
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool first = style == KVC_ROPE_HALF ? rfirst : (e & 1) == 0;
            const float dn = rope_rotated(first, d4[e], pd4[e], rcd[e], rsd[e]);
            const float sn = rope_rotated(first, s4[e], ps4[e], rcs[e], rss[e]);
            d4[e] = dn;
            s4[e] = sn;
          }
        }
      }
      split_bf16x2(d4[0] - s4[0], d4[1] - s4[1], hi[j][0], lo[j][0]);
      split_bf16x2(d4[2] - s4[2], d4[3] - s4[3], hi[j][1], lo[j][1]);
    }
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const uint32_t sel = (f & 1) ? 0x07060302u : 0x05040100u;
      u32x4 ch, cl;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        ch[k] = __builtin_amdgcn_perm(hi[2 * k + 1][f >> 1], hi[2 * k][f >> 1], sel);
        cl[k] = __builtin_amdgcn_perm(lo[2 * k + 1][f >> 1], lo[2 * k][f >> 1], sel);
      }
      buf[tg * kGLSlots + gl_swz(slot + f)] = ch;
      buf[(4 + tg) * kGLSlots + gl_swz(slot + f)] = cl;
    }
  };
  auto produce_step = [&](u32x4* buf) {
    if (wave_inside && present == all_rows) produce(buf, std::false_type{});
    else produce(buf, std::true_type{});
  };
  // the wave's 32 tiles of one step
  auto products = [&](const u32x4* buf) {
    bf16x8 ah[4], al[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = gl_swz(sA + 16 * i + lrow);
      ah[i] = as_bf16x8(buf[ltg * kGLSlots + c]);
      al[i] = as_bf16x8(buf[(4 + ltg) * kGLSlots + c]);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = gl_swz(sB + 16 * j + lrow);
      const bf16x8 bh = as_bf16x8(buf[ltg * kGLSlots + c]), bl = as_bf16x8(buf[(4 + ltg) * kGLSlots + c]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[i][j] = mfma16x16x32(al[i], bh, acc[i][j]);
        acc[i][j] = mfma16x16x32(ah[i], bl, acc[i][j]);
        acc[i][j] = mfma16x16x32(ah[i], bh, acc[i][j]);
      }
    }
  };

  const int nsteps = (t_end - t_begin + kGLStep - 1) / kGLStep;
  int2 td = make_int2(-1, -1), ts = make_int2(-1, -1);  // table entries of the next step to issue
  auto tables = [&](int k) {
    td = gl_blocks(pg, dst_tab, doff, t_begin + k * kGLStep + 8 * tg, t_end);
    if constexpr (DELTA) ts = gl_blocks(pg, src_tab, soff, t_begin + k * kGLStep + 8 * tg, t_end);
  };
  auto issue_step = [&](int k) {
    issue(t_begin + k * kGLStep, td, ts);
    if (k + 1 < nsteps) tables(k + 1);
  };
  // rows of step k (any k: past the sequence every row is missing) with missing rows read from the zero page, then
  // the table entries of step k + 1
  auto issue_zero = [&](int k) {
    const int t = t_begin + k * kGLStep + 8 * tg;
    const char* zero = reinterpret_cast<const char*>(gl_zero_page);
    auto rows = [&](const GLRows& x, uint2* dstv) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int64_t o = (j < x.n0 ? x.base0 : x.base1) + j * pg.token_stride;
        const char* row = (x.valid >> j) & 1u ? reinterpret_cast<const char*>(pool + o) : zero;
        dstv[j] = *reinterpret_cast<const uint2*>(row + fbytes);
      }
    };
    rows(gl_rows(pg, td, doff, t, t_end), rd);
    if constexpr (DELTA) rows(gl_rows(pg, ts, soff, t, t_end), rs);
    tables(k + 1);
  };
  if constexpr (FULL) {
    // every lane lies inside D and a missing row reads the zero page: one straight-line body per step, products of
    // step s, then the rows of step s + 1 (loaded one step earlier), then the loads of step s + 2.  Waves without a
    // block (diagonal pairs) run the products too and drop them; rows past the sequence load zeros.
    tables(0);
    issue_zero(0);
    produce(gl_lds, std::false_type{});
    issue_zero(1);
    __syncthreads();
    for (int s = 0; s < nsteps; ++s) {
      products(gl_lds + (s & 1) * kGLBufChunks);
      produce(gl_lds + ((s + 1) & 1) * kGLBufChunks, std::false_type{});
      // each of the 96 MFMAs followed by a share of the VALU work of the next step's rows
#pragma unroll
      for (int q = 0; q < 96; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // VALU
      }
      issue_zero(s + 2);
      __syncthreads();
    }
  } else {
    if (pact) {
      tables(0);
      issue_step(0);
      produce_step(gl_lds);
    }
    __syncthreads();
    for (int s = 0; s < nsteps; ++s) {
      const bool more = s + 1 < nsteps;
      if (pact && more) issue_step(s + 1);
      if (job) products(gl_lds + (s & 1) * kGLBufChunks);
      if (pact && more) produce_step(gl_lds + ((s + 1) & 1) * kGLBufChunks);
      __syncthreads();
    }
  }

  if (!job) return;
  float* P = a.partials + ((size_t)u * a.max_parts + part) * DL * DL;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int col = b2 * 128 + 16 * j + lrow;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = b1 * 128 + half * 64 + 16 * i + 4 * ltg + e;
        if (row < DL && col < DL) P[(size_t)row * DL + col] = acc[i][j][e];
      }
    }
}

// ---------------------------------------------------------------------------------------------------------------
// Gram, float32 caches: one 64 x 64 block of G over one token range per workgroup (VALU, 4 x 4 outputs per thread)
// ---------------------------------------------------------------------------------------------------------------

constexpr int kF32Block = 64, kF32Step = 16;

// Rotary angle tables of the float32 per-layer kernels in LDS: cos / sin at -pd, then at -ps, D / 2 each.
constexpr size_t kLayerRopeTableBytes = 4 * 64 * sizeof(float);
template <int D>
__device__ __forceinline__ void layer_rope_tables(const LayerFitArgs& a, const kvc_item* itp, float* t) {
  rope_table(a.pv.rope, D, -(double)itp->dst_position, t, t + D / 2);
  rope_table(a.pv.rope, D, -(double)itp->src_position, t + D, t + 3 * D / 2);
}
// Feature f of a key row in canonical coordinates, from the row at `row` (f32 pool) and the tables of one side.
template <int D>
__device__ __forceinline__ float layer_rope_value(const float* row, int f, int style, const float* c, const float* s) {
  const int i = rope_pair(style, D, f);
  return rope_rotated(rope_first(style, D, f), row[f], row[rope_partner(style, D, f)], c[i], s[i]);
}

template <int D>
__global__ __launch_bounds__(kLayerThreads) void gram_block_f32(LayerFitArgs a) {
  __shared__ float s_a[kF32Step][kF32Block + 1], s_b[kF32Step][kF32Block + 1];
  __shared__ float s_rope[4 * (D / 2)];
  const int H = a.pv.num_kv_heads, DL = H * D, nb = DL / kF32Block;
  const int bi = blockIdx.x / nb, bj = blockIdx.x - bi * nb;
  const int part = blockIdx.y, u = blockIdx.z;
  const LayerUnit lu = layer_unit(a, u);
  const kvc_item* itp = a.items + lu.item;
  const int r = itp->state.rank, Ts = itp->state.num_tokens;
  const int t_begin = part * a.part_tokens;
  if (r == 0 || t_begin >= Ts) return;  // whole workgroup
  const int t_end = min(Ts, t_begin + a.part_tokens);
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const float* pool = static_cast<const float*>(lu.kv ? a.layers.v[lu.lrel] : a.layers.k[lu.lrel]);
  const bool delta = a.mode == KVC_FIT_DELTA;
  const int tid = threadIdx.x, ti = tid / 16, tj = tid % 16;
  float acc[4][4] = {};
  // keys of a rotary cache in canonical coordinates: Z = R(-pd) C_dst - R(-ps) C_src (tables read after a barrier)
  const bool rot = a.pv.rope.style != KVC_ROPE_NONE && lu.kv == 0;
  const int style = a.pv.rope.style;
  if (rot) layer_rope_tables<D>(a, itp, s_rope);
  // every 64-feature block lies inside one head (64 divides d)
  auto z_of = [&](int t, int F) {
    const int h = F / D, f = F - h * D;
    const int64_t od = row_offset(a.pv, dst_tab, itp->dst_offset, t, h);
    float z = od >= 0 ? (rot ? layer_rope_value<D>(pool + od, f, style, s_rope, s_rope + D / 2) : pool[od + f]) : 0.0f;
    if (delta) {
      const int64_t os = row_offset(a.pv, src_tab, itp->src_offset, t, h);
      if (os >= 0) z -= rot ? layer_rope_value<D>(pool + os, f, style, s_rope + D, s_rope + 3 * D / 2) : pool[os + f];
    }
    return z;
  };
  __syncthreads();
  for (int t0 = t_begin; t0 < t_end; t0 += kF32Step) {
    for (int e = tid; e < kF32Step * kF32Block; e += kLayerThreads) {
      const int tk = e / kF32Block, c = e - tk * kF32Block, t = t0 + tk;
      s_a[tk][c] = t < t_end ? z_of(t, bi * kF32Block + c) : 0.0f;
      s_b[tk][c] = t < t_end ? z_of(t, bj * kF32Block + c) : 0.0f;
    }
    __syncthreads();
#pragma unroll 4
    for (int tk = 0; tk < kF32Step; ++tk) {
      float x[4], y[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[i] = s_a[tk][4 * ti + i];
        y[i] = s_b[tk][4 * tj + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(x[i], y[j], acc[i][j]);
    }
    __syncthreads();
  }
  float* P = a.partials + ((size_t)u * a.max_parts + part) * DL * DL;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      P[(size_t)(bi * kF32Block + 4 * ti + i) * DL + bj * kF32Block + 4 * tj + j] = acc[i][j];
}

// G = sum of the unit's partials in order, fp64, one 32 x 32 tile per workgroup.  With upper_only the partials hold
// the 128 x 128 blocks on and above the diagonal, and a tile below it is summed from its mirror and transposed in LDS.
__global__ __launch_bounds__(kLayerThreads) void gram_reduce(LayerFitArgs a, int upper_only) {
  __shared__ double tr[32][33];
  const int DL = a.pv.num_kv_heads * a.pv.head_dim, nt = DL / 32;
  const int u = blockIdx.y, I = blockIdx.x / nt, J = blockIdx.x - I * nt;
  const LayerUnit lu = layer_unit(a, u);
  const int Ts = a.items[lu.item].state.num_tokens;
  const int parts = min(a.max_parts, (Ts + a.part_tokens - 1) / a.part_tokens);
  const bool mirror = upper_only && (I >> 2) > (J >> 2);
  const int sI = mirror ? J : I, sJ = mirror ? I : J;
  const int rr = threadIdx.x >> 5, c = threadIdx.x & 31;
  const float* P = a.partials + (size_t)u * a.max_parts * DL * DL;
  double* G = a.gram + (size_t)u * DL * DL;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int row = rr + 8 * k;
    const size_t e = (size_t)(sI * 32 + row) * DL + sJ * 32 + c;
    double s = 0.0;
    for (int p = 0; p < parts; ++p) s += (double)P[(size_t)p * DL * DL + e];
    if (mirror) tr[row][c] = s;
    else G[(size_t)(I * 32 + row) * DL + J * 32 + c] = s;
  }
  if (!mirror) return;  // whole workgroup
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int row = rr + 8 * k;
    G[(size_t)(I * 32 + row) * DL + J * 32 + c] = tr[c][row];
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Subspace iteration on G (fp64 arithmetic)
// ---------------------------------------------------------------------------------------------------------------

__device__ __forceinline__ double hash_uniform(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t h = a * 0x9E3779B1u ^ (b + 0x7F4A7C15u) * 0x85EBCA77u ^ (c + 0x165667B1u) * 0xC2B2AE3Du;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  h *= 0x297A2D39u;
  h ^= h >> 15;
  return (double)h * (2.0 / 4294967296.0) - 1.0;
}

// Starting columns: deterministic pseudo-random entries in [-1, 1).
__global__ __launch_bounds__(kLayerThreads) void sub_init(LayerFitArgs a) {
  const int DL = a.pv.num_kv_heads * a.pv.head_dim;
  const int u = blockIdx.y;
  const int e = blockIdx.x * kLayerThreads + threadIdx.x;
  if (e == 0) {
    a.conv[u] = 0;
    a.iters[u] = 0;
  }
  if (e >= a.k * DL) return;
  a.y[(size_t)u * a.k * DL + e] = hash_uniform((uint32_t)u, (uint32_t)(e / DL), (uint32_t)(e % DL));
}

// Y = G X (fp64) for every unit on the matrix cores: a 128 x 64 tile of Y (features x columns) per workgroup of eight
// waves, each wave a 32 x 32 block as 2 x 2 products v_mfma_f64_16x16x4_f64 (operands: lane l holds A[l % 16][l / 16]
// and B[l / 16][l % 16]; result element v of lane l is D[l / 16 + 4 v][l % 16]).  16-wide slices of G and X are
// staged in LDS, the next slices loaded into registers while the current ones are multiplied.
constexpr int kGemmRows = 128, kGemmCols = 64, kGemmK = 16, kGemmMI = 2, kGemmNJ = 2;
constexpr int kGemmThreads = kGemmRows / (16 * kGemmMI) * (kGemmCols / (16 * kGemmNJ)) * kWave;
typedef double f64x4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(kGemmThreads) void sub_gemm(LayerFitArgs a) {
  constexpr int TR = kGemmRows, TC = kGemmCols, KB = kGemmK, MI = kGemmMI, NJ = kGemmNJ;
  constexpr int NG = TR * KB / kGemmThreads, NX = TC * KB / kGemmThreads;
  static_assert(NG * kGemmThreads == TR * KB && NX * kGemmThreads == TC * KB, "whole slices per thread");
  __shared__ double s_g[TR][KB + 1], s_x[TC][KB + 1];
  const int DL = a.pv.num_kv_heads * a.pv.head_dim;
  const int f0 = blockIdx.x * TR, c0 = blockIdx.y * TC, u = blockIdx.z;
  if (a.conv[u]) return;  // whole workgroup: the unit has stopped
  const double* G = a.gram + (size_t)u * DL * DL;
  const double* X = a.x + (size_t)u * a.k * DL;
  double* Y = a.y + (size_t)u * a.k * DL;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int WC = TC / (16 * NJ);  // waves across the columns
  const int wr = wave / WC, wc = wave % WC, li = lane & 15, lk = lane >> 4;
  double pg[NG], px[NX];
  auto load = [&](int k0) {
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      const int e = tid + q * kGemmThreads, i = e / KB, kk = e - i * KB;
      pg[q] = f0 + i < DL ? G[(size_t)(f0 + i) * DL + k0 + kk] : 0.0;
    }
#pragma unroll
    for (int q = 0; q < NX; ++q) {
      const int e = tid + q * kGemmThreads, i = e / KB, kk = e - i * KB;
      px[q] = X[(size_t)(c0 + i) * DL + k0 + kk];
    }
  };
  f64x4 acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
  load(0);
  for (int k0 = 0; k0 < DL; k0 += KB) {
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      const int e = tid + q * kGemmThreads, i = e / KB, kk = e - i * KB;
      s_g[i][kk] = pg[q];
    }
#pragma unroll
    for (int q = 0; q < NX; ++q) {
      const int e = tid + q * kGemmThreads, i = e / KB, kk = e - i * KB;
      s_x[i][kk] = px[q];
    }
    __syncthreads();
    if (k0 + KB < DL) load(k0 + KB);
#pragma unroll
    for (int kk = 0; kk < KB; kk += 4) {
      double ga[MI], xb[NJ];
#pragma unroll
      for (int t = 0; t < MI; ++t) ga[t] = s_g[16 * (MI * wr + t) + li][kk + lk];
#pragma unroll
      for (int t = 0; t < NJ; ++t) xb[t] = s_x[16 * (NJ * wc + t) + li][kk + lk];
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(ga[i], xb[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int c = c0 + 16 * (NJ * wc + j) + li;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int f = f0 + 16 * (MI * wr + i) + lk + 4 * v;
        if (f < DL) Y[(size_t)c * DL + f] = acc[i][j][v];
      }
    }
}

// Whole-workgroup sum (fixed order: waves in order), result in every thread.
template <int NW>
__device__ __forceinline__ double block_sum(double v, double* s_red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s_red[wave] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int w = 0; w < NW; ++w) s += s_red[w];
  return s;
}

// X = orthonormal columns spanning Y by Cholesky QR applied twice: S = Y^T Y (+ shift), S = R^T R, X = Y R^{-1}.
// The first pass carries a shift of the size of the rounding error of S (11 (D k + k (k + 1)) u ||Y||_F^2), which keeps
// the factorisation defined for ill-conditioned Y and leaves Y R^{-1} well enough conditioned for the exact second
// pass.  A perturbation of 1e-12 of Y's RMS (pseudo-random) keeps Y of full rank k when G has lower rank.  Four
// kernels per pass, each spread over the unit's features except the k x k factorisation:
//   cqr_scale   the perturbation size of each unit (first pass)
//   cqr_syrk    partial S over 256 features per workgroup (register blocks over LDS tiles of 32 features)
//   cqr_factor  one workgroup per unit: the partials summed in order, the shift, Cholesky and the inverse of R
//               (k = 64: the factorisation in one wave's registers, the inverse by four waves; k = 128: eight waves
//               on the matrix in LDS)
//   cqr_apply   X = Y R^{-1} for 64 features per workgroup (the tile is read whole before it is written, so the
//               second pass runs in place)
constexpr int kCqrThreads = 256, kCqrChunk = 256, kCqrSub = 32, kCqrRows = 64, kCqrWChunk = 32;

// The perturbed entry e of unit u's Y (every kernel of a pass forms it the same way).
__device__ __forceinline__ double cqr_perturbed(double y, double eps, uint32_t round, int u, size_t e) {
  return fma(eps, hash_uniform(0x51u + round, (uint32_t)u, (uint32_t)e), y);
}

constexpr int kScaleThreads = 1024;
__global__ __launch_bounds__(kScaleThreads) void cqr_scale(LayerFitArgs a, uint32_t round) {
  constexpr int NB = 8;
  __shared__ double red[kScaleThreads / kWave];
  const int DL = a.pv.num_kv_heads * a.pv.head_dim, u = blockIdx.x;
  if (a.conv[u]) return;  // whole workgroup: the unit has stopped
  const size_t n = (size_t)a.k * DL;
  const double* Y = a.y + (size_t)u * n;
  double ss[NB];
#pragma unroll
  for (int q = 0; q < NB; ++q) ss[q] = 0.0;
  for (size_t e0 = threadIdx.x; e0 < n; e0 += NB * kScaleThreads)
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const size_t e = e0 + q * kScaleThreads;
      const double y = e < n ? Y[e] : 0.0;
      ss[q] = fma(y, y, ss[q]);
    }
  double s = 0.0;
#pragma unroll
  for (int q = 0; q < NB; ++q) s += ss[q];
  s = block_sum<kScaleThreads / kWave>(s, red);
  const double rms = sqrt(s / (double)n);
  if (threadIdx.x == 0) a.eps[(round & 1u) * a.num_units + u] = rms > 0.0 ? 1e-12 * rms : 1.0;
}

template <int K>
__global__ __launch_bounds__(kCqrThreads) void cqr_syrk(LayerFitArgs a, const double* __restrict__ src, int perturb,
                                                         uint32_t round) {
  // the partial S = Y_c Y_c^T of 256 features on the matrix cores: each of the four waves takes a K/2 x K/2 quadrant
  // as (K/32)^2 products v_mfma_f64_16x16x4_f64 (lane layouts as in sub_gemm), both operands read from the staged
  // slice of Y
  constexpr int T = K / 32;
  static_assert(kCqrThreads == 4 * kWave, "four waves, one quadrant each");
  __shared__ double tile[K][kCqrSub + 1];
  const int DL = a.pv.num_kv_heads * a.pv.head_dim, nch = (DL + kCqrChunk - 1) / kCqrChunk;
  const int chunk = blockIdx.x, u = blockIdx.y, tid = threadIdx.x;
  if (a.conv[u]) return;  // whole workgroup: the unit has stopped
  const int lane = tid & 63, wave = tid >> 6, qi = wave >> 1, qj = wave & 1, li = lane & 15, lk = lane >> 4;
  const int f_begin = chunk * kCqrChunk, f_end = min(DL, f_begin + kCqrChunk);
  const double* Y = src + (size_t)u * K * DL;
  const double eps = perturb ? a.eps[(round & 1u) * a.num_units + u] : 0.0;
  f64x4 acc[T][T];
#pragma unroll
  for (int i = 0; i < T; ++i)
#pragma unroll
    for (int j = 0; j < T; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int f0 = f_begin; f0 < f_end; f0 += kCqrSub) {
    for (int e = tid; e < K * kCqrSub; e += kCqrThreads) {
      const int c = e / kCqrSub, ff = e - c * kCqrSub;
      const size_t idx = (size_t)c * DL + f0 + ff;
      const double y = Y[idx];
      tile[c][ff] = perturb ? cqr_perturbed(y, eps, round, u, idx) : y;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kCqrSub; kk += 4) {
      double ya[T], yb[T];
#pragma unroll
      for (int t = 0; t < T; ++t) {
        ya[t] = tile[qi * (K / 2) + 16 * t + li][kk + lk];
        yb[t] = tile[qj * (K / 2) + 16 * t + li][kk + lk];
      }
#pragma unroll
      for (int i = 0; i < T; ++i)
#pragma unroll
        for (int j = 0; j < T; ++j) acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(ya[i], yb[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  double* P = a.spart + ((size_t)u * nch + chunk) * K * K;
#pragma unroll
  for (int i = 0; i < T; ++i)
#pragma unroll
    for (int j = 0; j < T; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        P[(qi * (K / 2) + 16 * i + lk + 4 * v) * K + qj * (K / 2) + 16 * j + li] = acc[i][j][v];
}

// k = 64: wave 0 factorises, lane c holding column c of S in registers (entries k <= c are used).  Step j takes the
// pivot from lane j, every lane forms its entry R[j][c] and writes it to row j of R in LDS, and the trailing update
// reads that row back as broadcast loads (two entries per load) instead of one readlane pair per entry.  All four
// waves then form R^{-1} by back substitution, four lanes per column: with one lane per column the 64 accumulators
// of a lane left no registers to batch the inverse's LDS loads, which the compiler then waited on one at a time
// (67 us per launch at 8B/32K against 35 us now).
// Orders one wave's LDS accesses around points where lanes read values other lanes wrote.
__device__ __forceinline__ void wave_lds_sync_layer() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)b, lane), hi = __builtin_amdgcn_readlane((uint32_t)(b >> 32), lane);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// 64-bit broadcast of lane SEL of every quad (DPP quad_perm [SEL, SEL, SEL, SEL]; all lanes active).
template <int SEL>
__device__ __forceinline__ double quad_bcast_f64(double x) {
  constexpr int ctrl = SEL * 0x55;
  const unsigned long long b = __builtin_bit_cast(unsigned long long, x);
  const int lo = __builtin_amdgcn_mov_dpp((int)(unsigned)b, ctrl, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp((int)(unsigned)(b >> 32), ctrl, 0xF, 0xF, false);
  return __builtin_bit_cast(double, ((unsigned long long)(unsigned)hi << 32) | (unsigned)lo);
}

constexpr int kCqrFactorThreads = 256;

// The perturbation size of the next round's shifted pass, 1e-12 of the RMS of Y, from this shifted pass's trace of
// S = ||Y||_F^2: from the third round on, Y = G X in consecutive rounds with X of full rank and columns of about unit
// norm, so consecutive products have the same scale (the first two rounds measure Y itself: the random start, then
// the first product).  Slot (round + 1) mod 2 of eps; this round's passes read slot round mod 2.
__device__ __forceinline__ void cqr_next_eps(const LayerFitArgs& a, int u, uint32_t round, double tr, int DL, int K) {
  const double rms = sqrt(fmax(tr, 0.0) / ((double)DL * K));
  a.eps[((round + 1u) & 1u) * a.num_units + u] = rms > 0.0 ? 1e-12 * rms : 1.0;
}

__global__ __launch_bounds__(kCqrFactorThreads) void cqr_factor_reg64(LayerFitArgs a, int shifted, uint32_t round) {
  constexpr int K = 64, KP = K + 2;  // row stride: even, so that 16-byte loads stay aligned
  __shared__ __attribute__((aligned(16))) double s_r[K * KP];  // rows of R (the factorisation)
  __shared__ __attribute__((aligned(16))) double s_c[K * KP];  // columns of R above the diagonal, 0 on and below it
  __shared__ double s_ri[K];                                   // 1 / R[j][j]
  const int DL = a.pv.num_kv_heads * a.pv.head_dim, nch = (DL + kCqrChunk - 1) / kCqrChunk;
  const int u = blockIdx.x, tid = threadIdx.x;
  if (a.conv[u]) return;  // whole workgroup: the unit has stopped
  if (tid < kWave) {
    // the factorisation, by wave 0: lane c holds column c of S
    const int lane = tid;
    const double* P = a.spart + (size_t)u * nch * K * K;
    double col[K];
    double myinv = 0.0;  // 1 / R[lane][lane]
#pragma unroll
    for (int k = 0; k < K; ++k) col[k] = 0.0;
    for (int p = 0; p < nch; ++p)
#pragma unroll
      for (int k = 0; k < K; ++k) col[k] += P[(size_t)p * K * K + k * K + lane];
    if (shifted) {
      double d = 0.0;
#pragma unroll
      for (int k = 0; k < K; ++k) d = k == lane ? col[k] : d;
      double tr = 0.0;
#pragma unroll
      for (int c = 0; c < K; ++c) tr += readlane_f64(d, c);
      if (round >= 1u && lane == 0) cqr_next_eps(a, u, round, tr, DL, K);
      const double shift = 11.0 * ((double)DL * K + (double)K * (K + 1)) * 1.1102230246251565e-16 * tr;
#pragma unroll
      for (int k = 0; k < K; ++k) col[k] += k == lane ? shift : 0.0;
    }
    // entries below the diagonal of a lane's column are updated too but never read.  Pivots: 1 / sqrt from the
    // hardware reciprocal square root and one Newton step (relative error about 2^-47), R[j][j] = d / sqrt(d) and
    // row j of R = the column entries times 1 / sqrt(d).
#pragma unroll
    for (int j = 0; j < K; ++j) {
      const double d0 = readlane_f64(col[j], j);
      const double d = d0 > 1e-300 ? d0 : 1e-300;
      const double y0 = __builtin_amdgcn_rsq(d);
      const double inv = y0 * fma(-0.5 * d * y0, y0, 1.5);
      col[j] = lane == j ? d * inv : col[j] * inv;
      myinv = lane == j ? inv : myinv;
      s_r[j * KP + lane] = col[j];
      wave_lds_sync_layer();
#pragma unroll
      for (int k = j + 1; k < K; k += 2) {
        if (k + 1 < K) {
          const double2 rk = *reinterpret_cast<const double2*>(&s_r[j * KP + k]);
          col[k] -= rk.x * col[j];
          col[k + 1] -= rk.y * col[j];
        } else {
          col[k] -= s_r[j * KP + k] * col[j];
        }
      }
    }
    // column c of R (lane c) for the inverse, infinities clamped to the largest finite values so that a zero never
    // meets an infinity (a NaN from NaN input stays NaN)
#pragma unroll
    for (int i = 0; i < K; ++i) {
      constexpr double kMax = 1.7976931348623157e308;
      const double x = col[i];
      s_c[lane * KP + i] = i < lane ? (x == x ? fmin(fmax(x, -kMax), kMax) : x) : 0.0;
    }
    s_ri[lane] = myinv;
  }
  __syncthreads();
  // W = R^{-1} by column-oriented back substitution (R w = e_c): for j = K - 1 .. 0, w_j = acc_j / R[j][j], then
  // acc_i -= R[i][j] w_j for i < j.  Column c = tid / 4 is taken by the four lanes of a quad, lane s of the quad
  // holding rows 4 q + s (q = 0 .. 15, so that the triangle's work is spread evenly); w_j comes from the lane that
  // holds row j by a quad broadcast.  Every step updates all 16 rows of a lane: rows i >= j read the zeros of s_c
  // and stay unchanged (they are final by then).  For columns c < j, acc_j stays 0 and so w_j = 0 (W is upper
  // triangular).  Steps go in blocks of four (rows 4 J .. 4 J + 3), so that the broadcast's source lane is a
  // constant; cur follows row 4 J + s through the block.
  const int c = tid >> 2, sq = tid & 3;
  constexpr int QR = K / 4;
  double acc[QR];
#pragma unroll
  for (int q = 0; q < QR; ++q) acc[q] = 4 * q + sq == c ? 1.0 : 0.0;
  double* W = a.hmat + (size_t)u * K * K + c;
  for (int J = QR - 1; J >= 0; --J) {
    double cur = acc[0];
#pragma unroll
    for (int q = 1; q < QR; ++q) cur = q == J ? acc[q] : cur;
    auto step = [&](auto tc) {
      constexpr int t = decltype(tc)::value;
      const int j = 4 * J + t;
      const double wj = quad_bcast_f64<t>(cur * s_ri[j]);
      W[(size_t)j * K] = wj;  // row j of W (the quad's four lanes store the same value: no branch in the loop)
      const double* cj = s_c + j * KP + sq;
#pragma unroll
      for (int q = 0; q < QR; ++q) acc[q] = fma(-cj[4 * q], wj, acc[q]);
      cur = fma(-cj[4 * J], wj, cur);
    };
    step(std::integral_constant<int, 3>{});
    step(std::integral_constant<int, 2>{});
    step(std::integral_constant<int, 1>{});
    step(std::integral_constant<int, 0>{});
  }
}

// k = 128 (ranks above 48): S in LDS with rows padded to K + 1, eight waves.  The right-looking Cholesky (upper,
// S = R^T R; a pivot that is not positive is replaced by a tiny one) spreads each step's trailing update over 128
// columns x 4 row groups and reads the pivot row unscaled, so a step needs one barrier: row j is scaled after it,
// while the next step works on the rows below.  R^{-1} then comes by column-oriented back substitution as for k = 64
// (four lanes per column, 32 rows per lane), with the columns of R copied into the lower triangle of the LDS matrix
// so that each is contiguous.  (One wave for the whole factorisation took about 1 ms per launch at rank 64.)
constexpr int kCqrFactor128Threads = 512;

template <int K>
__global__ __launch_bounds__(kCqrFactor128Threads) void cqr_factor(LayerFitArgs a, int shifted, uint32_t round) {
  constexpr int KP = K + 1, NB = 8, NT = kCqrFactor128Threads;
  static_assert(NT == 4 * K && (K * K) % (NB * NT) == 0, "four lanes per column; whole load batches");
  extern __shared__ double fs[];  // [K][K + 1]
  __shared__ double s_ri[K];      // 1 / R[j][j]
  const int DL = a.pv.num_kv_heads * a.pv.head_dim, nch = (DL + kCqrChunk - 1) / kCqrChunk;
  const int u = blockIdx.x, tid = threadIdx.x;
  if (a.conv[u]) return;  // whole workgroup: the unit has stopped
  const double* P = a.spart + (size_t)u * nch * K * K;
  for (int e0 = tid; e0 < K * K; e0 += NB * NT) {
    double s[NB];
#pragma unroll
    for (int q = 0; q < NB; ++q) s[q] = 0.0;
    for (int p = 0; p < nch; ++p)
#pragma unroll
      for (int q = 0; q < NB; ++q) s[q] += P[(size_t)p * K * K + e0 + q * NT];
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int e = e0 + q * NT;
      fs[(e / K) * KP + e % K] = s[q];
    }
  }
  __syncthreads();
  if (shifted) {
    double tr = 0.0;
    for (int c = 0; c < K; ++c) tr += fs[c * KP + c];
    if (round >= 1u && tid == 0) cqr_next_eps(a, u, round, tr, DL, K);
    const double shift = 11.0 * ((double)DL * K + (double)K * (K + 1)) * 1.1102230246251565e-16 * tr;
    __syncthreads();
    for (int c = tid; c < K; c += NT) fs[c * KP + c] += shift;
    __syncthreads();
  }
  // Cholesky: thread (column cc, row group hg) updates S[k][cc] -= S[j][k] S[j][cc] / d for j < k <= cc, k = hg mod 4,
  // NB rows at a time with every load of the batch before its stores
  const int cc = tid & (K - 1), hg = tid / K;
  for (int j = 0; j < K; ++j) {
    const double d0 = fs[j * KP + j];
    const double d = d0 > 1e-300 ? d0 : 1e-300;
    const double y0 = __builtin_amdgcn_rsq(d);
    const double inv = y0 * fma(-0.5 * d * y0, y0, 1.5);  // 1 / sqrt(d), relative error about 2^-47
    if (cc > j) {
      const double sjc = fs[j * KP + cc] * (inv * inv);
      for (int k0 = j + 1 + ((hg - j - 1) & 3); k0 <= cc; k0 += 4 * NB) {
        double rj[NB], v[NB];
#pragma unroll
        for (int q = 0; q < NB; ++q) {
          const int k = k0 + 4 * q <= cc ? k0 + 4 * q : k0;
          rj[q] = fs[j * KP + k];
          v[q] = fs[k * KP + cc];
        }
#pragma unroll
        for (int q = 0; q < NB; ++q)
          if (k0 + 4 * q <= cc) fs[(k0 + 4 * q) * KP + cc] = v[q] - rj[q] * sjc;
      }
    }
    __syncthreads();
    if (tid == 0) s_ri[j] = inv;
    if (j + tid < K) fs[j * KP + j + tid] = tid == 0 ? d * inv : fs[j * KP + j + tid] * inv;
  }
  __syncthreads();
  // column j of R into row j left of the diagonal: fs[j KP + i] = R[i][j] for i < j
  for (int e = tid; e < K * K; e += NT) {
    const int j = e / K, i = e - j * K;
    if (i < j) fs[j * KP + i] = fs[i * KP + j];
  }
  __syncthreads();
  // W = R^{-1}, R w = e_c: for j = K - 1 .. 0, w_j = acc_j / R[j][j], then acc_i -= R[i][j] w_j for i < j.  Column
  // c = tid / 4 by the four lanes of a quad, lane s holding rows 4 q + s (q < 32); w_j by a quad broadcast from the
  // lane that holds row j.  Row j of the LDS matrix holds R[i][j] for i < j, then R[j][j] and row j of R: rows i >= j
  // take those values too, but they are final by then and the updates are never used.  For columns c < j, acc_j
  // stays 0 and so w_j = 0 (W is upper triangular).  Steps go in blocks of four so that the broadcast's source lane
  // is a constant; cur follows row 4 J + s through the block.
  const int c = tid >> 2, sq = tid & 3;
  constexpr int QR = K / 4;
  double acc[QR];
#pragma unroll
  for (int q = 0; q < QR; ++q) acc[q] = 4 * q + sq == c ? 1.0 : 0.0;
  double* W = a.hmat + (size_t)u * K * K + c;
  for (int J = QR - 1; J >= 0; --J) {
    double cur = acc[0];
#pragma unroll
    for (int q = 1; q < QR; ++q) cur = q == J ? acc[q] : cur;
    auto step = [&](auto tc) {
      constexpr int t = decltype(tc)::value;
      const int j = 4 * J + t;
      const double wj = quad_bcast_f64<t>(cur * s_ri[j]);
      W[(size_t)j * K] = wj;  // row j of W (the quad's four lanes store the same value: no branch in the loop)
      const double* cj = fs + j * KP + sq;
#pragma unroll
      for (int q = 0; q < QR; ++q) acc[q] = fma(-cj[4 * q], wj, acc[q]);
      cur = fma(-cj[4 * J], wj, cur);
    };
    step(std::integral_constant<int, 3>{});
    step(std::integral_constant<int, 2>{});
    step(std::integral_constant<int, 1>{});
    step(std::integral_constant<int, 0>{});
  }
}

size_t cqr_factor_lds(int k) { return (size_t)k * (k + 1) * sizeof(double); }
size_t cqr_apply_lds(int k) {
  return ((size_t)k * (kCqrRows + 1) + (size_t)kCqrWChunk * k) * sizeof(double);
}

// dst = (src (+ perturbation)) R^{-1} for 64 features; R^{-1} is streamed through LDS 32 rows at a time.
template <int K>
__global__ __launch_bounds__(kCqrThreads) void cqr_apply(LayerFitArgs a, const double* src, double* dst, int perturb,
                                                          uint32_t round) {
  extern __shared__ double as_[];
  double* ty = as_;                          // [K][kCqrRows + 1]
  double* tw = as_ + K * (kCqrRows + 1);     // [kCqrWChunk][K]
  const int DL = a.pv.num_kv_heads * a.pv.head_dim;
  const int f0 = blockIdx.x * kCqrRows, u = blockIdx.y, tid = threadIdx.x;
  if (a.conv[u]) return;  // whole workgroup: the unit has stopped
  const double* Y = src + (size_t)u * K * DL;
  const double* W = a.hmat + (size_t)u * K * K;
  const double eps = perturb ? a.eps[(round & 1u) * a.num_units + u] : 0.0;
  for (int e = tid; e < K * kCqrRows; e += kCqrThreads) {
    const int c = e / kCqrRows, ff = e - c * kCqrRows;
    const size_t idx = (size_t)c * DL + f0 + ff;
    const double y = Y[idx];
    ty[c * (kCqrRows + 1) + ff] = perturb ? cqr_perturbed(y, eps, round, u, idx) : y;
  }
  // on the matrix cores: wave (qi, qj) takes features 32 qi .. 32 qi + 31 and columns (K / 2) qj .. as 2 x K / 32
  // products v_mfma_f64_16x16x4_f64 (lane layouts as in sub_gemm)
  constexpr int NT = K / 32;
  const int lane = tid & 63, wave = tid >> 6, qi = wave >> 1, qj = wave & 1, li = lane & 15, lk = lane >> 4;
  f64x4 acc[2][NT];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int i0 = 0; i0 < K; i0 += kCqrWChunk) {
    __syncthreads();
    for (int e = tid; e < kCqrWChunk * K; e += kCqrThreads) tw[e] = W[(size_t)i0 * K + e];
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kCqrWChunk; kk += 4) {
      double ya[2], wb[NT];
#pragma unroll
      for (int t = 0; t < 2; ++t) ya[t] = ty[(i0 + kk + lk) * (kCqrRows + 1) + 32 * qi + 16 * t + li];
#pragma unroll
      for (int t = 0; t < NT; ++t) wb[t] = tw[(kk + lk) * K + (K / 2) * qj + 16 * t + li];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(ya[i], wb[j], acc[i][j], 0, 0, 0);
    }
  }
  double* X = dst + (size_t)u * K * DL;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        X[(size_t)((K / 2) * qj + 16 * j + li) * DL + f0 + 32 * qi + 16 * i + lk + 4 * v] = acc[i][j][v];
}

// Rayleigh-Ritz matrix H = (X^T Y + Y^T X) / 2 with Y = G X, in two steps: the partials X_c^T Y_c of 256 features
// per workgroup on the matrix cores (the layout of cqr_syrk, with X rows as the A operand and Y rows as B), written
// over the unit's Cholesky QR partials (idle until the next iteration; Y is kept for the residual check); then one
// workgroup per unit sums them in chunk order and takes the symmetric part.
template <int K>
__global__ __launch_bounds__(kCqrThreads) void sub_rayleigh(LayerFitArgs a) {
  constexpr int T = K / 32;
  constexpr int SW = K > 64 ? kCqrSub / 2 : kCqrSub;  // slice width: both slices within 64 KB of LDS
  __shared__ double tx[K][SW + 1], ty[K][SW + 1];
  const int DL = a.pv.num_kv_heads * a.pv.head_dim, nch = (DL + kCqrChunk - 1) / kCqrChunk;
  const int chunk = blockIdx.x, u = blockIdx.y, tid = threadIdx.x;
  if (a.conv[u]) return;  // whole workgroup: the unit has stopped
  const int lane = tid & 63, wave = tid >> 6, qi = wave >> 1, qj = wave & 1, li = lane & 15, lk = lane >> 4;
  const int f_begin = chunk * kCqrChunk, f_end = min(DL, f_begin + kCqrChunk);
  const double* X = a.x + (size_t)u * K * DL;
  const double* Y = a.y + (size_t)u * K * DL;
  f64x4 acc[T][T];
#pragma unroll
  for (int i = 0; i < T; ++i)
#pragma unroll
    for (int j = 0; j < T; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int f0 = f_begin; f0 < f_end; f0 += SW) {
    for (int e = tid; e < K * SW; e += kCqrThreads) {
      const int c = e / SW, ff = e - c * SW;
      tx[c][ff] = X[(size_t)c * DL + f0 + ff];
      ty[c][ff] = Y[(size_t)c * DL + f0 + ff];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < SW; kk += 4) {
      double xa[T], yb[T];
#pragma unroll
      for (int t = 0; t < T; ++t) {
        xa[t] = tx[qi * (K / 2) + 16 * t + li][kk + lk];
        yb[t] = ty[qj * (K / 2) + 16 * t + li][kk + lk];
      }
#pragma unroll
      for (int i = 0; i < T; ++i)
#pragma unroll
        for (int j = 0; j < T; ++j) acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(xa[i], yb[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  double* P = a.spart + ((size_t)u * nch + chunk) * K * K;
#pragma unroll
  for (int i = 0; i < T; ++i)
#pragma unroll
    for (int j = 0; j < T; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        P[(qi * (K / 2) + 16 * i + lk + 4 * v) * K + qj * (K / 2) + 16 * j + li] = acc[i][j][v];
}

template <int K>
__global__ __launch_bounds__(kCqrThreads) void sub_rayleigh_sum(LayerFitArgs a) {
  const int DL = a.pv.num_kv_heads * a.pv.head_dim, nch = (DL + kCqrChunk - 1) / kCqrChunk;
  const int u = blockIdx.x;
  if (a.conv[u]) return;  // whole workgroup: the unit has stopped
  const double* P = a.spart + (size_t)u * nch * K * K;
  double* Hm = a.hmat + (size_t)u * K * K;
  for (int e = threadIdx.x; e < K * K; e += kCqrThreads) {
    const int i = e / K, j = e - i * K;
    double sij = 0.0, sji = 0.0;
    for (int c = 0; c < nch; ++c) {
      sij += P[(size_t)c * K * K + i * K + j];
      sji += P[(size_t)c * K * K + j * K + i];
    }
    Hm[e] = 0.5 * (sij + sji);
  }
}

// Residual check of the top-r Ritz pairs: w_j = X v_j, z_j = Y v_j = G w_j (Y = G X of the last product), theta_j =
// w^T z / w^T w and resid_j = ||z - theta_j w|| / ||w|| = sqrt(z^T z - (w^T z)^2 / w^T w) / ||w||.  Each workgroup takes
// 256 features of a unit and all r pairs (kCheckBatch at a time), so X and Y are read once per unit; it writes its
// sums of w^T w, w^T z and z^T z over those features (in the syrk partials, free between the Rayleigh-Ritz sum and the
// next Cholesky QR pass), and sub_check_sum adds the feature chunks in order.  The expanded form of the squared
// residual carries the rounding of the sums, a few 1e-15 of z^T z; near the stopping tolerance (1e-6 of theta_1) the
// squared residual is at least 1e-12 of z^T z, so the decision moves by well under 1 % of the tolerance.  (The float32
// Ritz vectors put the residual's floor near 1e-7 theta_1.)
constexpr int kCheckBatch = 16;
__global__ __launch_bounds__(kLayerThreads) void sub_check(LayerFitArgs a) {
  constexpr int B = kCheckBatch, NV = 3 * B;
  __shared__ float s_v[B * 128];
  __shared__ double s_red[kLayerWaves][NV];
  const int DL = a.pv.num_kv_heads * a.pv.head_dim, k = a.k, r = a.rank;
  const int chunk = blockIdx.x, u = blockIdx.y, tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  if (a.conv[u]) return;  // whole workgroup
  const int nch = (DL + kLayerThreads - 1) / kLayerThreads;
  const int f = chunk * kLayerThreads + tid;
  const double* X = a.x + (size_t)u * k * DL;
  const double* Y = a.y + (size_t)u * k * DL;
  double* part = a.spart + ((size_t)u * nch + chunk) * r * 3;
  for (int j0 = 0; j0 < r; j0 += B) {
    const int nb = min(B, r - j0);
    __syncthreads();
    for (int e = tid; e < B * k; e += kLayerThreads)
      s_v[e] = e < nb * k ? a.vrows[((size_t)u * r + j0) * k + e] : 0.0f;
    __syncthreads();
    double w[B], z[B];
#pragma unroll
    for (int jj = 0; jj < B; ++jj) w[jj] = z[jj] = 0.0;
    if (f < DL) {
      for (int c = 0; c < k; ++c) {
        const double x = X[(size_t)c * DL + f], y = Y[(size_t)c * DL + f];
#pragma unroll
        for (int jj = 0; jj < B; ++jj) {
          const double v = (double)s_v[jj * k + c];
          w[jj] = fma(v, x, w[jj]);
          z[jj] = fma(v, y, z[jj]);
        }
      }
    }
    // per-lane terms, summed over the wave by a fixed butterfly, then over the four waves in order
    double t[NV];
#pragma unroll
    for (int jj = 0; jj < B; ++jj) {
      t[3 * jj] = w[jj] * w[jj];
      t[3 * jj + 1] = w[jj] * z[jj];
      t[3 * jj + 2] = z[jj] * z[jj];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
#pragma unroll
      for (int i = 0; i < NV; ++i) t[i] += __shfl_xor(t[i], o, kWave);
    if (lane == 0)
#pragma unroll
      for (int i = 0; i < NV; ++i) s_red[wave][i] = t[i];
    __syncthreads();
    if (tid < 3 * nb) {
      double sum = 0.0;
#pragma unroll
      for (int wv = 0; wv < kLayerWaves; ++wv) sum += s_red[wv][tid];
      part[(size_t)j0 * 3 + tid] = sum;
    }
  }
}

// resid_j of unit u from the feature chunks' sums (in chunk order).
__global__ __launch_bounds__(KVC_MAX_RANK) void sub_check_sum(LayerFitArgs a) {
  const int DL = a.pv.num_kv_heads * a.pv.head_dim, r = a.rank;
  const int u = blockIdx.x, j = threadIdx.x;
  if (a.conv[u] || j >= r) return;
  const int nch = (DL + kLayerThreads - 1) / kLayerThreads;
  const double* part = a.spart + (size_t)u * nch * r * 3;
  double ww = 0.0, wz = 0.0, zz = 0.0;
  for (int ch = 0; ch < nch; ++ch) {
    const double* p = part + ((size_t)ch * r + j) * 3;
    ww += p[0];
    wz += p[1];
    zz += p[2];
  }
  a.resid[(size_t)u * KVC_MAX_RANK + j] = ww > 0.0 ? sqrt(fmax(zz - wz * (wz / ww), 0.0) / ww) : 0.0;
}

// Stop a unit once every top-r residual is at most kLayerTol * theta_1 (theta_1 = sigma_1^2 of the Ritz step), or at
// the iteration cap; `done` is the number of subspace iterations so far.
__global__ __launch_bounds__(kWave) void sub_decide(LayerFitArgs a, int done, int last) {
  const int u = blockIdx.x, lane = threadIdx.x;
  if (a.conv[u]) return;  // whole wave
  double m = 0.0;
  for (int j = lane; j < a.rank; j += kWave) m = fmax(m, a.resid[(size_t)u * KVC_MAX_RANK + j]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmax(m, __shfl_xor(m, o, kWave));
  if (lane == 0) {
    const double s1 = (double)a.vsigma[(size_t)u * a.rank];
    const bool ok = m <= kLayerTol * s1 * s1;
    if (ok || last) {
      a.conv[u] = ok ? 1 : 2;
      a.iters[u] = done;
    }
  }
}

// Basis row j of unit u = (X^T v_j)^T with v_j the j-th Ritz vector, canonical sign (largest-magnitude entry
// positive, the first of the entries within 2^-20 of it), written with sigma to the item's per-layer state.
__global__ __launch_bounds__(kLayerThreads) void sub_basis(LayerFitArgs a) {
  __shared__ double s_red[kLayerWaves];
  __shared__ float s_v[128];
  const int D = a.pv.head_dim, DL = a.pv.num_kv_heads * D, k = a.k;
  const int j = blockIdx.x, u = blockIdx.y;
  const LayerUnit lu = layer_unit(a, u);
  const kvc_state& st = a.items[lu.item].state;
  const int r = st.rank;
  if (j >= r) return;  // whole workgroup
  const float* v = a.vrows + ((size_t)u * a.rank + j) * k;
  const double* X = a.x + (size_t)u * k * DL;
  for (int c = threadIdx.x; c < k; c += kLayerThreads) s_v[c] = v[c];
  __syncthreads();
  constexpr int MAXF = 1024 / kLayerThreads;
  double b[MAXF];
  double mx = 0.0;
#pragma unroll
  for (int q = 0; q < MAXF; ++q) {
    const int f = threadIdx.x + q * kLayerThreads;
    b[q] = 0.0;
    if (f < DL) {
      double s = 0.0;
      for (int c = 0; c < k; ++c) s = fma((double)s_v[c], X[(size_t)c * DL + f], s);
      b[q] = s;
      mx = fmax(mx, fabs(s));
    }
  }
  // largest magnitude over the row, then the first index within 2^-20 of it
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, kWave));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = mx;
  __syncthreads();
  for (int w = 0; w < kLayerWaves; ++w) mx = fmax(mx, s_red[w]);
  const double thr = mx * (1.0 - 0.00000095367431640625);  // 2^-20
  int first = DL;
#pragma unroll
  for (int q = 0; q < MAXF; ++q) {
    const int f = threadIdx.x + q * kLayerThreads;
    if (f < DL && fabs(b[q]) >= thr) first = min(first, f);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) first = min(first, __shfl_xor(first, o, kWave));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = (double)first;
  __syncthreads();
  for (int w = 0; w < kLayerWaves; ++w) first = min(first, (int)s_red[w]);
  // the sign of entry `first`, read from the thread that holds it
  __shared__ double s_sign;
#pragma unroll
  for (int q = 0; q < MAXF; ++q)
    if (threadIdx.x + q * kLayerThreads == first) s_sign = b[q] < 0.0 ? -1.0 : 1.0;
  __syncthreads();
  const double sg = s_sign;
  const int64_t lunit = (int64_t)lu.layer * 2 + lu.kv;
  float* brow = st.basis + (lunit * r + j) * DL;
#pragma unroll
  for (int q = 0; q < MAXF; ++q) {
    const int f = threadIdx.x + q * kLayerThreads;
    if (f < DL) brow[f] = (float)(sg * b[q]);
  }
  if (threadIdx.x == 0 && st.sigma) st.sigma[lunit * r + j] = a.vsigma[(size_t)u * a.rank + j];
}

// ---------------------------------------------------------------------------------------------------------------
// Projection coef = Z B^T over the heads
// ---------------------------------------------------------------------------------------------------------------

constexpr int kPLTiles = 2;                               // 16-token tiles per wave
constexpr int kPLWaves = 8;                               // waves per workgroup
constexpr int kPLThreads = kPLWaves * kWave;
constexpr int kPLChunk = kPLWaves * kPLTiles * 16;        // tokens per workgroup

// bf16: per head h the d columns of B (rank rows padded to RP = 16 MTR) are staged hi/lo in LDS (two buffers), the
// rows of h are read in MFMA B-operand layout and Z split hi/lo; the coefficient tiles accumulate over the heads.
// ROPE: key rows of a rotary cache enter Z in canonical coordinates (R(-pd) C_dst - R(-ps) C_src); the pairs of both
// styles lie inside a lane in this layout, and the angles come from two wave tables.
template <int D, int MTR, bool ROPE>
__global__ __launch_bounds__(kPLThreads) void proj_layer_bf16(LayerFitArgs a) {
  constexpr int KS = D / 32, RP = MTR * 16;
  extern __shared__ __attribute__((aligned(16))) unsigned char layer_lds[];
  uint16_t* s_b = reinterpret_cast<uint16_t*>(layer_lds);  // [2][hi, lo][RP][D]
  const int H = a.pv.num_kv_heads, DL = H * D;
  const int u = blockIdx.y;
  const LayerUnit lu = layer_unit(a, u);
  const kvc_item* itp = a.items + lu.item;
  const kvc_state& st = itp->state;
  const int r = st.rank, Ts = st.num_tokens;
  const int t_begin = blockIdx.x * kPLChunk;
  if (r == 0 || t_begin >= Ts) return;  // whole workgroup
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const uint16_t* pool = static_cast<const uint16_t*>(lu.kv ? a.layers.v[lu.lrel] : a.layers.k[lu.lrel]);
  const bool delta = a.mode == KVC_FIT_DELTA;
  const int64_t lunit = (int64_t)lu.layer * 2 + lu.kv;
  const float* basis = st.basis + lunit * r * DL;
  uint16_t* coef = static_cast<uint16_t*>(st.coef) + lunit * (int64_t)Ts * r;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, n = lane & 15;
  const bool rot = ROPE && lu.kv == 0;  // uniform over the workgroup
  const int style = a.pv.rope.style;
  float tcd = 1.0f, tsd = 0.0f, tcs = 1.0f, tss = 0.0f;  // wave tables for -pd (dst) and -ps (src)
  if (rot) {
    rope_wave_table<D>(a.pv.rope, -(double)itp->dst_position, lane, tcd, tsd);
    rope_wave_table<D>(a.pv.rope, -(double)itp->src_position, lane, tcs, tss);
  }

  f32x4 acc[kPLTiles][MTR];
#pragma unroll
  for (int j = 0; j < kPLTiles; ++j)
#pragma unroll
    for (int mt = 0; mt < MTR; ++mt) acc[j][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int h = 0; h < H; ++h) {
    uint16_t* s_hi = s_b + (h & 1) * 2 * RP * D;
    uint16_t* s_lo = s_hi + RP * D;
    for (int e = tid; e < RP * D; e += kPLThreads) {
      const int kk = e / D, f = e - kk * D;
      const float x = kk < r ? basis[(int64_t)kk * DL + h * D + f] : 0.f;
      uint32_t hb, lb;
      split_bf16(x, hb, lb);
      s_hi[e] = (uint16_t)hb;
      s_lo[e] = (uint16_t)lb;
    }
    __syncthreads();  // head h's columns are staged; the other buffer (head h - 1) is still read until here
#pragma unroll
    for (int j = 0; j < kPLTiles; ++j) {
      const int t0 = t_begin + (j * kPLWaves + wave) * 16;
      if (t0 >= Ts) continue;  // uniform over the wave
      const int t = t0 + n;
      const bool valid = t < Ts;
      const int64_t od = valid ? row_offset(a.pv, dst_tab, itp->dst_offset, t, h) : -1;
      const int64_t os = (valid && delta) ? row_offset(a.pv, src_tab, itp->src_offset, t, h) : -1;
      bf16x8 zh[KS], zl[KS];
      if (ROPE && rot) {  // uniform: the rotation reads the wave tables with shuffles
        f32x4 dv[2 * KS], sv[2 * KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const u32x4 d = od >= 0 ? *reinterpret_cast<const u32x4*>(pool + od + 32 * ks + 8 * g) : u32x4{0, 0, 0, 0};
          const u32x4 s = os >= 0 ? *reinterpret_cast<const u32x4*>(pool + os + 32 * ks + 8 * g) : u32x4{0, 0, 0, 0};
          dv[2 * ks] = f32x4{bf16_lo_to_f32(d[0]), bf16_hi_to_f32(d[0]), bf16_lo_to_f32(d[1]), bf16_hi_to_f32(d[1])};
          dv[2 * ks + 1] = f32x4{bf16_lo_to_f32(d[2]), bf16_hi_to_f32(d[2]), bf16_lo_to_f32(d[3]), bf16_hi_to_f32(d[3])};
          sv[2 * ks] = f32x4{bf16_lo_to_f32(s[0]), bf16_hi_to_f32(s[0]), bf16_lo_to_f32(s[1]), bf16_hi_to_f32(s[1])};
          sv[2 * ks + 1] = f32x4{bf16_lo_to_f32(s[2]), bf16_hi_to_f32(s[2]), bf16_lo_to_f32(s[3]), bf16_hi_to_f32(s[3])};
        }
        rope_rotate_rows_wave<D>(dv, style, g, tcd, tsd);
        rope_rotate_rows_wave<D>(sv, style, g, tcs, tss);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          u32x4 hw, lw;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const f32x4& dd = dv[2 * ks + (w >> 1)];
            const f32x4& ss = sv[2 * ks + (w >> 1)];
            uint32_t hh, ll;
            split_bf16x2(dd[2 * (w & 1)] - ss[2 * (w & 1)], dd[2 * (w & 1) + 1] - ss[2 * (w & 1) + 1], hh, ll);
            hw[w] = hh;
            lw[w] = ll;
          }
          zh[ks] = as_bf16x8(hw);
          zl[ks] = as_bf16x8(lw);
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const u32x4 d = od >= 0 ? *reinterpret_cast<const u32x4*>(pool + od + 32 * ks + 8 * g) : u32x4{0, 0, 0, 0};
          const u32x4 s = os >= 0 ? *reinterpret_cast<const u32x4*>(pool + os + 32 * ks + 8 * g) : u32x4{0, 0, 0, 0};
          u32x4 hw, lw;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            uint32_t hh, ll;
            split_bf16x2(bf16_lo_to_f32(d[w]) - bf16_lo_to_f32(s[w]), bf16_hi_to_f32(d[w]) - bf16_hi_to_f32(s[w]),
                         hh, ll);
            hw[w] = hh;
            lw[w] = ll;
          }
          zh[ks] = as_bf16x8(hw);
          zl[ks] = as_bf16x8(lw);
        }
      }
#pragma unroll
      for (int mt = 0; mt < MTR; ++mt) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int o = (16 * mt + n) * D + 32 * ks + 8 * g;
          const bf16x8 fh = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[o]));
          const bf16x8 fl = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[o]));
          acc[j][mt] = mfma16x16x32(fl, zh[ks], acc[j][mt]);
          acc[j][mt] = mfma16x16x32(fh, zl[ks], acc[j][mt]);
          acc[j][mt] = mfma16x16x32(fh, zh[ks], acc[j][mt]);
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kPLTiles; ++j) {
    const int t = t_begin + (j * kPLWaves + wave) * 16 + n;
    if (t >= Ts) continue;
#pragma unroll
    for (int mt = 0; mt < MTR; ++mt) {
      // lane holds coef[t][16 mt + 4 g + i], i = 0..3
      const int k0 = 16 * mt + 4 * g;
      uint16_t* cp = coef + (int64_t)t * r + k0;
      if ((r & 3) == 0 && k0 + 4 <= r) {
        uint2 w;
        w.x = pack_bf16x2(acc[j][mt][0], acc[j][mt][1]);
        w.y = pack_bf16x2(acc[j][mt][2], acc[j][mt][3]);
        *reinterpret_cast<uint2*>(cp) = w;
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (k0 + i < r) cp[i] = (uint16_t)f32_to_bf16_bits(acc[j][mt][i]);
      }
    }
  }
}

// float32: one thread per (token, rank), fp32 FMAs over the D = H d features; the basis [r][D] is in LDS.
template <int D>
__global__ __launch_bounds__(kLayerThreads) void proj_layer_f32(LayerFitArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char layer_lds[];
  float* s_b = reinterpret_cast<float*>(layer_lds);
  const int H = a.pv.num_kv_heads, DL = H * D;
  const int u = blockIdx.y;
  const LayerUnit lu = layer_unit(a, u);
  const kvc_item* itp = a.items + lu.item;
  const kvc_state& st = itp->state;
  const int r = st.rank, Ts = st.num_tokens;
  const int t_begin = blockIdx.x * kPLChunk;
  if (r == 0 || t_begin >= Ts) return;
  const int t_end = min(Ts, t_begin + kPLChunk);
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)lu.item * a.max_blocks : nullptr;
  const float* pool = static_cast<const float*>(lu.kv ? a.layers.v[lu.lrel] : a.layers.k[lu.lrel]);
  const bool delta = a.mode == KVC_FIT_DELTA;
  const int64_t lunit = (int64_t)lu.layer * 2 + lu.kv;
  const float* basis = st.basis + lunit * r * DL;
  float* coef = static_cast<float*>(st.coef) + lunit * (int64_t)Ts * r;
  float* s_rope = s_b + r * DL;  // keys of a rotary cache: the tables of -pd and -ps
  const bool rot = a.pv.rope.style != KVC_ROPE_NONE && lu.kv == 0;
  const int style = a.pv.rope.style;
  if (rot) layer_rope_tables<D>(a, itp, s_rope);
  for (int e = threadIdx.x; e < r * DL; e += kLayerThreads) s_b[e] = basis[e];
  __syncthreads();
  const int64_t total = (int64_t)(t_end - t_begin) * r;
  for (int64_t e = threadIdx.x; e < total; e += kLayerThreads) {
    const int t = t_begin + (int)(e / r), kk = (int)(e % r);
    float s = 0.f;
    for (int h = 0; h < H; ++h) {
      const int64_t od = row_offset(a.pv, dst_tab, itp->dst_offset, t, h);
      const int64_t os = delta ? row_offset(a.pv, src_tab, itp->src_offset, t, h) : -1;
      for (int f = 0; f < D; ++f) {
        float z = od >= 0 ? (rot ? layer_rope_value<D>(pool + od, f, style, s_rope, s_rope + D / 2) : pool[od + f]) : 0.f;
        if (os >= 0) z -= rot ? layer_rope_value<D>(pool + os, f, style, s_rope + D, s_rope + 3 * D / 2) : pool[os + f];
        s = fmaf(z, s_b[kk * DL + h * D + f], s);
      }
    }
    coef[(int64_t)t * r + kk] = s;
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------------------------------------------

template <int D, bool DELTA, bool FULL, bool ROPE>
static hipError_t launch_gl_one(const LayerFitArgs& a, dim3 grid, dim3 block, int pairs, int ng, hipStream_t stream) {
  hipError_t e = hipFuncSetAttribute((const void*)gram_layer_bf16<D, DELTA, FULL, ROPE>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)kGLLdsBytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gram_layer_bf16<D, DELTA, FULL, ROPE>), grid, block, kGLLdsBytes, stream, a, pairs, ng);
  return hipGetLastError();
}
template <int D, bool ROPE>
static hipError_t launch_gl(const LayerFitArgs& a, bool delta, bool full, dim3 grid, dim3 block, int pairs, int ng,
                            hipStream_t stream) {
  if (delta) return full ? launch_gl_one<D, true, true, ROPE>(a, grid, block, pairs, ng, stream)
                         : launch_gl_one<D, true, false, ROPE>(a, grid, block, pairs, ng, stream);
  return full ? launch_gl_one<D, false, true, ROPE>(a, grid, block, pairs, ng, stream)
              : launch_gl_one<D, false, false, ROPE>(a, grid, block, pairs, ng, stream);
}

hipError_t launch_layer_gram(const LayerFitArgs& a, kvc_dtype dtype, hipStream_t stream) {
  const int D = a.pv.head_dim, H = a.pv.num_kv_heads, DL = H * D;
  int upper_only = 0;
  // the LDS Gram addresses a lane's features within a row by a 32-bit byte offset
  const bool small_rows = 2 * ((int64_t)(H - 1) * a.pv.head_stride + D) < ((int64_t)1 << 31);
  if (dtype == KVC_BF16 && a.pv.block_shift >= 3 && small_rows) {
    const int NB = (DL + 127) / 128, NG = (NB + 1) / 2, pairs = NG * (NG + 1) / 2;
    const unsigned nwork = (unsigned)a.num_units * a.max_parts * pairs;
    const bool delta = a.mode == KVC_FIT_DELTA;
    // straight-line variant: every producing lane inside D and a row's lane offsets inside the zero page
    const bool full = DL % 256 == 0 && 2 * ((int64_t)(H - 1) * a.pv.head_stride + D) <= kGLZeroBytes;
    const bool rope = a.pv.rope.style != KVC_ROPE_NONE;
    const dim3 grid(nwork), block(kGLThreads);
    hipError_t e;
    if (D == 64) e = rope ? launch_gl<64, true>(a, delta, full, grid, block, pairs, NG, stream)
                          : launch_gl<64, false>(a, delta, full, grid, block, pairs, NG, stream);
    else e = rope ? launch_gl<128, true>(a, delta, full, grid, block, pairs, NG, stream)
                  : launch_gl<128, false>(a, delta, full, grid, block, pairs, NG, stream);
    if (e != hipSuccess) return e;
    upper_only = 1;
  } else if (dtype == KVC_BF16) {
    dim3 grid((a.max_parts + kLayerWaves / 2 - 1) / (kLayerWaves / 2), H * (H + 1) / 2, a.num_units);
    if (D == 64) hipLaunchKernelGGL(gram_pair_bf16<64>, grid, dim3(kLayerThreads), 0, stream, a);
    else hipLaunchKernelGGL(gram_pair_bf16<128>, grid, dim3(kLayerThreads), 0, stream, a);
  } else {
    const int nb = DL / kF32Block;
    dim3 grid(nb * nb, a.max_parts, a.num_units);
    if (D == 64) hipLaunchKernelGGL(gram_block_f32<64>, grid, dim3(kLayerThreads), 0, stream, a);
    else hipLaunchKernelGGL(gram_block_f32<128>, grid, dim3(kLayerThreads), 0, stream, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nt = DL / 32;
  hipLaunchKernelGGL(gram_reduce, dim3(nt * nt, a.num_units), dim3(kLayerThreads), 0, stream, a, upper_only);
  return hipGetLastError();
}

hipError_t launch_layer_subspace(const LayerFitArgs& a, const EigArgs& ea, hipStream_t stream) {
  const int DL = a.pv.num_kv_heads * a.pv.head_dim;
  hipLaunchKernelGGL(sub_init, dim3((a.k * DL + kLayerThreads - 1) / kLayerThreads, a.num_units),
                     dim3(kLayerThreads), 0, stream, a);
  const int nch = (DL + kCqrChunk - 1) / kCqrChunk;
  const size_t flds = cqr_factor_lds(a.k), alds = cqr_apply_lds(a.k);
  {
    const void* ap = a.k == 64 ? (const void*)cqr_apply<64> : (const void*)cqr_apply<128>;
    hipError_t e0 = hipFuncSetAttribute(ap, hipFuncAttributeMaxDynamicSharedMemorySize, (int)alds);
    if (e0 == hipSuccess && a.k == 128)
      e0 = hipFuncSetAttribute((const void*)cqr_factor<128>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)flds);
    if (e0 != hipSuccess) return e0;
  }
  const dim3 sgrid(nch, a.num_units), agrid(DL / kCqrRows, a.num_units);
  auto pass = [&](const double* src, double* dst, int first, uint32_t round) {
    if (a.k == 64) {
      hipLaunchKernelGGL(cqr_syrk<64>, sgrid, dim3(kCqrThreads), 0, stream, a, src, first, round);
      hipLaunchKernelGGL(cqr_factor_reg64, dim3(a.num_units), dim3(kCqrFactorThreads), 0, stream, a, first, round);
      hipLaunchKernelGGL(cqr_apply<64>, agrid, dim3(kCqrThreads), alds, stream, a, src, dst, first, round);
    } else {
      hipLaunchKernelGGL(cqr_syrk<128>, sgrid, dim3(kCqrThreads), 0, stream, a, src, first, round);
      hipLaunchKernelGGL(cqr_factor<128>, dim3(a.num_units), dim3(kCqrFactor128Threads), flds, stream, a, first,
                         round);
      hipLaunchKernelGGL(cqr_apply<128>, agrid, dim3(kCqrThreads), alds, stream, a, src, dst, first, round);
    }
  };
  // X = orth(Y): the perturbed, shifted pass from Y into X, then (`exact`) the exact pass on X in place.  Between two
  // Rayleigh-Ritz steps X only has to keep full rank (the iteration depends on span(X) alone), so the exact pass runs
  // before each Rayleigh-Ritz step only.
  auto orth = [&](uint32_t round, bool exact) {
    // the perturbation size: measured on Y in the first two rounds, then set by the previous round's factorisation
    if (round <= 1u) hipLaunchKernelGGL(cqr_scale, dim3(a.num_units), dim3(kScaleThreads), 0, stream, a, round);
    pass(a.y, a.x, 1, round);
    if (exact) pass(a.x, a.x, 0, round);
  };
  orth(0u, false);  // the random start is well conditioned, and X only has to keep full rank until the first check
  const dim3 ggrid((DL + kGemmRows - 1) / kGemmRows, a.k / kGemmCols, a.num_units);
  EigArgs es = ea;
  es.skip = a.conv;  // units that have stopped keep the Ritz pairs of their last check
  int done = 0;
  while (done < kLayerMaxIters) {
    const int n = done == 0 ? kLayerFirstIters : kLayerCheckEvery;
    for (int it = 0; it < n; ++it) {
      // after a Rayleigh-Ritz step Y already holds G X for this X (the Ritz step, the residual check and the
      // decision read X and Y and write neither), so the first product of every later round is that one
      if (done == 0 || it > 0) hipLaunchKernelGGL(sub_gemm, ggrid, dim3(kGemmThreads), 0, stream, a);
      orth((uint32_t)(++done), it + 1 == n);
    }
    // Rayleigh-Ritz on span(X) and the residuals of its top-r pairs (Y = G X is kept by the Ritz step)
    hipLaunchKernelGGL(sub_gemm, ggrid, dim3(kGemmThreads), 0, stream, a);
    if (a.k == 64) {
      hipLaunchKernelGGL(sub_rayleigh<64>, sgrid, dim3(kCqrThreads), 0, stream, a);
      hipLaunchKernelGGL(sub_rayleigh_sum<64>, dim3(a.num_units), dim3(kCqrThreads), 0, stream, a);
    } else {
      hipLaunchKernelGGL(sub_rayleigh<128>, sgrid, dim3(kCqrThreads), 0, stream, a);
      hipLaunchKernelGGL(sub_rayleigh_sum<128>, dim3(a.num_units), dim3(kCqrThreads), 0, stream, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = launch_eig(es, stream)) != hipSuccess) return e;
    hipLaunchKernelGGL(sub_check, dim3((DL + kLayerThreads - 1) / kLayerThreads, a.num_units), dim3(kLayerThreads), 0,
                       stream, a);
    hipLaunchKernelGGL(sub_check_sum, dim3(a.num_units), dim3(KVC_MAX_RANK), 0, stream, a);
    hipLaunchKernelGGL(sub_decide, dim3(a.num_units), dim3(kWave), 0, stream, a, done, done >= kLayerMaxIters);
  }
  hipLaunchKernelGGL(sub_basis, dim3(a.rank, a.num_units), dim3(kLayerThreads), 0, stream, a);
  return hipGetLastError();
}

// float32: the basis [rank][H d], then the rotary angle tables (cos / sin at -pd and -ps, D / 2 each)
size_t layer_proj_lds_bytes(int D, int H, int rank, kvc_dtype dtype) {
  if (dtype == KVC_BF16) return (size_t)2 * 2 * ((rank + 15) / 16 * 16) * D * sizeof(uint16_t);
  return (size_t)rank * H * D * sizeof(float) + kLayerRopeTableBytes;
}

template <int D, int MTR, bool ROPE>
static hipError_t launch_pl_one(const LayerFitArgs& a, dim3 grid, size_t lds, hipStream_t stream) {
  hipError_t e = hipFuncSetAttribute((const void*)proj_layer_bf16<D, MTR, ROPE>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((proj_layer_bf16<D, MTR, ROPE>), grid, dim3(kPLThreads), lds, stream, a);
  return hipGetLastError();
}

template <int D, bool ROPE>
static hipError_t launch_proj_layer_bf16(const LayerFitArgs& a, dim3 grid, size_t lds, hipStream_t stream) {
  const int mtr = (a.rank + 15) / 16;
  switch (mtr <= 1 ? 1 : mtr <= 2 ? 2 : mtr <= 4 ? 4 : 8) {
    case 1: return launch_pl_one<D, 1, ROPE>(a, grid, lds, stream);
    case 2: return launch_pl_one<D, 2, ROPE>(a, grid, lds, stream);
    case 4: return launch_pl_one<D, 4, ROPE>(a, grid, lds, stream);
    default: return launch_pl_one<D, 8, ROPE>(a, grid, lds, stream);
  }
}

hipError_t launch_layer_proj(const LayerFitArgs& a, kvc_dtype dtype, int max_tokens, hipStream_t stream) {
  const int D = a.pv.head_dim, H = a.pv.num_kv_heads;
  dim3 grid((max_tokens + kPLChunk - 1) / kPLChunk, a.num_units);
  // the bf16 kernel stages RP = 16 MTR rank rows (MTR in 1, 2, 4, 8) of one head, hi and lo, in two buffers
  const int mtr = (a.rank + 15) / 16, mtr_inst = mtr <= 1 ? 1 : mtr <= 2 ? 2 : mtr <= 4 ? 4 : 8;
  const size_t lds = (size_t)2 * 2 * 16 * mtr_inst * D * sizeof(uint16_t);
  if (dtype == KVC_BF16) {
    if (a.pv.rope.style != KVC_ROPE_NONE)
      return D == 64 ? launch_proj_layer_bf16<64, true>(a, grid, lds, stream)
                     : launch_proj_layer_bf16<128, true>(a, grid, lds, stream);
    return D == 64 ? launch_proj_layer_bf16<64, false>(a, grid, lds, stream)
                   : launch_proj_layer_bf16<128, false>(a, grid, lds, stream);
  }
  const size_t flds = layer_proj_lds_bytes(D, H, a.rank, dtype);
  const void* fn = D == 64 ? (const void*)proj_layer_f32<64> : (const void*)proj_layer_f32<128>;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)flds);
  if (e != hipSuccess) return e;
  if (D == 64) hipLaunchKernelGGL(proj_layer_f32<64>, grid, dim3(kLayerThreads), flds, stream, a);
  else hipLaunchKernelGGL(proj_layer_f32<128>, grid, dim3(kLayerThreads), flds, stream, a);
  return hipGetLastError();
}

}  // namespace kvc
