// kvc_apply kernels: C_dst[t] = C_src[t] + A[t] B for t < T_s, bit copy for T_s <= t < T (Eq. 4 with the source
// agent's cache as reference, Eq. 8 with one state, prefix coverage of Appendix A.3).
//
// bf16 caches: one workgroup of W wave64s over one (item, layer, K/V, head) unit and a chunk of 256 tokens (16 W tpw:
// 8 waves of 2 tiles for ranks up to 32, 4 waves of 4 tiles above, the fastest of the shapes measured on MI355X; a
// longer chunk per workgroup leaves fewer workgroups and a longer tail, a shorter one stages the basis more often;
// rotary keys take 1024-token chunks, see the launcher).  The
// correction of a 16-token tile is the MFMA contraction  D^T = B^T A^T + C^T  with M = feature (16 per tile), N =
// token, K = rank (32 per v_mfma_f32_16x16x32_bf16), and the accumulator C initialised with the source rows in fp32.
// B is staged once per workgroup in LDS as a bf16 hi/lo pair (about 16 significant bits of the fp32 basis) and read
// as MFMA A-fragments; the bf16 coefficients are the MFMA B-operand, loaded straight from the coefficient rows (one
// 16-byte load per lane and 32 ranks).  The M index of each tile is permuted so that the four lanes holding one token
// own 64 contiguous bytes of the row per 16-byte load: every global load and store of a cache row is 128-bit.
//
// Latency: the chunk's block-table entries are staged in LDS with the basis, so a row address needs no global load
// (a dependent global load would make the wave wait for every older memory operation, its earlier stores included,
// since one counter covers loads and stores); the tiles of a wave are software-pipelined in pairs, the loads of the
// next tile in flight while this tile is corrected and stored.
//
// float32 caches: a VALU kernel with the basis in LDS (float32 throughout, for the 1e-5 storage tolerance).
#include "kvc_device.h"
#include "kvc_launch.h"

namespace kvc {

constexpr int kApplyWaves = 4;
constexpr int kApplyThreads = kApplyWaves * kWave;
constexpr int kApplyTilesPerWave = 8;                                   // float32 kernel
constexpr int kApplyChunk = kApplyWaves * kApplyTilesPerWave * 16;      // tokens per workgroup (float32 kernel)
constexpr int kApplyChunkTokens = 256;                                  // bf16 kernel: tokens per workgroup
constexpr int kApplyRopeChunkTokens = 1024;                             // the same with rotary keys

int apply_chunk_tokens() { return kApplyChunk; }

// LDS of the bf16 kernel: basis hi/lo [D][KP] each, then the block-table slices of the workgroup's token chunk for
// the source and the destination sequence (nblk entries each: a chunk of c tokens spans at most c / bs + 1 blocks).
__host__ __device__ constexpr size_t apply_lds_bytes(int D, int KP, int nblk) {
  return (size_t)2 * D * KP * sizeof(uint16_t) + (size_t)2 * nblk * sizeof(int32_t);
}

// ROPE: the keys are rotary-encoded, corrected in canonical coordinates and rotated to the target positions,
// C_dst = R(pd - ps) C_src + (A B R(pd)^T): the accumulator starts from the source rotated by pd - ps and B is staged
// rotated by pd, so the rotation costs no extra pass (rows past T_s get the rotated source).
template <int D, int KS, int W, bool ROPE>
__global__ __launch_bounds__(W * kWave) void apply_bf16_mfma(ApplyArgs a, int tpw, int nblk) {
  constexpr int MT = D / 16;  // M-tiles per row
  constexpr int NQ = D / 32;  // 16-byte loads per lane per row
  constexpr int KP = KS * 32; // padded rank
  extern __shared__ __attribute__((aligned(16))) uint16_t s_dyn[];
  uint16_t* s_hi = s_dyn;
  uint16_t* s_lo = s_dyn + D * KP;
  int32_t* s_tab = reinterpret_cast<int32_t*>(s_dyn + 2 * D * KP);  // [2][nblk]: source, destination

  const int nl = a.num_layers;
  const int il = grid_item_layer(a.chunk_order);
  const int item_id = il / nl;
  const int lrel = il - item_id * nl;
  const int layer = a.layer_begin + lrel;
  const int H = a.pv.num_kv_heads;
  const int kv = a.kv_begin + (int)blockIdx.y / H;
  const int head = (int)blockIdx.y % H;

  const kvc_item* itp = a.items + item_id;
  const int T = itp->num_tokens;
  const int chunk = W * 16 * tpw;
  const int t_begin = grid_chunk(a.chunk_order) * chunk;
  if (t_begin >= T) return;  // whole workgroup
  const int t_end = min(T, t_begin + chunk);
  const int r = itp->state.rank;
  const int Tdecl = itp->state.num_tokens;
  const int Ts = r > 0 ? min(Tdecl, T) : 0;
  const int src_off = itp->src_offset, dst_off = itp->dst_offset;
  // a per-layer state shares the coefficient rows of a (layer, K/V) across heads; head h reads its d columns of the
  // basis rows of H d features
  const bool per_layer = itp->state.grouping == KVC_GROUP_LAYER;
  const int64_t unit = per_layer ? (int64_t)layer * 2 + kv : unit_index(layer, kv, head, H);
  const int bstride = per_layer ? H * D : D;
  const uint16_t* coef = static_cast<const uint16_t*>(itp->state.coef) + unit * (int64_t)Tdecl * r;
  const float* basis = itp->state.basis + unit * (int64_t)r * bstride + (per_layer ? head * D : 0);
  const uint16_t* src_pool = static_cast<const uint16_t*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]);
  uint16_t* dst_pool = static_cast<uint16_t*>(const_cast<void*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]));

  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int g = lane >> 4;
  const int n = lane & 15;
  const bool correct = t_begin < Ts;  // uniform over the workgroup

  // block ids of the chunk's logical blocks (the host checked that they lie inside the item's table row)
  const int bs = a.pv.block_size, bsh = a.pv.block_shift;
  auto lblock = [&](int p) { return bsh >= 0 ? p >> bsh : p / bs; };
  const int lb0s = lblock(src_off + t_begin), lb0d = lblock(dst_off + t_begin);
  {
    const int ns = lblock(src_off + t_end - 1) - lb0s + 1, nd = lblock(dst_off + t_end - 1) - lb0d + 1;
    const int32_t* st = a.src_tables ? a.src_tables + (int64_t)item_id * a.max_blocks : nullptr;
    const int32_t* dt = a.dst_tables ? a.dst_tables + (int64_t)item_id * a.max_blocks : nullptr;
    for (int i = threadIdx.x; i < ns; i += W * kWave) s_tab[i] = st ? st[lb0s + i] : lb0s + i;
    for (int i = threadIdx.x; i < nd; i += W * kWave) s_tab[nblk + i] = dt ? dt[lb0d + i] : lb0d + i;
  }

  // keys of a rotary cache: angle tables of the shift pd - ps (source rows) and of pd (the basis)
  __shared__ float s_rope[4][ROPE ? D / 2 : 1];
  const bool rope = ROPE && kv == 0;  // uniform over the workgroup
  const int style = a.pv.rope.style;
  bool shift = false;
  if (rope) {
    const int ps = itp->src_position, pd = itp->dst_position;
    shift = pd != ps;
    rope_table(a.pv.rope, D, (double)pd - (double)ps, s_rope[0], s_rope[1]);
    rope_table(a.pv.rope, D, (double)pd, s_rope[2], s_rope[3]);
    __syncthreads();
  }
  if (correct) {
    // Stage B^T as bf16 hi/lo, zero-padded to KP ranks: s[f * KP + k] = split(B[k][f]); one thread per (feature,
    // 8 consecutive ranks), one 16-byte LDS store per half.
    for (int e = threadIdx.x; e < D * (KP / 8); e += W * kWave) {
      const int f = e % D, k0 = 8 * (e / D);
      float x[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int k = k0 + i;
        x[i] = k < r ? basis[k * bstride + f] : 0.0f;
        if (rope && k < r) {  // B R(pd)^T: each basis row rotated like a key row at position pd
          const int pi = rope_pair(style, D, f);
          x[i] = rope_rotated(rope_first(style, D, f), x[i], basis[k * bstride + rope_partner(style, D, f)],
                              s_rope[2][pi], s_rope[3][pi]);
        }
      }
      u32x4 h, l;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t hh, ll;
        split_bf16x2(x[2 * i], x[2 * i + 1], hh, ll);
        h[i] = hh;
        l[i] = ll;
      }
      *reinterpret_cast<u32x4*>(&s_hi[f * KP + k0]) = h;
      *reinterpret_cast<u32x4*>(&s_lo[f * KP + k0]) = l;
    }
  }
  __syncthreads();
  const bool coef_vec = (r & 7) == 0;

  // Row offset of token t through the staged table slice (-1 when the block id is out of range).
  auto row_off = [&](int off, int lb0, const int32_t* tab, int t) -> int64_t {
    const int p = off + t, lb = lblock(p), slot = p - lb * bs;
    const int32_t blk = tab[lb - lb0];
    if (blk < 0 || blk >= a.pv.num_blocks) return -1;
    return (int64_t)blk * a.pv.block_stride + (int64_t)slot * a.pv.token_stride + (int64_t)head * a.pv.head_stride;
  };

  struct Tile {
    u32x4 raw[NQ];
    u32x4 cw[KS];
    int64_t dof;
  };
  auto tile_t0 = [&](int j) { return t_begin + (j * W + wave) * 16; };
  // Issue the loads of tile j (rows through the staged tables, coefficient rows); lanes past the chunk load nothing.
  auto load_tile = [&](int j, Tile& tl) __attribute__((always_inline)) {
    const int t = tile_t0(j) + n;
    const bool valid = t < t_end;
    const int64_t so = valid ? row_off(src_off, lb0s, s_tab, t) : -1;
    // a row whose source block id is out of range is neither read nor written
    tl.dof = so >= 0 ? row_off(dst_off, lb0d, s_tab + nblk, t) : -1;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      tl.raw[q] = u32x4{0, 0, 0, 0};
      if (so >= 0) tl.raw[q] = *reinterpret_cast<const u32x4*>(src_pool + so + 32 * q + 8 * g);
    }
    const bool crow = t < Ts;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int k0 = ks * 32 + 8 * g;
      u32x4 w = {0, 0, 0, 0};
      if (crow) {
        const uint16_t* cp = coef + (int64_t)t * r + k0;
        if (coef_vec && k0 + 8 <= r) {
          w = *reinterpret_cast<const u32x4*>(cp);
        } else {
          uint32_t e[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) e[i] = (k0 + i < r) ? cp[i] : 0u;
          w = u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16)};
        }
      }
      tl.cw[ks] = w;
    }
  };
  // Correct (rows t < Ts) or copy, then store through the destination table.
  auto finish_tile = [&](int j, const Tile& tl) __attribute__((always_inline)) {
    const int t0 = tile_t0(j);
    const int t = t0 + n;
    u32x4 outw[NQ];
    if (t0 < Ts) {
      f32x4 acc[MT];
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        acc[2 * q] = f32x4{bf16_lo_to_f32(tl.raw[q][0]), bf16_hi_to_f32(tl.raw[q][0]),
                           bf16_lo_to_f32(tl.raw[q][1]), bf16_hi_to_f32(tl.raw[q][1])};
        acc[2 * q + 1] = f32x4{bf16_lo_to_f32(tl.raw[q][2]), bf16_hi_to_f32(tl.raw[q][2]),
                               bf16_lo_to_f32(tl.raw[q][3]), bf16_hi_to_f32(tl.raw[q][3])};
      }
      if (ROPE && shift) rope_rotate_rows<D>(acc, style, g, s_rope[0], s_rope[1]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 cb = as_bf16x8(tl.cw[ks]);
          const int fo = mfma_row_feature(mt, n) * KP + ks * 32 + 8 * g;
          const bf16x8 fl = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[fo]));
          const bf16x8 fh = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[fo]));
          acc[mt] = mfma16x16x32(fl, cb, acc[mt]);
          acc[mt] = mfma16x16x32(fh, cb, acc[mt]);
        }
      }
      // rows past T_s had zero coefficients: with a shift they hold the rotated source, else they are bit copies
      const bool crow = t < Ts || (ROPE && shift);
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const f32x4 x = acc[2 * q], y = acc[2 * q + 1];
        const u32x4 c = {pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(y[0], y[1]),
                         pack_bf16x2(y[2], y[3])};
        outw[q] = crow ? c : tl.raw[q];
      }
    } else if (ROPE && shift) {  // uncovered tile: the re-aligned source
      f32x4 v[MT];
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        v[2 * q] = f32x4{bf16_lo_to_f32(tl.raw[q][0]), bf16_hi_to_f32(tl.raw[q][0]), bf16_lo_to_f32(tl.raw[q][1]),
                         bf16_hi_to_f32(tl.raw[q][1])};
        v[2 * q + 1] = f32x4{bf16_lo_to_f32(tl.raw[q][2]), bf16_hi_to_f32(tl.raw[q][2]),
                             bf16_lo_to_f32(tl.raw[q][3]), bf16_hi_to_f32(tl.raw[q][3])};
      }
      rope_rotate_rows<D>(v, style, g, s_rope[0], s_rope[1]);
#pragma unroll
      for (int q = 0; q < NQ; ++q)
        outw[q] = u32x4{pack_bf16x2(v[2 * q][0], v[2 * q][1]), pack_bf16x2(v[2 * q][2], v[2 * q][3]),
                        pack_bf16x2(v[2 * q + 1][0], v[2 * q + 1][1]), pack_bf16x2(v[2 * q + 1][2], v[2 * q + 1][3])};
    } else {
#pragma unroll
      for (int q = 0; q < NQ; ++q) outw[q] = tl.raw[q];
    }
    if (tl.dof >= 0) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) *reinterpret_cast<u32x4*>(dst_pool + tl.dof + 32 * q + 8 * g) = outw[q];
    }
  };

  // tiles of this wave in pairs: the loads of the next tile are in flight while this one is finished
  Tile ta, tb;
  if (tile_t0(0) >= t_end) return;  // whole wave
  load_tile(0, ta);
  for (int j = 0;; j += 2) {
    const bool m1 = j + 1 < tpw && tile_t0(j + 1) < t_end;
    if (m1) load_tile(j + 1, tb);
    finish_tile(j, ta);
    if (!m1) break;
    const bool m2 = j + 2 < tpw && tile_t0(j + 2) < t_end;
    if (m2) load_tile(j + 2, ta);
    finish_tile(j + 1, tb);
    if (!m2) break;
  }
}

// float32 caches: each thread owns 4 features of one token; the rank loop runs over B in LDS.
template <int D>
__global__ __launch_bounds__(kApplyThreads) void apply_f32_valu(ApplyArgs a) {
  extern __shared__ __attribute__((aligned(16))) float s_b[];  // [r][D]
  constexpr int LPT = D / 4;                                   // lanes per token
  constexpr int TPP = kApplyThreads / LPT;                     // tokens per pass

  const int nl = a.num_layers;
  const int il = grid_item_layer(a.chunk_order);
  const int item_id = il / nl;
  const int lrel = il - item_id * nl;
  const int layer = a.layer_begin + lrel;
  const int H = a.pv.num_kv_heads;
  const int kv = a.kv_begin + (int)blockIdx.y / H;
  const int head = (int)blockIdx.y % H;

  const kvc_item* itp = a.items + item_id;
  const int T = itp->num_tokens;
  const int t_begin = grid_chunk(a.chunk_order) * kApplyChunk;
  if (t_begin >= T) return;
  const int r = itp->state.rank;
  const int Tdecl = itp->state.num_tokens;
  const int Ts = r > 0 ? min(Tdecl, T) : 0;
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)item_id * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)item_id * a.max_blocks : nullptr;
  const bool per_layer = itp->state.grouping == KVC_GROUP_LAYER;
  const int64_t unit = per_layer ? (int64_t)layer * 2 + kv : unit_index(layer, kv, head, H);
  const int bstride = per_layer ? H * D : D;
  const float* coef = static_cast<const float*>(itp->state.coef) + unit * (int64_t)Tdecl * r;
  const float* basis = itp->state.basis + unit * (int64_t)r * bstride + (per_layer ? head * D : 0);
  const float* src_pool = static_cast<const float*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]);
  float* dst_pool = static_cast<float*>(const_cast<void*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]));

  // keys of a rotary cache: C_dst = R(pd - ps) C_src + A (B R(pd)^T), with the angle tables in LDS
  __shared__ float s_rope[4][D / 2];
  const bool rope = a.pv.rope.style != KVC_ROPE_NONE && kv == 0;  // uniform over the workgroup
  const int style = a.pv.rope.style;
  bool shift = false;
  if (rope) {
    const int ps = itp->src_position, pd = itp->dst_position;
    shift = pd != ps;
    rope_table(a.pv.rope, D, (double)pd - (double)ps, s_rope[0], s_rope[1]);
    rope_table(a.pv.rope, D, (double)pd, s_rope[2], s_rope[3]);
    __syncthreads();
  }
  const bool correct = t_begin < Ts;
  if (correct) {
    for (int e = threadIdx.x; e < r * D; e += kApplyThreads) {
      const int k = e / D, f = e - k * D;
      float x = basis[k * bstride + f];
      if (rope) {
        const int i = rope_pair(style, D, f);
        x = rope_rotated(rope_first(style, D, f), x, basis[k * bstride + rope_partner(style, D, f)], s_rope[2][i],
                         s_rope[3][i]);
      }
      s_b[e] = x;
    }
    __syncthreads();
  }
  const int sub = threadIdx.x / LPT;
  const int f0 = 4 * (threadIdx.x % LPT);
  const int t_end = min(T, t_begin + kApplyChunk);
  for (int t = t_begin + sub; t < t_end; t += TPP) {
    const int64_t so = row_offset(a.pv, src_tab, itp->src_offset, t, head);
    const int64_t dof = row_offset(a.pv, dst_tab, itp->dst_offset, t, head);
    if (so < 0 || dof < 0) continue;
    const f32x4 s = *reinterpret_cast<const f32x4*>(src_pool + so + f0);
    f32x4 o = s;
    if (shift) {  // the source rotated by pd - ps (the four features' partners: another quad, or inside this one)
      const int pf = rope_partner(style, D, f0) & ~3;
      const f32x4 y = *reinterpret_cast<const f32x4*>(src_pool + so + pf);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int f = f0 + j, i = rope_pair(style, D, f);
        const float partner = style == KVC_ROPE_HALF ? y[j] : s[j ^ 1];
        o[j] = rope_rotated(rope_first(style, D, f), s[j], partner, s_rope[0][i], s_rope[1][i]);
      }
    }
    if (t < Ts) {
      const float* crow = coef + (int64_t)t * r;
      for (int k = 0; k < r; ++k) {
        const float c = crow[k];
        const f32x4 b = *reinterpret_cast<const f32x4*>(&s_b[k * D + f0]);
        o[0] = fmaf(c, b[0], o[0]);
        o[1] = fmaf(c, b[1], o[1]);
        o[2] = fmaf(c, b[2], o[2]);
        o[3] = fmaf(c, b[3], o[3]);
      }
    }
    *reinterpret_cast<f32x4*>(dst_pool + dof + f0) = o;
  }
}

template <int D, int KS, int W, bool ROPE>
static hipError_t launch_bf16_w(const ApplyArgs& a, dim3 grid, int tpw, int nblk, hipStream_t stream) {
  const size_t lds = apply_lds_bytes(D, KS * 32, nblk);
  hipError_t e = hipFuncSetAttribute((const void*)apply_bf16_mfma<D, KS, W, ROPE>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((apply_bf16_mfma<D, KS, W, ROPE>), grid, dim3(W * kWave), lds, stream, a, tpw, nblk);
  return hipGetLastError();
}

// Waves per workgroup for a rank of KS 32-rank chunks.
constexpr int apply_waves(int ks) { return ks == 1 ? 8 : 4; }

// Keys of a rotary cache: every workgroup forms fp64 angle tables and stages a rotated basis, which a 1024-token chunk
// (4 waves of 16 tiles) amortises; values (and every unit of a plain cache) take 256-token chunks.
template <int D, int KS>
static hipError_t launch_bf16(const ApplyArgs& a0, int max_tokens, int num_items, hipStream_t stream) {
  ApplyArgs a = a0;
  const int H = a.pv.num_kv_heads;
  int nkv = 2;
  if (a.pv.rope.style != KVC_ROPE_NONE) {
    const int chunk = kApplyRopeChunkTokens;
    a.kv_begin = 0;
    const int chunks = (max_tokens + chunk - 1) / chunk;
    a.chunk_order = multi_item_order(num_items, chunks, kChunksRotated);
    const dim3 grid = chunk_grid(chunks, H, num_items * a.num_layers, a.chunk_order);
    const hipError_t e = launch_bf16_w<D, KS, 4, true>(a, grid, chunk / 64,
                                                       (chunk + a.pv.block_size - 1) / a.pv.block_size + 1, stream);
    if (e != hipSuccess) return e;
    a.kv_begin = 1;
    nkv = 1;
  }
  const int chunk = kApplyChunkTokens;
  constexpr int W = apply_waves(KS);
  const int chunks = (max_tokens + chunk - 1) / chunk;
  a.chunk_order = multi_item_order(num_items, chunks, kChunksRotated);
  const dim3 grid = chunk_grid(chunks, nkv * H, num_items * a.num_layers, a.chunk_order);
  return launch_bf16_w<D, KS, W, false>(a, grid, chunk / (16 * W), (chunk + a.pv.block_size - 1) / a.pv.block_size + 1,
                                        stream);
}

template <int D>
static hipError_t launch_bf16_ks(const ApplyArgs& a, int ks, int max_tokens, int num_items, hipStream_t stream) {
  switch (ks) {
    case 0:
    case 1: return launch_bf16<D, 1>(a, max_tokens, num_items, stream);
    case 2: return launch_bf16<D, 2>(a, max_tokens, num_items, stream);
    case 3: return launch_bf16<D, 3>(a, max_tokens, num_items, stream);
    default: return launch_bf16<D, 4>(a, max_tokens, num_items, stream);
  }
}

hipError_t launch_apply(const ApplyArgs& a, kvc_dtype dtype, int max_rank, int max_tokens, int num_items,
                        hipStream_t stream) {
  if (max_tokens == 0 || num_items == 0 || a.num_layers == 0) return hipSuccess;
  const int D = a.pv.head_dim;
  if (dtype == KVC_BF16) {
    const int ks = (max_rank + 31) / 32;
    return D == 64 ? launch_bf16_ks<64>(a, ks, max_tokens, num_items, stream)
                   : launch_bf16_ks<128>(a, ks, max_tokens, num_items, stream);
  }
  ApplyArgs b = a;
  const int chunks = (max_tokens + kApplyChunk - 1) / kApplyChunk;
  b.chunk_order = multi_item_order(num_items, chunks, kChunksRotated);
  const dim3 grid = chunk_grid(chunks, 2 * a.pv.num_kv_heads, num_items * a.num_layers, b.chunk_order);
  const size_t lds = (size_t)max_rank * D * sizeof(float);
  if (D == 64) {
    hipLaunchKernelGGL(apply_f32_valu<64>, grid, dim3(kApplyThreads), lds, stream, b);
  } else {
    hipLaunchKernelGGL(apply_f32_valu<128>, grid, dim3(kApplyThreads), lds, stream, b);
  }
  return hipGetLastError();
}

}  // namespace kvc
