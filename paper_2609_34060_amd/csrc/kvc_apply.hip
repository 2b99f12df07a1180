// kvc_apply kernels: C_dst[t] = C_src[t] + A[t] B for t < T_s, bit copy for T_s <= t < T (Eq. 4 with the source
// agent's cache as reference, Eq. 8 with one state, prefix coverage of Appendix A.3).
//
// bf16 caches: one workgroup = 4 wave64s over one (item, layer, K/V, head) unit and a chunk of 512 tokens.  The
// correction of a 16-token tile is the MFMA contraction  D^T = B^T A^T + C^T  with M = feature (16 per tile), N =
// token, K = rank (32 per v_mfma_f32_16x16x32_bf16), and the accumulator C initialised with the source rows in fp32.
// B is staged once per workgroup in LDS as a bf16 hi/lo pair (about 16 significant bits of the fp32 basis) and
// held in registers as MFMA A-fragments; the bf16 coefficients are the MFMA B-operand, loaded straight from the
// coefficient rows (one 16-byte load per lane and 32 ranks).  The M index of each tile is permuted so that the
// four lanes holding one token own 64 contiguous bytes of the row per 16-byte load: every global load and store of
// a cache row is 128-bit and a row is touched by whole 64-byte segments.
//
// float32 caches: a VALU kernel with the basis in LDS (float32 throughout, for the 1e-5 storage tolerance).
#include "kvc_device.h"
#include "kvc_launch.h"

namespace kvc {

constexpr int kApplyWaves = 4;
constexpr int kApplyThreads = kApplyWaves * kWave;
constexpr int kApplyTilesPerWave = 8;
constexpr int kApplyChunk = kApplyWaves * kApplyTilesPerWave * 16;  // tokens per workgroup

int apply_chunk_tokens() { return kApplyChunk; }

// Tuning knobs of the bf16 kernel (chosen by measurement on MI355X; see the launcher).
//   TPW   16-token tiles per wave per workgroup (a workgroup covers 4 * 16 * TPW tokens)
//   REGF  A-fragments held in registers for the whole chunk (true) or re-read from LDS per tile (false)
//   PF    software prefetch: the next tile's rows and coefficients are loaded before this tile's MFMAs
//   NTL   non-temporal loads of the streamed source rows (read exactly once)
//   NTS   non-temporal stores of the destination rows (written exactly once)
//   ROPE  the keys are rotary-encoded: corrected in canonical coordinates and rotated to the target positions,
//         C_dst = R(pd - ps) C_src + (A B R(pd)^T): the accumulator starts from the source rotated by pd - ps and B is
//         staged rotated by pd, so the rotation costs no extra pass (rows past T_s get the rotated source)
template <int D, int KS, int TPW, bool REGF, bool PF, bool NTL, bool NTS, bool ROPE>
__global__ __launch_bounds__(kApplyThreads) void apply_bf16_mfma(ApplyArgs a) {
  constexpr int MT = D / 16;  // M-tiles per row
  constexpr int NQ = D / 32;  // 16-byte loads per lane per row
  constexpr int KP = KS * 32; // padded rank
  constexpr int CHUNK = kApplyWaves * TPW * 16;
  __shared__ __attribute__((aligned(16))) uint16_t s_hi[D * KP];
  __shared__ __attribute__((aligned(16))) uint16_t s_lo[D * KP];

  const int nl = a.num_layers;
  const int item_id = blockIdx.z / nl;
  const int lrel = blockIdx.z - item_id * nl;
  const int layer = a.layer_begin + lrel;
  const int H = a.pv.num_kv_heads;
  const int kv = blockIdx.y / H;
  const int head = blockIdx.y - kv * H;

  const kvc_item* itp = a.items + item_id;
  const int T = itp->num_tokens;
  const int t_begin = blockIdx.x * CHUNK;
  if (t_begin >= T) return;
  const int r = itp->state.rank;
  const int Tdecl = itp->state.num_tokens;
  const int Ts = r > 0 ? min(Tdecl, T) : 0;
  const int src_off = itp->src_offset, dst_off = itp->dst_offset;
  const int32_t* src_tab = a.src_tables ? a.src_tables + (int64_t)item_id * a.max_blocks : nullptr;
  const int32_t* dst_tab = a.dst_tables ? a.dst_tables + (int64_t)item_id * a.max_blocks : nullptr;
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

  constexpr bool kRegFrags = REGF && KS <= 2;
  constexpr int FM = kRegFrags ? MT : 1, FK = kRegFrags ? KS : 1;
  bf16x8 ahi[FM][FK], alo[FM][FK];
  if (correct) {
    // Stage B^T as bf16 hi/lo, zero-padded to KP ranks: s[f * KP + k] = split(B[k][f]).
    for (int e = threadIdx.x; e < D * KP; e += kApplyThreads) {
      const int k = e / D, f = e - k * D;
      float x = k < r ? basis[k * bstride + f] : 0.0f;
      if (rope && k < r) {  // B R(pd)^T: each basis row rotated like a key row at position pd
        const int i = rope_pair(style, D, f);
        x = rope_rotated(rope_first(style, D, f), x, basis[k * bstride + rope_partner(style, D, f)], s_rope[2][i],
                         s_rope[3][i]);
      }
      uint32_t hb, lb;
      split_bf16(x, hb, lb);
      s_hi[f * KP + k] = (uint16_t)hb;
      s_lo[f * KP + k] = (uint16_t)lb;
    }
    __syncthreads();
    if constexpr (kRegFrags) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int f = mfma_row_feature(mt, n);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int k0 = ks * 32 + 8 * g;
          ahi[mt][ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[f * KP + k0]));
          alo[mt][ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[f * KP + k0]));
        }
      }
    }
  }
  const bool coef_vec = (r & 7) == 0;

  struct Tile {
    u32x4 raw[NQ];
    u32x4 cw[KS];
    int64_t dof;
  };
  // Issue the loads of tile j (rows through the block tables, coefficient rows); lanes past T load nothing.
  auto load_tile = [&](int j, Tile& tl) {
    const int t = t_begin + (j * kApplyWaves + wave) * 16 + n;
    const bool valid = t < T;
    const int64_t so = valid ? row_offset(a.pv, src_tab, src_off, t, head) : -1;
    // a row whose source block id is out of range is neither read nor written
    tl.dof = so >= 0 ? row_offset(a.pv, dst_tab, dst_off, t, head) : -1;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const u32x4* p = reinterpret_cast<const u32x4*>(src_pool + so + 32 * q + 8 * g);
      if (so >= 0) {
        tl.raw[q] = NTL ? __builtin_nontemporal_load(p) : *p;
      } else {
        tl.raw[q] = u32x4{0, 0, 0, 0};
      }
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
  auto finish_tile = [&](int j, const Tile& tl) {
    const int t0 = t_begin + (j * kApplyWaves + wave) * 16;
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
          if constexpr (kRegFrags) {
            acc[mt] = mfma16x16x32(alo[mt][ks], cb, acc[mt]);
            acc[mt] = mfma16x16x32(ahi[mt][ks], cb, acc[mt]);
          } else {
            const int fo = mfma_row_feature(mt, n) * KP + ks * 32 + 8 * g;
            const bf16x8 fl = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[fo]));
            const bf16x8 fh = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[fo]));
            acc[mt] = mfma16x16x32(fl, cb, acc[mt]);
            acc[mt] = mfma16x16x32(fh, cb, acc[mt]);
          }
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
      for (int q = 0; q < NQ; ++q) {
        u32x4* p = reinterpret_cast<u32x4*>(dst_pool + tl.dof + 32 * q + 8 * g);
        if (NTS) {
          __builtin_nontemporal_store(outw[q], p);
        } else {
          *p = outw[q];
        }
      }
    }
  };

  if constexpr (PF) {
    Tile cur, nxt;
    load_tile(0, cur);
    for (int j = 0; j < TPW; ++j) {
      if (t_begin + (j * kApplyWaves + wave) * 16 >= T) break;
      if (j + 1 < TPW && t_begin + ((j + 1) * kApplyWaves + wave) * 16 < T) load_tile(j + 1, nxt);
      finish_tile(j, cur);
      cur = nxt;
    }
  } else {
    for (int j = 0; j < TPW; ++j) {
      if (t_begin + (j * kApplyWaves + wave) * 16 >= T) break;
      Tile cur;
      load_tile(j, cur);
      finish_tile(j, cur);
    }
  }
}

// float32 caches: each thread owns 4 features of one token; the rank loop runs over B in LDS.
template <int D>
__global__ __launch_bounds__(kApplyThreads) void apply_f32_valu(ApplyArgs a) {
  extern __shared__ __attribute__((aligned(16))) float s_b[];  // [r][D]
  constexpr int LPT = D / 4;                                   // lanes per token
  constexpr int TPP = kApplyThreads / LPT;                     // tokens per pass

  const int nl = a.num_layers;
  const int item_id = blockIdx.z / nl;
  const int lrel = blockIdx.z - item_id * nl;
  const int layer = a.layer_begin + lrel;
  const int H = a.pv.num_kv_heads;
  const int kv = blockIdx.y / H;
  const int head = blockIdx.y - kv * H;

  const kvc_item* itp = a.items + item_id;
  const int T = itp->num_tokens;
  const int t_begin = blockIdx.x * kApplyChunk;
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

// Chosen configuration (tiles per wave, fragment placement, prefetch, non-temporal access).
constexpr int kTPW = 16;
constexpr bool kREGF = false, kPF = false, kNTL = false, kNTS = false;

template <int D, int KS>
static hipError_t launch_bf16(const ApplyArgs& a, dim3 grid, hipStream_t stream) {
  if (a.pv.rope.style != KVC_ROPE_NONE)
    hipLaunchKernelGGL((apply_bf16_mfma<D, KS, kTPW, kREGF, kPF, kNTL, kNTS, true>), grid, dim3(kApplyThreads), 0,
                       stream, a);
  else
    hipLaunchKernelGGL((apply_bf16_mfma<D, KS, kTPW, kREGF, kPF, kNTL, kNTS, false>), grid, dim3(kApplyThreads), 0,
                       stream, a);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_bf16_ks(const ApplyArgs& a, int ks, dim3 grid, hipStream_t stream) {
  switch (ks) {
    case 0:
    case 1: return launch_bf16<D, 1>(a, grid, stream);
    case 2: return launch_bf16<D, 2>(a, grid, stream);
    case 3: return launch_bf16<D, 3>(a, grid, stream);
    default: return launch_bf16<D, 4>(a, grid, stream);
  }
}

hipError_t launch_apply(const ApplyArgs& a, kvc_dtype dtype, int max_rank, int max_tokens, int num_items,
                        hipStream_t stream) {
  if (max_tokens == 0 || num_items == 0 || a.num_layers == 0) return hipSuccess;
  const int D = a.pv.head_dim;
  if (dtype == KVC_BF16) {
    const int chunk = kApplyWaves * kTPW * 16;
    dim3 grid((max_tokens + chunk - 1) / chunk, 2 * a.pv.num_kv_heads, num_items * a.num_layers);
    const int ks = (max_rank + 31) / 32;
    return D == 64 ? launch_bf16_ks<64>(a, ks, grid, stream) : launch_bf16_ks<128>(a, ks, grid, stream);
  }
  dim3 grid((max_tokens + kApplyChunk - 1) / kApplyChunk, 2 * a.pv.num_kv_heads, num_items * a.num_layers);
  const size_t lds = (size_t)max_rank * D * sizeof(float);
  if (D == 64) {
    hipLaunchKernelGGL(apply_f32_valu<64>, grid, dim3(kApplyThreads), lds, stream, a);
  } else {
    hipLaunchKernelGGL(apply_f32_valu<128>, grid, dim3(kApplyThreads), lds, stream, a);
  }
  return hipGetLastError();
}

}  // namespace kvc
