// Anchor-pool kernels (Section 3.3, Eq. 8-11, Appendix A.3).  One item per call; every kernel walks the item's
// rows through its block tables like kvc_apply.
//
//   weights  d_v[t] = mean over the layer's K (or V) row (all heads, all features) of |C_src[t] - (A_v B_v)[t]|,
//            A_v B_v anchor v's base state; w_v[t] = softmax_v(-d_v[t] / temperature).
//   apply    C_dst[t] = C_src[t] + sum_v w_v[t] A_v[t] B_v (Eq. 8, token-wise weights), bit copy past T_s.
//   gate     d_v = (sum over layers, heads, t < k, features of (V_src - V_v)^2)^(1/2) (Eq. 9), partial sums per
//            (layer, token chunk) added in a fixed order in fp64.
//
// bf16 caches: the reconstruction A_v B_v of a 16-token tile uses the layout of the apply kernel (MFMA with M =
// feature, N = token, K = rank; B staged in LDS as a bf16 hi/lo pair, about 16 significant bits).  In the anchored
// apply the weight multiplies the bf16 coefficients in fp32, so the scaled coefficients are split into hi/lo as
// well (hi*hi + hi*lo + lo*hi on the MFMA), and the correction of all anchors accumulates in fp32 before one
// rounding of C_src + correction.  float32 caches use VALU kernels in fp32.
#include <algorithm>

#include "kvc_device.h"
#include "kvc_launch.h"

namespace kvc {

constexpr int kAnchorWaves = 4;
constexpr int kAnchorThreads = kAnchorWaves * kWave;
constexpr int kAnchorTiles = 8;                                     // 16-token tiles per wave (distance kernels)
constexpr int kAnchorChunk = kAnchorWaves * kAnchorTiles * 16;      // 512 tokens per workgroup
constexpr int kAnchoredTiles = 4;                                   // tiles per wave in the anchored apply
constexpr int kAnchoredChunk = kAnchorWaves * kAnchoredTiles * 16;  // 256 tokens per workgroup
constexpr int kF32Chunk = 64;                                       // tokens per workgroup (float32 kernels)

int anchor_chunk_tokens() { return kAnchorChunk; }

// B^T of one unit staged as bf16 hi/lo, zero-padded to KP = 32 KSM ranks: s[f * KP + k] = split(B[k][f]).  A thread
// owns (feature f, eight ranks 8c .. 8c + 7) items, consecutive threads the consecutive 16-byte LDS granules, so the
// stores are conflict-free (the loads read 64-byte row segments).  The loads of the next basis are issued into
// registers before the current one is used (load) and written to the other LDS buffer one step later (store), so a
// workgroup waits once per basis at its barrier.
// ROPE: with `rot` set (keys of a rotary cache) each basis row is rotated like a key row by the angles of the table
// (c, s): the partner feature's values are loaded with the item's own and the rotation is applied at the store.
template <int D, int KSM, bool ROPE = false>
struct BasisStager {
  static constexpr int KP = 32 * KSM, KG = KP / 8;
  static constexpr int NI = D * KG / kAnchorThreads;  // items per thread
  static_assert(NI * kAnchorThreads == D * KG, "whole items per thread");
  float v[NI][8];
  float pv[ROPE ? NI : 1][8];
  __device__ __forceinline__ void load(const float* basis, int r, bool rot = false, int style = 0) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int idx = (int)threadIdx.x + i * kAnchorThreads;
      const int c = idx % KG, f = idx / KG;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[i][e] = 8 * c + e < r ? basis[(8 * c + e) * D + f] : 0.0f;
      if (ROPE && rot) {
        const int pf = rope_partner(style, D, f);
#pragma unroll
        for (int e = 0; e < 8; ++e) pv[i][e] = 8 * c + e < r ? basis[(8 * c + e) * D + pf] : 0.0f;
      }
    }
  }
  __device__ __forceinline__ void store(uint16_t* s_hi, uint16_t* s_lo, bool rot = false, int style = 0,
                                        const float* rc = nullptr, const float* rs = nullptr) const {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int idx = (int)threadIdx.x + i * kAnchorThreads;
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = v[i][e];
      if (ROPE && rot) {
        const int f = idx / KG, pi = rope_pair(style, D, f);
        const bool first = rope_first(style, D, f);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = rope_rotated(first, v[i][e], pv[i][e], rc[pi], rs[pi]);
      }
      u32x4 hi, lo;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        uint32_t hh, ll;
        split_bf16x2(x[2 * p], x[2 * p + 1], hh, ll);
        hi[p] = hh;
        lo[p] = ll;
      }
      *reinterpret_cast<u32x4*>(s_hi + 8 * idx) = hi;  // = s_hi + f * KP + 8 c
      *reinterpret_cast<u32x4*>(s_lo + 8 * idx) = lo;
    }
  }
};

// Eight bf16 coefficients of row t, ranks k0 .. k0 + 7 (zero past r).
__device__ __forceinline__ u32x4 load_coef8(const uint16_t* coef, int r, int t, int k0) {
  const uint16_t* cp = coef + (int64_t)t * r + k0;
  if ((r & 7) == 0 && k0 + 8 <= r) return *reinterpret_cast<const u32x4*>(cp);
  uint32_t e[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) e[i] = (k0 + i < r) ? cp[i] : 0u;
  return u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16)};
}

// One source row segment per lane: token t, features 32 q + 8 g .. + 7 for q < D / 32 (zero when the row is absent).
template <int NQ>
__device__ __forceinline__ void load_row_segments(const uint16_t* pool, int64_t off, int g, u32x4* raw) {
#pragma unroll
  for (int q = 0; q < NQ; ++q)
    raw[q] = off >= 0 ? *reinterpret_cast<const u32x4*>(pool + off + 32 * q + 8 * g) : u32x4{0u, 0u, 0u, 0u};
}

// ---------------------------------------------------------------------------------------------------------------
// distances (weights / gate), bf16
// ---------------------------------------------------------------------------------------------------------------

// ROPE: keys of a rotary cache are compared in canonical coordinates, R(-ps) C_src (the anchors are canonical).
template <int D, int KSM, bool GATE, bool ROPE>
__global__ __launch_bounds__(kAnchorThreads) void anchor_dist_bf16(AnchorArgs a) {
  constexpr int MT = D / 16, NQ = D / 32, KP = 32 * KSM;
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  uint16_t* s_b = reinterpret_cast<uint16_t*>(anchor_lds);   // [2 buffers][hi, lo][D * KP]
  float* s_d = reinterpret_cast<float*>(s_b + 4 * D * KP);     // GATE: [waves][V]; else [chunk][V]
  float* s_rope = s_d + (GATE ? kAnchorWaves : kAnchorChunk) * KVC_MAX_ANCHORS;  // cos / sin of -ps

  const int lrel = blockIdx.z, layer = a.layer_begin + lrel;
  const int kv = GATE ? 1 : blockIdx.y;
  const int H = a.pv.num_kv_heads, V = a.num_anchors;
  const int Tl = a.num_weighted;
  const int t_begin = blockIdx.x * kAnchorChunk;
  if (t_begin >= Tl) return;  // whole workgroup
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave, g = lane >> 4, n = lane & 15;
  const uint16_t* pool = static_cast<const uint16_t*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]);
  const int nd = GATE ? kAnchorWaves * V : kAnchorChunk * V;
  for (int e = threadIdx.x; e < nd; e += kAnchorThreads) s_d[e] = 0.0f;
  const bool rot = ROPE && kv == 0;  // uniform; read after the first barrier below
  const int style = a.pv.rope.style;
  if (rot) rope_table(a.pv.rope, D, -(double)a.src_position, s_rope, s_rope + D / 2);

  BasisStager<D, KSM> stager;
  auto basis_of = [&](int hv) {
    const int h = hv / V, v = hv - h * V;
    return a.basis[v] + unit_index(layer, kv, h, H) * (int64_t)a.rank[v] * D;
  };
  // the gate (value rows only) takes one KV head per workgroup; the weights walk every head of the layer row
  const int hv0 = GATE ? (int)blockIdx.y * V : 0, hv1 = GATE ? hv0 + V : H * V;
  stager.load(basis_of(hv0), a.rank[hv0 % V]);
  for (int hv = hv0; hv < hv1; ++hv) {
    const int h = hv / V, v = hv - h * V;
    const int r = a.rank[v], KS = (r + 31) / 32;
    uint16_t* s_hi = s_b + (hv & 1) * 2 * D * KP;
    uint16_t* s_lo = s_hi + D * KP;
    stager.store(s_hi, s_lo);
    __syncthreads();  // this basis is in LDS; the other buffer is no longer read (and s_d is initialised)
    if (hv + 1 < hv1) stager.load(basis_of(hv + 1), a.rank[(hv + 1) % V]);
    const int64_t unit = unit_index(layer, kv, h, H);
    const uint16_t* coef = static_cast<const uint16_t*>(a.coef[v]) + unit * (int64_t)a.tokens[v] * r;
    float part = 0.0f;
    for (int j = 0; j < kAnchorTiles; ++j) {
      const int tile = j * kAnchorWaves + wave;
      const int t0 = t_begin + tile * 16;
      if (t0 >= Tl) break;
      const int t = t0 + n;
      const bool valid = t < Tl;
      u32x4 raw[NQ];
      load_row_segments<NQ>(pool, valid ? row_offset(a.pv, a.src_table, a.src_offset, t, h) : -1, g, raw);
      f32x4 acc[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KSM; ++ks) {
        if (ks >= KS) break;
        const bf16x8 cb = as_bf16x8(valid ? load_coef8(coef, r, t, ks * 32 + 8 * g) : u32x4{0u, 0u, 0u, 0u});
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int fo = mfma_row_feature(mt, n) * KP + ks * 32 + 8 * g;
          acc[mt] = mfma16x16x32(as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[fo])), cb, acc[mt]);
          acc[mt] = mfma16x16x32(as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[fo])), cb, acc[mt]);
        }
      }
      f32x4 xv[MT];
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        xv[2 * q] = f32x4{bf16_lo_to_f32(raw[q][0]), bf16_hi_to_f32(raw[q][0]), bf16_lo_to_f32(raw[q][1]),
                          bf16_hi_to_f32(raw[q][1])};
        xv[2 * q + 1] = f32x4{bf16_lo_to_f32(raw[q][2]), bf16_hi_to_f32(raw[q][2]), bf16_lo_to_f32(raw[q][3]),
                              bf16_hi_to_f32(raw[q][3])};
      }
      if (ROPE && rot) rope_rotate_rows<D>(xv, style, g, s_rope, s_rope + D / 2);
      float s = 0.0f;
#pragma unroll
      for (int m = 0; m < MT; ++m) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float diff = xv[m][e] - acc[m][e];
          s += GATE ? diff * diff : fabsf(diff);
        }
      }
      s += __shfl_xor(s, 16, kWave);
      s += __shfl_xor(s, 32, kWave);
      if (GATE) {
        part += valid ? s : 0.0f;
      } else if (g == 0 && valid) {
        s_d[(tile * 16 + n) * V + v] += s;  // this lane owns the token: no race
      }
    }
    if (GATE) {
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) part += __shfl_xor(part, o, kWave);
      if (lane == 0) s_d[wave * V + v] += part;
    }
  }
  __syncthreads();
  if (GATE) {
    if (threadIdx.x < V) {
      const int v = threadIdx.x;
      float s = 0.0f;
      for (int w = 0; w < kAnchorWaves; ++w) s += s_d[w * V + v];
      a.gate_partials[((int64_t)lrel * a.gate_chunks + blockIdx.x * gridDim.y + blockIdx.y) * V + v] = s;
    }
  } else {
    const float inv_feat = 1.0f / (float)(H * D);
    for (int tok = threadIdx.x; tok < kAnchorChunk; tok += kAnchorThreads) {
      const int t = t_begin + tok;
      if (t >= Tl) break;
      float dmin = INFINITY;
      for (int v = 0; v < V; ++v) dmin = fminf(dmin, s_d[tok * V + v] * inv_feat);
      float sum = 0.0f;
      for (int v = 0; v < V; ++v) sum += __expf(-(s_d[tok * V + v] * inv_feat - dmin) * a.inv_temperature);
      const float inv = 1.0f / sum;
      float* wout = a.weights + ((int64_t)(lrel * 2 + kv) * Tl + t) * V;
      for (int v = 0; v < V; ++v) wout[v] = __expf(-(s_d[tok * V + v] * inv_feat - dmin) * a.inv_temperature) * inv;
    }
  }
}

// ---------------------------------------------------------------------------------------------------------------
// distances, float32 (VALU): D / 4 lanes per token, four features per lane
// ---------------------------------------------------------------------------------------------------------------

template <int D, bool GATE, bool ROPE>
__global__ __launch_bounds__(kAnchorThreads) void anchor_dist_f32(AnchorArgs a) {
  constexpr int LPT = D / 4, TPP = kAnchorThreads / LPT;
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  float* s_b = reinterpret_cast<float*>(anchor_lds);           // [max_rank][D]
  float* s_d = s_b + a.max_rank * D;                            // GATE: [TPP][V]; else [chunk][V]
  float* s_rope = s_d + (GATE ? TPP : kF32Chunk) * KVC_MAX_ANCHORS;  // cos / sin of -ps (rotary keys)
  const int lrel = blockIdx.z, layer = a.layer_begin + lrel;
  const int kv = GATE ? 1 : blockIdx.y;
  const int H = a.pv.num_kv_heads, V = a.num_anchors;
  const int Tl = a.num_weighted;
  const int t_begin = blockIdx.x * kF32Chunk;
  if (t_begin >= Tl) return;
  const int sub = threadIdx.x / LPT, f0 = 4 * (threadIdx.x % LPT);
  const float* pool = static_cast<const float*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]);
  const int nd = GATE ? TPP * V : kF32Chunk * V;
  for (int e = threadIdx.x; e < nd; e += kAnchorThreads) s_d[e] = 0.0f;
  const bool rot = ROPE && kv == 0;  // canonical source keys R(-ps) C_src; the table is read after a barrier
  const int style = a.pv.rope.style;
  if (rot) rope_table(a.pv.rope, D, -(double)a.src_position, s_rope, s_rope + D / 2);
  for (int h = 0; h < H; ++h) {
    const int64_t unit = unit_index(layer, kv, h, H);
    for (int v = 0; v < V; ++v) {
      const int r = a.rank[v];
      __syncthreads();
      for (int e = threadIdx.x; e < r * D; e += kAnchorThreads) s_b[e] = a.basis[v][unit * (int64_t)r * D + e];
      __syncthreads();
      const float* coef = static_cast<const float*>(a.coef[v]) + unit * (int64_t)a.tokens[v] * r;
      float part = 0.0f;
      for (int tok = sub; tok < kF32Chunk; tok += TPP) {
        const int t = t_begin + tok;
        float s = 0.0f;
        if (t < Tl) {
          const int64_t so = row_offset(a.pv, a.src_table, a.src_offset, t, h);
          f32x4 x = so >= 0 ? *reinterpret_cast<const f32x4*>(pool + so + f0) : f32x4{0.f, 0.f, 0.f, 0.f};
          if (ROPE && rot && so >= 0) {
            const f32x4 y = *reinterpret_cast<const f32x4*>(pool + so + (rope_partner(style, D, f0) & ~3));
            f32x4 xc;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int f = f0 + j, i = rope_pair(style, D, f);
              const float partner = style == KVC_ROPE_HALF ? y[j] : x[j ^ 1];
              xc[j] = rope_rotated(rope_first(style, D, f), x[j], partner, s_rope[i], s_rope[D / 2 + i]);
            }
            x = xc;
          }
          const float* crow = coef + (int64_t)t * r;
          for (int k = 0; k < r; ++k) {
            const float c = crow[k];
            const f32x4 b = *reinterpret_cast<const f32x4*>(&s_b[k * D + f0]);
            x[0] = fmaf(-c, b[0], x[0]);
            x[1] = fmaf(-c, b[1], x[1]);
            x[2] = fmaf(-c, b[2], x[2]);
            x[3] = fmaf(-c, b[3], x[3]);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) s += GATE ? x[i] * x[i] : fabsf(x[i]);
        }
#pragma unroll
        for (int o = 1; o < LPT; o <<= 1) s += __shfl_xor(s, o, kWave);  // LPT lanes of one token
        if (GATE) part += s;
        else if (threadIdx.x % LPT == 0 && t < Tl) s_d[tok * V + v] += s;
      }
      if (GATE && threadIdx.x % LPT == 0) s_d[sub * V + v] += part;
    }
  }
  __syncthreads();
  if (GATE) {
    if (threadIdx.x < V) {
      const int v = threadIdx.x;
      float s = 0.0f;
      for (int w = 0; w < TPP; ++w) s += s_d[w * V + v];
      a.gate_partials[((int64_t)lrel * a.gate_chunks + blockIdx.x) * V + v] = s;
    }
  } else {
    const float inv_feat = 1.0f / (float)(H * D);
    for (int tok = threadIdx.x; tok < kF32Chunk; tok += kAnchorThreads) {
      const int t = t_begin + tok;
      if (t >= Tl) break;
      float dmin = INFINITY;
      for (int v = 0; v < V; ++v) dmin = fminf(dmin, s_d[tok * V + v] * inv_feat);
      float sum = 0.0f;
      for (int v = 0; v < V; ++v) sum += expf(-(s_d[tok * V + v] * inv_feat - dmin) * a.inv_temperature);
      const float inv = 1.0f / sum;
      float* wout = a.weights + ((int64_t)(lrel * 2 + kv) * Tl + t) * V;
      for (int v = 0; v < V; ++v) wout[v] = expf(-(s_d[tok * V + v] * inv_feat - dmin) * a.inv_temperature) * inv;
    }
  }
}

// Gate: d_v = sqrt(sum of the partials of every (layer, chunk[, head])) in a fixed order, fp64.  Wave w takes
// anchors v = w, w + 4, ...; lane l adds the partials l, l + 64, ... in order and a fixed xor butterfly combines the
// lanes, so the sum does not depend on scheduling.
__global__ __launch_bounds__(kAnchorThreads) void gate_finish(AnchorArgs a) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t n = (int64_t)a.num_layers * a.gate_chunks;
  for (int v = wave; v < a.num_anchors; v += kAnchorWaves) {  // uniform over the wave
    double s = 0.0;
    for (int64_t i = lane; i < n; i += kWave) s += (double)a.gate_partials[i * a.num_anchors + v];
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) s += __shfl_xor(s, o, kWave);
    if (lane == 0) a.distances[v] = (float)sqrt(s);
  }
}

// ---------------------------------------------------------------------------------------------------------------
// anchored apply, bf16: the correction of every anchor accumulates in registers over an outer loop on the anchors
// (one basis staging per anchor and workgroup), then C_src + correction is rounded once and stored
// ---------------------------------------------------------------------------------------------------------------

// ROPE: keys of a rotary cache, C_dst = R(pd - ps) C_src + sum_v w_v A_v (B_v R(pd)^T) (bases staged rotated).
template <int D, int KSM, bool ROPE>
__global__ __launch_bounds__(kAnchorThreads) void apply_anchored_bf16(AnchorArgs a) {
  constexpr int MT = D / 16, NQ = D / 32, TPW = kAnchoredTiles, KP = 32 * KSM;
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  uint16_t* s_b = reinterpret_cast<uint16_t*>(anchor_lds);  // [2 buffers][hi, lo][D * KP]
  float* s_rope = reinterpret_cast<float*>(s_b + 4 * D * KP);  // cos / sin of pd - ps, then of pd

  const int lrel = blockIdx.z, layer = a.layer_begin + lrel;
  const int H = a.pv.num_kv_heads;
  const int kv = blockIdx.y / H, head = blockIdx.y - kv * H;
  const int T = a.num_tokens, Ts = a.num_weighted, V = a.num_anchors;
  const int t_begin = blockIdx.x * kAnchoredChunk;
  if (t_begin >= T) return;  // whole workgroup
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave, g = lane >> 4, n = lane & 15;
  const int64_t unit = unit_index(layer, kv, head, H);
  const uint16_t* src_pool = static_cast<const uint16_t*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]);
  uint16_t* dst_pool = static_cast<uint16_t*>(const_cast<void*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]));
  const float* wrow = a.weights + (int64_t)(lrel * 2 + kv) * Ts * V;
  const bool rot = ROPE && kv == 0;  // uniform over the workgroup
  const bool shift = rot && a.dst_position != a.src_position;
  const int style = a.pv.rope.style;
  if (rot) {
    rope_table(a.pv.rope, D, (double)a.dst_position - (double)a.src_position, s_rope, s_rope + D / 2);
    rope_table(a.pv.rope, D, (double)a.dst_position, s_rope + D, s_rope + 3 * D / 2);
    __syncthreads();
  }

  f32x4 acc[TPW][MT];
#pragma unroll
  for (int j = 0; j < TPW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (t_begin < Ts) {  // whole workgroup
    BasisStager<D, KSM, ROPE> stager;
    stager.load(a.basis[0] + unit * (int64_t)a.rank[0] * D, a.rank[0], rot, style);
    for (int v = 0; v < V; ++v) {
      const int r = a.rank[v], KS = (r + 31) / 32;
      uint16_t* s_hi = s_b + (v & 1) * 2 * D * KP;
      uint16_t* s_lo = s_hi + D * KP;
      stager.store(s_hi, s_lo, rot, style, s_rope + D, s_rope + 3 * D / 2);
      __syncthreads();  // this basis is in LDS; the other buffer is no longer read
      if (v + 1 < V) stager.load(a.basis[v + 1] + unit * (int64_t)a.rank[v + 1] * D, a.rank[v + 1], rot, style);
      const uint16_t* coef = static_cast<const uint16_t*>(a.coef[v]) + unit * (int64_t)a.tokens[v] * r;
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        const int t0 = t_begin + (j * kAnchorWaves + wave) * 16;
        if (t0 >= Ts) continue;  // uniform over the wave
        const int t = t0 + n;
        const bool valid = t < Ts;
        const float w = valid ? wrow[(int64_t)t * V + v] : 0.0f;
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks) {
          if (ks >= KS) break;
          const u32x4 cw = valid ? load_coef8(coef, r, t, ks * 32 + 8 * g) : u32x4{0u, 0u, 0u, 0u};
          u32x4 ch, cl;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            uint32_t hh, ll;
            split_bf16x2(w * bf16_lo_to_f32(cw[i]), w * bf16_hi_to_f32(cw[i]), hh, ll);
            ch[i] = hh;
            cl[i] = ll;
          }
          const bf16x8 bh = as_bf16x8(ch), bl = as_bf16x8(cl);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const int fo = mfma_row_feature(mt, n) * KP + ks * 32 + 8 * g;
            const bf16x8 fl = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[fo]));
            const bf16x8 fh = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[fo]));
            acc[j][mt] = mfma16x16x32(fl, bh, acc[j][mt]);
            acc[j][mt] = mfma16x16x32(fh, bl, acc[j][mt]);
            acc[j][mt] = mfma16x16x32(fh, bh, acc[j][mt]);
          }
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    const int t0 = t_begin + (j * kAnchorWaves + wave) * 16;
    if (t0 >= T) break;
    const int t = t0 + n;
    const bool valid = t < T;
    u32x4 raw[NQ];
    const int64_t so = valid ? row_offset(a.pv, a.src_table, a.src_offset, t, head) : -1;
    load_row_segments<NQ>(src_pool, so, g, raw);
    // a row whose source block id is out of range is neither read nor written
    const int64_t dof = so >= 0 ? row_offset(a.pv, a.dst_table, a.dst_offset, t, head) : -1;
    u32x4 outw[NQ];
    // rows past T_s have a zero correction: the re-aligned source with a shift, else bit copies
    const bool crow = t < Ts || shift;
    f32x4 xv[MT];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      xv[2 * q] = f32x4{bf16_lo_to_f32(raw[q][0]), bf16_hi_to_f32(raw[q][0]), bf16_lo_to_f32(raw[q][1]),
                        bf16_hi_to_f32(raw[q][1])};
      xv[2 * q + 1] = f32x4{bf16_lo_to_f32(raw[q][2]), bf16_hi_to_f32(raw[q][2]), bf16_lo_to_f32(raw[q][3]),
                            bf16_hi_to_f32(raw[q][3])};
    }
    if (ROPE && shift) rope_rotate_rows<D>(xv, style, g, s_rope, s_rope + D / 2);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const f32x4 x = xv[2 * q] + acc[j][2 * q], y = xv[2 * q + 1] + acc[j][2 * q + 1];
      const u32x4 c = {pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(y[0], y[1]),
                       pack_bf16x2(y[2], y[3])};
      outw[q] = crow ? c : raw[q];
    }
    if (dof >= 0) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) *reinterpret_cast<u32x4*>(dst_pool + dof + 32 * q + 8 * g) = outw[q];
    }
  }
}

// anchored apply, float32 (VALU): D / 4 lanes per token; the tokens of a workgroup accumulate over the anchors
template <int D, bool ROPE>
__global__ __launch_bounds__(kAnchorThreads) void apply_anchored_f32(AnchorArgs a) {
  constexpr int LPT = D / 4, TPP = kAnchorThreads / LPT, NP = kF32Chunk / TPP;
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  float* s_b = reinterpret_cast<float*>(anchor_lds);  // [max_rank][D]
  float* s_rope = s_b + a.max_rank * D;               // cos / sin of pd - ps, then of pd (rotary keys)
  const int lrel = blockIdx.z, layer = a.layer_begin + lrel;
  const int H = a.pv.num_kv_heads;
  const int kv = blockIdx.y / H, head = blockIdx.y - kv * H;
  const int T = a.num_tokens, Ts = a.num_weighted, V = a.num_anchors;
  const int t_begin = blockIdx.x * kF32Chunk;
  if (t_begin >= T) return;
  const int sub = threadIdx.x / LPT, f0 = 4 * (threadIdx.x % LPT);
  const int64_t unit = unit_index(layer, kv, head, H);
  const float* src_pool = static_cast<const float*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]);
  float* dst_pool = static_cast<float*>(const_cast<void*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]));
  const float* wrow = a.weights + (int64_t)(lrel * 2 + kv) * Ts * V;
  const bool rot = ROPE && kv == 0;  // uniform over the workgroup
  const bool shift = rot && a.dst_position != a.src_position;
  const int style = a.pv.rope.style;
  if (rot) {
    rope_table(a.pv.rope, D, (double)a.dst_position - (double)a.src_position, s_rope, s_rope + D / 2);
    rope_table(a.pv.rope, D, (double)a.dst_position, s_rope + D, s_rope + 3 * D / 2);
    __syncthreads();
  }
  f32x4 acc[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) acc[p] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (t_begin < Ts) {
    for (int v = 0; v < V; ++v) {
      const int r = a.rank[v];
      __syncthreads();
      const float* bv = a.basis[v] + unit * (int64_t)r * D;
      for (int e = threadIdx.x; e < r * D; e += kAnchorThreads) {
        float x = bv[e];
        if (rot) {  // B_v R(pd)^T
          const int k = e / D, f = e - k * D, i = rope_pair(style, D, f);
          x = rope_rotated(rope_first(style, D, f), x, bv[k * D + rope_partner(style, D, f)], s_rope[D + i],
                           s_rope[3 * D / 2 + i]);
        }
        s_b[e] = x;
      }
      __syncthreads();
      const float* coef = static_cast<const float*>(a.coef[v]) + unit * (int64_t)a.tokens[v] * r;
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        const int t = t_begin + p * TPP + sub;
        if (t >= Ts) continue;
        const float w = wrow[(int64_t)t * V + v];
        const float* crow = coef + (int64_t)t * r;
        f32x4 s = {0.f, 0.f, 0.f, 0.f};
        for (int k = 0; k < r; ++k) {
          const float c = crow[k];
          const f32x4 b = *reinterpret_cast<const f32x4*>(&s_b[k * D + f0]);
          s[0] = fmaf(c, b[0], s[0]);
          s[1] = fmaf(c, b[1], s[1]);
          s[2] = fmaf(c, b[2], s[2]);
          s[3] = fmaf(c, b[3], s[3]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[p][i] = fmaf(w, s[i], acc[p][i]);
      }
    }
  }
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int t = t_begin + p * TPP + sub;
    if (t >= T) continue;
    const int64_t so = row_offset(a.pv, a.src_table, a.src_offset, t, head);
    const int64_t dof = row_offset(a.pv, a.dst_table, a.dst_offset, t, head);
    if (so < 0 || dof < 0) continue;
    f32x4 x = *reinterpret_cast<const f32x4*>(src_pool + so + f0);
    if (ROPE && shift) {  // the source rotated by pd - ps
      const f32x4 y = *reinterpret_cast<const f32x4*>(src_pool + so + (rope_partner(style, D, f0) & ~3));
      f32x4 xr;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int f = f0 + j, i = rope_pair(style, D, f);
        const float partner = style == KVC_ROPE_HALF ? y[j] : x[j ^ 1];
        xr[j] = rope_rotated(rope_first(style, D, f), x[j], partner, s_rope[i], s_rope[D / 2 + i]);
      }
      x = xr;
    }
    f32x4 o = x;
    if (t < Ts) {
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = x[i] + acc[p][i];
    }
    *reinterpret_cast<f32x4*>(dst_pool + dof + f0) = o;
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Resident-basis kernels, bf16: the bases of every anchor of one unit sit in LDS at once (the anchors' ranks cut
// into 32-rank chunks, at most kResMaxChunks of them and 160 KB as hi/lo), so a wave streams its tokens through
// all anchors in one pass, the way kvc_apply streams them through one state.  Used whenever the chunks fit; the
// kernels above (one anchor's basis at a time) take the rest.
// ---------------------------------------------------------------------------------------------------------------

constexpr int kResWaves = 8;
constexpr int kResThreads = kResWaves * kWave;
// 16-token tiles per wave: 16 for the anchored apply and the gate (2048 tokens per workgroup), 8 for the weights,
// whose per-tile distances stay in registers (1024 tokens)
constexpr int kResTiles = 16, kResDistTiles = 8;
constexpr int kResChunk = kResWaves * kResTiles * 16;
constexpr int kResDistChunk = kResWaves * kResDistTiles * 16;
int anchor_resident_chunk_tokens() { return kResDistChunk; }  // the shorter chunk (more partials)
constexpr size_t kResMaxLds = 160 * 1024;

// LDS holds hi [D][32 NC] then lo; the 16-byte granule (8 ranks) q of feature row f sits at q ^ res_swz(f), a
// swizzle inside each 32-rank chunk that spreads the staging stores (consecutive f) and the fragment reads (the
// features of one MFMA tile) over the banks.
__device__ __forceinline__ int res_swz(int f) { return ((f >> 1) & 1) | (((f >> 3) & 1) << 1); }

__device__ __forceinline__ bf16x8 res_frag(const uint16_t* s, int kpt, int f, int c, int g) {
  return as_bf16x8(*reinterpret_cast<const u32x4*>(s + f * kpt + 8 * (4 * c + (g ^ res_swz(f)))));
}

// The resident kernels fill the LDS with bases, so per-workgroup tables live in registers and are read with lane
// shuffles (no global load, hence no wait on the wave's earlier stores, inside the tile loop).
//
// Block ids of the chunk's logical blocks lb0 .. lb0 + 127: lane k holds those of lb0 + k (e0) and lb0 + 64 + k (e1).
// A chunk spanning more blocks (block sizes below 9 at 1024 tokens) reads the table from global memory instead.
struct LaneTable {
  int32_t e0, e1;
  int lb0;
  bool regs;
};
__device__ __forceinline__ int lane_lblock(const PoolView& pv, int p) {
  return pv.block_shift >= 0 ? p >> pv.block_shift : p / pv.block_size;
}
__device__ __forceinline__ LaneTable lane_table(const PoolView& pv, const int32_t* __restrict__ table, int off,
                                                int t_begin, int t_end, int lane) {
  LaneTable lt;
  lt.lb0 = lane_lblock(pv, off + t_begin);
  const int nb = lane_lblock(pv, off + t_end - 1) - lt.lb0 + 1;  // the host checked these lie in the table row
  lt.regs = nb <= 2 * kWave;
  const int i0 = lane, i1 = lane + kWave;
  lt.e0 = lt.regs && i0 < nb ? (table ? table[lt.lb0 + i0] : lt.lb0 + i0) : -1;
  lt.e1 = lt.regs && i1 < nb ? (table ? table[lt.lb0 + i1] : lt.lb0 + i1) : -1;
  return lt;
}
// Row offset of token t (-1 when absent or out of range).  Call from converged control flow (lane shuffles).
__device__ __forceinline__ int64_t lane_row_offset(const PoolView& pv, const LaneTable& lt,
                                                   const int32_t* __restrict__ table, int off, int t, bool valid,
                                                   int head) {
  const int p = off + t, lb = lane_lblock(pv, p), k = lb - lt.lb0;
  const int a0 = __shfl(lt.e0, k & (kWave - 1), kWave), a1 = __shfl(lt.e1, k & (kWave - 1), kWave);
  if (!valid) return -1;
  const int32_t blk = lt.regs ? (k < kWave ? a0 : a1) : (table ? table[lb] : lb);
  if (blk < 0 || blk >= pv.num_blocks) return -1;
  return (int64_t)blk * pv.block_stride + (int64_t)(p - lb * pv.block_size) * pv.token_stride +
         (int64_t)head * pv.head_stride;
}

// Every chunk of unit `unit` into LDS: a thread takes (feature f, eight ranks of one chunk); the lanes of a wave
// take 64 consecutive features, so each of the eight 4-byte loads is one coalesced 256-byte row segment.  A thread
// always takes the same feature (kResThreads is a multiple of D).  ROPE with `rot`: each basis row is rotated like a
// key row at position `pos` (B R(pos)^T), from the partner feature's values and one angle per thread.
template <int D, bool ROPE = false>
__device__ __forceinline__ void stage_stacked(const AnchorArgs& a, int64_t unit, uint16_t* s_hi, uint16_t* s_lo,
                                              bool rot = false, double pos = 0.0) {
  static_assert(kResThreads % D == 0, "one feature per thread");
  const int NC = a.num_chunks, kpt = 32 * NC, items = D * 4 * NC;
  const int style = a.pv.rope.style;
  const int fth = (int)threadIdx.x % D;
  float rc = 1.0f, rs = 0.0f;
  if (ROPE && rot) {
    double sn, cs;
    sincos(pos * a.pv.rope.inv_freq[rope_pair(style, D, fth)], &sn, &cs);
    rc = (float)cs;
    rs = (float)sn;
  }
  for (int base = 0; base < items; base += kResThreads) {
    const int idx = base + (int)threadIdx.x;
    if (idx >= items) break;  // whole waves: items is a multiple of 64
    const int q = __builtin_amdgcn_readfirstlane(idx / D);  // the same for the 64 lanes of a wave
    const int f = idx - q * D;
    const int c = q >> 2, v = a.chunk_anchor[c], k0 = a.chunk_k0[c] + 8 * (q & 3), r = a.rank[v];
    const float* b = a.basis[v] + unit * (int64_t)r * D + f;
    float x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = k0 + e < r ? b[(int64_t)(k0 + e) * D] : 0.0f;
    if (ROPE && rot) {
      const float* bp = a.basis[v] + unit * (int64_t)r * D + rope_partner(style, D, f);
      const bool first = rope_first(style, D, f);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        x[e] = rope_rotated(first, x[e], k0 + e < r ? bp[(int64_t)(k0 + e) * D] : 0.0f, rc, rs);
    }
    u32x4 hi, lo;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t hh, ll;
      split_bf16x2(x[2 * p], x[2 * p + 1], hh, ll);
      hi[p] = hh;
      lo[p] = ll;
    }
    const int off = f * kpt + 8 * ((q & ~3) | ((q & 3) ^ res_swz(f)));
    *reinterpret_cast<u32x4*>(s_hi + off) = hi;
    *reinterpret_cast<u32x4*>(s_lo + off) = lo;
  }
}

// Eq. 8 with every anchor resident: per 16-token tile the accumulator starts from the source rows in fp32 and
// takes w_v[t] (A_v[t, chunk c] B_v[chunk c]) over all chunks (the bf16 coefficients are exact MFMA operands against
// the basis hi/lo, two MFMAs per fragment, and the product is scaled by the token's weight in fp32), then one
// rounding.
// ROPE: keys of a rotary cache, C_dst = R(pd - ps) C_src + sum_v w_v A_v (B_v R(pd)^T) (bases staged rotated, the
// source rotated in the accumulator; rows past T_s get the rotated source).
template <int D, bool ROPE>
__global__ __launch_bounds__(kResThreads) void apply_anchored_res_bf16(AnchorArgs a) {
  constexpr int MT = D / 16, NQ = D / 32, NCM = kResMaxChunks;
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  const int NC = a.num_chunks, kpt = 32 * NC;
  uint16_t* s_hi = reinterpret_cast<uint16_t*>(anchor_lds);
  uint16_t* s_lo = s_hi + D * kpt;

  const int lrel = blockIdx.z, layer = a.layer_begin + lrel;
  const int H = a.pv.num_kv_heads;
  const int kv = blockIdx.y / H, head = blockIdx.y - kv * H;
  const int T = a.num_tokens, Ts = a.num_weighted, V = a.num_anchors;
  const int t_begin = blockIdx.x * kResChunk;
  if (t_begin >= T) return;  // whole workgroup
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave, g = lane >> 4, n = lane & 15;
  const int64_t unit = unit_index(layer, kv, head, H);
  const uint16_t* src_pool = static_cast<const uint16_t*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]);
  uint16_t* dst_pool = static_cast<uint16_t*>(const_cast<void*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]));
  const float* wrow = a.weights + (int64_t)(lrel * 2 + kv) * Ts * V;
  const bool rope = ROPE && kv == 0;  // uniform over the workgroup
  const int style = a.pv.rope.style;
  const bool shift = rope && a.dst_position != a.src_position;
  float tc = 1.0f, ts = 0.0f;  // this lane's entry of the wave's angle table for pd - ps
  if (shift) rope_wave_table<D>(a.pv.rope, (double)a.dst_position - (double)a.src_position, lane, tc, ts);
  if (t_begin < Ts) {  // whole workgroup
    stage_stacked<D, ROPE>(a, unit, s_hi, s_lo, rope, (double)a.dst_position);
    __syncthreads();
  }
  const int t_end = min(T, t_begin + kResChunk);
  const LaneTable lts = lane_table(a.pv, a.src_table, a.src_offset, t_begin, t_end, lane);
  const LaneTable ltd = lane_table(a.pv, a.dst_table, a.dst_offset, t_begin, t_end, lane);

  struct Tile {
    u32x4 raw[NQ];
    u32x4 cw[NCM];
    float w[NCM];
    int64_t dof;
  };
  auto load_tile = [&](int j, Tile& tl) __attribute__((always_inline)) {
    const int t = t_begin + (j * kResWaves + wave) * 16 + n;
    const bool valid = t < T, crow = t < Ts;
    const int64_t so = lane_row_offset(a.pv, lts, a.src_table, a.src_offset, t, valid, head);
    // a row whose source block id is out of range is neither read nor written
    const int64_t dof = lane_row_offset(a.pv, ltd, a.dst_table, a.dst_offset, t, valid, head);
    tl.dof = so >= 0 ? dof : -1;
    load_row_segments<NQ>(src_pool, so, g, tl.raw);
#pragma unroll
    for (int c = 0; c < NCM; ++c) {
      tl.cw[c] = u32x4{0u, 0u, 0u, 0u};
      tl.w[c] = 0.0f;
      if (c < NC && crow) {
        const int v = a.chunk_anchor[c], r = a.rank[v];
        const uint16_t* coef = static_cast<const uint16_t*>(a.coef[v]) + unit * (int64_t)a.tokens[v] * r;
        tl.cw[c] = load_coef8(coef, r, t, a.chunk_k0[c] + 8 * g);
        tl.w[c] = wrow[(int64_t)t * V + v];
      }
    }
  };
  // the corrected (or copied) rows of tile j, ready to store
  auto finish_tile = [&](int j, const Tile& tl, u32x4* outw) __attribute__((always_inline)) {
    const int t0 = t_begin + (j * kResWaves + wave) * 16, t = t0 + n;
    if (t0 < Ts || shift) {  // uniform over the wave
      f32x4 acc[MT];
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        acc[2 * q] = f32x4{bf16_lo_to_f32(tl.raw[q][0]), bf16_hi_to_f32(tl.raw[q][0]),
                           bf16_lo_to_f32(tl.raw[q][1]), bf16_hi_to_f32(tl.raw[q][1])};
        acc[2 * q + 1] = f32x4{bf16_lo_to_f32(tl.raw[q][2]), bf16_hi_to_f32(tl.raw[q][2]),
                               bf16_lo_to_f32(tl.raw[q][3]), bf16_hi_to_f32(tl.raw[q][3])};
      }
      if (ROPE && shift) rope_rotate_rows_wave<D>(acc, style, g, tc, ts);
#pragma unroll
      for (int c = 0; c < NCM; ++c) {
        if (t0 >= Ts) break;  // uniform: a tile past the coverage takes the rotated source only
        if (c >= NC) break;
        int kc = kpt;
        asm volatile("" : "+s"(kc));  // keeps the fragment reads in this chunk's step (not hoisted out of the tiles)
        // the chunk's reconstruction from the exact bf16 coefficients (basis hi/lo), then scaled by the lane's
        // token weight in fp32: lane (g, n) holds rows 4g .. 4g + 3 of token n's column
        const bf16x8 cb = as_bf16x8(tl.cw[c]);
        const float wc = tl.w[c];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int f = mfma_row_feature(mt, n);
          const bf16x8 fl = res_frag(s_lo, kc, f, c, g), fh = res_frag(s_hi, kc, f, c, g);
          f32x4 p = mfma16x16x32(fl, cb, f32x4{0.f, 0.f, 0.f, 0.f});
          p = mfma16x16x32(fh, cb, p);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[mt][e] = fmaf(wc, p[e], acc[mt][e]);
        }
      }
      // rows past T_s have a zero correction: the rotated source with a shift, else bit copies
      const bool crow = t < Ts || shift;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const f32x4 x = acc[2 * q], y = acc[2 * q + 1];
        const u32x4 c = {pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(y[0], y[1]),
                         pack_bf16x2(y[2], y[3])};
        outw[q] = crow ? c : tl.raw[q];
      }
    } else {
#pragma unroll
      for (int q = 0; q < NQ; ++q) outw[q] = tl.raw[q];
    }
  };

  // the next tile's loads are issued before this tile's stores, so waiting for them never waits for the stores
  if (t_begin + wave * 16 >= T) return;  // whole wave
  Tile cur;
  load_tile(0, cur);
  for (int j = 0; j < kResTiles; ++j) {
    u32x4 outw[NQ];
    finish_tile(j, cur, outw);
    const int64_t dof = cur.dof;
    const bool more = j + 1 < kResTiles && t_begin + ((j + 1) * kResWaves + wave) * 16 < T;  // uniform
    if (more) load_tile(j + 1, cur);
    if (dof >= 0) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) *reinterpret_cast<u32x4*>(dst_pool + dof + 32 * q + 8 * g) = outw[q];
    }
    if (!more) break;
  }
}

// Distances with every anchor of one head resident: a workgroup covers 1024 tokens of one (layer, K/V) and walks
// the heads, staging each head's anchors once.  Per tile and anchor the reconstruction A_v B_v accumulates over the
// anchor's chunks (bf16 coefficients are exact MFMA operands, B as hi/lo), then |x - recon| (weights) or
// (x - recon)^2 (gate) is summed over the row.  Lane (g, n) keeps the sums of anchors v = 4u + g of its tiles'
// token n in registers across heads.
// ROPE (weights): keys of a rotary cache are compared in canonical coordinates, R(-ps) C_src (the bases are canonical).
template <int D, bool GATE, bool ROPE>
__global__ __launch_bounds__(kResThreads) void anchor_dist_res_bf16(AnchorArgs a) {
  constexpr int MT = D / 16, NQ = D / 32, NCM = kResMaxChunks, TPW = GATE ? kResTiles : kResDistTiles;
  constexpr int CH = kResWaves * TPW * 16;  // tokens per workgroup
  static_assert(KVC_MAX_ANCHORS <= 16, "four anchors per lane group");
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  const int NC = a.num_chunks, kpt = 32 * NC;
  uint16_t* s_hi = reinterpret_cast<uint16_t*>(anchor_lds);
  uint16_t* s_lo = s_hi + D * kpt;

  const int lrel = blockIdx.z, layer = a.layer_begin + lrel;
  const int kv = GATE ? 1 : blockIdx.y;
  const int H = a.pv.num_kv_heads, V = a.num_anchors;
  // the gate reads value rows only, so its launch spreads the heads over the grid (one head per workgroup); the
  // weights need every head of a token in one workgroup (the mean runs over the whole layer row)
  const int h_lo = GATE ? (int)blockIdx.y : 0, h_hi = GATE ? h_lo + 1 : H;
  const int Tl = a.num_weighted;
  const int t_begin = blockIdx.x * CH;
  if (t_begin >= Tl) return;  // whole workgroup
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave, g = lane >> 4, n = lane & 15;
  const uint16_t* pool = static_cast<const uint16_t*>(kv ? a.layers.v[lrel] : a.layers.k[lrel]);

  // per-tile distances (the weights need each token's); the gate only needs their sum, so it keeps one set
  constexpr int ND = GATE ? 1 : TPW;
  float dist[ND][4];
#pragma unroll
  for (int j = 0; j < ND; ++j)
#pragma unroll
    for (int u = 0; u < 4; ++u) dist[j][u] = 0.0f;
  const bool rot = ROPE && !GATE && kv == 0;  // uniform over the workgroup
  const int style = a.pv.rope.style;
  float tc = 1.0f, ts = 0.0f;  // this lane's entry of the wave's angle table for -ps
  if (rot) rope_wave_table<D>(a.pv.rope, -(double)a.src_position, lane, tc, ts);
  const LaneTable lts = lane_table(a.pv, a.src_table, a.src_offset, t_begin, min(Tl, t_begin + CH), lane);

  struct Tile {
    u32x4 raw[NQ];
    u32x4 cw[NCM];
  };
  for (int h = h_lo; h < h_hi; ++h) {
    const int64_t unit = unit_index(layer, kv, h, H);
    if (h > h_lo) __syncthreads();  // every wave is done with the previous head's bases
    stage_stacked<D>(a, unit, s_hi, s_lo);
    __syncthreads();
    auto load_tile = [&](int j, Tile& tl) __attribute__((always_inline)) {
      const int t = t_begin + (j * kResWaves + wave) * 16 + n;
      const bool valid = t < Tl;
      load_row_segments<NQ>(pool, lane_row_offset(a.pv, lts, a.src_table, a.src_offset, t, valid, h), g, tl.raw);
#pragma unroll
      for (int c = 0; c < NCM; ++c) {
        tl.cw[c] = u32x4{0u, 0u, 0u, 0u};
        if (c < NC && valid) {
          const int v = a.chunk_anchor[c], r = a.rank[v];
          const uint16_t* coef = static_cast<const uint16_t*>(a.coef[v]) + unit * (int64_t)a.tokens[v] * r;
          tl.cw[c] = load_coef8(coef, r, t, a.chunk_k0[c] + 8 * g);
        }
      }
    };
    // dist[0] always belongs to the current tile (the weights): the array is rotated by one after every tile (static
    // register indices with a rolled tile loop), so after TPW tiles dist[j] is tile j's again
#pragma unroll 1
    for (int j = 0; j < TPW; ++j) {
      const int t0 = t_begin + (j * kResWaves + wave) * 16;
      if (t0 < Tl) {  // uniform over the wave
        Tile cur;
        load_tile(j, cur);
        const bool valid = t0 + n < Tl;
        // ROPE: the canonical source rows R(-ps) C_src in fp32 (the rotary instantiation only)
        f32x4 xv[ROPE ? MT : 1];
        if constexpr (ROPE) {
#pragma unroll
          for (int q = 0; q < NQ; ++q) {
            xv[2 * q] = f32x4{bf16_lo_to_f32(cur.raw[q][0]), bf16_hi_to_f32(cur.raw[q][0]),
                              bf16_lo_to_f32(cur.raw[q][1]), bf16_hi_to_f32(cur.raw[q][1])};
            xv[2 * q + 1] = f32x4{bf16_lo_to_f32(cur.raw[q][2]), bf16_hi_to_f32(cur.raw[q][2]),
                                  bf16_lo_to_f32(cur.raw[q][3]), bf16_hi_to_f32(cur.raw[q][3])};
          }
          if (rot) rope_rotate_rows_wave<D>(xv, style, g, tc, ts);
        }
        f32x4 acc[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NCM; ++c) {
          if (c < NC) {  // a guard, not a break: the loop must unroll fully (cw stays in registers)
          int kc = kpt;
          asm volatile("" : "+s"(kc));  // keeps the fragment reads in this chunk's step
          const bf16x8 cb = as_bf16x8(cur.cw[c]);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const int f = mfma_row_feature(mt, n);
            acc[mt] = mfma16x16x32(res_frag(s_lo, kc, f, c, g), cb, acc[mt]);
            acc[mt] = mfma16x16x32(res_frag(s_hi, kc, f, c, g), cb, acc[mt]);
          }
          if (a.chunk_last[c]) {  // uniform: anchor v's reconstruction is complete
            float s = 0.0f;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const uint32_t w = cur.raw[q][e >> 1];
                const float x = ROPE ? xv[ROPE ? 2 * q + (e >> 2) : 0][e & 3]
                                     : ((e & 1) ? bf16_hi_to_f32(w) : bf16_lo_to_f32(w));
                const float diff = x - acc[2 * q + (e >> 2)][e & 3];
                s += GATE ? diff * diff : fabsf(diff);
              }
            }
            s += __shfl_xor(s, 16, kWave);
            s += __shfl_xor(s, 32, kWave);
            s = valid ? s : 0.0f;
            const int v = a.chunk_anchor[c];
#pragma unroll
            for (int u = 0; u < 4; ++u) dist[0][u] += (v == 4 * u + g) ? s : 0.0f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
          }
        }
      }
      if constexpr (!GATE) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float d0 = dist[0][u];
#pragma unroll
          for (int jj = 0; jj + 1 < TPW; ++jj) dist[jj][u] = dist[jj + 1][u];
          dist[TPW - 1][u] = d0;
        }
      }
    }
  }
  __syncthreads();  // the bases are no longer read: LDS now holds the per-token (or per-wave) sums
  float* s_d = reinterpret_cast<float*>(anchor_lds);
  if (GATE) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      float p = dist[0][u];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) p += __shfl_xor(p, o, kWave);
      if (n == 0 && 4 * u + g < V) s_d[wave * V + 4 * u + g] = p;
    }
    __syncthreads();
    if (threadIdx.x < V) {
      const int v = threadIdx.x;
      float s = 0.0f;
      for (int w = 0; w < kResWaves; ++w) s += s_d[w * V + v];
      a.gate_partials[((int64_t)lrel * a.gate_chunks + blockIdx.x * gridDim.y + blockIdx.y) * V + v] = s;
    }
  } else {
#pragma unroll
    for (int j = 0; j < ND; ++j) {
      const int tok = (j * kResWaves + wave) * 16 + n;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (4 * u + g < V) s_d[tok * V + 4 * u + g] = dist[j][u];
    }
    __syncthreads();
    const float inv_feat = 1.0f / (float)(H * D);
    for (int tok = threadIdx.x; tok < CH; tok += kResThreads) {
      const int t = t_begin + tok;
      if (t >= Tl) break;
      float dmin = INFINITY;
      for (int v = 0; v < V; ++v) dmin = fminf(dmin, s_d[tok * V + v] * inv_feat);
      float sum = 0.0f;
      for (int v = 0; v < V; ++v) sum += __expf(-(s_d[tok * V + v] * inv_feat - dmin) * a.inv_temperature);
      const float inv = 1.0f / sum;
      float* wout = a.weights + ((int64_t)(lrel * 2 + kv) * Tl + t) * V;
      for (int v = 0; v < V; ++v) wout[v] = __expf(-(s_d[tok * V + v] * inv_feat - dmin) * a.inv_temperature) * inv;
    }
  }
}

// ---------------------------------------------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------------------------------------------

// which: 0 weights, 1 apply, 2 gate.  Every layout ends with room for the rotary angle tables (4 x 64 floats).
size_t anchor_lds_bytes(int D, int max_rank, kvc_dtype dtype, int which) {
  const int V = KVC_MAX_ANCHORS;
  const size_t rope = 4 * 64 * sizeof(float);
  if (dtype == KVC_BF16) {
    const size_t kp = 32 * (size_t)((max_rank + 31) / 32);
    const size_t basis = 4 * (size_t)D * kp * sizeof(uint16_t);  // two buffers of hi/lo
    if (which == 1) return basis + rope;
    return basis + (size_t)(which == 2 ? kAnchorWaves : kAnchorChunk) * V * sizeof(float) + rope;
  }
  const size_t basis = (size_t)max_rank * D * sizeof(float);
  if (which == 1) return basis + rope;
  return basis + (size_t)(which == 2 ? kAnchorThreads / (D / 4) : kF32Chunk) * V * sizeof(float) + rope;
}

template <typename K>
static hipError_t launch_with_lds(K kernel, dim3 grid, size_t lds, const AnchorArgs& a, hipStream_t stream,
                                  int threads = kAnchorThreads) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kernel, grid, dim3(threads), lds, stream, a);
  return hipGetLastError();
}

// The chunk map of the resident-basis kernels (bf16); false when the anchors' chunks do not fit.
static bool plan_resident(AnchorArgs& a) {
  int nc = 0;
  for (int v = 0; v < a.num_anchors; ++v) {
    const int ks = std::max(1, (a.rank[v] + 31) / 32);
    for (int k = 0; k < ks; ++k) {
      if (nc == kResMaxChunks) return false;
      a.chunk_anchor[nc] = v;
      a.chunk_k0[nc] = 32 * k;
      a.chunk_last[nc] = k == ks - 1;
      ++nc;
    }
  }
  a.num_chunks = nc;
  return (size_t)a.pv.head_dim * 32 * nc * 2 * sizeof(uint16_t) <= kResMaxLds;
}

// which: 0 weights, 1 apply, 2 gate
static size_t res_lds_bytes(const AnchorArgs& a, int which) {
  const size_t basis = (size_t)a.pv.head_dim * 32 * a.num_chunks * 2 * sizeof(uint16_t);
  const size_t sums = which == 0   ? (size_t)kResDistChunk * a.num_anchors * sizeof(float)
                      : which == 2 ? (size_t)kResWaves * a.num_anchors * sizeof(float)
                                   : 0;
  return std::max(basis, sums);
}

template <int D, bool GATE, bool ROPE>
static hipError_t launch_dist_bf16(const AnchorArgs& a, dim3 grid, size_t lds, hipStream_t stream) {
  switch ((a.max_rank + 31) / 32) {
    case 1: return launch_with_lds(anchor_dist_bf16<D, 1, GATE, ROPE>, grid, lds, a, stream);
    case 2: return launch_with_lds(anchor_dist_bf16<D, 2, GATE, ROPE>, grid, lds, a, stream);
    case 3: return launch_with_lds(anchor_dist_bf16<D, 3, GATE, ROPE>, grid, lds, a, stream);
    default: return launch_with_lds(anchor_dist_bf16<D, 4, GATE, ROPE>, grid, lds, a, stream);
  }
}

template <int D, bool ROPE>
static hipError_t launch_anchored_bf16(const AnchorArgs& a, dim3 grid, size_t lds, hipStream_t stream) {
  switch ((a.max_rank + 31) / 32) {
    case 1: return launch_with_lds(apply_anchored_bf16<D, 1, ROPE>, grid, lds, a, stream);
    case 2: return launch_with_lds(apply_anchored_bf16<D, 2, ROPE>, grid, lds, a, stream);
    case 3: return launch_with_lds(apply_anchored_bf16<D, 3, ROPE>, grid, lds, a, stream);
    default: return launch_with_lds(apply_anchored_bf16<D, 4, ROPE>, grid, lds, a, stream);
  }
}

template <bool ROPE>
static hipError_t launch_weights_variant(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream) {
  const int D = a.pv.head_dim;
  const size_t lds = anchor_lds_bytes(D, a.max_rank, dtype, 0);
  if (dtype == KVC_BF16) {
    AnchorArgs r = a;
    if (plan_resident(r)) {
      dim3 grid((a.num_weighted + kResDistChunk - 1) / kResDistChunk, 2, a.num_layers);
      const size_t rl = res_lds_bytes(r, 0);
      return D == 64 ? launch_with_lds(anchor_dist_res_bf16<64, false, ROPE>, grid, rl, r, stream, kResThreads)
                     : launch_with_lds(anchor_dist_res_bf16<128, false, ROPE>, grid, rl, r, stream, kResThreads);
    }
    dim3 grid((a.num_weighted + kAnchorChunk - 1) / kAnchorChunk, 2, a.num_layers);
    return D == 64 ? launch_dist_bf16<64, false, ROPE>(a, grid, lds, stream)
                   : launch_dist_bf16<128, false, ROPE>(a, grid, lds, stream);
  }
  dim3 grid((a.num_weighted + kF32Chunk - 1) / kF32Chunk, 2, a.num_layers);
  return D == 64 ? launch_with_lds(anchor_dist_f32<64, false, ROPE>, grid, lds, a, stream)
                 : launch_with_lds(anchor_dist_f32<128, false, ROPE>, grid, lds, a, stream);
}

hipError_t launch_anchor_weights(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream) {
  if (a.num_weighted == 0 || a.num_layers == 0) return hipSuccess;
  return a.pv.rope.style != KVC_ROPE_NONE ? launch_weights_variant<true>(a, dtype, stream)
                                          : launch_weights_variant<false>(a, dtype, stream);
}

// The gate reads value rows only, which carry no rotary encoding.
hipError_t launch_gate_distances(const AnchorArgs& args, kvc_dtype dtype, hipStream_t stream) {
  AnchorArgs a = args;
  a.pv.rope.style = KVC_ROPE_NONE;
  const int D = a.pv.head_dim;
  const size_t lds = anchor_lds_bytes(D, a.max_rank, dtype, 2);
  hipError_t e;
  dim3 grid(a.gate_chunks, 1, a.num_layers);
  if (dtype == KVC_BF16 && plan_resident(a)) {
    // one partial per (layer, 2048-token chunk, KV head): within what the workspace query sizes (1024-token chunks)
    grid.x = (a.num_weighted + kResChunk - 1) / kResChunk;
    grid.y = a.pv.num_kv_heads;
    a.gate_chunks = (int)(grid.x * grid.y);
    const size_t rl = res_lds_bytes(a, 2);
    e = D == 64 ? launch_with_lds(anchor_dist_res_bf16<64, true, false>, grid, rl, a, stream, kResThreads)
                : launch_with_lds(anchor_dist_res_bf16<128, true, false>, grid, rl, a, stream, kResThreads);
  } else if (dtype == KVC_BF16) {
    // one partial per (layer, 512-token chunk, KV head), as the workspace query sizes
    grid.y = a.pv.num_kv_heads;
    a.gate_chunks = (int)(grid.x * grid.y);
    e = D == 64 ? launch_dist_bf16<64, true, false>(a, grid, lds, stream)
                : launch_dist_bf16<128, true, false>(a, grid, lds, stream);
  } else {
    e = D == 64 ? launch_with_lds(anchor_dist_f32<64, true, false>, grid, lds, a, stream)
                : launch_with_lds(anchor_dist_f32<128, true, false>, grid, lds, a, stream);
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(gate_finish, dim3(1), dim3(kAnchorThreads), 0, stream, a);
  return hipGetLastError();
}

template <bool ROPE>
static hipError_t launch_anchored_variant(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream) {
  const int D = a.pv.head_dim;
  const size_t lds = anchor_lds_bytes(D, a.max_rank, dtype, 1);
  if (dtype == KVC_BF16) {
    AnchorArgs r = a;
    if (plan_resident(r)) {
      dim3 grid((a.num_tokens + kResChunk - 1) / kResChunk, 2 * a.pv.num_kv_heads, a.num_layers);
      const size_t rl = res_lds_bytes(r, 1);
      return D == 64 ? launch_with_lds(apply_anchored_res_bf16<64, ROPE>, grid, rl, r, stream, kResThreads)
                     : launch_with_lds(apply_anchored_res_bf16<128, ROPE>, grid, rl, r, stream, kResThreads);
    }
    dim3 grid((a.num_tokens + kAnchoredChunk - 1) / kAnchoredChunk, 2 * a.pv.num_kv_heads, a.num_layers);
    return D == 64 ? launch_anchored_bf16<64, ROPE>(a, grid, lds, stream)
                   : launch_anchored_bf16<128, ROPE>(a, grid, lds, stream);
  }
  dim3 grid((a.num_tokens + kF32Chunk - 1) / kF32Chunk, 2 * a.pv.num_kv_heads, a.num_layers);
  return D == 64 ? launch_with_lds(apply_anchored_f32<64, ROPE>, grid, lds, a, stream)
                 : launch_with_lds(apply_anchored_f32<128, ROPE>, grid, lds, a, stream);
}

hipError_t launch_apply_anchored(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream) {
  if (a.num_tokens == 0 || a.num_layers == 0) return hipSuccess;
  return a.pv.rope.style != KVC_ROPE_NONE ? launch_anchored_variant<true>(a, dtype, stream)
                                          : launch_anchored_variant<false>(a, dtype, stream);
}

}  // namespace kvc
