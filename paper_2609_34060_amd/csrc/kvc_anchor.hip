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

// B^T of one unit staged as bf16 hi/lo, zero-padded to KP = 32 KSM ranks: s[f * KP + k] = split(B[k][f]).  The
// float4 loads of the next basis are issued into registers before the current one is used (load), and written to
// the other LDS buffer one step later (store), so a workgroup waits once per basis at its barrier.
template <int D, int KSM>
struct BasisStager {
  static constexpr int KP = 32 * KSM;
  static constexpr int N4 = D * KP / (kAnchorThreads * 4);  // float4 per thread
  f32x4 v[N4];
  __device__ __forceinline__ void load(const float* basis, int r) {
#pragma unroll
    for (int i = 0; i < N4; ++i) {
      const int e = 4 * ((int)threadIdx.x + i * kAnchorThreads);
      const int k = e / D, f = e - k * D;
      v[i] = k < r ? *reinterpret_cast<const f32x4*>(basis + k * D + f) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
  __device__ __forceinline__ void store(uint16_t* s_hi, uint16_t* s_lo) const {
#pragma unroll
    for (int i = 0; i < N4; ++i) {
      const int e = 4 * ((int)threadIdx.x + i * kAnchorThreads);
      const int k = e / D, f = e - k * D;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        uint32_t hb, lb;
        split_bf16(v[i][c], hb, lb);
        s_hi[(f + c) * KP + k] = (uint16_t)hb;
        s_lo[(f + c) * KP + k] = (uint16_t)lb;
      }
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

template <int D, int KSM, bool GATE>
__global__ __launch_bounds__(kAnchorThreads) void anchor_dist_bf16(AnchorArgs a) {
  constexpr int MT = D / 16, NQ = D / 32, KP = 32 * KSM;
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  uint16_t* s_b = reinterpret_cast<uint16_t*>(anchor_lds);   // [2 buffers][hi, lo][D * KP]
  float* s_d = reinterpret_cast<float*>(s_b + 4 * D * KP);     // GATE: [waves][V]; else [chunk][V]

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

  BasisStager<D, KSM> stager;
  auto basis_of = [&](int hv) {
    const int h = hv / V, v = hv - h * V;
    return a.basis[v] + unit_index(layer, kv, h, H) * (int64_t)a.rank[v] * D;
  };
  stager.load(basis_of(0), a.rank[0]);
  for (int hv = 0; hv < H * V; ++hv) {
    const int h = hv / V, v = hv - h * V;
    const int r = a.rank[v], KS = (r + 31) / 32;
    uint16_t* s_hi = s_b + (hv & 1) * 2 * D * KP;
    uint16_t* s_lo = s_hi + D * KP;
    stager.store(s_hi, s_lo);
    __syncthreads();  // this basis is in LDS; the other buffer is no longer read (and s_d is initialised)
    if (hv + 1 < H * V) stager.load(basis_of(hv + 1), a.rank[(hv + 1) % V]);
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
      float s = 0.0f;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t w = raw[q][e >> 1];
          const float x = (e & 1) ? bf16_hi_to_f32(w) : bf16_lo_to_f32(w);
          const float diff = x - acc[2 * q + (e >> 2)][e & 3];
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
      a.gate_partials[((int64_t)lrel * a.gate_chunks + blockIdx.x) * V + v] = s;
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

template <int D, bool GATE>
__global__ __launch_bounds__(kAnchorThreads) void anchor_dist_f32(AnchorArgs a) {
  constexpr int LPT = D / 4, TPP = kAnchorThreads / LPT;
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  float* s_b = reinterpret_cast<float*>(anchor_lds);           // [max_rank][D]
  float* s_d = s_b + a.max_rank * D;                            // GATE: [TPP][V]; else [chunk][V]
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

// Gate: d_v = sqrt(sum of the partials of every (layer, chunk)) in a fixed order, fp64.
__global__ __launch_bounds__(kAnchorThreads) void gate_finish(AnchorArgs a) {
  const int v = threadIdx.x;
  if (v >= a.num_anchors) return;
  double s = 0.0;
  for (int64_t i = 0; i < (int64_t)a.num_layers * a.gate_chunks; ++i) s += (double)a.gate_partials[i * a.num_anchors + v];
  a.distances[v] = (float)sqrt(s);
}

// ---------------------------------------------------------------------------------------------------------------
// anchored apply, bf16: the correction of every anchor accumulates in registers over an outer loop on the anchors
// (one basis staging per anchor and workgroup), then C_src + correction is rounded once and stored
// ---------------------------------------------------------------------------------------------------------------

template <int D, int KSM>
__global__ __launch_bounds__(kAnchorThreads) void apply_anchored_bf16(AnchorArgs a) {
  constexpr int MT = D / 16, NQ = D / 32, TPW = kAnchoredTiles, KP = 32 * KSM;
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  uint16_t* s_b = reinterpret_cast<uint16_t*>(anchor_lds);  // [2 buffers][hi, lo][D * KP]

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

  f32x4 acc[TPW][MT];
#pragma unroll
  for (int j = 0; j < TPW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (t_begin < Ts) {  // whole workgroup
    BasisStager<D, KSM> stager;
    stager.load(a.basis[0] + unit * (int64_t)a.rank[0] * D, a.rank[0]);
    for (int v = 0; v < V; ++v) {
      const int r = a.rank[v], KS = (r + 31) / 32;
      uint16_t* s_hi = s_b + (v & 1) * 2 * D * KP;
      uint16_t* s_lo = s_hi + D * KP;
      stager.store(s_hi, s_lo);
      __syncthreads();  // this basis is in LDS; the other buffer is no longer read
      if (v + 1 < V) stager.load(a.basis[v + 1] + unit * (int64_t)a.rank[v + 1] * D, a.rank[v + 1]);
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
    load_row_segments<NQ>(src_pool, valid ? row_offset(a.pv, a.src_table, a.src_offset, t, head) : -1, g, raw);
    const int64_t dof = valid ? row_offset(a.pv, a.dst_table, a.dst_offset, t, head) : -1;
    u32x4 outw[NQ];
    const bool crow = t < Ts;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const f32x4 x = acc[j][2 * q], y = acc[j][2 * q + 1];
      const u32x4 c = {pack_bf16x2(bf16_lo_to_f32(raw[q][0]) + x[0], bf16_hi_to_f32(raw[q][0]) + x[1]),
                       pack_bf16x2(bf16_lo_to_f32(raw[q][1]) + x[2], bf16_hi_to_f32(raw[q][1]) + x[3]),
                       pack_bf16x2(bf16_lo_to_f32(raw[q][2]) + y[0], bf16_hi_to_f32(raw[q][2]) + y[1]),
                       pack_bf16x2(bf16_lo_to_f32(raw[q][3]) + y[2], bf16_hi_to_f32(raw[q][3]) + y[3])};
      outw[q] = crow ? c : raw[q];
    }
    if (dof >= 0) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) *reinterpret_cast<u32x4*>(dst_pool + dof + 32 * q + 8 * g) = outw[q];
    }
  }
}

// anchored apply, float32 (VALU): D / 4 lanes per token; the tokens of a workgroup accumulate over the anchors
template <int D>
__global__ __launch_bounds__(kAnchorThreads) void apply_anchored_f32(AnchorArgs a) {
  constexpr int LPT = D / 4, TPP = kAnchorThreads / LPT, NP = kF32Chunk / TPP;
  extern __shared__ __attribute__((aligned(16))) unsigned char anchor_lds[];
  float* s_b = reinterpret_cast<float*>(anchor_lds);  // [max_rank][D]
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
  f32x4 acc[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) acc[p] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (t_begin < Ts) {
    for (int v = 0; v < V; ++v) {
      const int r = a.rank[v];
      __syncthreads();
      for (int e = threadIdx.x; e < r * D; e += kAnchorThreads) s_b[e] = a.basis[v][unit * (int64_t)r * D + e];
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
    const f32x4 x = *reinterpret_cast<const f32x4*>(src_pool + so + f0);
    f32x4 o = x;
    if (t < Ts) {
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = x[i] + acc[p][i];
    }
    *reinterpret_cast<f32x4*>(dst_pool + dof + f0) = o;
  }
}

// ---------------------------------------------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------------------------------------------

// which: 0 weights, 1 apply, 2 gate
size_t anchor_lds_bytes(int D, int max_rank, kvc_dtype dtype, int which) {
  const int V = KVC_MAX_ANCHORS;
  if (dtype == KVC_BF16) {
    const size_t kp = 32 * (size_t)((max_rank + 31) / 32);
    const size_t basis = 4 * (size_t)D * kp * sizeof(uint16_t);  // two buffers of hi/lo
    if (which == 1) return basis;
    return basis + (size_t)(which == 2 ? kAnchorWaves : kAnchorChunk) * V * sizeof(float);
  }
  const size_t basis = (size_t)max_rank * D * sizeof(float);
  if (which == 1) return basis;
  return basis + (size_t)(which == 2 ? kAnchorThreads / (D / 4) : kF32Chunk) * V * sizeof(float);
}

template <typename K>
static hipError_t launch_with_lds(K kernel, dim3 grid, size_t lds, const AnchorArgs& a, hipStream_t stream) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kernel, grid, dim3(kAnchorThreads), lds, stream, a);
  return hipGetLastError();
}

template <int D, bool GATE>
static hipError_t launch_dist_bf16(const AnchorArgs& a, dim3 grid, size_t lds, hipStream_t stream) {
  switch ((a.max_rank + 31) / 32) {
    case 1: return launch_with_lds(anchor_dist_bf16<D, 1, GATE>, grid, lds, a, stream);
    case 2: return launch_with_lds(anchor_dist_bf16<D, 2, GATE>, grid, lds, a, stream);
    case 3: return launch_with_lds(anchor_dist_bf16<D, 3, GATE>, grid, lds, a, stream);
    default: return launch_with_lds(anchor_dist_bf16<D, 4, GATE>, grid, lds, a, stream);
  }
}

template <int D>
static hipError_t launch_anchored_bf16(const AnchorArgs& a, dim3 grid, size_t lds, hipStream_t stream) {
  switch ((a.max_rank + 31) / 32) {
    case 1: return launch_with_lds(apply_anchored_bf16<D, 1>, grid, lds, a, stream);
    case 2: return launch_with_lds(apply_anchored_bf16<D, 2>, grid, lds, a, stream);
    case 3: return launch_with_lds(apply_anchored_bf16<D, 3>, grid, lds, a, stream);
    default: return launch_with_lds(apply_anchored_bf16<D, 4>, grid, lds, a, stream);
  }
}

hipError_t launch_anchor_weights(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream) {
  if (a.num_weighted == 0 || a.num_layers == 0) return hipSuccess;
  const int D = a.pv.head_dim;
  const size_t lds = anchor_lds_bytes(D, a.max_rank, dtype, 0);
  if (dtype == KVC_BF16) {
    dim3 grid((a.num_weighted + kAnchorChunk - 1) / kAnchorChunk, 2, a.num_layers);
    return D == 64 ? launch_dist_bf16<64, false>(a, grid, lds, stream) : launch_dist_bf16<128, false>(a, grid, lds, stream);
  }
  dim3 grid((a.num_weighted + kF32Chunk - 1) / kF32Chunk, 2, a.num_layers);
  return D == 64 ? launch_with_lds(anchor_dist_f32<64, false>, grid, lds, a, stream)
                 : launch_with_lds(anchor_dist_f32<128, false>, grid, lds, a, stream);
}

hipError_t launch_gate_distances(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream) {
  const int D = a.pv.head_dim;
  const size_t lds = anchor_lds_bytes(D, a.max_rank, dtype, 2);
  hipError_t e;
  dim3 grid(a.gate_chunks, 1, a.num_layers);
  if (dtype == KVC_BF16) {
    e = D == 64 ? launch_dist_bf16<64, true>(a, grid, lds, stream) : launch_dist_bf16<128, true>(a, grid, lds, stream);
  } else {
    e = D == 64 ? launch_with_lds(anchor_dist_f32<64, true>, grid, lds, a, stream)
                : launch_with_lds(anchor_dist_f32<128, true>, grid, lds, a, stream);
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(gate_finish, dim3(1), dim3(kAnchorThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_apply_anchored(const AnchorArgs& a, kvc_dtype dtype, hipStream_t stream) {
  if (a.num_tokens == 0 || a.num_layers == 0) return hipSuccess;
  const int D = a.pv.head_dim;
  const size_t lds = anchor_lds_bytes(D, a.max_rank, dtype, 1);
  if (dtype == KVC_BF16) {
    dim3 grid((a.num_tokens + kAnchoredChunk - 1) / kAnchoredChunk, 2 * a.pv.num_kv_heads, a.num_layers);
    return D == 64 ? launch_anchored_bf16<64>(a, grid, lds, stream) : launch_anchored_bf16<128>(a, grid, lds, stream);
  }
  dim3 grid((a.num_tokens + kF32Chunk - 1) / kF32Chunk, 2 * a.pv.num_kv_heads, a.num_layers);
  return D == 64 ? launch_with_lds(apply_anchored_f32<64>, grid, lds, a, stream)
                 : launch_with_lds(apply_anchored_f32<128>, grid, lds, a, stream);
}

}  // namespace kvc
