// kvc_chain kernels: compose S1 = (A1, B1) = Delta_{j<-i} and S2 = (A2, B2) = Delta_{k<-j} into the rank-r_out
// truncated SVD of M = A1 B1 + A2 B2 (Eq. 6 then Eq. 7) without forming M.  With A = [A1 A2] (T x m, m = r1 + r2)
// and K = [B1; B2]^T (d x m), M = A K^T and M^T M = K (A^T A) K^T, so
//   cgram     H = A^T A from the coefficient rows (one pass over T; rows past a state's T are zero), partial per
//             token chunk.  bf16 coefficients are exact MFMA operands; fp32 ones use the bf16 hi/lo split.
//   assemble  G = K H K^T in fp64 (d x d), the Gram of M.
//   eig       the shared eigensolver: top r_out eigenvectors R of G, sigma = sqrt(lambda) -> out.basis, out.sigma.
//   ymat      Y = K^T R (m x r_out), so that the new coefficients are M R = A Y (operands staged in LDS).
//   cproj     A_out = A Y, a second pass over the coefficient rows on MFMA (Y as a bf16 hi/lo pair).
#include <utility>

#include "kvc_device.h"
#include "kvc_launch.h"

namespace kvc {

constexpr int kChainThreads = 256;
constexpr int kChainWaves = kChainThreads / kWave;

struct ChainUnit {
  int lrel, layer, kv, head;
  int64_t idx;  // unit index within the states
};

__device__ __forceinline__ ChainUnit chain_unit(const ChainArgs& a, int u) {
  ChainUnit c;
  const int H = a.first.num_kv_heads;
  c.lrel = u / (2 * H);
  int rem = u - c.lrel * 2 * H;
  c.kv = rem / H;
  c.head = rem - c.kv * H;
  c.layer = a.layer_begin + c.lrel;
  c.idx = unit_index(c.layer, c.kv, c.head, H);
  return c;
}

// Concatenated coefficient [A1 A2][t][l] as a float (0 outside either state's rows).
template <bool F32>
__device__ __forceinline__ float cat_coef(const ChainArgs& a, const void* A1, const void* A2, int t, int l) {
  const int r1 = a.first.rank, r2 = a.second.rank;
  if (l < r1) {
    if (t >= a.first.num_tokens) return 0.f;
    return F32 ? static_cast<const float*>(A1)[(int64_t)t * r1 + l]
               : bf16_lo_to_f32(static_cast<const uint16_t*>(A1)[(int64_t)t * r1 + l]);
  }
  l -= r1;
  if (l >= r2 || t >= a.second.num_tokens) return 0.f;
  return F32 ? static_cast<const float*>(A2)[(int64_t)t * r2 + l]
             : bf16_lo_to_f32(static_cast<const uint16_t*>(A2)[(int64_t)t * r2 + l]);
}

__device__ __forceinline__ float cat_basis(const ChainArgs& a, int64_t idx, int l, int f) {
  const int r1 = a.first.rank, d = a.first.head_dim;
  if (l < r1) return a.first.basis[(idx * r1 + l) * d + f];
  return a.second.basis[(idx * a.second.rank + (l - r1)) * d + f];
}

// ---------------------------------------------------------------------------------------------------------------
// cgram: partial H over a token chunk, tiles on or above the diagonal
// ---------------------------------------------------------------------------------------------------------------

template <int FT, bool F32>
__global__ __launch_bounds__(kChainThreads) void chain_gram(ChainArgs a) {
  constexpr int MP = FT * 16;
  constexpr int NT = FT * (FT + 1) / 2;
  constexpr int TPWV = (NT + kChainWaves - 1) / kChainWaves;
  constexpr int STEP = 32, LDT = STEP + 8;
  __shared__ __attribute__((aligned(16))) uint16_t s_hi[MP * LDT];
  __shared__ __attribute__((aligned(16))) uint16_t s_lo[F32 ? MP * LDT : 8];

  const int u = blockIdx.y;
  const ChainUnit cu = chain_unit(a, u);
  const int T = a.out.num_tokens;
  const int t_begin = blockIdx.x * a.part_tokens;
  if (t_begin >= T) return;
  const int t_end = min(T, t_begin + a.part_tokens);
  const int esz = F32 ? 4 : 2;
  const void* A1 = static_cast<const char*>(a.first.coef) + cu.idx * (int64_t)a.first.num_tokens * a.first.rank * esz;
  const void* A2 =
      static_cast<const char*>(a.second.coef) + cu.idx * (int64_t)a.second.num_tokens * a.second.rank * esz;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, n = lane & 15;

  f32x4 acc[TPWV];
#pragma unroll
  for (int q = 0; q < TPWV; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int t0 = t_begin; t0 < t_end; t0 += STEP) {
    for (int e = tid; e < STEP * MP; e += kChainThreads) {
      const int tk = e / MP, l = e - tk * MP;
      const int t = t0 + tk;
      const float x = (t < t_end) ? cat_coef<F32>(a, A1, A2, t, l) : 0.f;
      if (F32) {
        uint32_t hb, lb;
        split_bf16(x, hb, lb);
        s_hi[l * LDT + tk] = (uint16_t)hb;
        s_lo[l * LDT + tk] = (uint16_t)lb;
      } else {
        s_hi[l * LDT + tk] = (uint16_t)(__float_as_uint(x) >> 16);  // exact: x came from a bf16
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < TPWV; ++q) {
      const int idx = wave + q * kChainWaves;
      if (idx < NT) {
        int fi = 0, rem = idx;
        while (rem >= FT - fi) {
          rem -= FT - fi;
          ++fi;
        }
        const int fj = fi + rem;
        const int oa = (16 * fi + n) * LDT + 8 * g, ob = (16 * fj + n) * LDT + 8 * g;
        const bf16x8 ah = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[oa]));
        const bf16x8 bh = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[ob]));
        if constexpr (F32) {
          const bf16x8 al = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[oa]));
          const bf16x8 bl = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[ob]));
          acc[q] = mfma16x16x32(al, bh, acc[q]);
          acc[q] = mfma16x16x32(ah, bl, acc[q]);
        }
        acc[q] = mfma16x16x32(ah, bh, acc[q]);
      }
    }
    __syncthreads();
  }
  float* P = a.partials + ((size_t)u * a.max_parts + blockIdx.x) * MP * MP;
#pragma unroll
  for (int q = 0; q < TPWV; ++q) {
    const int idx = wave + q * kChainWaves;
    if (idx < NT) {
      int fi = 0, rem = idx;
      while (rem >= FT - fi) {
        rem -= FT - fi;
        ++fi;
      }
      const int fj = fi + rem;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * fi + 4 * g + i, col = 16 * fj + n;
        P[row * MP + col] = acc[q][i];
        P[col * MP + row] = acc[q][i];
      }
    }
  }
}

// cgram without LDS for bf16 coefficients with r1, r2 multiples of FT and m <= 16 FT: one wave per token range,
// the same permuted feature order as the fit's Gram (lane (g, m) holds features FT m .. FT m + FT - 1 of tokens
// 8 g + j), one exact bf16 product per tile.
template <int FT, int Q>
__device__ __forceinline__ void cgram_tile(f32x4* acc, const typename GramSeg<FT>::T* seg) {
  constexpr int fi = tile_fi(Q, FT), fj = tile_fj(Q, FT);
  acc[Q] = mfma16x16x32(gram_fragment<FT, fi>(seg), gram_fragment<FT, fj>(seg), acc[Q]);
}
template <int FT, int... Qs>
__device__ __forceinline__ void cgram_tiles(f32x4* acc, const typename GramSeg<FT>::T* seg,
                                            std::integer_sequence<int, Qs...>) {
  (cgram_tile<FT, Qs>(acc, seg), ...);
}

template <int FT>
__global__ __launch_bounds__(kChainThreads) void chain_gram_wave(ChainArgs a) {
  constexpr int NT = FT * (FT + 1) / 2;
  constexpr int MP = 16 * FT;
  constexpr int STEP = 32;
  using Seg = typename GramSeg<FT>::T;
  const int u = blockIdx.y;
  const ChainUnit cu = chain_unit(a, u);
  const int T = a.out.num_tokens;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int part = blockIdx.x * kChainWaves + wave;
  const int t_begin = part * a.part_tokens;
  if (t_begin >= T) return;  // per wave: no barrier in this kernel
  const int t_end = min(T, t_begin + a.part_tokens);
  const int r1 = a.first.rank, r2 = a.second.rank, T1 = a.first.num_tokens, T2 = a.second.num_tokens;
  const uint16_t* A1 = static_cast<const uint16_t*>(a.first.coef) + cu.idx * (int64_t)T1 * r1;
  const uint16_t* A2 = static_cast<const uint16_t*>(a.second.coef) + cu.idx * (int64_t)T2 * r2;
  const int g = lane >> 4, n = lane & 15;
  const int l0 = FT * n;  // first concatenated rank of this lane's segment

  f32x4 acc[NT];
#pragma unroll
  for (int q = 0; q < NT; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
  // rows of two steps ahead in flight (two register sets): step s + 2 is issued before step s is multiplied
  Seg sa[8], sb[8];
  auto load = [&](int t0, Seg* seg) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int t = t0 + 8 * g + j;
      Seg v{};
      if (t < t_end) {
        if (l0 < r1) {
          if (t < T1) v = *reinterpret_cast<const Seg*>(A1 + (int64_t)t * r1 + l0);
        } else if (l0 < r1 + r2) {
          if (t < T2) v = *reinterpret_cast<const Seg*>(A2 + (int64_t)t * r2 + (l0 - r1));
        }
      }
      seg[j] = v;
    }
  };
  auto step = [&](int t0, Seg* seg) {
    Seg cur[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) cur[j] = seg[j];
    if (t0 + 2 * STEP < t_end) load(t0 + 2 * STEP, seg);
    cgram_tiles<FT>(acc, cur, std::make_integer_sequence<int, NT>{});
  };
  load(t_begin, sa);
  if (t_begin + STEP < t_end) load(t_begin + STEP, sb);
  for (int t0 = t_begin; t0 < t_end; t0 += 2 * STEP) {
    step(t0, sa);
    if (t0 + STEP >= t_end) break;
    step(t0 + STEP, sb);
  }
  float* P = a.partials + ((size_t)u * a.max_parts + part) * MP * MP;
#pragma unroll
  for (int q = 0; q < NT; ++q) {
    const int fi = tile_fi(q, FT), fj = tile_fj(q, FT);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = FT * (4 * g + i) + fi, col = FT * n + fj;
      P[row * MP + col] = acc[q][i];
      P[col * MP + row] = acc[q][i];
    }
  }
}

// ---------------------------------------------------------------------------------------------------------------
// assemble: H = sum of partials (fp64), P = H K^T (m x d), G = K P (d x d)
// ---------------------------------------------------------------------------------------------------------------

// LDS version for m <= 128: H (fp64 sum of the partials, kept as fp32) and K^T = [B1; B2] staged in LDS (H needs
// M8 x M8 floats, more than P's M8 x d when the rank sum exceeds the head dimension); P = H K^T
// with fp64 accumulation in registers (8 x 4 tiles), written back over H; G = K P in 8 x 8 tiles on or above the
// diagonal, staged in LDS as fp32 (the precision the eigensolver keeps) with each tile's mirror, then written out in
// whole rows.
__global__ __launch_bounds__(kChainThreads) void chain_assemble_lds(ChainArgs a) {
  extern __shared__ __attribute__((aligned(16))) float s_asm[];
  const int u = blockIdx.x;
  const ChainUnit cu = chain_unit(a, u);
  const int m = a.first.rank + a.second.rank, MP = a.mp, d = a.first.head_dim;
  const int M8 = (m + 7) / 8 * 8;
  const int T = a.out.num_tokens;
  const int parts = (T + a.part_tokens - 1) / a.part_tokens;
  const float* PP = a.partials + (size_t)u * a.max_parts * MP * MP;
  const int RW = M8 > d ? M8 : d;  // the first region holds H [M8][M8], later P [M8][d]
  float* R = s_asm;
  float* Bs = s_asm + M8 * RW;     // K^T [M8][d]
  const int tid = threadIdx.x;
  // H: the partials summed in fp64 in order c = 0, 1, ...; a batch of entries per thread has all its loads of one
  // partial in flight together
  constexpr int HB = 16;
  for (int e0 = 0; e0 < M8 * M8; e0 += HB * kChainThreads) {
    double s[HB];
    int off[HB];
#pragma unroll
    for (int q = 0; q < HB; ++q) {
      const int e = e0 + tid + q * kChainThreads;
      const int i = e / M8, j = e - i * M8;
      s[q] = 0.0;
      off[q] = e < M8 * M8 && i < m && j < m ? i * MP + j : -1;
    }
    for (int c = 0; c < parts; ++c) {
      float v[HB];
#pragma unroll
      for (int q = 0; q < HB; ++q) v[q] = off[q] >= 0 ? PP[(size_t)c * MP * MP + off[q]] : 0.0f;
#pragma unroll
      for (int q = 0; q < HB; ++q) s[q] += (double)v[q];
    }
#pragma unroll
    for (int q = 0; q < HB; ++q) {
      const int e = e0 + tid + q * kChainThreads;
      if (e < M8 * M8) R[e] = (float)s[q];
    }
  }
  constexpr int BB = 32;
  for (int e0 = 0; e0 < M8 * d; e0 += BB * kChainThreads) {
    float v[BB];
#pragma unroll
    for (int q = 0; q < BB; ++q) {
      const int e = e0 + tid + q * kChainThreads;
      const int l = e / d, f = e - l * d;
      v[q] = e < M8 * d && l < m ? cat_basis(a, cu.idx, l, f) : 0.f;
    }
#pragma unroll
    for (int q = 0; q < BB; ++q) {
      const int e = e0 + tid + q * kChainThreads;
      if (e < M8 * d) Bs[e] = v[q];
    }
  }
  __syncthreads();
  // P = H K^T: tile (8 rows l, 4 columns f); at most two tiles per thread (M8 <= 128)
  const int ntp = (M8 / 8) * (d / 4);
  double pacc[2][8][4];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int tile = tid + s * kChainThreads;
    if (tile < ntp) {
      const int l0 = 8 * (tile / (d / 4)), f0 = 4 * (tile % (d / 4));
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) pacc[s][i][c] = 0.0;
      for (int k = 0; k < m; ++k) {
        const float4 b = *reinterpret_cast<const float4*>(&Bs[k * d + f0]);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const double h = R[(l0 + i) * M8 + k];
          pacc[s][i][0] += h * b.x;
          pacc[s][i][1] += h * b.y;
          pacc[s][i][2] += h * b.z;
          pacc[s][i][3] += h * b.w;
        }
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int tile = tid + s * kChainThreads;
    if (tile < ntp) {
      const int l0 = 8 * (tile / (d / 4)), f0 = 4 * (tile % (d / 4));
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *reinterpret_cast<float4*>(&R[(l0 + i) * d + f0]) =
            make_float4((float)pacc[s][i][0], (float)pacc[s][i][1], (float)pacc[s][i][2], (float)pacc[s][i][3]);
    }
  }
  __syncthreads();
  // G = K P: tiles (8 rows i, 8 columns j) with i0 <= j0, one per thread (at most 136 for d <= 128); staged in LDS
  // over H and K^T (whose reads end at the barrier) as the fp32 values the eigensolver takes, with their mirrors, then
  // written out in whole rows
  const int nb = d / 8;
  const int tile = tid;
  const bool has_tile = tile < nb * (nb + 1) / 2;
  int i0 = 0, j0 = 0;
  double g[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) g[i][j] = 0.0;
  if (has_tile) {
    int bi = 0, rem = tile;
    while (rem >= nb - bi) {
      rem -= nb - bi;
      ++bi;
    }
    i0 = 8 * bi;
    j0 = 8 * (bi + rem);
    for (int l = 0; l < m; ++l) {
      const float4 b0 = *reinterpret_cast<const float4*>(&Bs[l * d + i0]);
      const float4 b1 = *reinterpret_cast<const float4*>(&Bs[l * d + i0 + 4]);
      const float4 p0 = *reinterpret_cast<const float4*>(&R[l * d + j0]);
      const float4 p1 = *reinterpret_cast<const float4*>(&R[l * d + j0 + 4]);
      const double bi8[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
      const double pj8[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) g[i][j] += bi8[i] * pj8[j];
    }
  }
  __syncthreads();
  float* Gs = s_asm;  // [d][d]
  if (has_tile) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        // the diagonal tiles are computed twice (i, j) and (j, i) with different rounding; keep the upper value
        // and mirror it so that G is exactly symmetric
        if (i0 == j0 && j < i) continue;
        const float v = (float)g[i][j];
        Gs[(i0 + i) * d + j0 + j] = v;
        Gs[(j0 + j) * d + i0 + i] = v;
      }
  }
  __syncthreads();
  double* G = a.gram + (size_t)u * d * d;
  for (int e = tid; e < d * d / 2; e += kChainThreads) {
    const float2 v = *reinterpret_cast<const float2*>(&Gs[2 * e]);
    *reinterpret_cast<double2*>(&G[2 * e]) = make_double2((double)v.x, (double)v.y);
  }
}

size_t chain_assemble_lds_bytes(int m, int d) {
  const size_t m8 = (size_t)(m + 7) / 8 * 8;
  const size_t hk = m8 * (m8 > (size_t)d ? m8 : (size_t)d) + m8 * d;  // H (later P) and K^T
  return (hk > (size_t)d * d ? hk : (size_t)d * d) * sizeof(float);  // then G
}

__global__ __launch_bounds__(kChainThreads) void chain_assemble(ChainArgs a) {
  const int u = blockIdx.x;
  const ChainUnit cu = chain_unit(a, u);
  const int m = a.first.rank + a.second.rank, MP = a.mp, d = a.first.head_dim;
  const int T = a.out.num_tokens;
  const int parts = (T + a.part_tokens - 1) / a.part_tokens;
  const float* PP = a.partials + (size_t)u * a.max_parts * MP * MP;
  double* Hs = a.hsum + (size_t)u * m * m;
  double* Pm = a.pmat + (size_t)u * m * d;
  double* G = a.gram + (size_t)u * d * d;
  for (int e = threadIdx.x; e < m * m; e += kChainThreads) {
    const int i = e / m, j = e - i * m;
    double s = 0.0;
    for (int c = 0; c < parts; ++c) s += (double)PP[(size_t)c * MP * MP + i * MP + j];
    Hs[e] = s;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < m * d; e += kChainThreads) {
    const int l = e / d, f = e - l * d;
    double s = 0.0;
    for (int k = 0; k < m; ++k) s += Hs[l * m + k] * (double)cat_basis(a, cu.idx, k, f);
    Pm[e] = s;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < d * d; e += kChainThreads) {
    const int i = e / d, j = e - i * d;
    if (j < i) continue;
    double s = 0.0;
    for (int l = 0; l < m; ++l) s += (double)cat_basis(a, cu.idx, l, i) * Pm[l * d + j];
    G[i * d + j] = s;
    G[j * d + i] = s;
  }
}

// ---------------------------------------------------------------------------------------------------------------
// ymat: Y = K^T R with R = out.basis^T (fp64 accumulation, stored fp32)
// ---------------------------------------------------------------------------------------------------------------

__global__ __launch_bounds__(kChainThreads) void chain_ymat(ChainArgs a) {
  const int u = blockIdx.x;
  const ChainUnit cu = chain_unit(a, u);
  const int m = a.first.rank + a.second.rank, ro = a.out.rank, d = a.first.head_dim;
  const float* Bo = a.out.basis + cu.idx * (int64_t)ro * d;
  float* Y = a.ymat + (size_t)u * m * ro;
  for (int e = threadIdx.x; e < m * ro; e += kChainThreads) {
    const int l = e / ro, k = e - l * ro;
    double s = 0.0;
    for (int f = 0; f < d; ++f) s += (double)cat_basis(a, cu.idx, l, f) * (double)Bo[k * d + f];
    Y[e] = (float)s;
  }
}

// The same product with K^T and R^T staged in LDS (rows padded to d + 1 floats): lanes take consecutive output
// columns k of one row l, so the R^T reads fall in distinct banks and the K^T read is a broadcast; the sums run
// over f in the same order as chain_ymat (identical results).
__global__ __launch_bounds__(kChainThreads) void chain_ymat_lds(ChainArgs a) {
  extern __shared__ float s_ym[];
  const int u = blockIdx.x;
  const ChainUnit cu = chain_unit(a, u);
  const int m = a.first.rank + a.second.rank, ro = a.out.rank, d = a.first.head_dim, dp = d + 1;
  const float* Bo = a.out.basis + cu.idx * (int64_t)ro * d;
  float* Ks = s_ym;
  float* Rs = s_ym + m * dp;
  for (int e = threadIdx.x; e < m * d; e += kChainThreads) {
    const int l = e / d, f = e - l * d;
    Ks[l * dp + f] = cat_basis(a, cu.idx, l, f);
  }
  for (int e = threadIdx.x; e < ro * d; e += kChainThreads) {
    const int k = e / d, f = e - k * d;
    Rs[k * dp + f] = Bo[e];
  }
  __syncthreads();
  float* Y = a.ymat + (size_t)u * m * ro;
  for (int e = threadIdx.x; e < m * ro; e += kChainThreads) {
    const int l = e / ro, k = e - l * ro;
    const float* kr = Ks + l * dp;
    const float* rr = Rs + k * dp;
    double s = 0.0;
#pragma unroll 8
    for (int f = 0; f < d; ++f) s += (double)kr[f] * (double)rr[f];
    Y[e] = (float)s;
  }
}

size_t chain_ymat_lds_bytes(int m, int ro, int d) { return (size_t)(m + ro) * (d + 1) * sizeof(float); }

// ---------------------------------------------------------------------------------------------------------------
// cproj: A_out = [A1 A2] Y on MFMA.  M = output rank (16 per tile), N = token (16), K = concatenated rank (32 per
// step).  Y^T is staged in LDS as a bf16 hi/lo pair; the coefficient rows are the B operand.
// ---------------------------------------------------------------------------------------------------------------

// 2048 tokens per workgroup: Y^T is staged once per 2048 tokens (0.652 ms at 8B/32K against 0.715 ms with 512 and
// 0.663 ms with 1024)
constexpr int kCprojTilesPerWave = 32;
constexpr int kCprojChunk = kChainWaves * kCprojTilesPerWave * 16;

// VEC (bf16, r1 and r2 multiples of 8, r_out a multiple of 4): 16-byte coefficient loads and 8-byte stores.
template <int MTR, bool F32, bool VEC>
__global__ __launch_bounds__(kChainThreads) void chain_proj(ChainArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint16_t s_y[];  // hi [MTR*16][KP], lo [MTR*16][KP]
  const int u = blockIdx.y;
  const ChainUnit cu = chain_unit(a, u);
  const int T = a.out.num_tokens;
  const int t_begin = blockIdx.x * kCprojChunk;
  if (t_begin >= T) return;
  const int m = a.first.rank + a.second.rank, ro = a.out.rank;
  const int KSC = (m + 31) / 32, KP = KSC * 32;
  uint16_t* s_hi = s_y;
  uint16_t* s_lo = s_y + MTR * 16 * KP;
  const float* Y = a.ymat + (size_t)u * m * ro;
  for (int e = threadIdx.x; e < MTR * 16 * KP; e += kChainThreads) {
    const int k = e / KP, l = e - k * KP;
    const float y = (k < ro && l < m) ? Y[l * ro + k] : 0.f;
    uint32_t hb, lb;
    split_bf16(y, hb, lb);
    s_hi[e] = (uint16_t)hb;
    s_lo[e] = (uint16_t)lb;
  }
  __syncthreads();
  const int esz = F32 ? 4 : 2;
  const void* A1 = static_cast<const char*>(a.first.coef) + cu.idx * (int64_t)a.first.num_tokens * a.first.rank * esz;
  const void* A2 =
      static_cast<const char*>(a.second.coef) + cu.idx * (int64_t)a.second.num_tokens * a.second.rank * esz;
  void* Co = static_cast<char*>(a.out.coef) + cu.idx * (int64_t)T * ro * esz;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, n = lane & 15;

  for (int j = 0; j < kCprojTilesPerWave; ++j) {
    const int t0 = t_begin + (j * kChainWaves + wave) * 16;
    if (t0 >= T) break;
    const int t = t0 + n;
    f32x4 acc[MTR];
#pragma unroll
    for (int mt = 0; mt < MTR; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks < KSC; ++ks) {
      uint32_t ch[4], cl[4];
      if constexpr (VEC) {
        const int l = 32 * ks + 8 * g;
        const int r1 = a.first.rank;
        u32x4 v = {0, 0, 0, 0};
        if (t < T) {
          if (l < r1) {
            if (t < a.first.num_tokens)
              v = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(A1) + (int64_t)t * r1 + l);
          } else if (l < m) {
            if (t < a.second.num_tokens)
              v = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(A2) +
                                                  (int64_t)t * a.second.rank + (l - r1));
          }
        }
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          ch[w] = v[w];
          cl[w] = 0;
        }
      } else {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int l = 32 * ks + 8 * g + 2 * w;
        const float x0 = (t < T) ? cat_coef<F32>(a, A1, A2, t, l) : 0.f;
        const float x1 = (t < T) ? cat_coef<F32>(a, A1, A2, t, l + 1) : 0.f;
        if (F32) {
          split_bf16x2(x0, x1, ch[w], cl[w]);
        } else {
          ch[w] = (__float_as_uint(x0) >> 16) | (__float_as_uint(x1) & 0xffff0000u);
          cl[w] = 0;
        }
      }
      }
      const bf16x8 bh = as_bf16x8(u32x4{ch[0], ch[1], ch[2], ch[3]});
      const bf16x8 bl = as_bf16x8(u32x4{cl[0], cl[1], cl[2], cl[3]});
#pragma unroll
      for (int mt = 0; mt < MTR; ++mt) {
        const int o = (16 * mt + n) * KP + 32 * ks + 8 * g;
        const bf16x8 yh = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_hi[o]));
        const bf16x8 yl = as_bf16x8(*reinterpret_cast<const u32x4*>(&s_lo[o]));
        acc[mt] = mfma16x16x32(yl, bh, acc[mt]);
        if constexpr (F32) acc[mt] = mfma16x16x32(yh, bl, acc[mt]);
        acc[mt] = mfma16x16x32(yh, bh, acc[mt]);
      }
    }
    if (t < T && VEC) {
#pragma unroll
      for (int mt = 0; mt < MTR; ++mt) {
        const int k0 = 16 * mt + 4 * g;
        if (k0 < ro) {
          uint2 w;
          w.x = pack_bf16x2(acc[mt][0], acc[mt][1]);
          w.y = pack_bf16x2(acc[mt][2], acc[mt][3]);
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(Co) + (int64_t)t * ro + k0) = w;
        }
      }
    } else if (t < T) {
#pragma unroll
      for (int mt = 0; mt < MTR; ++mt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k = 16 * mt + 4 * g + i;
          if (k < ro) {
            if (F32) static_cast<float*>(Co)[(int64_t)t * ro + k] = acc[mt][i];
            else static_cast<uint16_t*>(Co)[(int64_t)t * ro + k] = (uint16_t)f32_to_bf16_bits(acc[mt][i]);
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------------------------------------------

template <int FT, bool F32>
static void launch_cgram_one(dim3 grid, hipStream_t stream, const ChainArgs& a) {
  hipLaunchKernelGGL((chain_gram<FT, F32>), grid, dim3(kChainThreads), 0, stream, a);
}

template <bool F32, int... FTs>
static void launch_cgram_ft(int ft, dim3 grid, hipStream_t stream, const ChainArgs& a,
                            std::integer_sequence<int, FTs...>) {
  ((ft == FTs + 1 ? launch_cgram_one<FTs + 1, F32>(grid, stream, a) : void()), ...);
}

template <bool F32, bool VEC>
static void launch_cproj_mtr(int mtr, dim3 grid, size_t lds, hipStream_t stream, const ChainArgs& a) {
  switch (mtr) {
    case 1: hipLaunchKernelGGL((chain_proj<1, F32, VEC>), grid, dim3(kChainThreads), lds, stream, a); break;
    case 2: hipLaunchKernelGGL((chain_proj<2, F32, VEC>), grid, dim3(kChainThreads), lds, stream, a); break;
    case 3:
    case 4: hipLaunchKernelGGL((chain_proj<4, F32, VEC>), grid, dim3(kChainThreads), lds, stream, a); break;
    default: hipLaunchKernelGGL((chain_proj<8, F32, VEC>), grid, dim3(kChainThreads), lds, stream, a); break;
  }
}

template <int FT>
static void launch_cgram_wave(dim3 grid, hipStream_t stream, const ChainArgs& a) {
  hipLaunchKernelGGL((chain_gram_wave<FT>), grid, dim3(kChainThreads), 0, stream, a);
}

hipError_t launch_chain(const ChainArgs& a, const EigArgs& ea, hipStream_t stream) {
  const bool f32 = a.first.coef_dtype == KVC_F32;
  const int T = a.out.num_tokens;
  const int m = a.first.rank + a.second.rank;
  const int d = a.first.head_dim;
  hipError_t e;
  if (a.gram_wave_ft > 0) {
    dim3 ggrid((a.max_parts + kChainWaves - 1) / kChainWaves, a.num_units);
    switch (a.gram_wave_ft) {
      case 2: launch_cgram_wave<2>(ggrid, stream, a); break;
      case 4: launch_cgram_wave<4>(ggrid, stream, a); break;
      default: launch_cgram_wave<8>(ggrid, stream, a); break;
    }
  } else {
    dim3 ggrid(a.max_parts, a.num_units);
    const int ft = a.mp / 16;
    if (f32) launch_cgram_ft<true>(ft, ggrid, stream, a, std::make_integer_sequence<int, 16>{});
    else launch_cgram_ft<false>(ft, ggrid, stream, a, std::make_integer_sequence<int, 16>{});
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (m <= 128) {
    const size_t lds = chain_assemble_lds_bytes(m, d);
    e = hipFuncSetAttribute((const void*)chain_assemble_lds, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(chain_assemble_lds, dim3(a.num_units), dim3(kChainThreads), lds, stream, a);
  } else {
    hipLaunchKernelGGL(chain_assemble, dim3(a.num_units), dim3(kChainThreads), 0, stream, a);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = launch_eig(ea, stream)) != hipSuccess) return e;
  const size_t ylds = chain_ymat_lds_bytes(m, a.out.rank, d);
  if (ylds <= 160 * 1024) {
    e = hipFuncSetAttribute((const void*)chain_ymat_lds, hipFuncAttributeMaxDynamicSharedMemorySize, (int)ylds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(chain_ymat_lds, dim3(a.num_units), dim3(kChainThreads), ylds, stream, a);
  } else {
    hipLaunchKernelGGL(chain_ymat, dim3(a.num_units), dim3(kChainThreads), 0, stream, a);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int mtr = (a.out.rank + 15) / 16;
  const int mtr_inst = mtr <= 2 ? mtr : (mtr <= 4 ? 4 : 8);
  const size_t lds = (size_t)mtr_inst * 16 * ((m + 31) / 32 * 32) * 2 * sizeof(uint16_t);
  dim3 pgrid((T + kCprojChunk - 1) / kCprojChunk, a.num_units);
  const bool vec = !f32 && a.first.rank % 8 == 0 && a.second.rank % 8 == 0 && a.out.rank % 4 == 0;
  const void* big = f32 ? (const void*)chain_proj<8, true, false>
                        : (vec ? (const void*)chain_proj<8, false, true> : (const void*)chain_proj<8, false, false>);
  e = hipFuncSetAttribute(big, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  if (f32) launch_cproj_mtr<true, false>(mtr, pgrid, lds, stream, a);
  else if (vec) launch_cproj_mtr<false, true>(mtr, pgrid, lds, stream, a);
  else launch_cproj_mtr<false, false>(mtr, pgrid, lds, stream, a);
  return hipGetLastError();
}

}  // namespace kvc
