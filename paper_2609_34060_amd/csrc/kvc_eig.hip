// Top-r eigenpairs of the per-unit d x d Gram matrices in fp64: the right singular vectors R_r and singular values
// of Eq. 7 (Z^T Z = R Sigma^2 R^T).  One workgroup of 1024 threads per (layer, K/V, head) unit:
//   1. G = sum of the unit's fp32 partial Grams in a fixed order in fp64 (or a dense fp64 matrix), into LDS.
//   2. Householder tridiagonalisation G = Q T Q^T in fp64 arithmetic; the trailing matrix is kept in LDS in fp32
//      (the Gram itself carries fp32 accuracy), which lets two units share a CU; the reflectors go to the workspace.
//   3. Multisection bisection with Sturm counts for the r largest eigenvalues of T (groups of lanes per
//      eigenvalue, one ballot per step).
//   4. Inverse iteration on T (LDL^T without pivoting, tiny pivots replaced) from pseudo-random starts, one lane
//      per eigenvector; then modified Gram-Schmidt over the r vectors.  Vectors of tightly clustered eigenvalues
//      come out as an orthonormal basis of the cluster's invariant subspace (where the SVD itself is not unique).
//   5. Back-transformation by the reflectors, canonical sign (largest-magnitude entry positive, first index on
//      near-ties), basis rows and sigma = sqrt(lambda) written to the state.
#include <algorithm>
#include <type_traits>

#include "kvc_device.h"
#include "kvc_launch.h"

namespace kvc {

constexpr int kEigThreads = 1024;
constexpr int kEigWaves = kEigThreads / kWave;
constexpr int kReflChunk = 16;  // reflectors staged in LDS per back-transformation chunk
constexpr int kInvBatch = 32;   // eigenvectors per inverse-iteration batch (one lane each)

// fp64 cross-lane moves by DPP (two 32-bit halves); lanes whose row is masked off receive 0.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ double dpp64(double x) {
  const unsigned long long b = __builtin_bit_cast(unsigned long long, x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(unsigned)b, CTRL, ROW_MASK, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(unsigned)(b >> 32), CTRL, ROW_MASK, 0xF, false);
  return __builtin_bit_cast(double, ((unsigned long long)(unsigned)hi << 32) | (unsigned)lo);
}
constexpr int kDppRor1 = 0x121, kDppRor2 = 0x122, kDppRor4 = 0x124, kDppRor8 = 0x128;
constexpr int kDppBcast15 = 0x142, kDppBcast31 = 0x143;

// Sum over each group of G consecutive lanes (G = 16, 32 or 64); the group's last lane holds the total (other lanes
// hold partial sums).  A fixed order, so the result is deterministic.  Called with the whole wave active.
template <int G>
__device__ __forceinline__ double group_sum(double x) {
  x += dpp64<kDppRor8>(x);
  x += dpp64<kDppRor4>(x);
  x += dpp64<kDppRor2>(x);
  x += dpp64<kDppRor1>(x);
  if (G >= 32) x += dpp64<kDppBcast15, 0xA>(x);
  if (G >= 64) x += dpp64<kDppBcast31, 0xC>(x);
  return x;
}
__device__ __forceinline__ double lane_value(double x, int l) {
  const unsigned long long b = __builtin_bit_cast(unsigned long long, x);
  const unsigned lo = __builtin_amdgcn_readlane((int)(unsigned)b, l);
  const unsigned hi = __builtin_amdgcn_readlane((int)(unsigned)(b >> 32), l);
  return __builtin_bit_cast(double, ((unsigned long long)hi << 32) | lo);
}
// Whole-wave sum and maximum, returned in every lane.
__device__ __forceinline__ double wave_sum(double x) { return lane_value(group_sum<64>(x), 63); }
__device__ __forceinline__ double wave_max(double x) {
  x = fmax(x, dpp64<kDppRor8>(x));
  x = fmax(x, dpp64<kDppRor4>(x));
  x = fmax(x, dpp64<kDppRor2>(x));
  x = fmax(x, dpp64<kDppRor1>(x));
  return fmax(fmax(lane_value(x, 0), lane_value(x, 16)), fmax(lane_value(x, 32), lane_value(x, 48)));
}

// Reductions over groups of eight consecutive lanes (every lane of the group gets the result; fp32 addition is
// commutative, so all eight agree).
template <int CTRL>
__device__ __forceinline__ float dpp32(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp32i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141;
__device__ __forceinline__ float sum8(float x) {
  x += dpp32<kDppXor1>(x);
  x += dpp32<kDppXor2>(x);
  return x + dpp32<kDppHalfMirror>(x);
}
__device__ __forceinline__ float max8(float x) {
  x = fmaxf(x, dpp32<kDppXor1>(x));
  x = fmaxf(x, dpp32<kDppXor2>(x));
  return fmaxf(x, dpp32<kDppHalfMirror>(x));
}
__device__ __forceinline__ int min8(int x) {
  x = min(x, dpp32i<kDppXor1>(x));
  x = min(x, dpp32i<kDppXor2>(x));
  return min(x, dpp32i<kDppHalfMirror>(x));
}

struct UnitTarget {
  int rank;
  int tokens;
  float* basis;
  float* sigma;
};

__device__ __forceinline__ UnitTarget eig_target(const EigArgs& a, int u) {
  const int H = a.num_kv_heads;
  const int per_item = a.num_layers * 2 * H;
  const int item = u / per_item;
  int rem = u - item * per_item;
  const int lrel = rem / (2 * H);
  rem -= lrel * 2 * H;
  const int kv = rem / H, head = rem - kv * H;
  const kvc_state* st = a.items ? &a.items[item].state : &a.state;
  const int64_t idx = unit_index(a.layer_begin + lrel, kv, head, H);
  UnitTarget t;
  t.rank = st->rank;
  t.tokens = st->num_tokens;
  t.basis = st->basis + idx * st->rank * a.n;
  t.sigma = st->sigma ? st->sigma + idx * st->rank : nullptr;
  return t;
}

__device__ __forceinline__ uint32_t hash3(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t h = a * 0x9E3779B1u ^ (b + 0x7F4A7C15u) * 0x85EBCA77u ^ (c + 0x165667B1u) * 0xC2B2AE3Du;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  h *= 0x297A2D39u;
  h ^= h >> 15;
  return h;
}

// 1 / q from the hardware reciprocal and one Newton step (relative error about 2^-52).
__device__ __forceinline__ double recip(double q) {
  const double r0 = __builtin_amdgcn_rcp(q);
  return fma(r0, fma(-q, r0, 1.0), r0);
}

// Scalars of one Householder step from x_0 and s = ||x||^2: out = {alpha, v_0, beta} with alpha = -sign(x_0) ||x||,
// v = x - alpha e_1 and beta = 2 / v^T v = 1 / (||x|| (||x|| + |x_0|)) (0 when x = 0: the step is the identity).
__device__ __forceinline__ void reflector_scalars(double x0, double s, double* out) {
  const double nrm = sqrt(s);
  const double alpha = nrm == 0.0 ? 0.0 : -copysign(nrm, x0);
  out[0] = alpha;
  out[1] = x0 - alpha;
  out[2] = nrm == 0.0 ? 0.0 : recip(nrm * (nrm + fabs(x0)));
}

// Number of eigenvalues of T below x (ratio form of the Sturm sequence; pivots smaller than pivmin are replaced
// by -pivmin, so that b^2 / q stays finite).
template <int N>
__device__ __forceinline__ int sturm_count(const double* sa, const double* sb2, double x, double pivmin) {
  double q = sa[0] - x;
  if (fabs(q) < pivmin) q = -pivmin;
  int c = q < 0.0;
#pragma unroll 4
  for (int i = 1; i < N; ++i) {
    q = (sa[i] - x) - sb2[i - 1] * recip(q);
    if (fabs(q) < pivmin) q = -pivmin;
    c += q < 0.0;
  }
  return c;
}

// ---- Householder tridiagonalisation steps ----------------------------------------------------------------------
// Step k reflects x = row k beyond the diagonal (the matrix is symmetric) onto alpha e_1 with H_k = I - beta v v^T,
// v = x - alpha e_1; with p = beta A22 v, K = beta v^T p / 2 and w = p - K v, A22 <- A22 - v w^T - w v^T.
// The matrix lives in LDS as fp32 [N][N]; the rank-2 update is two fp32 fmas per entry (v and w rounded to fp32),
// everything else (p, K, w, the scalars, the reflectors) is fp64.  Per step:
//   pivot (wave 0): p of step k from the row-group partials, K, w; row k + 1 under step k (the next x); the scalars
//       of step k + 1; {v_C, w_C, x'_C} of every column to s_vw; the reflector to the workspace.
//   sweep (all threads): rows C > k + 1 under step k; from the updated entries, the row-group partial sums of the
//       next step's A22 v' (no scaling by beta yet).  Thread (g, R) owns column R of rows g, g + RG, ...; a row
//       group is whole waves, so row skips are uniform; partial[g][R] goes to LDS, summed by the next pivot.
// Step k's scalars {alpha, v_0, beta} are in s_ab + 4 (k & 1).

// Wave 0.  Before the first step (k = -1) only the scalars of step 0 and s_vw are formed.  Every LDS load is issued
// up front (indices stay in range), so the pivot waits for LDS once.
template <int N>
__device__ __forceinline__ void tri_pivot(float* A, const double* partial, const double* s_kp, float4* s_vw,
                                          double* s_ab, double* s_b, double* refl, double* refl_beta, int k, int lane) {
  constexpr int RG = kEigThreads / N;  // row groups of the sweep
  constexpr int Q = N / kWave;         // columns per lane
  const int kn = k + 1;
  const int kr = k < 0 ? 0 : k;
  const double* ab = s_ab + 4 * (kr & 1);
  const double alpha = ab[0], v0 = k < 0 ? 0.0 : ab[1], beta = k < 0 ? 0.0 : ab[2];
  double psum[Q];
  float xk[Q], xn[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int C = lane + kWave * q;
    xk[q] = A[kr * N + C];
    xn[q] = A[kn * N + C];
    double sum = 0.0;
#pragma unroll
    for (int gi = 0; gi < RG; ++gi) sum += partial[gi * N + C];
    psum[q] = k < 0 ? 0.0 : sum;  // (before the first step the partials hold nothing yet)
  }
  // K = (beta / 2) v^T p = (beta^2 / 2) sum of the sweep's per-wave shares
  double kk = 0.0;
#pragma unroll
  for (int i = 0; i < kEigWaves; ++i) kk += s_kp[i];
  const double K = k < 0 ? 0.0 : 0.5 * beta * beta * kk;
  double vq[Q], wq[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int C = lane + kWave * q;
    vq[q] = k < 0 ? 0.0 : (C > kn ? (double)xk[q] : (C == kn ? v0 : 0.0));
    wq[q] = C >= kn ? beta * psum[q] - K * vq[q] : 0.0;
  }
  const double wR = k < 0 ? 0.0 : lane_value(wq[kn / kWave], kn % kWave);  // w of row k + 1 (its v is v_0)
  // row k + 1 under step k (same arithmetic as the sweep; columns below k + 1 do not change), its norm beyond the
  // diagonal, the next scalars; s_vw[C] = {v_C, w_C, v'_C} with v' the next step's v
  const float v0f = (float)v0, wRf = (float)wR;
  double s = 0.0;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int C = lane + kWave * q;
    xn[q] = fmaf(-v0f, (float)wq[q], fmaf(-wRf, (float)vq[q], xn[q]));
    A[kn * N + C] = xn[q];
    s += C > kn ? (double)xn[q] * (double)xn[q] : 0.0;
    s_vw[C] = make_float4((float)vq[q], (float)wq[q], C > kn + 1 ? xn[q] : 0.0f, 0.0f);
  }
  s = wave_sum(s);
  const double x0 = lane_value((double)xn[((kn + 1) % N) / kWave], (kn + 1) % kWave);
  if (lane == 0) {
    double* abn = s_ab + 4 * (kn & 1);
    reflector_scalars(kn + 1 < N ? x0 : 0.0, s, abn);
    if (kn + 1 < N) s_vw[kn + 1].z = (float)abn[1];  // v'_{k+2} = v_0 of the next step
  }
  if (k >= 0) {
    double* refl_k = refl + __builtin_amdgcn_readfirstlane(k * N);
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int C = lane + kWave * q;
      if (C >= kn) refl_k[C - kn] = vq[q];
    }
    if (lane == 0) {
      s_b[k] = alpha;
      refl_beta[k] = beta;
    }
  }
}

// All threads: rows C > k + 1 under step k (UPD; without UPD, k = -1 and nothing is updated), then the row-group
// partial sums of A22 v' for step k + 1 and each wave's share of v'^T (A22 v').
template <int N, bool UPD>
__device__ __forceinline__ void tri_sweep(float* A, double* partial, double* s_kp, const float4* s_vw, int k,
                                          int tid, int lane, int wave) {
  constexpr int RG = kEigThreads / N;
  constexpr int RPT = N / RG;
  const int R = tid & (N - 1);
  const int g = __builtin_amdgcn_readfirstlane(tid / N);  // uniform: a row group is whole waves
  const int kn = k + 1;
  const float4 vwR = s_vw[R];
  // first live row of this thread: g + RG t > k + 1.  Entries of eliminated columns (R <= k + 1) are updated too
  // (with v_R = w_R = 0 they do not change, and column k + 1 is not read again), so that stores need no mask.
  const int t0 = kn < g ? 0 : (kn - g) / RG + 1;
  float acc = 0.0f;
  // rows in batches of four: every load of a batch is issued before its stores
  auto rows = [&](int t, auto nb) {
    constexpr int NB = decltype(nb)::value;
    float4 vwC[NB];
    float a[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int C = g + RG * (t + j);
      vwC[j] = s_vw[C];
      a[j] = A[C * N + R];
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int C = g + RG * (t + j);
      if (UPD) {
        a[j] = fmaf(-vwC[j].x, vwR.y, fmaf(-vwC[j].y, vwR.x, a[j]));
        A[C * N + R] = a[j];
      }
      acc = fmaf(a[j], vwC[j].z, acc);
    }
  };
  int t = t0;
  for (; t + 4 <= RPT; t += 4) rows(t, std::integral_constant<int, 4>());
  for (; t < RPT; ++t) rows(t, std::integral_constant<int, 1>());
  partial[g * N + R] = acc;
  const double kp = group_sum<kWave>((double)acc * (double)vwR.z);
  if (lane == kWave - 1) s_kp[wave] = kp;
}

// LDS layout (bytes): the matrix region MREG holds, in turn, G / the trailing matrix as fp32 [N][N] (phases 1-2),
// the inverse-iteration scratch fp64 [N][kInvBatch] x 2 (phase 4), X fp32 [r][N] (MGS, back-transformation); then
// fp64 scalars and vectors; then the staging region: the sweep's row-group partials fp64 [RG][N] during phase 2, a
// chunk of reflectors during phase 5.  About 79 KB for N = 128, so two units share a CU.
template <int N>
struct EigLds {
  static constexpr size_t kMat = (size_t)N * N * 4;
  static constexpr size_t kScratch = (size_t)2 * N * kInvBatch * 8;
  static constexpr size_t kX = (size_t)KVC_MAX_RANK * N * 4;
  static constexpr size_t kMreg = ((kMat > kScratch ? (kMat > kX ? kMat : kX) : (kScratch > kX ? kScratch : kX)) +
                                   15) / 16 * 16;
  // s_a, s_b [N]; s_lam [KVC_MAX_RANK]; s_ab [2][4]; s_kp [kEigWaves]; s_misc [8]; s_vw float4 [N] (later b^2 [N])
  static constexpr size_t kSmall = (size_t)(2 * N + KVC_MAX_RANK + 8 + kEigWaves + 8) * 8 + (size_t)N * 16;
  static constexpr size_t kPartial = (size_t)(kEigThreads / N) * N * 8;
  static constexpr size_t kReflStage = (size_t)kReflChunk * (N + 1) * 4;
  static constexpr size_t kStage = kPartial > kReflStage ? kPartial : kReflStage;
  static constexpr size_t kTotal = kMreg + kSmall + kStage;
};

// Eight waves per SIMD (at most 64 VGPRs) so that two 1024-thread units share a CU.
template <int N>
__global__ __launch_bounds__(kEigThreads) __attribute__((amdgpu_waves_per_eu(8))) void eig_topr(EigArgs a) {
  using Lay = EigLds<N>;
  constexpr int LD = N;
  extern __shared__ __attribute__((aligned(16))) double smem[];
  char* base = reinterpret_cast<char*>(smem);
  float* A = reinterpret_cast<float*>(base);             // G, then the trailing matrix (fp32 storage)
  double* invd = reinterpret_cast<double*>(base);        // inverse-iteration scratch [N][kInvBatch]
  double* xv = invd + N * kInvBatch;                     // [N][kInvBatch]
  float* X = reinterpret_cast<float*>(base);             // eigenvectors, vector j in row j (fp32 storage)
  double* s_a = reinterpret_cast<double*>(base + Lay::kMreg);  // diagonal of T
  double* s_b = s_a + N;                    // off-diagonal of T: b[i] couples i and i + 1
  double* s_lam = s_b + N;                  // eigenvalues, descending
  double* s_ab = s_lam + KVC_MAX_RANK;      // reflector scalars {alpha, v_0, beta, -}, by step parity [2][4]
  double* s_kp = s_ab + 8;                  // per-wave shares of v^T A22 v from the sweep [kEigWaves]
  double* s_misc = s_kp + kEigWaves;        // scalars
  float4* s_vw = reinterpret_cast<float4*>(s_misc + 8);  // {v_C, w_C, x'_C, -} of the current step
  double* s_b2 = reinterpret_cast<double*>(s_vw);        // b^2 (after the tridiagonalisation)
  double* partial = reinterpret_cast<double*>(base + Lay::kMreg + Lay::kSmall);  // sweep partials [RG][N]
  float* s_rb = reinterpret_cast<float*>(partial);  // reflector chunk fp32 [kReflChunk][N] (back-transformation)
  float* s_rbeta = s_rb + kReflChunk * N;

  const int u = blockIdx.x;
  if (a.skip && a.skip[u]) return;  // whole workgroup
  const UnitTarget tg = eig_target(a, u);
  const int r = tg.rank;
  if (r <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  double* refl = a.reflect + (size_t)u * N * N;          // v_k in row k
  double* refl_beta = a.reflect_beta + (size_t)u * N;
  double* gvec = a.vecs + (size_t)u * N * KVC_MAX_RANK;  // eigenvectors of T, vector j in row j

  // ---- 1. load G ------------------------------------------------------------------------------------------
  if (a.partials) {
    const int parts = (tg.tokens + a.part_tokens - 1) / a.part_tokens;
    const float* P = a.partials + (size_t)u * a.max_parts * N * N;
    for (int e = tid; e < N * N; e += kEigThreads) {
      double s = 0.0;
      for (int c = 0; c < parts; ++c) s += (double)P[(size_t)c * N * N + e];
      A[(e / N) * LD + (e % N)] = (float)s;
    }
  } else {
    const double* Dm = a.dense + (size_t)u * N * N;
    for (int e = tid; e < N * N; e += kEigThreads) A[(e / N) * LD + (e % N)] = (float)Dm[e];
  }
  __syncthreads();

  // ---- 2. Householder tridiagonalisation -----------------------------------------------------------------------
  if (wave == 0) tri_pivot<N>(A, partial, s_kp, s_vw, s_ab, s_b, refl, refl_beta, -1, lane);
  __syncthreads();
  tri_sweep<N, false>(A, partial, s_kp, s_vw, -1, tid, lane, wave);
  __syncthreads();
  for (int k = 0; k < N - 2; ++k) {
    if (wave == 0) tri_pivot<N>(A, partial, s_kp, s_vw, s_ab, s_b, refl, refl_beta, k, lane);
    __syncthreads();
    tri_sweep<N, true>(A, partial, s_kp, s_vw, k, tid, lane, wave);
    __syncthreads();
  }
  for (int i = tid; i < N; i += kEigThreads) s_a[i] = A[i * LD + i];
  if (tid == 0) s_b[N - 2] = A[(N - 2) * LD + N - 1];
  __syncthreads();
  for (int i = tid; i < N - 1; i += kEigThreads) s_b2[i] = s_b[i] * s_b[i];
  if (tid == 0) {
    double lo = s_a[0], hi = s_a[0], bmax2 = 0.0;
    for (int i = 0; i < N; ++i) {
      const double rad = (i > 0 ? fabs(s_b[i - 1]) : 0.0) + (i < N - 1 ? fabs(s_b[i]) : 0.0);
      lo = fmin(lo, s_a[i] - rad);
      hi = fmax(hi, s_a[i] + rad);
      if (i < N - 1) bmax2 = fmax(bmax2, s_b[i] * s_b[i]);
    }
    const double tnorm = fmax(fabs(lo), fabs(hi));
    const double pivmin = 2.2250738585072014e-308 * fmax(1.0, bmax2);
    const double pad = 2.0 * 2.220446049250313e-16 * tnorm * N + pivmin;
    s_misc[1] = lo - pad;
    s_misc[2] = hi + pad;
    s_misc[3] = tnorm;
    s_misc[4] = pivmin;
  }
  __syncthreads();
  const double tnorm = s_misc[3];

  if (tnorm == 0.0) {
    // Z = 0: every eigenvalue is 0; take the unit vectors (the product is zero whatever the basis).
    for (int e = tid; e < r * N; e += kEigThreads) X[e] = (e / N) == (e % N) ? 1.0f : 0.0f;
    for (int j = tid; j < r; j += kEigThreads) s_lam[j] = 0.0;
    __syncthreads();
  } else {
    // ---- 3. multisection bisection for the r largest eigenvalues ---------------------------------------
    {
      int rp = 1;
      while (rp < r) rp <<= 1;
      // lanes per eigenvalue (a power of two dividing 64): 8 lanes and 11 steps of 9-way splitting (88 Sturm counts
      // per eigenvalue) measured faster than 16 lanes and 8 steps (128 counts) or 4 lanes and 14 steps (56)
      const int P = min(8, kEigThreads / rp);
      // each step shrinks the bracket (P + 1)-fold; stop below 2^-32 of the Gershgorin interval, under the
      // perturbation that fp32 storage of the matrix already carries
      const int iters = P >= 16 ? 8 : P >= 8 ? 11 : P >= 4 ? 14 : P >= 2 ? 21 : 32;
      const int grp = tid / P, s = tid - grp * P;
      const int kasc = N - 1 - grp;                  // ascending index of the target eigenvalue
      const double pivmin = s_misc[4];
      double lo = s_misc[1], hi = s_misc[2];
      for (int it = 0; it < iters; ++it) {
        const double x = lo + (hi - lo) * (double)(s + 1) / (double)(P + 1);
        const int c = grp < r ? sturm_count<N>(s_a, s_b2, x, pivmin) : 0;
        const uint64_t mask = __ballot(c <= kasc);
        const uint64_t gmask = P == kWave ? mask : (mask >> ((lane / P) * P)) & ((1ull << P) - 1ull);
        const int sstar = __popcll(gmask);
        const double nlo = sstar == 0 ? lo : lo + (hi - lo) * (double)sstar / (double)(P + 1);
        const double nhi = sstar == P ? hi : lo + (hi - lo) * (double)(sstar + 1) / (double)(P + 1);
        lo = nlo;
        hi = nhi;
      }
      if (grp < r && s == 0) s_lam[grp] = 0.5 * (lo + hi);
    }
    __syncthreads();

    // ---- 4. inverse iteration, kInvBatch vectors per batch, one lane each ------------------------------
    const double piv = 2.220446049250313e-16 * tnorm;
    for (int j0 = 0; j0 < r; j0 += kInvBatch) {
      const int j = j0 + tid;
      if (tid < kInvBatch && j < r) {
        const double lam = s_lam[j];
        double d = s_a[0] - lam;
        if (fabs(d) < piv) d = copysign(piv, d);
        invd[tid] = 1.0 / d;
#pragma unroll 2
        for (int i = 1; i < N; ++i) {
          const double l = s_b[i - 1] * invd[(i - 1) * kInvBatch + tid];
          d = (s_a[i] - lam) - l * s_b[i - 1];
          if (fabs(d) < piv) d = copysign(piv, d);
          invd[i * kInvBatch + tid] = 1.0 / d;
        }
#pragma unroll 2
        for (int i = 0; i < N; ++i) {
          const uint32_t h = hash3(a.seed ^ (uint32_t)u, (uint32_t)j, (uint32_t)i);
          xv[i * kInvBatch + tid] = (double)(h >> 11) * (1.0 / 2097152.0) - 1.0;
        }
        for (int itr = 0; itr < 3; ++itr) {
          double z = xv[tid];
#pragma unroll 2
          for (int i = 1; i < N; ++i) {
            z = xv[i * kInvBatch + tid] - s_b[i - 1] * invd[(i - 1) * kInvBatch + tid] * z;
            xv[i * kInvBatch + tid] = z;
          }
          double x = xv[(N - 1) * kInvBatch + tid] * invd[(N - 1) * kInvBatch + tid];
          xv[(N - 1) * kInvBatch + tid] = x;
          double mx = fabs(x);
#pragma unroll 2
          for (int i = N - 2; i >= 0; --i) {
            x = (xv[i * kInvBatch + tid] - s_b[i] * x) * invd[i * kInvBatch + tid];
            xv[i * kInvBatch + tid] = x;
            mx = fmax(mx, fabs(x));
          }
          const double sc = mx > 0.0 ? 1.0 / mx : 1.0;
          double ss = 0.0;
#pragma unroll 2
          for (int i = 0; i < N; ++i) {
            const double y = xv[i * kInvBatch + tid] * sc;
            ss += y * y;
          }
          const double f = sc / sqrt(ss);
#pragma unroll 2
          for (int i = 0; i < N; ++i) xv[i * kInvBatch + tid] *= f;
        }
#pragma unroll 2
        for (int i = 0; i < N; ++i) gvec[(size_t)j * N + i] = xv[i * kInvBatch + tid];
      }
      __syncthreads();
    }
    // X[j][i] in LDS (fp32 storage, fp64 arithmetic below)
    for (int e = tid; e < r * N; e += kEigThreads) X[e] = (float)gvec[e];
    __syncthreads();

    // modified Gram-Schmidt
    for (int j = 0; j < r; ++j) {
      if (wave == 0) {
        double s = 0.0;
        for (int i = lane; i < N; i += kWave) s += (double)X[j * N + i] * X[j * N + i];
        s = wave_sum(s);
        const double f = 1.0 / sqrt(s);
        for (int i = lane; i < N; i += kWave) X[j * N + i] = (float)(X[j * N + i] * f);
      }
      __syncthreads();
      for (int k = j + 1 + wave; k < r; k += kEigWaves) {
        double s = 0.0;
        for (int i = lane; i < N; i += kWave) s += (double)X[j * N + i] * X[k * N + i];
        s = wave_sum(s);
        for (int i = lane; i < N; i += kWave) X[k * N + i] = (float)(X[k * N + i] - s * X[j * N + i]);
      }
      __syncthreads();
    }

    __syncthreads();
  }

  // ---- 5. back-transformation X <- H_0 H_1 ... H_{N-3} X, canonical sign, output ---------------------------------
  // Eight lanes per vector: vector jv = tid / 8 keeps positions sub * PB .. sub * PB + PB - 1 (sub = tid % 8) in fp32
  // registers.  Reflectors are staged kReflChunk at a time at their absolute positions (zero up to k), so the steps
  // inside a chunk need no barrier.
  constexpr int PB = N / 8;
  const int jv = tid >> 3, sub = tid & 7;
  const bool wave_act = wave * (kWave / 8) < r;  // uniform
  float xr[PB];
  if (jv < r) {
#pragma unroll
    for (int i = 0; i < PB; i += 4) {
      const float4 x4 = *reinterpret_cast<const float4*>(&X[jv * N + sub * PB + i]);
      xr[i] = x4.x;
      xr[i + 1] = x4.y;
      xr[i + 2] = x4.z;
      xr[i + 3] = x4.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < PB; ++i) xr[i] = 0.0f;
  }
  if (tnorm != 0.0) {
    for (int kc = N - 3; kc >= 0; kc -= kReflChunk) {
      const int nk = min(kReflChunk, kc + 1);
      __syncthreads();
      for (int e = tid; e < nk * N; e += kEigThreads) {
        const int c = e / N, pos = e - c * N;
        const int k = kc - c;
        s_rb[c * N + pos] = pos > k ? (float)refl[k * N + pos - k - 1] : 0.0f;
      }
      for (int c = tid; c < nk; c += kEigThreads) s_rbeta[c] = (float)refl_beta[kc - c];
      __syncthreads();
      if (wave_act) {
        for (int c = 0; c < nk; ++c) {
          const float beta = s_rbeta[c];
          float v[PB];
#pragma unroll
          for (int i = 0; i < PB; i += 4) {
            const float4 v4 = *reinterpret_cast<const float4*>(&s_rb[c * N + sub * PB + i]);
            v[i] = v4.x;
            v[i + 1] = v4.y;
            v[i + 2] = v4.z;
            v[i + 3] = v4.w;
          }
          float d0 = 0.0f, d1 = 0.0f;
#pragma unroll
          for (int i = 0; i < PB; i += 2) {
            d0 = fmaf(xr[i], v[i], d0);
            d1 = fmaf(xr[i + 1], v[i + 1], d1);
          }
          const float sc = beta * sum8(d0 + d1);
#pragma unroll
          for (int i = 0; i < PB; ++i) xr[i] = fmaf(-sc, v[i], xr[i]);
        }
      }
    }
  }

  // canonical sign: the largest-magnitude entry positive; entries within 2^-20 of it count as ties, the first wins
  if (wave_act) {
    float mx = 0.0f;
#pragma unroll
    for (int i = 0; i < PB; ++i) mx = fmaxf(mx, fabsf(xr[i]));
    mx = max8(mx);
    const float thr = (float)((double)mx * (1.0 - 9.5367431640625e-07));
    int key = 2 * N;  // 2 * position + sign bit of the first entry at or above the threshold
#pragma unroll
    for (int i = PB - 1; i >= 0; --i)
      if (fabsf(xr[i]) >= thr) key = 2 * (sub * PB + i) + (xr[i] < 0.0f ? 1 : 0);
    key = min8(key);
    const float sgn = (key < 2 * N && (key & 1)) ? -1.0f : 1.0f;
    if (jv < r) {
#pragma unroll
      for (int i = 0; i < PB; i += 4)
        *reinterpret_cast<float4*>(&tg.basis[(size_t)jv * N + sub * PB + i]) =
            make_float4(sgn * xr[i], sgn * xr[i + 1], sgn * xr[i + 2], sgn * xr[i + 3]);
      if (sub == 0 && tg.sigma) tg.sigma[jv] = (float)sqrt(fmax(s_lam[jv], 0.0));
    }
  }
}

size_t eig_lds_bytes(int n) { return n == 64 ? EigLds<64>::kTotal : EigLds<128>::kTotal; }

hipError_t launch_eig(const EigArgs& a, hipStream_t stream) {
  if (a.num_units == 0) return hipSuccess;
  const size_t lds = eig_lds_bytes(a.n);
  hipError_t e;
  if (a.n == 64) {
    e = hipFuncSetAttribute((const void*)eig_topr<64>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(eig_topr<64>, dim3(a.num_units), dim3(kEigThreads), lds, stream, a);
  } else {
    e = hipFuncSetAttribute((const void*)eig_topr<128>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(eig_topr<128>, dim3(a.num_units), dim3(kEigThreads), lds, stream, a);
  }
  return hipGetLastError();
}

}  // namespace kvc
