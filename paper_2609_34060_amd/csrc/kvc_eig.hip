// Top-r eigenpairs of the per-unit d x d Gram matrices in fp64: the right singular vectors R_r and singular values
// of Eq. 7 (Z^T Z = R Sigma^2 R^T).  One workgroup of 1024 threads per (layer, K/V, head) unit:
//   1. G = sum of the unit's fp32 partial Grams in a fixed order in fp64 (or a dense fp64 matrix), into LDS.
//   2. Householder tridiagonalisation G = Q T Q^T in fp64 arithmetic; the trailing matrix is kept in LDS in fp32
//      (the Gram itself carries fp32 accuracy), which lets two units share a CU; the reflectors go to the workspace.
//   3. Multisection bisection with Sturm counts for the r largest eigenvalues of T: a first step shared by all
//      targets (every lane's shifts cut the whole interval), then groups of lanes per eigenvalue, kBisShifts
//      shifts per lane, one ballot per shift.
//   4. Inverse iteration on T (LDL^T without pivoting, tiny pivots replaced) from pseudo-random starts, one lane
//      per eigenvector; then modified Gram-Schmidt within each cluster of close eigenvalues.  Vectors of tightly
//      clustered eigenvalues come out as an orthonormal basis of the cluster's invariant subspace (where the SVD
//      itself is not unique).
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
constexpr int kBisShifts = 2;   // Sturm counts per lane and bisection step (even: whole int2 slices below)
// Inverse-iteration solves per eigenvector: with lambda within about 2^-24 of the spectrum's width, each solve
// shrinks the other eigenvectors' components by that error over their gap, so two solves leave a residual far
// below the fp32 rounding of the reduced matrix (about 1e-11 of the width in an fp64 simulation of the recurrence
// on decaying and flat spectra).
constexpr int kInvSolves = 2;

// fp64 cross-lane move by DPP (two 32-bit halves).  Lanes whose row is masked off keep an undefined value: the only
// user reads a lane that every step writes.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ double dpp64(double x) {
  const unsigned long long b = __builtin_bit_cast(unsigned long long, x);
  const int lo = __builtin_amdgcn_mov_dpp((int)(unsigned)b, CTRL, ROW_MASK, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp((int)(unsigned)(b >> 32), CTRL, ROW_MASK, 0xF, false);
  return __builtin_bit_cast(double, ((unsigned long long)(unsigned)hi << 32) | (unsigned)lo);
}
constexpr int kDppRor1 = 0x121, kDppRor2 = 0x122, kDppRor4 = 0x124, kDppRor8 = 0x128;
constexpr int kDppBcast15 = 0x142, kDppBcast31 = 0x143;

__device__ __forceinline__ double lane_value(double x, int l) {
  const unsigned long long b = __builtin_bit_cast(unsigned long long, x);
  const unsigned lo = __builtin_amdgcn_readlane((int)(unsigned)b, l);
  const unsigned hi = __builtin_amdgcn_readlane((int)(unsigned)(b >> 32), l);
  return __builtin_bit_cast(double, ((unsigned long long)hi << 32) | lo);
}
// Whole-wave reduction by op in a fixed order (deterministic), returned in every lane: within rows of 16 lanes,
// then the row broadcasts carry rows 0-2 into row 3, whose last lane holds the result.  Called with the whole wave
// active.
template <class Op>
__device__ __forceinline__ double wave_reduce(double x, Op op) {
  x = op(x, dpp64<kDppRor8>(x));
  x = op(x, dpp64<kDppRor4>(x));
  x = op(x, dpp64<kDppRor2>(x));
  x = op(x, dpp64<kDppRor1>(x));
  x = op(x, dpp64<kDppBcast15, 0xA>(x));
  x = op(x, dpp64<kDppBcast31, 0xC>(x));
  return lane_value(x, 63);
}
__device__ __forceinline__ double wave_sum(double x) {
  return wave_reduce(x, [](double u, double v) { return u + v; });
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
__device__ __forceinline__ int sum8i(int x) {
  x += dpp32i<kDppXor1>(x);
  x += dpp32i<kDppXor2>(x);
  return x + dpp32i<kDppHalfMirror>(x);
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
  // ||x|| from the hardware reciprocal square root and one Newton step (s is 0 or a normal number)
  const double y0 = __builtin_amdgcn_rsq(s);
  const double g0 = s * y0, h0 = 0.5 * y0;
  const double nrm = s == 0.0 ? 0.0 : fma(g0, fma(-g0, h0, 0.5), g0);
  const double alpha = nrm == 0.0 ? 0.0 : -copysign(nrm, x0);
  out[0] = alpha;
  out[1] = x0 - alpha;
  out[2] = nrm == 0.0 ? 0.0 : recip(nrm * (nrm + fabs(x0)));
}

// Numbers of eigenvalues of T below each of the M shifts x[m]: the ratio form of the Sturm sequence, q_i = (a_i - x)
// - b_{i-1}^2 / q_{i-1}, with the hardware reciprocal (relative error below 2^-24, measured on random fp64 inputs)
// and IEEE infinities in place of a pivot guard: a zero pivot makes the next one -inf (counted), and the one after
// that is plain a - x again, the same count the classical replacement of tiny pivots gives.  b^2 is floored at the
// smallest normal number so that b^2 times an infinite reciprocal is never 0 * inf.  Each count is exact for T with
// every b^2 perturbed by at most 2^-24 relative, below the perturbation fp32 storage of the matrix carries.  The M
// recurrences are independent, so their latencies overlap, and they share the loads of T.
template <int N, int M>
__device__ __forceinline__ void sturm_counts(const double* sa, const double* sb2, const double* x, int* cnt) {
  double q[M];
#pragma unroll
  for (int m = 0; m < M; ++m) {
    q[m] = sa[0] - x[m];
    cnt[m] = q[m] < 0.0;
  }
#pragma unroll 4
  for (int i = 1; i < N; ++i) {
    const double ai = sa[i], bi = sb2[i - 1];
#pragma unroll
    for (int m = 0; m < M; ++m) {
      q[m] = fma(-bi, __builtin_amdgcn_rcp(q[m]), ai - x[m]);
      cnt[m] += q[m] < 0.0;
    }
  }
}

// ---- Householder tridiagonalisation ----------------------------------------------------------------------------
// Step k reflects x = row k beyond the diagonal (the matrix is symmetric) onto alpha e_1 with H_k = I - beta v v^T,
// v = x - alpha e_1; with p = A22 v, K = (beta^2 / 2) v^T p and w = beta p - K v, A22 <- A22 - v w^T - w v^T.
// The matrix lives in LDS as fp32 [N][N]; the rank-2 update is two fp32 fmas per entry (v and w rounded to fp32),
// each wave's share of A22 v is an fp32 sum over its rows, and the rest (the shares' total p, K, w, the scalars,
// the reflectors) is fp64.
//
// kTriWaves waves (one per SIMD) run the reduction with one workgroup barrier per step.  Lane l of every wave owns
// the CPL = N / 64 consecutive columns CPL l ..; row R belongs to wave R mod kTriWaves.  The update of step k - 1 is
// applied lazily: step k
//   1. brings row k up to date in registers (every wave, from the same LDS row), forms the reflector (every wave
//      the same scalars; wave 0 writes the reflector, alpha and the diagonal entry),
//   2. sweeps the wave's rows R > k: applies the pending update to them and accumulates the wave's share of A22 v
//      (fp32 fmas of the fp32 entries and the fp32 copy of v over the wave's rows; the shares are summed in fp64),
//   3. after the barrier, sums the shares in a fixed order, so K and w, the next pending update, come out
//      identical in every wave.
// s_vw[R] = {v_R, w_R} of the pending update and v'_R of the current step; every wave writes the same values to
// it, each before reading them (LDS operations of one wave complete in issue order; the fences below stop the
// compiler from moving LDS accesses across the points where other lanes' values are read).  The shares are double
// buffered by step parity: a wave writes step k + 1's share only after the barrier that follows every wave's reads
// of step k - 1's.
constexpr int kTriWaves = 4;

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Waves 0 .. kTriWaves - 1 of the workgroup; the other waves meet the same N - 2 barriers.  Writes s_a (the diagonal
// of T), s_b[0 .. N - 2] (its off-diagonal), the reflectors (v of step k in refl[k N ..]) and their beta.
template <int N>
__device__ __forceinline__ void tri_reduce(float* A, float4* s_vw, double* share, double* s_a, double* s_b,
                                           double* refl, double* refl_beta, int lane, int wave) {
  constexpr int CPL = N / kWave;
  constexpr int W = kTriWaves;
  if (wave >= W) {
    for (int k = 0; k < N - 2; ++k) __syncthreads();
    return;
  }
  float vpf[CPL], wpf[CPL];  // pending update of the lane's columns (fp32, as applied)
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    vpf[c] = wpf[c] = 0.0f;
    *reinterpret_cast<float2*>(&s_vw[CPL * lane + c]) = make_float2(0.0f, 0.0f);
  }
  auto upd = [&](float a, const float4& vw, int c) { return fmaf(-vw.x, wpf[c], fmaf(-vw.y, vpf[c], a)); };
  // row k as the sweep of step k - 1 left it (loaded right after that step's barrier) and its pending-update
  // scalars {v_k, w_k} (taken from the lane that holds column k, not through LDS)
  float ak[CPL];
  float4 vwk = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
  for (int c = 0; c < CPL; ++c) ak[c] = A[CPL * lane + c];
  for (int k = 0; k < N - 2; ++k) {
    const int k1 = k + 1;
    // 1. row k under the pending update; its entries beyond the diagonal are x
    double x[CPL];
    double ss = 0.0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int C = CPL * lane + c;
      const float a = upd(ak[c], vwk, c);
      if (wave == 0 && C == k) s_a[k] = (double)a;
      x[c] = C > k ? (double)a : 0.0;
      ss += x[c] * x[c];
    }
    ss = wave_sum(ss);
    const double x0 = lane_value(x[k1 % CPL], k1 / CPL);
    double ab[3];
    reflector_scalars(x0, ss, ab);
    const double beta = ab[2];
    double v[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int C = CPL * lane + c;
      v[c] = C > k1 ? x[c] : (C == k1 ? ab[1] : 0.0);
      s_vw[C].z = (float)v[c];
    }
    if (wave == 0) {
      double* refl_k = refl + __builtin_amdgcn_readfirstlane(k * N);
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        if (CPL * lane + c >= k1) refl_k[CPL * lane + c - k1] = v[c];
      if (lane == 0) {
        s_b[k] = ab[0];
        refl_beta[k] = beta;
      }
    }
    wave_lds_sync();
    // 2. the wave's rows R > k: the pending update, then p += a v'_R
    float pf[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) pf[c] = 0.0f;
    const int R0 = k1 + ((wave - k1) % W + W) % W;  // first row > k of this wave
    int R = R0;
    for (; R + 3 * W < N; R += 4 * W) {
      float4 vw[4];
      float a[4][CPL];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        vw[j] = s_vw[R + j * W];
#pragma unroll
        for (int c = 0; c < CPL; ++c) a[j][c] = A[(R + j * W) * N + CPL * lane + c];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          a[j][c] = upd(a[j][c], vw[j], c);
          A[(R + j * W) * N + CPL * lane + c] = a[j][c];
          pf[c] = fmaf(a[j][c], vw[j].z, pf[c]);
        }
    }
    if (R < N) {
      // the last 1 - 3 rows, loaded together (a missing row re-reads row R and is neither stored nor counted)
      const int m = (N - 1 - R) / W + 1;
      float4 vw[3];
      float a[3][CPL];
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        const int Rj = j < m ? R + j * W : R;
        vw[j] = s_vw[Rj];
#pragma unroll
        for (int c = 0; c < CPL; ++c) a[j][c] = A[Rj * N + CPL * lane + c];
      }
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        if (j < m) {
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            a[j][c] = upd(a[j][c], vw[j], c);
            A[(R + j * W) * N + CPL * lane + c] = a[j][c];
            pf[c] = fmaf(a[j][c], vw[j].z, pf[c]);
          }
        }
      }
    }
    double* sh = share + (k & 1) * W * N;
#pragma unroll
    for (int c = 0; c < CPL; ++c) sh[wave * N + CPL * lane + c] = (double)pf[c];
    __syncthreads();
#pragma unroll
    for (int c = 0; c < CPL; ++c) ak[c] = A[k1 * N + CPL * lane + c];
    // 3. p = the sum of the shares; K = (beta^2 / 2) v^T p; w = beta p - K v becomes the pending update
    double kk = 0.0, p[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      double t = sh[CPL * lane + c];
#pragma unroll
      for (int w = 1; w < W; ++w) t += sh[w * N + CPL * lane + c];
      p[c] = t;
      kk += CPL * lane + c > k ? v[c] * t : 0.0;
    }
    const double K = 0.5 * beta * beta * wave_sum(kk);
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int C = CPL * lane + c;
      vpf[c] = (float)v[c];
      wpf[c] = C > k ? (float)(beta * p[c] - K * v[c]) : 0.0f;
      *reinterpret_cast<float2*>(&s_vw[C]) = make_float2(vpf[c], wpf[c]);
    }
    float vsel = vpf[0], wsel = wpf[0];
#pragma unroll
    for (int c = 1; c < CPL; ++c)
      if (k1 % CPL == c) {
        vsel = vpf[c];
        wsel = wpf[c];
      }
    vwk.x = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, vsel), k1 / CPL));
    vwk.y = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wsel), k1 / CPL));
  }
  // the last pending update on the trailing 2 x 2 block
  if (wave == 0) {
    wave_lds_sync();
#pragma unroll
    for (int R = N - 2; R < N; ++R) {
      const float4 vw = s_vw[R];
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int C = CPL * lane + c;
        const float a = upd(A[R * N + C], vw, c);
        if (C == R) s_a[R] = (double)a;
        if (R == N - 2 && C == N - 1) s_b[N - 2] = (double)a;
      }
    }
  }
}

// LDS layout (bytes): the matrix region MREG holds, in turn, G / the trailing matrix as fp32 [N][N] (phases 1-2),
// the inverse-iteration scratch fp64 [N][kInvBatch] x 2 (phase 4), X fp32 [r][N] (MGS, back-transformation); then
// fp64 scalars and vectors; then the staging region: the sweep's per-wave shares of A22 v, fp64 [2][kTriWaves][N],
// during phase 2, a chunk of reflectors during phase 5.  About 79 KB for N = 128, so two units share a CU.
template <int N>
struct EigLds {
  static constexpr size_t kMat = (size_t)N * N * 4;
  static constexpr size_t kScratch = (size_t)2 * N * kInvBatch * 8;
  static constexpr size_t kX = (size_t)KVC_MAX_RANK * N * 4;
  static constexpr size_t kMreg = ((kMat > kScratch ? (kMat > kX ? kMat : kX) : (kScratch > kX ? kScratch : kX)) +
                                   15) / 16 * 16;
  // s_a, s_b [N]; s_lam [KVC_MAX_RANK]; s_misc [8]; s_vw float4 [N] (later b^2 [N])
  static constexpr size_t kSmall = (size_t)(2 * N + KVC_MAX_RANK + 8) * 8 + (size_t)N * 16;
  static constexpr size_t kShare = (size_t)2 * kTriWaves * N * 8;
  static constexpr size_t kReflStage = (size_t)kReflChunk * (N + 1) * 4;
  static constexpr size_t kStage = kShare > kReflStage ? kShare : kReflStage;
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
  double* s_misc = s_lam + KVC_MAX_RANK;    // scalars
  float4* s_vw = reinterpret_cast<float4*>(s_misc + 8);  // {v_C, w_C, v'_C, -} of the tridiagonalisation
  double* s_b2 = reinterpret_cast<double*>(s_vw);        // b^2 (after the tridiagonalisation)
  double* share = reinterpret_cast<double*>(base + Lay::kMreg + Lay::kSmall);  // shares of A22 v [2][W][N]
  float* s_rb = reinterpret_cast<float*>(share);  // reflector chunk fp32 [kReflChunk][N] (back-transformation)
  float* s_rbeta = s_rb + kReflChunk * N;

  const int u = blockIdx.x;
  if (a.skip && a.skip[u]) return;  // whole workgroup
  const UnitTarget tg = eig_target(a, u);
  const int r = tg.rank;
  if (r <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  double* refl = a.reflect + (size_t)u * N * N;          // v_k in row k
  double* refl_beta = a.reflect_beta + (size_t)u * N;
  double* gvec = a.vecs + (size_t)u * N * KVC_MAX_RANK;  // eigenvectors of T, vector j in row j

  // ---- 1. load G ------------------------------------------------------------------------------------------
  // Each thread takes Q groups of 4 consecutive entries; every load of a partial (or of the dense matrix) is issued
  // before its values are added, and the partials are added in order c = 0, 1, ... in fp64.
  static_assert(LD == N && (N * N) % (4 * kEigThreads) == 0, "whole float4 groups per thread");
  constexpr int Q = N * N / (4 * kEigThreads);
  if (a.partials) {
    const int parts = (tg.tokens + a.part_tokens - 1) / a.part_tokens;
    const float4* P4 = reinterpret_cast<const float4*>(a.partials + (size_t)u * a.max_parts * N * N);
    double acc[Q][4];
#pragma unroll
    for (int q = 0; q < Q; ++q) acc[q][0] = acc[q][1] = acc[q][2] = acc[q][3] = 0.0;
#pragma unroll 2
    for (int c = 0; c < parts; ++c) {
      float4 v[Q];
#pragma unroll
      for (int q = 0; q < Q; ++q) v[q] = P4[(size_t)c * (N * N / 4) + tid + q * kEigThreads];
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        acc[q][0] += (double)v[q].x;
        acc[q][1] += (double)v[q].y;
        acc[q][2] += (double)v[q].z;
        acc[q][3] += (double)v[q].w;
      }
    }
#pragma unroll
    for (int q = 0; q < Q; ++q)
      reinterpret_cast<float4*>(A)[tid + q * kEigThreads] =
          make_float4((float)acc[q][0], (float)acc[q][1], (float)acc[q][2], (float)acc[q][3]);
  } else {
    const double2* D2 = reinterpret_cast<const double2*>(a.dense + (size_t)u * N * N);
    double2 v[2 * Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      v[2 * q] = D2[2 * (tid + q * kEigThreads)];
      v[2 * q + 1] = D2[2 * (tid + q * kEigThreads) + 1];
    }
#pragma unroll
    for (int q = 0; q < Q; ++q)
      reinterpret_cast<float4*>(A)[tid + q * kEigThreads] =
          make_float4((float)v[2 * q].x, (float)v[2 * q].y, (float)v[2 * q + 1].x, (float)v[2 * q + 1].y);
  }
  __syncthreads();

  // ---- 2. Householder tridiagonalisation ------------------------------------------------------------------------
  tri_reduce<N>(A, s_vw, share, s_a, s_b, refl, refl_beta, lane, wave);
  __syncthreads();
  for (int i = tid; i < N - 1; i += kEigThreads) s_b2[i] = fmax(s_b[i] * s_b[i], 2.2250738585072014e-308);
  if (wave == 0) {
    // Gershgorin interval of T (minima and maxima: any order gives the same result)
    double lo = s_a[0], hi = s_a[0];
#pragma unroll
    for (int q = 0; q < N / kWave; ++q) {
      const int i = lane + kWave * q;
      const double rad = (i > 0 ? fabs(s_b[i - 1]) : 0.0) + (i < N - 1 ? fabs(s_b[i]) : 0.0);
      lo = fmin(lo, s_a[i] - rad);
      hi = fmax(hi, s_a[i] + rad);
    }
    lo = wave_reduce(lo, [](double x, double y) { return fmin(x, y); });
    hi = wave_reduce(hi, [](double x, double y) { return fmax(x, y); });
    if (lane == 0) {
      const double tnorm = fmax(fabs(lo), fabs(hi));
      const double pad = 2.0 * 2.220446049250313e-16 * tnorm * N + 2.2250738585072014e-308;
      s_misc[1] = lo - pad;
      s_misc[2] = hi + pad;
      s_misc[3] = tnorm;
    }
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
      // P lanes per eigenvalue, each evaluating kBisShifts shifts: the bracket is cut into S = P kBisShifts + 1
      // pieces per step
      constexpr int P = 8;
      static_assert(kEigThreads / KVC_MAX_RANK >= P, "P lanes for every eigenvalue");
      constexpr int S = P * kBisShifts + 1;
      // (tid passes through an empty asm so that the compiler does not keep tid / P live until the
      // back-transformation, which takes the same quotient, and spill it)
      int tidb = tid;
      asm volatile("" : "+v"(tidb));
      const int grp = tidb / P, s = tidb - grp * P;
      const int kasc = N - 1 - grp;                  // ascending index of the target eigenvalue
      double lo = s_misc[1], hi = s_misc[2];
      // First step, shared by all targets: the rp P lanes cut the Gershgorin interval at M = rp P kBisShifts
      // points (counts to LDS, in the matrix region, free since the reduction); each target's lanes then count
      // the cut points left of it, so every bracket starts at 1 / (M + 1) of the interval.
      const int M = rp * P * kBisShifts;
      int* s_cnt = reinterpret_cast<int*>(A);
      if (tid < rp * P) {
        double x[kBisShifts];
        int c[kBisShifts];
#pragma unroll
        for (int m = 0; m < kBisShifts; ++m) {
          x[m] = lo + (hi - lo) * (double)(tid * kBisShifts + m + 1) / (double)(M + 1);
          c[m] = 0;
        }
        sturm_counts<N, kBisShifts>(s_a, s_b2, x, c);
#pragma unroll
        for (int m = 0; m < kBisShifts; ++m) s_cnt[tid * kBisShifts + m] = c[m];
      }
      __syncthreads();
      if (grp < rp) {
        // counts do not decrease along the cut points, so those left of the target are a prefix; lane s scans
        // the s-th of P equal slices
        const int per = M / P;  // rp kBisShifts, even
        int left = 0;
#pragma unroll 4
        for (int j = s * per; j < (s + 1) * per; j += 2) {
          const int2 c2 = *reinterpret_cast<const int2*>(&s_cnt[j]);
          left += (c2.x <= kasc) + (c2.y <= kasc);
        }
        left = sum8i(left);
        const double nlo = left == 0 ? lo : lo + (hi - lo) * (double)left / (double)(M + 1);
        const double nhi = left == M ? hi : lo + (hi - lo) * (double)(left + 1) / (double)(M + 1);
        lo = nlo;
        hi = nhi;
      }
      // then S-way steps per target until the bracket is below 2^-25 of the Gershgorin interval, the accuracy of
      // the counts themselves
      int iters = 0;
      for (double w = (double)(M + 1); w < 33554432.0; w *= S) ++iters;
      for (int it = 0; it < iters; ++it) {
        double x[kBisShifts];
        int c[kBisShifts];
#pragma unroll
        for (int m = 0; m < kBisShifts; ++m) {
          x[m] = lo + (hi - lo) * (double)(s * kBisShifts + m + 1) / (double)S;
          c[m] = 0;
        }
        if (grp < r) sturm_counts<N, kBisShifts>(s_a, s_b2, x, c);
        // shifts left of the target form a prefix of the S - 1 cut points; sstar counts them
        int sstar = 0;
#pragma unroll
        for (int m = 0; m < kBisShifts; ++m) {
          const uint64_t mask = __ballot(c[m] <= kasc);
          sstar += __popcll((mask >> ((lane / P) * P)) & ((1ull << P) - 1ull));
        }
        const double nlo = sstar == 0 ? lo : lo + (hi - lo) * (double)sstar / (double)S;
        const double nhi = sstar == S - 1 ? hi : lo + (hi - lo) * (double)(sstar + 1) / (double)S;
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
        // LDL^T of T - lam I without pivoting (tiny pivots replaced): invd[i] = 1 / d_i, in one pass with the
        // pseudo-random start x and the first solve's forward substitution z_i = x_i - b_{i-1} z_{i-1} / d_{i-1}
        // (which needs 1 / d_{i-1} only), so the start is never stored and the forward chain and the start's hash
        // run beside the reciprocals.  The recurrences read T and the scratch in chunks loaded ahead of the chunk's
        // stores, so one LDS round trip serves a chunk instead of each step waiting for its own loads behind the
        // previous store.
        static_assert(N % 4 == 0, "whole chunks");
        {
          double id = 0.0, z = 0.0;
          for (int i0 = 0; i0 < N; i0 += 4) {
            double av[4], bv[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              av[t] = s_a[i0 + t];
              bv[t] = s_b[i0 + t > 0 ? i0 + t - 1 : 0];
            }
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int i = i0 + t;
              const uint32_t h = hash3(a.seed ^ (uint32_t)u, (uint32_t)j, (uint32_t)i);
              const double x0 = (double)(h >> 11) * (1.0 / 2097152.0) - 1.0;
              z = i > 0 ? x0 - bv[t] * id * z : x0;
              xv[i * kInvBatch + tid] = z;
              double d = i > 0 ? (av[t] - lam) - bv[t] * id * bv[t] : av[t] - lam;
              if (fabs(d) < piv) d = copysign(piv, d);
              id = recip(d);
              invd[i * kInvBatch + tid] = id;
            }
          }
        }
        // kInvSolves solves (T - lam I) x_new = x; each right-hand side is scaled by 1 / max|x| on the way in (the
        // first solve's forward substitution is done above, with scale 1)
        double sc = 1.0;
        for (int itr = 0; itr < kInvSolves; ++itr) {
          double z = 0.0;
          for (int i0 = 0; itr > 0 && i0 < N; i0 += 4) {
            double xw[4], bw[4], iw[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int i = i0 + t, im = i > 0 ? i - 1 : 0;
              xw[t] = xv[i * kInvBatch + tid];
              bw[t] = s_b[im];
              iw[t] = invd[im * kInvBatch + tid];
            }
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              z = i0 + t > 0 ? xw[t] * sc - bw[t] * iw[t] * z : xw[t] * sc;
              xv[(i0 + t) * kInvBatch + tid] = z;
            }
          }
          double x = 0.0, mx = 0.0;
          for (int i1 = N - 1; i1 >= 0; i1 -= 4) {
            double xw[4], bw[4], iw[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int i = i1 - t;
              xw[t] = xv[i * kInvBatch + tid];
              bw[t] = s_b[i < N - 1 ? i : 0];
              iw[t] = invd[i * kInvBatch + tid];
            }
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              x = i1 - t == N - 1 ? xw[t] * iw[t] : (xw[t] - bw[t] * x) * iw[t];
              xv[(i1 - t) * kInvBatch + tid] = x;
              mx = fmax(mx, fabs(x));
            }
          }
          sc = mx > 0.0 ? 1.0 / mx : 1.0;
        }
        double ss = 0.0;
#pragma unroll 4
        for (int i = 0; i < N; ++i) {
          const double y = xv[i * kInvBatch + tid] * sc;
          ss += y * y;
        }
        const double f = sc / sqrt(ss);
#pragma unroll 4
        for (int i = 0; i < N; ++i) gvec[(size_t)j * N + i] = xv[i * kInvBatch + tid] * f;
      }
      __syncthreads();
    }
    // X[j][i] in LDS (fp32 storage, fp64 arithmetic below)
    for (int e = tid; e < r * N; e += kEigThreads) X[e] = (float)gvec[e];
    __syncthreads();

    // modified Gram-Schmidt within clusters, one barrier per vector that has a later cluster member: the wave that
    // takes vector j + 1 in round j (wave 0) also normalises it, so vector j is normalised when round j starts
    constexpr int QN = N / kWave;
    auto normalise = [&](float* x) {
      double s = 0.0;
#pragma unroll
      for (int q = 0; q < QN; ++q) s += (double)x[q] * x[q];
      s = wave_sum(s);
      // 1 / sqrt(s) from the hardware reciprocal square root and one Newton step
      const double y0 = __builtin_amdgcn_rsq(s);
      const double f = y0 * fma(-0.5 * s * y0, y0, 1.5);
#pragma unroll
      for (int q = 0; q < QN; ++q) x[q] = (float)(x[q] * f);
    };
    // Clusters: runs of eigenvalues whose consecutive gaps are at most 1e-3 of the norm of T (the reorthogonalisation
    // criterion of LAPACK's inverse iteration, stein).  A vector is orthogonalised against the earlier vectors of its
    // cluster only: the bisection's eigenvalues lie within about 2^-24 of the norm of T of the exact ones, so each
    // inverse-iteration solve scales a vector's components along eigenvectors at least 1e-3 away by at most
    // 2^-24 / 1e-3 relative to its own, and the two solves leave vectors of different clusters orthogonal to about
    // 4e-9 of the start's components.  The first vector of a cluster keeps the inverse iteration's normalisation.
    // Bit j of the mask: vectors j and j + 1 share a cluster.
    const double ctol = 1e-3 * tnorm;
    static_assert(KVC_MAX_RANK <= 2 * kWave, "two mask words");
    const uint64_t m0 = __ballot(lane + 1 < r && s_lam[lane] - s_lam[lane + 1] <= ctol);
    const uint64_t m1 = __ballot(lane + kWave + 1 < r && s_lam[lane + kWave] - s_lam[lane + kWave + 1] <= ctol);
    auto joined = [&](int j) { return ((j < kWave ? m0 >> j : m1 >> (j - kWave)) & 1ull) != 0; };
    int cend = 0;  // last index of the cluster of vector j (uniform)
    for (int j = 0; j < r; ++j) {
      if (!joined(j)) continue;
      if (cend <= j) {
        cend = j + 1;
        while (joined(cend)) ++cend;
      }
      for (int k = j + 1 + wave; k <= cend; k += kEigWaves) {
        float xj[QN], xk[QN];
        double s = 0.0;
#pragma unroll
        for (int q = 0; q < QN; ++q) {
          xj[q] = X[j * N + lane + kWave * q];
          xk[q] = X[k * N + lane + kWave * q];
          s += (double)xj[q] * xk[q];
        }
        s = wave_sum(s);
#pragma unroll
        for (int q = 0; q < QN; ++q) xk[q] = (float)(xk[q] - s * xj[q]);
        if (k == j + 1) normalise(xk);
#pragma unroll
        for (int q = 0; q < QN; ++q) X[k * N + lane + kWave * q] = xk[q];
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
    // each chunk's reflectors are read from the workspace into registers one chunk ahead, so that the global
    // loads run while the previous chunk is applied
    constexpr int EPT = (kReflChunk * N + kEigThreads - 1) / kEigThreads;
    static_assert(kReflChunk <= kEigThreads, "one beta per thread");
    float pre[EPT], preb = 0.0f;
    auto fetch = [&](int kc) {
      const int nk = min(kReflChunk, kc + 1);
#pragma unroll
      for (int q = 0; q < EPT; ++q) {
        const int e = tid + q * kEigThreads;
        float v = 0.0f;
        if (e < nk * N) {
          const int c = e / N, pos = e - c * N;
          const int k = kc - c;
          if (pos > k) v = (float)refl[k * N + pos - k - 1];
        }
        pre[q] = v;
      }
      preb = tid < nk ? (float)refl_beta[kc - tid] : 0.0f;
    };
    fetch(N - 3);
    for (int kc = N - 3; kc >= 0; kc -= kReflChunk) {
      const int nk = min(kReflChunk, kc + 1);
      __syncthreads();
#pragma unroll
      for (int q = 0; q < EPT; ++q) {
        const int e = tid + q * kEigThreads;
        if (e < nk * N) s_rb[e] = pre[q];
      }
      if (tid < nk) s_rbeta[tid] = preb;
      __syncthreads();
      if (kc >= kReflChunk) fetch(kc - kReflChunk);
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
