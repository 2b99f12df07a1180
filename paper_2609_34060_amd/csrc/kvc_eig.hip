// Top-r eigenpairs of the per-unit d x d Gram matrices in fp64: the right singular vectors R_r and singular values
// of Eq. 7 (Z^T Z = R Sigma^2 R^T).  One workgroup of 1024 threads per (layer, K/V, head) unit:
//   1. G = sum of the unit's fp32 partial Grams in a fixed order (or a dense fp64 matrix), into LDS.
//   2. Householder tridiagonalisation G = Q T Q^T in LDS; the reflectors go to the workspace.
//   3. Multisection bisection with Sturm counts for the r largest eigenvalues of T (groups of lanes per
//      eigenvalue, one ballot per step).
//   4. Inverse iteration on T (LDL^T without pivoting, tiny pivots replaced) from pseudo-random starts, one lane
//      per eigenvector; then modified Gram-Schmidt over the r vectors.  Vectors of tightly clustered eigenvalues
//      come out as an orthonormal basis of the cluster's invariant subspace (where the SVD itself is not unique).
//   5. Back-transformation by the reflectors, canonical sign (largest-magnitude entry positive, first index on
//      near-ties), basis rows and sigma = sqrt(lambda) written to the state.
#include <algorithm>

#include "kvc_device.h"
#include "kvc_launch.h"

namespace kvc {

constexpr int kEigThreads = 1024;
constexpr int kEigWaves = kEigThreads / kWave;
constexpr int kReflChunk = 16;  // reflectors staged in LDS per back-transformation chunk

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, kWave);
  return x;
}
__device__ __forceinline__ double wave_max(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmax(x, __shfl_xor(x, o, kWave));
  return x;
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

template <int N>
__global__ __launch_bounds__(kEigThreads) void eig_topr(EigArgs a) {
  constexpr int LD = N + 1;
  // the matrix region also holds the inverse-iteration scratch (2 x N x 64) and X (r x N)
  constexpr int AREG = N * LD > 2 * N * kWave ? N * LD : 2 * N * kWave;
  extern __shared__ __attribute__((aligned(16))) double smem[];
  double* A = smem;                     // N x LD (phase 1-2); scratch / X afterwards
  double* s_a = A + AREG;               // diagonal of T
  double* s_b = s_a + N;                // off-diagonal of T: b[i] couples i and i + 1
  double* s_b2 = s_b + N;               // b^2
  double* s_lam = s_b2 + N;             // eigenvalues, descending
  double* s_v = s_lam + KVC_MAX_RANK;   // current reflector
  double* s_p = s_v + N;                // p / w
  double* s_misc = s_p + N;             // scalars
  double* s_rb = s_misc + 8;            // a chunk of reflectors for the back-transformation [kReflChunk][N]
  double* s_rbeta = s_rb + kReflChunk * N;

  const int u = blockIdx.x;
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
      A[(e / N) * LD + (e % N)] = s;
    }
  } else {
    const double* Dm = a.dense + (size_t)u * N * N;
    for (int e = tid; e < N * N; e += kEigThreads) A[(e / N) * LD + (e % N)] = Dm[e];
  }
  __syncthreads();

  // ---- 2. Householder tridiagonalisation ------------------------------------------------------------------
  for (int k = 0; k < N - 2; ++k) {
    const int m = N - k - 1;
    if (wave == 0) {
      double s = 0.0;
      for (int i = lane; i < m; i += kWave) {
        const double x = A[(k + 1 + i) * LD + k];
        s += x * x;
      }
      s = wave_sum(s);
      const double x0 = A[(k + 1) * LD + k];
      const double nrm = sqrt(s);
      const double alpha = nrm == 0.0 ? 0.0 : -copysign(nrm, x0);
      const double v0 = x0 - alpha;
      const double vtv = (s - x0 * x0) + v0 * v0;
      const double beta = vtv > 0.0 ? 2.0 / vtv : 0.0;
      for (int i = lane; i < m; i += kWave) {
        const double vi = i == 0 ? v0 : A[(k + 1 + i) * LD + k];
        s_v[i] = vi;
        refl[k * N + i] = vi;
      }
      if (lane == 0) {
        s_b[k] = alpha;
        s_misc[0] = beta;
        refl_beta[k] = beta;
      }
    }
    __syncthreads();
    const double beta = s_misc[0];
    if (beta == 0.0) {  // x = 0: H_k = I
      __syncthreads();  // everyone has read s_misc[0] before wave 0 rewrites it
      continue;
    }
    {
      // p = beta * A22 v, eight lanes per row
      const int i = tid >> 3, sub = tid & 7;
      double s = 0.0;
      if (i < m) {
        const double* row = &A[(k + 1 + i) * LD + k + 1];
        for (int j = sub; j < m; j += 8) s += row[j] * s_v[j];
      }
      s += __shfl_xor(s, 1, kWave);
      s += __shfl_xor(s, 2, kWave);
      s += __shfl_xor(s, 4, kWave);
      if (i < m && sub == 0) s_p[i] = beta * s;
    }
    __syncthreads();
    {
      // w = p - (beta / 2) (v^T p) v; every wave forms the scalar itself
      double s = 0.0;
      for (int i = lane; i < m; i += kWave) s += s_v[i] * s_p[i];
      s = wave_sum(s);
      const double K = 0.5 * beta * s;
      __syncthreads();
      for (int i = tid; i < m; i += kEigThreads) s_p[i] = s_p[i] - K * s_v[i];
    }
    __syncthreads();
    // A22 -= v w^T + w v^T, with the same rounding for (i, j) and (j, i) to keep A exactly symmetric
    for (int i = tid >> 5; i < m; i += kEigThreads >> 5) {
      const double vi = s_v[i], wi = s_p[i];
      double* row = &A[(k + 1 + i) * LD + k + 1];
      for (int j = tid & 31; j < m; j += 32) {
        const double t = __dadd_rn(__dmul_rn(vi, s_p[j]), __dmul_rn(wi, s_v[j]));
        row[j] = __dsub_rn(row[j], t);
      }
    }
    __syncthreads();
  }
  for (int i = tid; i < N; i += kEigThreads) s_a[i] = A[i * LD + i];
  if (tid == 0) s_b[N - 2] = A[(N - 1) * LD + N - 2];
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
    for (int e = tid; e < r * N; e += kEigThreads) A[e] = (e / N) == (e % N) ? 1.0 : 0.0;
    for (int j = tid; j < r; j += kEigThreads) s_lam[j] = 0.0;
    __syncthreads();
  } else {
    // ---- 3. multisection bisection for the r largest eigenvalues ---------------------------------------
    {
      int rp = 1;
      while (rp < r) rp <<= 1;
      // lanes per eigenvalue (a power of two dividing 64); 16 trades latency (iterations) against the fp64 work
      const int P = min(16, kEigThreads / rp);
      int bits = 0;
      while ((2 << bits) <= P + 1) ++bits;          // floor(log2(P + 1))
      const int iters = 66 / bits + 1;
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

    // ---- 4. inverse iteration, 64 vectors per batch, one lane each ------------------------------------
    double* invd = A;                  // [N][64]
    double* xv = A + N * kWave;        // [N][64]
    const double piv = 2.220446049250313e-16 * tnorm;
    for (int j0 = 0; j0 < r; j0 += kWave) {
      const int j = j0 + tid;
      if (tid < kWave && j < r) {
        const double lam = s_lam[j];
        double d = s_a[0] - lam;
        if (fabs(d) < piv) d = copysign(piv, d);
        invd[tid] = 1.0 / d;
        #pragma unroll 2
        for (int i = 1; i < N; ++i) {
          const double l = s_b[i - 1] * invd[(i - 1) * kWave + tid];
          d = (s_a[i] - lam) - l * s_b[i - 1];
          if (fabs(d) < piv) d = copysign(piv, d);
          invd[i * kWave + tid] = 1.0 / d;
        }
        #pragma unroll 2
        for (int i = 0; i < N; ++i) {
          const uint32_t h = hash3(a.seed ^ (uint32_t)u, (uint32_t)j, (uint32_t)i);
          xv[i * kWave + tid] = (double)(h >> 11) * (1.0 / 2097152.0) - 1.0;
        }
        for (int itr = 0; itr < 3; ++itr) {
          double z = xv[tid];
          #pragma unroll 2
          for (int i = 1; i < N; ++i) {
            z = xv[i * kWave + tid] - s_b[i - 1] * invd[(i - 1) * kWave + tid] * z;
            xv[i * kWave + tid] = z;
          }
          double x = xv[(N - 1) * kWave + tid] * invd[(N - 1) * kWave + tid];
          xv[(N - 1) * kWave + tid] = x;
          double mx = fabs(x);
          #pragma unroll 2
          for (int i = N - 2; i >= 0; --i) {
            x = (xv[i * kWave + tid] - s_b[i] * x) * invd[i * kWave + tid];
            xv[i * kWave + tid] = x;
            mx = fmax(mx, fabs(x));
          }
          const double sc = mx > 0.0 ? 1.0 / mx : 1.0;
          double ss = 0.0;
          #pragma unroll 2
          for (int i = 0; i < N; ++i) {
            const double y = xv[i * kWave + tid] * sc;
            ss += y * y;
          }
          const double f = sc / sqrt(ss);
          #pragma unroll 2
          for (int i = 0; i < N; ++i) xv[i * kWave + tid] *= f;
        }
        #pragma unroll 2
        for (int i = 0; i < N; ++i) gvec[(size_t)j * N + i] = xv[i * kWave + tid];
      }
      __syncthreads();
    }
    // X[j][i] in LDS
    for (int e = tid; e < r * N; e += kEigThreads) A[e] = gvec[e];
    __syncthreads();

    // modified Gram-Schmidt
    for (int j = 0; j < r; ++j) {
      if (wave == 0) {
        double s = 0.0;
        for (int i = lane; i < N; i += kWave) s += A[j * N + i] * A[j * N + i];
        s = wave_sum(s);
        const double f = 1.0 / sqrt(s);
        for (int i = lane; i < N; i += kWave) A[j * N + i] *= f;
      }
      __syncthreads();
      for (int k = j + 1 + wave; k < r; k += kEigWaves) {
        double s = 0.0;
        for (int i = lane; i < N; i += kWave) s += A[j * N + i] * A[k * N + i];
        s = wave_sum(s);
        for (int i = lane; i < N; i += kWave) A[k * N + i] -= s * A[j * N + i];
      }
      __syncthreads();
    }

    // ---- 5. back-transformation X <- H_0 H_1 ... H_{N-3} X ---------------------------------------------
    // Reflectors are staged kReflChunk at a time; each wave owns whole columns of X, so the steps inside a chunk
    // need no barrier.
    for (int kc = N - 3; kc >= 0; kc -= kReflChunk) {
      const int nk = min(kReflChunk, kc + 1);
      __syncthreads();
      for (int e = tid; e < nk * N; e += kEigThreads) {
        const int c = e / N, i = e - c * N;
        const int k = kc - c;
        s_rb[c * N + i] = i < N - k - 1 ? refl[k * N + i] : 0.0;
      }
      for (int c = tid; c < nk; c += kEigThreads) s_rbeta[c] = refl_beta[kc - c];
      __syncthreads();
      for (int c = 0; c < nk; ++c) {
        const int k = kc - c;
        const int m = N - k - 1;
        const double beta = s_rbeta[c];
        if (beta == 0.0) continue;
        const double* v = &s_rb[c * N];
        for (int j = wave; j < r; j += kEigWaves) {
          double s = 0.0;
          for (int i = lane; i < m; i += kWave) s += v[i] * A[j * N + k + 1 + i];
          s = wave_sum(s) * beta;
          for (int i = lane; i < m; i += kWave) A[j * N + k + 1 + i] -= s * v[i];
        }
      }
    }
    __syncthreads();
  }

  // ---- canonical sign and output ----------------------------------------------------------------------------
  for (int j = wave; j < r; j += kEigWaves) {
    double mx = 0.0;
    for (int i = lane; i < N; i += kWave) mx = fmax(mx, fabs(A[j * N + i]));
    mx = wave_max(mx);
    const double thr = mx * (1.0 - 9.5367431640625e-07);  // 2^-20
    int first = N;
    for (int i0 = 0; i0 < N; i0 += kWave) {
      const int i = i0 + lane;
      const uint64_t m = __ballot(i < N && fabs(A[j * N + i]) >= thr);
      if (m) {
        first = i0 + __ffsll((long long)m) - 1;
        break;
      }
    }
    const double sgn = (first < N && A[j * N + first] < 0.0) ? -1.0 : 1.0;
    for (int i = lane; i < N; i += kWave) tg.basis[(size_t)j * N + i] = (float)(sgn * A[j * N + i]);
    if (lane == 0 && tg.sigma) tg.sigma[j] = (float)sqrt(fmax(s_lam[j], 0.0));
  }
}

size_t eig_lds_bytes(int n) {
  const size_t areg = std::max((size_t)n * (n + 1), (size_t)2 * n * kWave);
  return (areg + 5 * (size_t)n + KVC_MAX_RANK + 8 + (size_t)kReflChunk * (n + 1)) * sizeof(double);
}

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
