// Binary64 dense helpers shared by the ISO-Merger and TSV paths (internal): one-sided
// Jacobi SVD, a strided tiled GEMM with optional split-K partials, and small element-wise
// kernels.  Each translation unit gets its own copy (anonymous namespace).
#pragma once

#include <algorithm>

#include "iso_device.h"

namespace iso {
namespace {

constexpr int kJacobiThreads = 1024;
constexpr int kJacobiMaxSweeps = 60;

// ---- one-sided Jacobi SVD ------------------------------------------------------------------------
// A: r x c col-major (r >= c), overwritten by A V = U Sigma; V: c x c col-major, written.
struct JacobiJob {
  double* a;
  double* v;
  int64_t r, c;
};

__device__ __forceinline__ double wave_sum_f64(double x) {
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

__global__ void __launch_bounds__(kJacobiThreads) k_jacobi(const JacobiJob* __restrict__ jobs, uint32_t* status) {
  __shared__ int s_rot;
  const JacobiJob J = jobs[blockIdx.x];
  const int64_t r = J.r, c = J.c;
  double* A = J.a;
  double* V = J.v;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int64_t e = threadIdx.x; e < c * c; e += blockDim.x) V[e] = ((e % c) == (e / c)) ? 1.0 : 0.0;
  __syncthreads();
  const int64_t cp = c + (c & 1);          // even count: a phantom column pairs with nobody
  const double tol = (double)r * 1.1102230246251565e-16;   // r * unit roundoff
  bool converged = (c < 2);
  for (int sweep = 0; sweep < kJacobiMaxSweeps && !converged; ++sweep) {
    if (threadIdx.x == 0) s_rot = 0;
    __syncthreads();
    for (int64_t round = 0; round < cp - 1; ++round) {
      // round-robin pairing: position 0 fixed, positions 1..cp-1 rotate
      for (int64_t pr = wid; pr < cp / 2; pr += nw) {
        int64_t x = (pr == 0) ? 0 : 1 + (pr - 1 + round) % (cp - 1);
        int64_t y = 1 + (cp - 2 - pr + round) % (cp - 1);
        if (x >= c || y >= c) continue;
        int64_t p = min(x, y), q = max(x, y);
        double* ap = A + p * r;
        double* aq = A + q * r;
        double al = 0.0, be = 0.0, ga = 0.0;
        for (int64_t t = lane; t < r; t += 64) {
          double u = ap[t], w = aq[t];
          al += u * u;
          be += w * w;
          ga += u * w;
        }
        al = wave_sum_f64(al);
        be = wave_sum_f64(be);
        ga = wave_sum_f64(ga);
        if (fabs(ga) > tol * sqrt(al * be) && ga != 0.0) {
          const double zeta = (be - al) / (2.0 * ga);
          const double t = ((zeta >= 0.0) ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
          const double cs = 1.0 / sqrt(1.0 + t * t);
          const double sn = cs * t;
          for (int64_t i = lane; i < r; i += 64) {
            double u = ap[i], w = aq[i];
            ap[i] = cs * u - sn * w;
            aq[i] = sn * u + cs * w;
          }
          double* vp = V + p * c;
          double* vq = V + q * c;
          for (int64_t i = lane; i < c; i += 64) {
            double u = vp[i], w = vq[i];
            vp[i] = cs * u - sn * w;
            vq[i] = sn * u + cs * w;
          }
          if (lane == 0) s_rot = 1;
        }
      }
      __syncthreads();
    }
    converged = (s_rot == 0);
    __syncthreads();
  }
  if (!converged && threadIdx.x == 0) flag_status(status, kStatusInternal);
}

// Sorted thin factors from a converged Jacobi job: left (r x c) = A's columns normalised,
// right (c x c) = V, s (c), all permuted to nonincreasing s.  Zero columns give zero vectors.
__global__ void __launch_bounds__(1024) k_svd_finalize(const JacobiJob* __restrict__ jobs, double* const* left,
                                                       double* const* right, double* const* sv) {
  extern __shared__ double sh[];           // c norms + c ranks
  const JacobiJob J = jobs[blockIdx.x];
  const int64_t r = J.r, c = J.c;
  double* nrm = sh;
  int* rank = (int*)(sh + c);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int64_t j = wid; j < c; j += nw) {
    double s = 0.0;
    for (int64_t t = lane; t < r; t += 64) s += J.a[j * r + t] * J.a[j * r + t];
    s = wave_sum_f64(s);
    if (lane == 0) nrm[j] = sqrt(s);
  }
  __syncthreads();
  for (int64_t j = threadIdx.x; j < c; j += blockDim.x) {
    int rk = 0;
    for (int64_t k = 0; k < c; ++k) rk += (nrm[k] > nrm[j]) || (nrm[k] == nrm[j] && k < j);
    rank[j] = rk;
  }
  __syncthreads();
  double* L = left[blockIdx.x];
  double* R = right[blockIdx.x];
  double* S = sv[blockIdx.x];
  for (int64_t j = wid; j < c; j += nw) {
    const int64_t d = rank[j];
    const double s = nrm[j];
    const double inv = (s > 0.0) ? 1.0 / s : 0.0;
    for (int64_t t = lane; t < r; t += 64) L[d * r + t] = J.a[j * r + t] * inv;
    for (int64_t t = lane; t < c; t += 64) R[d * c + t] = J.v[j * c + t];
    if (lane == 0) S[d] = s;
  }
}

// out = x - y (elementwise, n entries)
__global__ void k_sub(double* __restrict__ out, const double* __restrict__ x, const double* __restrict__ y, int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
    out[e] = x[e] - y[e];
}

__global__ void k_add(double* __restrict__ out, const double* __restrict__ x, const double* __restrict__ y, int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
    out[e] = x[e] + y[e];
}

__global__ void k_copy(double* __restrict__ out, const double* __restrict__ x, int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
    out[e] = x[e];
}

// Normalise the columns of an r x q col-major A into L (zero columns stay zero).
__global__ void __launch_bounds__(1024) k_normalize_cols(double* __restrict__ L, const double* __restrict__ A, int64_t r,
                                                         int64_t q) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int64_t j = (int64_t)blockIdx.x * nw + wid; j < q; j += (int64_t)gridDim.x * nw) {
    double s = 0.0;
    for (int64_t t = lane; t < r; t += 64) s += A[j * r + t] * A[j * r + t];
    s = wave_sum_f64(s);
    const double inv = (s > 0.0) ? 1.0 / sqrt(s) : 0.0;
    for (int64_t t = lane; t < r; t += 64) L[j * r + t] = A[j * r + t] * inv;
  }
}

unsigned grid_for(int64_t n) { return (unsigned)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 4096)); }


// C(i,j) = alpha * sum_k A(i,k) B(k,j) + beta * C(i,j); X(i,k) at X[i*xs0 + k*xs1].
// With blockIdx.z > 0 splits: block z sums k in [z*kz, (z+1)*kz) and writes C + z*cz (beta ignored).
constexpr int GT = 64, GK = 16;
__global__ void __launch_bounds__(256) k_gemm(int64_t M, int64_t N, int64_t Kd, double alpha, const double* __restrict__ A,
                                              int64_t as0, int64_t as1, const double* __restrict__ B, int64_t bs0,
                                              int64_t bs1, double beta, double* __restrict__ C, int64_t cs0,
                                              int64_t cs1, int64_t kz, int64_t cz) {
  __shared__ double As[GK][GT + 1];
  __shared__ double Bs[GK][GT + 1];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int64_t i0 = (int64_t)blockIdx.x * GT, j0 = (int64_t)blockIdx.y * GT;
  const int64_t kb = (gridDim.z > 1) ? (int64_t)blockIdx.z * kz : 0;
  const int64_t ke = (gridDim.z > 1) ? std::min(Kd, kb + kz) : Kd;
  double* Cz = C + ((gridDim.z > 1) ? (int64_t)blockIdx.z * cz : 0);
  double acc[4][4] = {};
  for (int64_t k0 = kb; k0 < ke; k0 += GK) {
    for (int e = threadIdx.x; e < GK * GT; e += 256) {
      const int kk = e / GT, ii = e % GT;
      const int64_t gi = i0 + ii, gk = k0 + kk, gj = j0 + ii;
      As[kk][ii] = (gi < M && gk < ke) ? A[gi * as0 + gk * as1] : 0.0;
      Bs[kk][ii] = (gj < N && gk < ke) ? B[gk * bs0 + gj * bs1] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GK; ++kk) {
      double a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) { a[u] = As[kk][tx + 16 * u]; b[u] = Bs[kk][ty + 16 * u]; }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = acc[u][v] + a[u] * b[v];
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t gi = i0 + tx + 16 * u, gj = j0 + ty + 16 * v;
      if (gi < M && gj < N) {
        double* cp = Cz + gi * cs0 + gj * cs1;
        *cp = (beta == 0.0 || gridDim.z > 1) ? alpha * acc[u][v] : alpha * acc[u][v] + beta * *cp;
      }
    }
}

// out[e] = sum_z parts[z*stride + e], z in order (deterministic split-K reduction)
__global__ void k_sum_parts(double* __restrict__ out, const double* __restrict__ parts, int nz, int64_t stride,
                            int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    double s = 0.0;
    for (int z = 0; z < nz; ++z) s = s + parts[(int64_t)z * stride + e];
    out[e] = s;
  }
}

inline void gemm(int64_t M, int64_t N, int64_t Kd, double alpha, const double* A, int64_t as0, int64_t as1,
                 const double* B, int64_t bs0, int64_t bs1, double beta, double* C, int64_t cs0, int64_t cs1,
                 hipStream_t s) {
  dim3 grid((unsigned)((M + GT - 1) / GT), (unsigned)((N + GT - 1) / GT), 1);
  k_gemm<<<grid, 256, 0, s>>>(M, N, Kd, alpha, A, as0, as1, B, bs0, bs1, beta, C, cs0, cs1, 0, 0);
}

// C (M x N, written with strides cs0/cs1 = contiguous parts of size M*N) = A B summed over nz
// K-slabs; `parts` holds nz * M * N doubles.
inline void gemm_splitk(int64_t M, int64_t N, int64_t Kd, const double* A, int64_t as0, int64_t as1, const double* B,
                        int64_t bs0, int64_t bs1, double* C, double* parts, int nz, hipStream_t s) {
  const int64_t kz = ((Kd + nz - 1) / nz + GK - 1) / GK * GK;
  nz = (int)std::max<int64_t>(1, (Kd + kz - 1) / kz);
  dim3 grid((unsigned)((M + GT - 1) / GT), (unsigned)((N + GT - 1) / GT), (unsigned)nz);
  if (nz == 1) {
    k_gemm<<<grid, 256, 0, s>>>(M, N, Kd, 1.0, A, as0, as1, B, bs0, bs1, 0.0, C, N, 1, 0, 0);
    return;
  }
  k_gemm<<<grid, 256, 0, s>>>(M, N, Kd, 1.0, A, as0, as1, B, bs0, bs1, 0.0, parts, N, 1, kz, M * N);
  k_sum_parts<<<grid_for(M * N), 256, 0, s>>>(C, parts, nz, M * N, M * N);
}

}  // namespace
}  // namespace iso

namespace iso {
namespace {

// A batch of independent GEMMs in one launch: grid.z indexes the job; blocks outside a
// job's M x N exit.  C(i,j) = alpha * sum_k A(i,k) B(k,j) + beta * C(i,j) with X(i,k) at
// X[i*xs0 + k*xs1].  `upper`: only the tiles on or above the diagonal are computed (for a
// symmetric product whose lower triangle the caller fills in).
struct GemmJob {
  const double* A;
  const double* B;
  double* C;
  int64_t as0, as1, bs0, bs1, cs0, cs1;
  int64_t M, N, K;
  double alpha, beta;
  int upper;
};

typedef double gemm_f64x4_t __attribute__((ext_vector_type(4)));

// 64 x 64 output tile per workgroup on v_mfma_f64_16x16x4_f64 (lane (ln, g) supplies A[ln][g]
// and B[g][ln], receives D[g + 4v][ln] in register pair v): four waves as 2 x 2, each a 32 x 32 block of four
// MFMA tiles; k in steps of 16 staged in LDS.  Operands are loaded along whichever of their
// strides is 1, so row- and column-major inputs both read whole cache lines.  LDS rows are 80
// doubles apart, which puts the four k rows of a fragment read on disjoint bank halves.
constexpr int GJP = 80;
__global__ void __launch_bounds__(256) k_gemm_jobs(const GemmJob* __restrict__ jobs) {
  __shared__ double As[GK][GJP];
  __shared__ double Bs[GK][GJP];
  const GemmJob J = jobs[blockIdx.z];
  const int64_t i0 = (int64_t)blockIdx.x * GT, j0 = (int64_t)blockIdx.y * GT;
  if (i0 >= J.M || j0 >= J.N || (J.upper && i0 > j0)) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  const int wm = w >> 1, wn = w & 1;
  const bool a_kfast = J.as1 == 1, b_kfast = J.bs0 == 1;
  gemm_f64x4_t acc[2][2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) acc[rb][cb] = gemm_f64x4_t{0.0, 0.0, 0.0, 0.0};
  // the next k-tile is loaded into registers while the current one is multiplied
  constexpr int PT = (GK * GT) / 256;
  double pa[PT], pb[PT];
  auto load = [&](int64_t k0) {
#pragma unroll
    for (int q = 0; q < PT; ++q) {
      const int e = threadIdx.x + 256 * q;
      const int ka = a_kfast ? (e & 15) : (e >> 6), ia = a_kfast ? (e >> 4) : (e & 63);
      const int kb = b_kfast ? (e & 15) : (e >> 6), jb = b_kfast ? (e >> 4) : (e & 63);
      const int64_t gi = i0 + ia, gka = k0 + ka, gj = j0 + jb, gkb = k0 + kb;
      pa[q] = (gi < J.M && gka < J.K) ? J.A[gi * J.as0 + gka * J.as1] : 0.0;
      pb[q] = (gj < J.N && gkb < J.K) ? J.B[gkb * J.bs0 + gj * J.bs1] : 0.0;
    }
  };
  load(0);
  for (int64_t k0 = 0; k0 < J.K; k0 += GK) {
#pragma unroll
    for (int q = 0; q < PT; ++q) {
      const int e = threadIdx.x + 256 * q;
      const int ka = a_kfast ? (e & 15) : (e >> 6), ia = a_kfast ? (e >> 4) : (e & 63);
      const int kb = b_kfast ? (e & 15) : (e >> 6), jb = b_kfast ? (e >> 4) : (e & 63);
      As[ka][ia] = pa[q];
      Bs[kb][jb] = pb[q];
    }
    __syncthreads();
    if (k0 + GK < J.K) load(k0 + GK);
#pragma unroll
    for (int sub = 0; sub < GK / 4; ++sub) {
      double a[2], b[2];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) a[rb] = As[4 * sub + g][32 * wm + 16 * rb + ln];
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) b[cb] = Bs[4 * sub + g][32 * wn + 16 * cb + ln];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[rb], b[cb], acc[rb][cb], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t gi = i0 + 32 * wm + 16 * rb + g + 4 * v, gj = j0 + 32 * wn + 16 * cb + ln;
        if (gi < J.M && gj < J.N) {
          double* cp = J.C + gi * J.cs0 + gj * J.cs1;
          *cp = (J.beta == 0.0) ? J.alpha * acc[rb][cb][v] : J.alpha * acc[rb][cb][v] + J.beta * *cp;
        }
      }
}

}  // namespace
}  // namespace iso
