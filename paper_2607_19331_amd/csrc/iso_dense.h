// Binary64 dense helpers shared by the ISO-Merger and TSV paths (internal): one-sided
// Jacobi SVD, a strided tiled GEMM with optional split-K partials, and small element-wise
// kernels.  Each translation unit gets its own copy (anonymous namespace).
#pragma once

#include <algorithm>
#include <mutex>
#include <vector>

#include "iso_device.h"

namespace iso {
namespace {

constexpr int kJacobiThreads = 1024;
constexpr int kJacobiMaxSweeps = 60;

// ---- one-sided Jacobi SVD ------------------------------------------------------------------------

__device__ __forceinline__ double wave_sum_f64(double x) {
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Sum over the 16 lanes of a DPP row (xor 1, xor 2, then the half-row and row mirrors pair
// the quads and the halves), the result in every lane of the row.
__device__ __forceinline__ double row16_sum_f64(double x) {
  auto step = [](double v, int ctrl) {
    const uint64_t b = __double_as_longlong(v);
    int lo = (int)(uint32_t)b, hi = (int)(uint32_t)(b >> 32);
    switch (ctrl) {
      case 0: lo = __builtin_amdgcn_mov_dpp(lo, 0xB1, 0xF, 0xF, false); hi = __builtin_amdgcn_mov_dpp(hi, 0xB1, 0xF, 0xF, false); break;
      case 1: lo = __builtin_amdgcn_mov_dpp(lo, 0x4E, 0xF, 0xF, false); hi = __builtin_amdgcn_mov_dpp(hi, 0x4E, 0xF, 0xF, false); break;
      case 2: lo = __builtin_amdgcn_mov_dpp(lo, 0x141, 0xF, 0xF, false); hi = __builtin_amdgcn_mov_dpp(hi, 0x141, 0xF, 0xF, false); break;
      default: lo = __builtin_amdgcn_mov_dpp(lo, 0x140, 0xF, 0xF, false); hi = __builtin_amdgcn_mov_dpp(hi, 0x140, 0xF, 0xF, false); break;
    }
    return v + __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
  };
  x = step(x, 0);
  x = step(x, 1);
  x = step(x, 2);
  return step(x, 3);
}

// Rotation of the column pair (p, q) of A (r rows) and V (c rows) by one 16-lane row of the
// workgroup.  RT > 0: the lane keeps its RT entries of each A column in registers between the
// dot products and the rotation (r <= 16 RT); RT = 0: two passes over memory.
template <int RT>
__device__ __forceinline__ bool jacobi_pair(double* A, double* V, int r, int c, int p, int q, int sub, double tol) {
  double* ap = A + (int64_t)p * r;
  double* aq = A + (int64_t)q * r;
  double al = 0.0, be = 0.0, ga = 0.0;
  double xu[RT > 0 ? RT : 1], xw[RT > 0 ? RT : 1];
  if constexpr (RT > 0) {
#pragma unroll
    for (int e = 0; e < RT; ++e) {
      const int t = sub + 16 * e;
      xu[e] = (t < r) ? ap[t] : 0.0;
      xw[e] = (t < r) ? aq[t] : 0.0;
    }
#pragma unroll
    for (int e = 0; e < RT; ++e) {
      al += xu[e] * xu[e];
      be += xw[e] * xw[e];
      ga += xu[e] * xw[e];
    }
  } else {
#pragma unroll 4
    for (int t = sub; t < r; t += 16) {
      const double u = ap[t], w = aq[t];
      al += u * u;
      be += w * w;
      ga += u * w;
    }
  }
  al = row16_sum_f64(al);
  be = row16_sum_f64(be);
  ga = row16_sum_f64(ga);
  if (!(fabs(ga) > tol * sqrt(al * be) && ga != 0.0)) return false;
  const double zeta = (be - al) / (2.0 * ga);
  const double t = ((zeta >= 0.0) ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
  const double cs = 1.0 / sqrt(1.0 + t * t);
  const double sn = cs * t;
  if constexpr (RT > 0) {
#pragma unroll
    for (int e = 0; e < RT; ++e) {
      const int i = sub + 16 * e;
      if (i < r) {
        ap[i] = cs * xu[e] - sn * xw[e];
        aq[i] = sn * xu[e] + cs * xw[e];
      }
    }
  } else {
#pragma unroll 4
    for (int i = sub; i < r; i += 16) {
      const double u = ap[i], w = aq[i];
      ap[i] = cs * u - sn * w;
      aq[i] = sn * u + cs * w;
    }
  }
  double* vp = V + (int64_t)p * c;
  double* vq = V + (int64_t)q * c;
#pragma unroll 4
  for (int i = sub; i < c; i += 16) {
    const double u = vp[i], w = vq[i];
    vp[i] = cs * u - sn * w;
    vq[i] = sn * u + cs * w;
  }
  return true;
}

// One-sided Jacobi sweeps on A (r x c col-major, r >= c), rotations accumulated into V (c x c,
// the identity on entry), until a sweep rotates nothing (relative tolerance r * u) or
// kJacobiMaxSweeps.  Columns are paired round-robin (position 0 fixed, the others rotating; a
// phantom column when c is odd); one 16-lane row of the workgroup per pair, so a wave rotates
// four pairs at once.  Block-uniform result: converged.
template <int RT>
__device__ bool jacobi_sweeps(double* A, double* V, int r, int c, int* s_rot, int max_sweeps = kJacobiMaxSweeps) {
  const int sub = threadIdx.x & 15, grp = threadIdx.x >> 4, ngrp = blockDim.x >> 4;
  const int cp = c + (c & 1);
  const double tol = (double)r * 1.1102230246251565e-16;
  bool converged = (c < 2);
  for (int sweep = 0; sweep < max_sweeps && !converged; ++sweep) {
    if (threadIdx.x == 0) *s_rot = 0;
    __syncthreads();
    for (int round = 0; round < cp - 1; ++round) {
      for (int pr = grp; pr < cp / 2; pr += ngrp) {
        const int x = (pr == 0) ? 0 : 1 + (pr - 1 + round) % (cp - 1);
        const int y = 1 + (cp - 2 - pr + round) % (cp - 1);
        if (x >= c || y >= c) continue;                    // the whole 16-lane row skips
        if (jacobi_pair<RT>(A, V, r, c, min(x, y), max(x, y), sub, tol) && sub == 0) *s_rot = 1;
      }
      __syncthreads();
    }
    converged = (*s_rot == 0);
    __syncthreads();
  }
  return converged;
}

// A: r x c col-major (r >= c), overwritten by A V = U Sigma; V: c x c col-major, written.
// tr: the row count that scales the convergence test (r * u), when A stands for a taller matrix
// with the same Gram (a Cholesky factor of its A^T A); 0: r itself.
struct JacobiJob {
  double* a;
  double* v;
  int64_t r, c;
  int64_t tr;
};

__device__ __forceinline__ double jacobi_tol(const JacobiJob& J) {
  return (double)(J.tr > 0 ? J.tr : J.r) * 1.1102230246251565e-16;
}

__global__ void __launch_bounds__(kJacobiThreads) k_jacobi(const JacobiJob* __restrict__ jobs, uint32_t* status) {
  __shared__ int s_rot;
  const JacobiJob J = jobs[blockIdx.x];
  const int r = (int)J.r, c = (int)J.c;
  for (int64_t e = threadIdx.x; e < (int64_t)c * c; e += blockDim.x) J.v[e] = ((e % c) == (e / c)) ? 1.0 : 0.0;
  __syncthreads();
  const bool converged = (r <= 256) ? jacobi_sweeps<16>(J.a, J.v, r, c, &s_rot) : jacobi_sweeps<0>(J.a, J.v, r, c, &s_rot);
  if (!converged && threadIdx.x == 0) flag_status(status, kStatusInternal);
}

// ---- the same sweeps spread over many workgroups ---------------------------------------------------
// The pairs of one round are independent, so each round is one launch over all jobs (16 pairs per
// 256-thread workgroup): the kernel boundary is the barrier between rounds.  Per job, `rot` records
// a rotation in the current sweep and `done` a sweep that rotated nothing; converged jobs' rounds
// exit at once.  Same pairing, rotation and stopping rule as jacobi_sweeps.
struct JacobiState {
  int rot, done;
};

// V <- I unless v_given (V then holds a starting orthogonal factor: the rotations multiply it)
__global__ void k_jacobi_begin(const JacobiJob* __restrict__ jobs, JacobiState* __restrict__ st, int v_given = 0) {
  const JacobiJob J = jobs[blockIdx.y];
  const int64_t c = J.c, cc = c * c;
  if (!v_given)
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < cc; e += (int64_t)gridDim.x * blockDim.x)
      J.v[e] = ((e % c) == (e / c)) ? 1.0 : 0.0;
  if (blockIdx.x == 0 && threadIdx.x == 0) st[blockIdx.y] = JacobiState{0, c < 2 ? 1 : 0};
}

__global__ void __launch_bounds__(256) k_jacobi_round(const JacobiJob* __restrict__ jobs, JacobiState* st, int round) {
  const int job = blockIdx.y;
  if (st[job].done) return;
  const JacobiJob J = jobs[job];
  const int r = (int)J.r, c = (int)J.c, cp = c + (c & 1);
  if (round >= cp - 1) return;
  const int sub = threadIdx.x & 15, pr = blockIdx.x * 16 + (threadIdx.x >> 4);
  if (pr >= cp / 2) return;                            // whole 16-lane rows
  const int x = (pr == 0) ? 0 : 1 + (pr - 1 + round) % (cp - 1);
  const int y = 1 + (cp - 2 - pr + round) % (cp - 1);
  if (x >= c || y >= c) return;
  const double tol = jacobi_tol(J);
  const bool rot = (r <= 256) ? jacobi_pair<16>(J.a, J.v, r, c, min(x, y), max(x, y), sub, tol)
                              : jacobi_pair<0>(J.a, J.v, r, c, min(x, y), max(x, y), sub, tol);
  if (rot && sub == 0) st[job].rot = 1;                // every writer stores 1
}

__global__ void k_jacobi_sweep_end(JacobiState* st, int njobs) {
  for (int j = threadIdx.x; j < njobs; j += blockDim.x)
    if (!st[j].done) {
      if (st[j].rot == 0) st[j].done = 1;
      st[j].rot = 0;
    }
}

__global__ void k_jacobi_check(const JacobiState* st, int njobs, uint32_t* status) {
  for (int j = threadIdx.x; j < njobs; j += blockDim.x)
    if (!st[j].done) flag_status(status, kStatusInternal);
}

constexpr int kJacobiCheckSweeps = 4;   // sweeps queued between host checks of the done flags

// Runs the Jacobi sweeps of njobs jobs (device table, max_c the largest column count).  The host
// reads the done flags every kJacobiCheckSweeps sweeps and stops queueing once all are set, so
// the call synchronises the stream a few times.
inline hipError_t jacobi_multi(const JacobiJob* jobs, int njobs, int64_t max_c, JacobiState* st, uint32_t* status,
                               hipStream_t s) {
  const unsigned gb = (unsigned)std::max<int64_t>(1, std::min<int64_t>((max_c * max_c + 255) / 256, 4096));
  k_jacobi_begin<<<dim3(gb, (unsigned)njobs), 256, 0, s>>>(jobs, st);
  const int cpm = (int)(max_c + (max_c & 1));
  const dim3 g((unsigned)std::max(1, (cpm / 2 + 15) / 16), (unsigned)njobs);
  std::vector<JacobiState> h(njobs);
  for (int sweep = 0; sweep < kJacobiMaxSweeps;) {
    for (int b = 0; b < kJacobiCheckSweeps && sweep < kJacobiMaxSweeps; ++b, ++sweep) {
      for (int round = 0; round < cpm - 1; ++round) k_jacobi_round<<<g, 256, 0, s>>>(jobs, st, round);
      k_jacobi_sweep_end<<<1, 256, 0, s>>>(st, njobs);
    }
    hipError_t e = hipMemcpyAsync(h.data(), st, sizeof(JacobiState) * njobs, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return e;
    bool all = true;
    for (int j = 0; j < njobs; ++j) all = all && h[j].done;
    if (all) break;
  }
  k_jacobi_check<<<1, 256, 0, s>>>(st, njobs, status);
  return hipGetLastError();
}

// ---- block one-sided Jacobi ------------------------------------------------------------------------
// Columns in blocks of w (the last may be short; a phantom block when the count is odd), blocks
// paired round-robin.  Per outer round, each workgroup takes one pair of blocks, stages their
// (at most 2w) columns of A and V in LDS, runs one round-robin sweep over them (inner pairs, one
// 16-lane row each) and writes them back; every column pair is checked at least once per outer
// sweep, so a sweep that rotates nothing means the whole job has converged (same test as
// jacobi_sweeps).  Far fewer launches than one per column round.
__global__ void __launch_bounds__(256) k_bjacobi_round(const JacobiJob* __restrict__ jobs, JacobiState* st, int round,
                                                       int w) {
  extern __shared__ double bsh[];
  __shared__ int s_rot;
  const int job = blockIdx.y;
  if (st[job].done) return;
  const JacobiJob J = jobs[job];
  const int r = (int)J.r, c = (int)J.c;
  const int nb = (c + w - 1) / w, nbp = nb + (nb & 1);
  if (round >= nbp - 1) return;
  const int pr = blockIdx.x;
  if (pr >= nbp / 2) return;
  const int bx = (pr == 0) ? 0 : 1 + (pr - 1 + round) % (nbp - 1);
  const int by = 1 + (nbp - 2 - pr + round) % (nbp - 1);
  // a block paired with the phantom sweeps its own column pairs (a job of one block has no other
  // pairs at all)
  const bool alone = bx >= nb || by >= nb;
  const int c0 = min(bx, by) * w, c1 = alone ? c0 : max(bx, by) * w;
  const int n0 = min(w, c - c0), n1 = alone ? 0 : min(w, c - c1), nc = n0 + n1;
  double* A = bsh;                                  // nc columns of r
  double* V = bsh + (int64_t)2 * w * r;             // nc columns of c
  auto gcol = [&](int l) { return (l < n0) ? c0 + l : c1 + (l - n0); };
  for (int l = 0; l < nc; ++l) {
    const int g = gcol(l);
    for (int i = threadIdx.x; i < r; i += blockDim.x) A[(int64_t)l * r + i] = J.a[(int64_t)g * r + i];
    for (int i = threadIdx.x; i < c; i += blockDim.x) V[(int64_t)l * c + i] = J.v[(int64_t)g * c + i];
  }
  if (threadIdx.x == 0) s_rot = 0;
  __syncthreads();
  const int sub = threadIdx.x & 15, grp = threadIdx.x >> 4, ngrp = blockDim.x >> 4;
  const int cp = nc + (nc & 1);
  const double tol = jacobi_tol(J);
  for (int ir = 0; ir < cp - 1; ++ir) {
    for (int q = grp; q < cp / 2; q += ngrp) {
      const int x = (q == 0) ? 0 : 1 + (q - 1 + ir) % (cp - 1);
      const int y = 1 + (cp - 2 - q + ir) % (cp - 1);
      if (x >= nc || y >= nc) continue;
      const bool rot = (r <= 256) ? jacobi_pair<16>(A, V, r, c, min(x, y), max(x, y), sub, tol)
                                  : jacobi_pair<0>(A, V, r, c, min(x, y), max(x, y), sub, tol);
      if (rot && sub == 0) s_rot = 1;
    }
    __syncthreads();
  }
  for (int l = 0; l < nc; ++l) {
    const int g = gcol(l);
    for (int i = threadIdx.x; i < r; i += blockDim.x) J.a[(int64_t)g * r + i] = A[(int64_t)l * r + i];
    for (int i = threadIdx.x; i < c; i += blockDim.x) J.v[(int64_t)g * c + i] = V[(int64_t)l * c + i];
  }
  if (threadIdx.x == 0 && s_rot) st[job].rot = 1;
}

// ---- block Jacobi step through the pair's Gram matrix (long columns) --------------------------------
// For columns too long to stage: the pair's (at most 64) columns stay in global memory.  Their
// 64 x 64 Gram matrix is formed on v_mfma_f64_16x16x4_f64 (lane (ln, g) supplies A[ln][g] and
// B[g][ln] and receives D[g + 4v][ln]) from 64-row chunks staged in LDS; if some column pair fails
// the rotation test, one-sided Jacobi on the Gram itself gives a rotation Q towards its
// eigenvectors (for a symmetric positive semidefinite matrix the right singular vectors are the
// eigenvectors), and the columns of A and of V are multiplied by Q, chunk by chunk, again on MFMA
// through LDS.
typedef double jac_f64x4_t __attribute__((ext_vector_type(4)));
constexpr int kGW = 32, kGN = 64, kGP = kGN + 1;
// Sweeps of the inner Jacobi on a block pair's Gram matrix.  One sweep suffices: the block pair
// comes round again in the next outer sweep, and the outer test (every scaled off-diagonal Gram
// entry below tolerance) is what ends the iteration, so an inner solve run to convergence only
// buys fewer outer sweeps at a higher price each (at 2048 x 2048 one inner sweep is 18% faster
// end to end than full inner convergence, with identical merged weights).
constexpr int kGramInnerSweeps = 1;

// Row chunk loads: thread t holds entries e = t + 256 u (u < 16) of a kGN x kGN chunk, column
// l = e / kGN (the l-th of the pair's columns), row i = e % kGN: each wave reads one column's 64
// consecutive rows.
constexpr int kGChunkPer = kGN * kGN / 256;

__device__ __forceinline__ void gram_load(double (&pf)[kGChunkPer], const double* X, int64_t ld, int nrows,
                                          const int* gc, int nc, int k0) {
#pragma unroll
  for (int u = 0; u < kGChunkPer; ++u) {
    const int e = threadIdx.x + 256 * u, l = e / kGN, i = e % kGN;
    pf[u] = (l < nc && k0 + i < nrows) ? gmem(X)[(int64_t)gc[l] * ld + k0 + i] : 0.0;
  }
}

__device__ __forceinline__ void gram_stage(double* ch, const double (&pf)[kGChunkPer]) {
#pragma unroll
  for (int u = 0; u < kGChunkPer; ++u) {
    const int e = threadIdx.x + 256 * u;
    ch[(e / kGN) * kGP + e % kGN] = pf[u];
  }
}

// X[row0:nrows, cols] <- X[row0:nrows, cols] Q (X col-major with leading dimension ld); ch is a
// kGN x kGP LDS chunk, q the kGN x kGN LDS rotation (col-major).  The next chunk is loaded into
// registers while the current one is multiplied.
__device__ __forceinline__ void gram_apply(double* X, int64_t ld, int row0, int nrows, const int* gc, int nc,
                                           double* ch, const double* q) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  double pf[kGChunkPer];
  gram_load(pf, X, ld, nrows, gc, nc, row0);
  for (int k0 = row0; k0 < nrows; k0 += kGN) {
    gram_stage(ch, pf);
    __syncthreads();
    if (k0 + kGN < nrows) gram_load(pf, X, ld, nrows, gc, nc, k0 + kGN);
    jac_f64x4_t acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = jac_f64x4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
    for (int s = 0; s < kGN / 4; ++s) {
      const double a = ch[(4 * s + g) * kGP + 16 * w + ln];          // chunk row 16w + ln, k = 4s + g
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, q[(16 * t + ln) * kGN + 4 * s + g], acc[t], 0, 0, 0);
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) ch[(16 * t + ln) * kGP + 16 * w + g + 4 * v] = acc[t][v];
    __syncthreads();
    for (int e = threadIdx.x; e < kGN * kGN; e += blockDim.x) {
      const int l = e / kGN, i = e % kGN;
      if (l < nc && k0 + i < nrows) gmem(X)[(int64_t)gc[l] * ld + k0 + i] = ch[l * kGP + i];
    }
    __syncthreads();
  }
}

__global__ void __launch_bounds__(256) k_bjacobi_gram(const JacobiJob* __restrict__ jobs, JacobiState* st, int round) {
  // GC: the row chunk [column][row] while the Gram is formed and while A and V are multiplied by
  // Q; in between the Gram (col-major, leading dimension kGN), then the Jacobi matrix.  About
  // 66 KB in all: two workgroups per CU.
  __shared__ double GC[kGN * kGP];
  __shared__ double Q[kGN * kGN];          // rotations (col-major)
  __shared__ int gc[kGN];
  __shared__ int s_need, s_rot;
  double* const G = GC;
  double* const ch = GC;
  const int job = blockIdx.y;
  if (st[job].done) return;
  const JacobiJob J = jobs[job];
  const int r = (int)J.r, c = (int)J.c;
  const int nb = (c + kGW - 1) / kGW, nbp = nb + (nb & 1);
  if (round >= nbp - 1) return;
  const int pr = blockIdx.x;
  if (pr >= nbp / 2) return;
  const int bx = (pr == 0) ? 0 : 1 + (pr - 1 + round) % (nbp - 1);
  const int by = 1 + (nbp - 2 - pr + round) % (nbp - 1);
  const bool alone = bx >= nb || by >= nb;        // paired with the phantom: the block's own pairs
  const int c0 = min(bx, by) * kGW, c1 = alone ? c0 : max(bx, by) * kGW;
  const int n0 = min(kGW, c - c0), n1 = alone ? 0 : min(kGW, c - c1), nc = n0 + n1;
  if (threadIdx.x < kGN) gc[threadIdx.x] = (threadIdx.x < n0) ? c0 + threadIdx.x : c1 + (threadIdx.x - n0);
  if (threadIdx.x == 0) { s_need = 0; s_rot = 0; }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  // 1. Gram: wave w owns the tile row w (four 16 x 16 tiles)
  jac_f64x4_t acc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) acc[t] = jac_f64x4_t{0.0, 0.0, 0.0, 0.0};
  __syncthreads();
  double pf[kGChunkPer];
  gram_load(pf, J.a, r, r, gc, nc, 0);
  for (int k0 = 0; k0 < r; k0 += kGN) {
    gram_stage(ch, pf);
    __syncthreads();
    if (k0 + kGN < r) gram_load(pf, J.a, r, r, gc, nc, k0 + kGN);
#pragma unroll 4
    for (int s = 0; s < kGN / 4; ++s) {
      const double a = ch[(16 * w + ln) * kGP + 4 * s + g];          // X^T[16w + ln][k]
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, ch[(16 * t + ln) * kGP + 4 * s + g], acc[t], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int v = 0; v < 4; ++v) G[(16 * t + ln) * kGN + 16 * w + g + 4 * v] = acc[t][v];   // G[i][j] at j*64+i
  __syncthreads();
  // 2. rotation test on every column pair (the test of jacobi_pair)
  const double tol = jacobi_tol(J);
  for (int e = threadIdx.x; e < kGN * kGN; e += blockDim.x) {
    const int i = e % kGN, j = e / kGN;
    if (i < j && j < nc) {
      const double gij = G[j * kGN + i];
      if (fabs(gij) > tol * sqrt(G[i * kGN + i] * G[j * kGN + j]) && gij != 0.0) s_need = 1;
    }
  }
  for (int e = threadIdx.x; e < kGN * kGN; e += blockDim.x) Q[e] = ((e % kGN) == (e / kGN)) ? 1.0 : 0.0;
  __syncthreads();
  if (!s_need) return;
  // 3. rotations that diagonalise G: one-sided Jacobi on G (its columns orthogonalised, one sweep),
  //    accumulated into Q
  jacobi_sweeps<4>(G, Q, kGN, kGN, &s_rot, kGramInnerSweeps);
  __syncthreads();
  // 4. A and V columns times Q (G is no longer needed: its space takes the row chunks)
  gram_apply(J.a, r, 0, r, gc, nc, ch, Q);
  gram_apply(J.v, c, 0, c, gc, nc, ch, Q);
  if (threadIdx.x == 0) st[job].rot = 1;
}

// ---- the same step with the rows of a block pair split over workgroups ---------------------------
// Three launches per round: partial Grams of row slices of A (one workgroup per pair
// and slice), the sum of a pair's partials in slice order with the rotation test and the inner
// sweep (one workgroup per pair; the rotation and a flag go to global memory), and the rotation of
// every slice of A and of V (one workgroup per pair and slice).  Long columns then take many
// short workgroups instead of one long one; the result is the same step.
// Rows per slice, one value for a whole job set: 512 while the set's longest column is at most
// 8192 rows (more workgroups per round for the mid-sized matrices, where the rounds are short),
// 1024 beyond (fewer partial Grams for each rotation step to sum).
constexpr int64_t kGSliceSmallMax = 8192;
inline int gram_slice_rows(int64_t max_r) { return max_r <= kGSliceSmallMax ? 512 : 1024; }
// Slices of a job set of at most max_r rows, or of any set with fewer rows (which may take the
// smaller slice): the count the split scratch is sized for.
inline int64_t gram_slices_bound(int64_t max_r) {
  const int64_t own = (max_r + gram_slice_rows(max_r) - 1) / gram_slice_rows(max_r);
  const int64_t small = (std::min(max_r, kGSliceSmallMax) + 511) / 512;
  return std::max(own, small);
}

struct GramPair {     // the block pair a workgroup of round `round` works on, or none
  int ok, nc;
  int c0, n0, c1;
};

__device__ __forceinline__ GramPair gram_pair_of(int c, int pr, int round) {
  GramPair P{0, 0, 0, 0, 0};
  const int nb = (c + kGW - 1) / kGW, nbp = nb + (nb & 1);
  if (round >= nbp - 1 || pr >= nbp / 2) return P;
  const int bx = (pr == 0) ? 0 : 1 + (pr - 1 + round) % (nbp - 1);
  const int by = 1 + (nbp - 2 - pr + round) % (nbp - 1);
  const bool alone = bx >= nb || by >= nb;        // paired with the phantom: the block's own pairs
  P.c0 = min(bx, by) * kGW;
  P.c1 = alone ? P.c0 : max(bx, by) * kGW;
  P.n0 = min(kGW, c - P.c0);
  P.nc = P.n0 + (alone ? 0 : min(kGW, c - P.c1));
  P.ok = 1;
  return P;
}

struct GramSplit {
  double* part;     // njobs x npairs x nslices x kGN^2: partial Grams
  double* qrot;     // njobs x npairs x kGN^2: rotations
  int* need;        // njobs x npairs: 1 if the pair rotates this round
  int npairs, nslices;
  int slice;        // rows per slice (gram_slice_rows of the set)
};

__global__ void __launch_bounds__(256) k_bjg_part(const JacobiJob* __restrict__ jobs, const JacobiState* st,
                                                  int round, GramSplit S) {
  __shared__ double ch[kGN * kGP];
  __shared__ int gc[kGN];
  const int job = blockIdx.y;
  if (st[job].done) return;
  const JacobiJob J = jobs[job];
  const int r = (int)J.r, c = (int)J.c;
  const int pr = blockIdx.x / S.nslices, z = blockIdx.x % S.nslices;
  const GramPair P = gram_pair_of(c, pr, round);
  const int row0 = z * S.slice, row1 = min(r, row0 + S.slice);
  if (!P.ok || row0 >= r) return;
  if (threadIdx.x < kGN) gc[threadIdx.x] = (threadIdx.x < P.n0) ? P.c0 + threadIdx.x : P.c1 + (threadIdx.x - P.n0);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  // the Gram is symmetric: only its 10 tiles on and above the diagonal are formed, three per wave
  // for waves 0 and 1 and two for waves 2 and 3 (tile (R, C) as the nibble 4R + C of a packed list)
  constexpr unsigned kTiles[4] = {0x0 | (0x1 << 4) | (0x2 << 8), 0x3 | (0x5 << 4) | (0x6 << 8),
                                  0x7 | (0xA << 4), 0xB | (0xF << 4)};
  const unsigned tl = kTiles[w];
  const int nt = (w < 2) ? 3 : 2;
  int tr[3], tc[3];
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const unsigned e = (tl >> (4 * j)) & 0xFu;
    tr[j] = (int)(e >> 2);
    tc[j] = (int)(e & 3u);
  }
  jac_f64x4_t acc[3];
#pragma unroll
  for (int j = 0; j < 3; ++j) acc[j] = jac_f64x4_t{0.0, 0.0, 0.0, 0.0};
  __syncthreads();
  // two row chunks in flight, as in k_bjg_apply
  double pf0[kGChunkPer], pf1[kGChunkPer];
  gram_load(pf0, J.a, r, row1, gc, P.nc, row0);
  if (row0 + kGN < row1) gram_load(pf1, J.a, r, row1, gc, P.nc, row0 + kGN);
  auto chunk = [&](int k0, double (&pf)[kGChunkPer]) {
    gram_stage(ch, pf);
    __syncthreads();
    if (k0 + 2 * kGN < row1) gram_load(pf, J.a, r, row1, gc, P.nc, k0 + 2 * kGN);
#pragma unroll 4
    for (int s = 0; s < kGN / 4; ++s) {
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        if (j < nt) {
          const double a = ch[(16 * tr[j] + ln) * kGP + 4 * s + g];     // X^T[16R + ln][k]
          const double b = ch[(16 * tc[j] + ln) * kGP + 4 * s + g];     // X[k][16C + ln]
          acc[j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc[j], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  };
  for (int k0 = row0; k0 < row1; k0 += 2 * kGN) {
    chunk(k0, pf0);
    if (k0 + kGN < row1) chunk(k0 + kGN, pf1);
  }
  // G[i][j] at j * kGN + i; a tile above the diagonal also fills its mirror below it
  double* out = S.part + (((size_t)job * S.npairs + pr) * S.nslices + z) * (kGN * kGN);
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    if (j < nt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int gi = 16 * tr[j] + g + 4 * v, gj = 16 * tc[j] + ln;
        out[gj * kGN + gi] = acc[j][v];
        if (tr[j] != tc[j]) out[gi * kGN + gj] = acc[j][v];
      }
    }
  }
}

// 512 threads: 32 sixteen-lane rows, one per column pair of the 64 x 64 inner sweep
__global__ void __launch_bounds__(512) k_bjg_rot(const JacobiJob* __restrict__ jobs, JacobiState* st, int round,
                                                 GramSplit S) {
  __shared__ double G[kGN * kGN];
  __shared__ double Q[kGN * kGN];
  __shared__ int s_need, s_rot;
  const int job = blockIdx.y, pr = blockIdx.x;
  if (st[job].done) return;
  const JacobiJob J = jobs[job];
  const int r = (int)J.r, c = (int)J.c;
  const GramPair P = gram_pair_of(c, pr, round);
  int* need = S.need + (size_t)job * S.npairs + pr;
  if (!P.ok) {
    if (threadIdx.x == 0 && pr < S.npairs) *need = 0;
    return;
  }
  const int ns = (r + S.slice - 1) / S.slice;
  const double* part = S.part + ((size_t)job * S.npairs + pr) * S.nslices * (kGN * kGN);
  for (int e = threadIdx.x; e < kGN * kGN; e += blockDim.x) {
    double x = 0.0;
    for (int z = 0; z < ns; ++z) x += part[(size_t)z * (kGN * kGN) + e];
    G[e] = x;
  }
  if (threadIdx.x == 0) { s_need = 0; s_rot = 0; }
  __syncthreads();
  const double tol = jacobi_tol(J);
  for (int e = threadIdx.x; e < kGN * kGN; e += blockDim.x) {
    const int i = e % kGN, j = e / kGN;
    if (i < j && j < P.nc) {
      const double gij = G[j * kGN + i];
      if (fabs(gij) > tol * sqrt(G[i * kGN + i] * G[j * kGN + j]) && gij != 0.0) s_need = 1;
    }
  }
  for (int e = threadIdx.x; e < kGN * kGN; e += blockDim.x) Q[e] = ((e % kGN) == (e / kGN)) ? 1.0 : 0.0;
  __syncthreads();
  if (threadIdx.x == 0) *need = s_need;
  if (!s_need) return;
  jacobi_sweeps<4>(G, Q, kGN, kGN, &s_rot, kGramInnerSweeps);
  __syncthreads();
  double* q = S.qrot + ((size_t)job * S.npairs + pr) * (kGN * kGN);
  for (int e = threadIdx.x; e < kGN * kGN; e += blockDim.x) q[e] = Q[e];
  if (threadIdx.x == 0) st[job].rot = 1;
}

__global__ void __launch_bounds__(256) k_bjg_apply(const JacobiJob* __restrict__ jobs, const JacobiState* st,
                                                   int round, GramSplit S, int slices_a, int slices_v) {
  constexpr int QS = kGN + 2;                      // Q row stride: the 16 rows of a fragment read
  __shared__ double ch[kGN * kGP];                 // start 4 banks apart, so a half-wave is conflict-free
  __shared__ double qs[kGN * QS];
  __shared__ int gc[kGN];
  const int job = blockIdx.y;
  if (st[job].done) return;
  const JacobiJob J = jobs[job];
  const int r = (int)J.r, c = (int)J.c;
  const int per = slices_a + slices_v;
  const int pr = blockIdx.x / per, z = blockIdx.x % per;
  const GramPair P = gram_pair_of(c, pr, round);
  if (!P.ok || S.need[(size_t)job * S.npairs + pr] == 0) return;
  const bool on_a = z < slices_a;
  const int rows = on_a ? r : c;
  const int row0 = (on_a ? z : z - slices_a) * S.slice, row1 = min(rows, row0 + S.slice);
  if (row0 >= rows) return;
  if (threadIdx.x < kGN) gc[threadIdx.x] = (threadIdx.x < P.n0) ? P.c0 + threadIdx.x : P.c1 + (threadIdx.x - P.n0);
  const double* q = S.qrot + ((size_t)job * S.npairs + pr) * (kGN * kGN);
  // Q (the same for every chunk) in LDS, which leaves the registers to the chunks in flight
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  for (int e = threadIdx.x; e < kGN * kGN; e += blockDim.x) qs[(e / kGN) * QS + e % kGN] = q[e];
  __syncthreads();
  double* X = on_a ? J.a : J.v;
  // two row chunks in flight: chunk k is loaded into pf[k & 1] while chunk k - 1 is rotated
  double pf0[kGChunkPer], pf1[kGChunkPer];
  gram_load(pf0, X, rows, row1, gc, P.nc, row0);
  if (row0 + kGN < row1) gram_load(pf1, X, rows, row1, gc, P.nc, row0 + kGN);
  auto chunk = [&](int k0, double (&pf)[kGChunkPer]) {
    gram_stage(ch, pf);
    __syncthreads();
    if (k0 + 2 * kGN < row1) gram_load(pf, X, rows, row1, gc, P.nc, k0 + 2 * kGN);
    jac_f64x4_t acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = jac_f64x4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int s4 = 0; s4 < kGN / 4; ++s4) {
      const double a = ch[(4 * s4 + g) * kGP + 16 * w + ln];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, qs[(16 * t + ln) * QS + 4 * s4 + g], acc[t], 0, 0, 0);
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) ch[(16 * t + ln) * kGP + 16 * w + g + 4 * v] = acc[t][v];
    __syncthreads();
    for (int e = threadIdx.x; e < kGN * kGN; e += blockDim.x) {
      const int l = e / kGN, i = e % kGN;
      if (l < P.nc && k0 + i < row1) gmem(X)[(int64_t)gc[l] * rows + k0 + i] = ch[l * kGP + i];
    }
    __syncthreads();
  };
  for (int k0 = row0; k0 < row1; k0 += 2 * kGN) {
    chunk(k0, pf0);
    if (k0 + kGN < row1) chunk(k0 + kGN, pf1);
  }
}

// Scratch of the split step for njobs jobs of at most max_r rows and max_c columns.
inline size_t gram_split_bytes(int njobs, int64_t max_r, int64_t max_c) {
  const int64_t nb = (max_c + kGW - 1) / kGW, np = (nb + (nb & 1)) / 2;
  const int64_t ns = gram_slices_bound(max_r);
  return ((size_t)njobs * np * (size_t)(ns + 1) * kGN * kGN) * sizeof(double) + (size_t)njobs * np * sizeof(int) + 256;
}

// Job groups of the split Jacobi step, each on a stream of its own.
constexpr int kJacobiGroups = 4;

// Stream i (0 <= i < kJacobiGroups - 1) of the current device besides the caller's (default
// priority, created on first use and kept until the process ends), or null if it cannot be created.
inline hipStream_t aux_stream(int i) {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static hipStream_t per[kMaxDev][kJacobiGroups] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev || i < 0 || i >= kJacobiGroups) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (per[dev][i] == nullptr && hipStreamCreateWithFlags(&per[dev][i], hipStreamNonBlocking) != hipSuccess)
    per[dev][i] = nullptr;
  return per[dev][i];
}

// Independent per-item work fanned out over the caller's stream s and the extra streams of this
// device: begin() makes the extra streams wait for what s holds so far, at(e) is item e's stream
// (round-robin), end() makes s wait for all of them.  Without the extra streams or their events,
// everything stays on s.  If end() was not reached (an error return), the destructor waits for the
// extra streams, so that no work of this call is left running.
struct Fan {
  hipStream_t st[kJacobiGroups] = {};
  hipEvent_t fork = nullptr, join[kJacobiGroups] = {};
  int n = 1;
  bool open = false;
  hipError_t begin(hipStream_t s, int items) {
    st[0] = s;
    n = 1;
    const int want = std::min(kJacobiGroups, std::max(1, items));
    if (want < 2 || hipEventCreateWithFlags(&fork, hipEventDisableTiming) != hipSuccess) {
      fork = nullptr;
      return hipSuccess;
    }
    for (int i = 1; i < want; ++i) {
      hipStream_t x = aux_stream(i - 1);
      if (x == nullptr || hipEventCreateWithFlags(&join[i], hipEventDisableTiming) != hipSuccess) {
        join[i] = nullptr;
        break;
      }
      st[i] = x;
      n = i + 1;
    }
    if (n < 2) return hipSuccess;
    open = true;
    hipError_t e = hipEventRecord(fork, s);
    for (int i = 1; i < n && e == hipSuccess; ++i) e = hipStreamWaitEvent(st[i], fork, 0);
    return e;
  }
  hipStream_t at(int e) const { return st[e % n]; }
  hipError_t end() {
    hipError_t e = hipSuccess;
    for (int i = 1; i < n && e == hipSuccess; ++i) {
      e = hipEventRecord(join[i], st[i]);
      if (e == hipSuccess) e = hipStreamWaitEvent(st[0], join[i], 0);
    }
    if (e == hipSuccess) open = false;
    return e;
  }
  ~Fan() {
    if (open)
      for (int i = 1; i < n; ++i) (void)hipStreamSynchronize(st[i]);
    if (fork != nullptr) (void)hipEventDestroy(fork);
    for (int i = 0; i < kJacobiGroups; ++i)
      if (join[i] != nullptr) (void)hipEventDestroy(join[i]);
  }
};

// With scratch (the split step) and at least two jobs, the job set runs as up to kJacobiGroups
// contiguous groups, group 0 on s and the others on aux_stream(): a round's rotation launch has
// one workgroup per block pair and leaves most of the chip idle, and the other groups' Gram and
// apply launches fill it meanwhile.  The groups share no job, state entry or scratch.  In each
// block of sweeps between host checks, group g + 1 starts once group g's first Gram launch of the
// block is done (a phase apart), and every group joins s before the check.  Concurrent calls on
// one device share the extra streams, which orders their groups but keeps each call's
// dependencies on its own events.
inline hipError_t jacobi_gram(const JacobiJob* jobs, int njobs, int64_t max_r, int64_t max_c, JacobiState* st,
                              uint32_t* status, hipStream_t s, bool v_given, void* scratch) {
  const unsigned gb = (unsigned)std::max<int64_t>(1, std::min<int64_t>((max_c * max_c + 255) / 256, 4096));
  k_jacobi_begin<<<dim3(gb, (unsigned)njobs), 256, 0, s>>>(jobs, st, v_given ? 1 : 0);
  const int nb = (int)((max_c + kGW - 1) / kGW), nbp = nb + (nb & 1);
  const dim3 g((unsigned)std::max(1, nbp / 2), (unsigned)njobs);
  GramSplit S{};
  if (scratch != nullptr) {
    S.npairs = std::max(1, nbp / 2);
    S.slice = gram_slice_rows(max_r);
    S.nslices = (int)((max_r + S.slice - 1) / S.slice);
    S.part = (double*)scratch;
    S.qrot = S.part + (size_t)njobs * S.npairs * S.nslices * kGN * kGN;
    S.need = (int*)(S.qrot + (size_t)njobs * S.npairs * kGN * kGN);
  }
  const int slices_a = S.nslices, slices_v = S.slice ? (int)((max_c + S.slice - 1) / S.slice) : 0;
  // a sweep of the split step is three launches per round and job group, milliseconds even once
  // every job has converged (their launches return at once), and so is a sweep over more than
  // 2^26 matrix entries: check the flags after each one
  const int check = (scratch != nullptr || (double)max_r * (double)max_c * njobs > 67108864.0) ? 1 : kJacobiCheckSweeps;
  struct Group {
    const JacobiJob* jobs;
    JacobiState* st;
    GramSplit S;
    int n;
    hipStream_t s;
    hipEvent_t started, joined;   // after the group's first Gram launch of a block; at its end
  };
  Group grp[kJacobiGroups] = {};
  int ng = (scratch != nullptr) ? std::min(kJacobiGroups, njobs) : 1;
  for (int i = 0; i < ng; ++i) {
    hipStream_t si = (i == 0) ? s : aux_stream(i - 1);      // s may be the null stream
    if ((i > 0 && si == nullptr) || (ng > 1 && (hipEventCreateWithFlags(&grp[i].started, hipEventDisableTiming) != hipSuccess ||
                                     hipEventCreateWithFlags(&grp[i].joined, hipEventDisableTiming) != hipSuccess))) {
      ng = i;            // run with the groups set up so far (at least group 0 on s)
      break;
    }
    grp[i].s = si;
  }
  if (ng == 0) ng = 1;
  if (ng == 1) {
    for (int i = 0; i < kJacobiGroups; ++i) {
      if (grp[i].started != nullptr) (void)hipEventDestroy(grp[i].started);
      if (grp[i].joined != nullptr) (void)hipEventDestroy(grp[i].joined);
      grp[i].started = grp[i].joined = nullptr;
    }
  }
  for (int i = 0, j0 = 0; i < ng; ++i) {
    const int j1 = (int)((int64_t)njobs * (i + 1) / ng);
    GramSplit Si = S;
    if (scratch != nullptr) {
      Si.part += (size_t)j0 * S.npairs * S.nslices * kGN * kGN;
      Si.qrot += (size_t)j0 * S.npairs * kGN * kGN;
      Si.need += (size_t)j0 * S.npairs;
    }
    grp[i].jobs = jobs + j0;
    grp[i].st = st + j0;
    grp[i].S = Si;
    grp[i].n = j1 - j0;
    grp[i].s = (i == 0) ? s : grp[i].s;
    j0 = j1;
  }
  auto run = [&]() -> hipError_t {
    std::vector<JacobiState> h(njobs);
    for (int sweep = 0; sweep < kJacobiMaxSweeps;) {
      hipError_t e = hipSuccess;
      const int sweep0 = sweep;
      for (int gi = 0; gi < ng; ++gi) {
        const Group& G = grp[gi];
        if (gi > 0 && (e = hipStreamWaitEvent(G.s, grp[gi - 1].started, 0)) != hipSuccess) return e;
        for (int b = 0, sw = sweep0; b < check && sw < kJacobiMaxSweeps; ++b, ++sw) {
          for (int round = 0; round < nbp - 1; ++round) {
            if (scratch == nullptr) {
              k_bjacobi_gram<<<g, 256, 0, G.s>>>(G.jobs, G.st, round);
            } else {
              k_bjg_part<<<dim3((unsigned)(G.S.npairs * G.S.nslices), (unsigned)G.n), 256, 0, G.s>>>(G.jobs, G.st,
                                                                                                     round, G.S);
              if (ng > 1 && b == 0 && round == 0 && (e = hipEventRecord(G.started, G.s)) != hipSuccess) return e;
              k_bjg_rot<<<dim3((unsigned)G.S.npairs, (unsigned)G.n), 512, 0, G.s>>>(G.jobs, G.st, round, G.S);
              k_bjg_apply<<<dim3((unsigned)(G.S.npairs * (slices_a + slices_v)), (unsigned)G.n), 256, 0, G.s>>>(
                  G.jobs, G.st, round, G.S, slices_a, slices_v);
            }
          }
          k_jacobi_sweep_end<<<1, 256, 0, G.s>>>(G.st, G.n);
        }
      }
      for (int b = 0; b < check && sweep < kJacobiMaxSweeps; ++b) ++sweep;
      for (int gi = 1; gi < ng; ++gi) {
        e = hipEventRecord(grp[gi].joined, grp[gi].s);
        if (e == hipSuccess) e = hipStreamWaitEvent(s, grp[gi].joined, 0);
        if (e != hipSuccess) return e;
      }
      e = hipMemcpyAsync(h.data(), st, sizeof(JacobiState) * njobs, hipMemcpyDeviceToHost, s);
      if (e == hipSuccess) e = hipStreamSynchronize(s);
      if (e != hipSuccess) return e;
      bool all = true;
      for (int j = 0; j < njobs; ++j) all = all && h[j].done;
      if (all) break;
    }
    return hipSuccess;
  };
  hipError_t e = run();
  for (int gi = 0; gi < kJacobiGroups; ++gi) {
    // every group joins s before each host check, so the extra streams have drained when run()
    // returns normally
    if (e != hipSuccess && gi > 0 && gi < ng) (void)hipStreamSynchronize(grp[gi].s);
    if (grp[gi].started != nullptr) (void)hipEventDestroy(grp[gi].started);
    if (grp[gi].joined != nullptr) (void)hipEventDestroy(grp[gi].joined);
  }
  if (e != hipSuccess) return e;
  k_jacobi_check<<<1, 256, 0, s>>>(st, njobs, status);
  return hipGetLastError();
}

constexpr size_t kBJacobiLds = 150 * 1024;

// Column block width of jacobi_block for the given largest row and column counts, and how many
// of its workgroups one CU holds at once (LDS bound).
inline void jacobi_block_shape(int64_t max_r, int64_t max_c, int64_t* width, int64_t* per_cu) {
  const int64_t w = std::min<int64_t>(16, (int64_t)(kBJacobiLds / (16 * (size_t)(max_r + max_c))));
  if (w < 16) {
    *width = kGW;
    *per_cu = 2;
  } else {
    *width = w;
    *per_cu = std::max<int64_t>(1, std::min<int64_t>(8, (int64_t)((160 * 1024) / (16 * w * (max_r + max_c)))));
  }
}

// Block one-sided Jacobi over njobs jobs (max_r, max_c the largest row and column counts): the
// block width is the largest that lets 2w columns of A and V fit the LDS budget (at most 16);
// longer columns take the Gram-based step.  As jacobi_multi, the host checks the done flags every
// kJacobiCheckSweeps sweeps.  v_given: each job's V already holds an orthogonal starting factor
// (A then being the matrix times it), which the rotations multiply.
inline hipError_t jacobi_block(const JacobiJob* jobs, int njobs, int64_t max_r, int64_t max_c, JacobiState* st,
                               uint32_t* status, hipStream_t s, bool v_given = false, void* split = nullptr) {
  const int w = (int)std::min<int64_t>(16, (int64_t)(kBJacobiLds / (16 * (size_t)(max_r + max_c))));
  if (w < 16) return jacobi_gram(jobs, njobs, max_r, max_c, st, status, s, v_given, split);
  const size_t lds = sizeof(double) * 2 * (size_t)w * (size_t)(max_r + max_c);
  const unsigned gb = (unsigned)std::max<int64_t>(1, std::min<int64_t>((max_c * max_c + 255) / 256, 4096));
  k_jacobi_begin<<<dim3(gb, (unsigned)njobs), 256, 0, s>>>(jobs, st, v_given ? 1 : 0);
  const int nb = (int)((max_c + w - 1) / w), nbp = nb + (nb & 1);
  const dim3 g((unsigned)std::max(1, nbp / 2), (unsigned)njobs);
  std::vector<JacobiState> h(njobs);
  for (int sweep = 0; sweep < kJacobiMaxSweeps;) {
    for (int b = 0; b < kJacobiCheckSweeps && sweep < kJacobiMaxSweeps; ++b, ++sweep) {
      for (int round = 0; round < nbp - 1; ++round) k_bjacobi_round<<<g, 256, lds, s>>>(jobs, st, round, w);
      k_jacobi_sweep_end<<<1, 256, 0, s>>>(st, njobs);
    }
    hipError_t e = hipMemcpyAsync(h.data(), st, sizeof(JacobiState) * njobs, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return e;
    bool all = true;
    for (int j = 0; j < njobs; ++j) all = all && h[j].done;
    if (all) break;
  }
  k_jacobi_check<<<1, 256, 0, s>>>(st, njobs, status);
  return hipGetLastError();
}

// Sorted thin factors from converged Jacobi jobs: left (r x c) = A's columns normalised, right
// (c x c) = V, s (c), all permuted to nonincreasing s (equal norms keep their column order); zero
// columns give zero vectors; a null left pointer skips that job's left factor.  Three launches with one wave per column and blockIdx.y the job, so
// that long columns are spread over the chip: the column norms into s (unsorted), the scatter of
// every column to its rank (the norms staged in LDS), then s itself sorted by one workgroup per job.
__global__ void __launch_bounds__(1024) k_svd_norms(const JacobiJob* __restrict__ jobs, double* const* sv) {
  const JacobiJob J = jobs[blockIdx.y];
  const int64_t r = J.r, c = J.c;
  const int lane = threadIdx.x & 63;
  const int64_t j = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 6);
  if (j >= c) return;
  double s = 0.0;
  for (int64_t t = lane; t < r; t += 64) s += J.a[j * r + t] * J.a[j * r + t];
  s = wave_sum_f64(s);
  if (lane == 0) sv[blockIdx.y][j] = sqrt(s);
}

// Position of column j among c norms sorted nonincreasing: the columns with a larger norm, or an
// equal norm and a smaller index, come first.
__device__ __forceinline__ int64_t svd_rank(const double* nrm, int64_t c, int64_t j, int lane) {
  const double s = nrm[j];
  double cnt = 0.0;
  for (int64_t k = lane; k < c; k += 64) cnt += ((nrm[k] > s) || (nrm[k] == s && k < j)) ? 1.0 : 0.0;
  return (int64_t)wave_sum_f64(cnt);
}

__global__ void __launch_bounds__(1024) k_svd_scatter(const JacobiJob* __restrict__ jobs, double* const* left,
                                                      double* const* right, double* const* sv) {
  extern __shared__ double nrm[];          // c column norms (8 c bytes: 128 KiB at c = 16384)
  const JacobiJob J = jobs[blockIdx.y];
  const int64_t r = J.r, c = J.c;
  if ((int64_t)blockIdx.x * 16 >= c) return;
  const double* S = sv[blockIdx.y];
  for (int64_t k = threadIdx.x; k < c; k += blockDim.x) nrm[k] = S[k];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t j = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 6);
  if (j >= c) return;
  const int64_t d = svd_rank(nrm, c, j, lane);
  const double inv = (nrm[j] > 0.0) ? 1.0 / nrm[j] : 0.0;
  double* L = left[blockIdx.y];
  double* R = right[blockIdx.y];
  if (L != nullptr)
    for (int64_t t = lane; t < r; t += 64) L[d * r + t] = J.a[j * r + t] * inv;
  for (int64_t t = lane; t < c; t += 64) R[d * c + t] = J.v[j * c + t];
}

__global__ void __launch_bounds__(1024) k_svd_sort(const JacobiJob* __restrict__ jobs, double* const* sv) {
  extern __shared__ double nrm[];
  const int64_t c = jobs[blockIdx.x].c;
  double* S = sv[blockIdx.x];
  for (int64_t k = threadIdx.x; k < c; k += blockDim.x) nrm[k] = S[k];
  __syncthreads();
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int64_t j = wid; j < c; j += nw) {
    const int64_t d = svd_rank(nrm, c, j, lane);
    if (lane == 0) S[d] = nrm[j];
  }
}

// left/right/sv hold one pointer per job; max_c is the largest column count of the jobs.
inline void svd_finalize(const JacobiJob* jobs, double* const* left, double* const* right, double* const* sv,
                         int njobs, int64_t max_c, hipStream_t s) {
  const dim3 g((unsigned)((max_c + 15) / 16), (unsigned)njobs);
  const size_t lds = sizeof(double) * (size_t)max_c;
  k_svd_norms<<<g, 1024, 0, s>>>(jobs, sv);
  k_svd_scatter<<<g, 1024, lds, s>>>(jobs, left, right, sv);
  k_svd_sort<<<njobs, 1024, lds, s>>>(jobs, sv);
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


constexpr int GT = 64, GK = 16;

}  // namespace
}  // namespace iso

namespace iso {
namespace {

// A batch of independent GEMMs in one launch: grid.z indexes the job; blocks outside a
// job's M x N exit.  C(i,j) = alpha * sum_k A(i,k) B(k,j) + beta * C(i,j) with X(i,k) at
// X[i*xs0 + k*xs1].  `upper`: only the tiles on or above the diagonal are computed (for a
// symmetric product whose lower triangle the caller fills in).  `skip`: if set and *skip is
// nonzero when the kernel runs, the job is left out (an iteration whose job has converged).
struct GemmJob {
  const double* A;
  const double* B;
  double* C;
  int64_t as0, as1, bs0, bs1, cs0, cs1;
  int64_t M, N, K;
  double alpha, beta;
  int upper;
  const int* skip;
};

typedef double gemm_f64x4_t __attribute__((ext_vector_type(4)));

// One output tile of C = alpha A B + beta C on v_mfma_f64_16x16x4_f64 (lane (ln, g) supplies
// A[ln][g] and B[g][ln], receives D[g + 4v][ln] in register pair v).  W MFMA blocks per wave side:
// the four waves (2 x 2) each own a 16W x 16W block of the 32W x 32W tile; W = 2 gives 64 x 64
// tiles, W = 4 gives 128 x 128 tiles (16 MFMAs per 4-deep k step per wave, and each k-tile load
// feeds twice the rows and columns).  k in steps of GK = 16 staged in LDS, double-buffered: the
// next k-tile is loaded into registers before the current one's MFMAs and written to the other
// buffer after them, one barrier per step.  Operands are loaded along whichever of their strides
// is 1, so row- and column-major inputs both read whole cache lines, and staged in the layout that
// load writes without bank conflicts: k-major ([k][i], rows of PAD doubles, padded so that the four
// k rows of a fragment read fall on different bank halves) for an operand read along i, i-major
// ([i][k], rows of SK = GK + 2 doubles) for one read along k.  In the i-major layout the sixteen
// rows of a fragment read start 36 banks apart (mod 64), so they and the two k of a half-wave
// cover the 64 banks once; a k-major store of a k-fast operand would put 16 k rows 1152 bytes apart
// (8-way conflicts).
template <int W>
struct GemmTile {
  static constexpr int TM = 32 * W, TW = 16 * W, PAD = (W == 2) ? 80 : TM + 16, PT = GK * TM / 256;
  static constexpr int SK = GK + 2;
  static constexpr int BUF = (GK * PAD > TM * SK) ? GK * PAD : TM * SK;
};

// AK / BK: A / B is read along k, else along its rows / columns; a template parameter, so that
// each instantiation holds only its own address arithmetic.
template <int W, bool AK, bool BK>
__device__ __forceinline__ void gemm_tile_l(const GemmJob& J, int64_t i0, int64_t j0, double (*As)[GemmTile<W>::BUF],
                                            double (*Bs)[GemmTile<W>::BUF]) {
  using T = GemmTile<W>;
  constexpr int TM = T::TM, TW = T::TW, PAD = T::PAD, PT = T::PT, SK = T::SK;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  const int wm = w >> 1, wn = w & 1;
  constexpr bool a_kfast = AK, b_kfast = BK;
  gemm_f64x4_t acc[W][W];
#pragma unroll
  for (int rb = 0; rb < W; ++rb)
#pragma unroll
    for (int cb = 0; cb < W; ++cb) acc[rb][cb] = gemm_f64x4_t{0.0, 0.0, 0.0, 0.0};
  double pa[PT], pb[PT];
  // element e of a k-tile: 16 consecutive k of one row (k-fast operand) or TM consecutive rows
  // of one k (the other)
  auto load = [&](int64_t k0) {
#pragma unroll
    for (int q = 0; q < PT; ++q) {
      const int e = threadIdx.x + 256 * q;
      const int ka = a_kfast ? (e & 15) : (e / TM), ia = a_kfast ? (e >> 4) : (e % TM);
      const int kb = b_kfast ? (e & 15) : (e / TM), jb = b_kfast ? (e >> 4) : (e % TM);
      const int64_t gi = i0 + ia, gka = k0 + ka, gj = j0 + jb, gkb = k0 + kb;
      pa[q] = (gi < J.M && gka < J.K) ? gmem(J.A)[gi * J.as0 + gka * J.as1] : 0.0;
      pb[q] = (gj < J.N && gkb < J.K) ? gmem(J.B)[gkb * J.bs0 + gj * J.bs1] : 0.0;
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int q = 0; q < PT; ++q) {
      const int e = threadIdx.x + 256 * q;
      const int ka = a_kfast ? (e & 15) : (e / TM), ia = a_kfast ? (e >> 4) : (e % TM);
      const int kb = b_kfast ? (e & 15) : (e / TM), jb = b_kfast ? (e >> 4) : (e % TM);
      As[buf][a_kfast ? ia * SK + ka : ka * PAD + ia] = pa[q];
      Bs[buf][b_kfast ? jb * SK + kb : kb * PAD + jb] = pb[q];
    }
  };
  load(0);
  store(0);
  __syncthreads();
  int buf = 0;
  for (int64_t k0 = 0; k0 < J.K; k0 += GK) {
    const bool more = k0 + GK < J.K;
    if (more) load(k0 + GK);
#pragma unroll
    for (int sub = 0; sub < GK / 4; ++sub) {
      __builtin_amdgcn_sched_barrier(0);
      double a[W], b[W];
#pragma unroll
      for (int rb = 0; rb < W; ++rb) {
        const int i = TW * wm + 16 * rb + ln, k = 4 * sub + g;
        a[rb] = As[buf][a_kfast ? i * SK + k : k * PAD + i];
      }
#pragma unroll
      for (int cb = 0; cb < W; ++cb) {
        const int j = TW * wn + 16 * cb + ln, k = 4 * sub + g;
        b[cb] = Bs[buf][b_kfast ? j * SK + k : k * PAD + j];
      }
#pragma unroll
      for (int rb = 0; rb < W; ++rb)
#pragma unroll
        for (int cb = 0; cb < W; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[rb], b[cb], acc[rb][cb], 0, 0, 0);
    }
    // the other buffer was last read before the previous step's barrier
    if (more) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
#pragma unroll
  for (int rb = 0; rb < W; ++rb) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int cb = 0; cb < W; ++cb)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t gi = i0 + TW * wm + 16 * rb + g + 4 * v, gj = j0 + TW * wn + 16 * cb + ln;
        if (gi < J.M && gj < J.N) {
          auto cp = gmem(J.C) + gi * J.cs0 + gj * J.cs1;
          *cp = (J.beta == 0.0) ? J.alpha * acc[rb][cb][v] : J.alpha * acc[rb][cb][v] + J.beta * *cp;
        }
      }
  }
}

template <int W>
__device__ __forceinline__ void gemm_tile(const GemmJob& J, int64_t bx, int64_t by) {
  using T = GemmTile<W>;
  __shared__ double As[2][T::BUF];
  __shared__ double Bs[2][T::BUF];
  const int64_t i0 = bx * T::TM, j0 = by * T::TM;
  if (i0 >= J.M || j0 >= J.N || (J.upper && i0 > j0)) return;
  if (J.skip != nullptr && *J.skip != 0) return;
  if (J.as1 == 1) {
    if (J.bs0 == 1) gemm_tile_l<W, true, true>(J, i0, j0, As, Bs);
    else gemm_tile_l<W, true, false>(J, i0, j0, As, Bs);
  } else {
    if (J.bs0 == 1) gemm_tile_l<W, false, true>(J, i0, j0, As, Bs);
    else gemm_tile_l<W, false, false>(J, i0, j0, As, Bs);
  }
}

// A batch of jobs: grid.z indexes the job.
template <int W>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) k_gemm_jobs(const GemmJob* __restrict__ jobs) {
  const GemmJob J = jobs[blockIdx.z];
  gemm_tile<W>(J, blockIdx.x, blockIdx.y);
}

// One job passed by value.
template <int W>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) k_gemm_one(GemmJob J) {
  gemm_tile<W>(J, blockIdx.x, blockIdx.y);
}

// 128 x 128 tiles once the outputs are at least 256 on both sides, else 64 x 64.
inline bool gemm_big(int64_t M, int64_t N) { return M >= 256 && N >= 256; }

// njobs jobs from a device table, at most max_m x max_n outputs each.
inline void gemm_jobs(const GemmJob* jobs, int njobs, int64_t max_m, int64_t max_n, hipStream_t s) {
  if (gemm_big(max_m, max_n)) {
    const dim3 g((unsigned)((max_m + 127) / 128), (unsigned)((max_n + 127) / 128), (unsigned)njobs);
    k_gemm_jobs<4><<<g, 256, 0, s>>>(jobs);
  } else {
    const dim3 g((unsigned)((max_m + 63) / 64), (unsigned)((max_n + 63) / 64), (unsigned)njobs);
    k_gemm_jobs<2><<<g, 256, 0, s>>>(jobs);
  }
}

// C(i,j) = alpha * sum_k A(i,k) B(k,j) + beta * C(i,j); X(i,k) at X[i*xs0 + k*xs1].
inline void gemm(int64_t M, int64_t N, int64_t Kd, double alpha, const double* A, int64_t as0, int64_t as1,
                 const double* B, int64_t bs0, int64_t bs1, double beta, double* C, int64_t cs0, int64_t cs1,
                 hipStream_t s) {
  const GemmJob J{A, B, C, as0, as1, bs0, bs1, cs0, cs1, M, N, Kd, alpha, beta, 0, nullptr};
  if (gemm_big(M, N)) {
    k_gemm_one<4><<<dim3((unsigned)((M + 127) / 128), (unsigned)((N + 127) / 128)), 256, 0, s>>>(J);
  } else {
    k_gemm_one<2><<<dim3((unsigned)((M + 63) / 64), (unsigned)((N + 63) / 64)), 256, 0, s>>>(J);
  }
}

// One job with every field given (a sub-block product, the `upper` tiles).
inline void gemm_job(const GemmJob& J, hipStream_t s) {
  if (gemm_big(J.M, J.N)) {
    k_gemm_one<4><<<dim3((unsigned)((J.M + 127) / 128), (unsigned)((J.N + 127) / 128)), 256, 0, s>>>(J);
  } else {
    k_gemm_one<2><<<dim3((unsigned)((J.M + 63) / 64), (unsigned)((J.N + 63) / 64)), 256, 0, s>>>(J);
  }
}

// ---- Cholesky factor of a symmetric positive definite matrix ------------------------------------
// G = R^T R with R upper triangular, G q x q col-major and only its upper triangle read, R written
// over it (zeros below the diagonal), for a table of jobs at once.  Right-looking in 64-column
// panels: each job's diagonal block factored in LDS by one workgroup, its panel's block row solved
// against it (one thread per column), the trailing upper triangles updated on the batched MFMA
// GEMM.  A pivot that is not positive and finite sets the job's fail flag (its factor is then
// zeroed, so that what follows stays finite).
constexpr int kCholB = 64;

struct CholJob {
  double* g;          // q x q col-major, upper triangle holding G on entry, R on exit
  int64_t q;
  int* fail;          // 0 on entry
};

__global__ void __launch_bounds__(256) k_chol_diag_jobs(const CholJob* __restrict__ jobs, int64_t kb) {
  const CholJob J = jobs[blockIdx.x];
  if (kb >= J.q) return;
  __shared__ double a[kCholB][kCholB + 1];
  __shared__ int bad;
  const int nb = (int)min<int64_t>(kCholB, J.q - kb);
  double* g = J.g;
  const int64_t q = J.q;
  for (int e = threadIdx.x; e < nb * nb; e += blockDim.x) {
    const int i = e % nb, l = e / nb;
    a[i][l] = (i <= l) ? g[(kb + i) + (kb + l) * q] : 0.0;
  }
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  for (int j = 0; j < nb; ++j) {
    if (threadIdx.x == 0) {
      double d = a[j][j];
      if (!(d > 0.0) || !isfinite(d)) {
        bad = 1;
        d = 1.0;
      }
      a[j][j] = sqrt(d);
    }
    __syncthreads();
    const double rjj = a[j][j];
    for (int l = j + 1 + (int)threadIdx.x; l < nb; l += blockDim.x) a[j][l] /= rjj;
    __syncthreads();
    for (int e = threadIdx.x; e < nb * nb; e += blockDim.x) {
      const int i = e % nb, l = e / nb;
      if (i > j && i <= l) a[i][l] -= a[j][i] * a[j][l];
    }
    __syncthreads();
  }
  for (int e = threadIdx.x; e < nb * nb; e += blockDim.x) {
    const int i = e % nb, l = e / nb;
    g[(kb + i) + (kb + l) * q] = (i <= l) ? a[i][l] : 0.0;
  }
  if (threadIdx.x == 0 && bad) *J.fail = 1;
}

__global__ void __launch_bounds__(256) k_chol_panel_jobs(const CholJob* __restrict__ jobs, int64_t kb) {
  const CholJob J = jobs[blockIdx.y];
  if (kb + kCholB >= J.q) return;                  // no columns right of this job's last panel
  __shared__ double rk[kCholB][kCholB + 1];
  double* g = J.g;
  const int64_t q = J.q;
  for (int e = threadIdx.x; e < kCholB * kCholB; e += blockDim.x) {
    const int i = e % kCholB, l = e / kCholB;
    rk[i][l] = (i <= l) ? g[(kb + i) + (kb + l) * q] : 0.0;
  }
  __syncthreads();
  for (int64_t c = kb + kCholB + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < q;
       c += (int64_t)gridDim.x * blockDim.x) {
    auto col = gmem(g) + kb + c * q;
    double x[kCholB];
#pragma unroll
    for (int i = 0; i < kCholB; ++i) x[i] = col[i];
#pragma unroll
    for (int i = 0; i < kCholB; ++i) {
      double t = x[i];
#pragma unroll
      for (int l = 0; l < i; ++l) t -= rk[l][i] * x[l];
      x[i] = t / rk[i][i];
    }
#pragma unroll
    for (int i = 0; i < kCholB; ++i) col[i] = x[i];
  }
}

// The trailing-update products of panel kb, one per job (M = 0 for a job with nothing right of it).
__global__ void k_chol_trail_jobs(const CholJob* __restrict__ jobs, int njobs, int64_t kb, GemmJob* __restrict__ out) {
  for (int j = threadIdx.x; j < njobs; j += blockDim.x) {
    const CholJob J = jobs[j];
    const int64_t t0 = kb + kCholB, rem = J.q - t0;
    GemmJob G{};
    if (rem > 0) {
      const double* rp = J.g + kb + t0 * J.q;
      G = GemmJob{rp, rp, J.g + t0 + t0 * J.q, J.q, 1, 1, J.q, 1, J.q, rem, rem, kCholB, -1.0, 1.0, 1, nullptr};
    }
    out[j] = G;
  }
}

__global__ void k_chol_finish_jobs(const CholJob* __restrict__ jobs) {
  const CholJob J = jobs[blockIdx.y];
  const bool zero = *J.fail != 0;
  const int64_t q = J.q;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < q * q; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e % q, j = e / q;
    if (zero || i > j) J.g[e] = 0.0;
  }
}

// The factors of njobs jobs (device table; max_q the largest q; trail: scratch for njobs GemmJobs),
// panel by panel over all jobs at once.  A job's last panel may be short (the diagonal kernel takes
// any width up to 64); it has no columns to its right, so the panel solve and the trailing update
// only ever see full panels.
inline void cholesky_upper_jobs(const CholJob* jobs, int njobs, int64_t max_q, GemmJob* trail, hipStream_t s) {
  for (int64_t kb = 0; kb < max_q; kb += kCholB) {
    k_chol_diag_jobs<<<(unsigned)njobs, 256, 0, s>>>(jobs, kb);
    const int64_t rem = max_q - kb - kCholB;
    if (rem <= 0) continue;
    k_chol_panel_jobs<<<dim3((unsigned)((rem + 255) / 256), (unsigned)njobs), 256, 0, s>>>(jobs, kb);
    k_chol_trail_jobs<<<1, 256, 0, s>>>(jobs, njobs, kb, trail);
    gemm_jobs(trail, njobs, rem, rem, s);
  }
  k_chol_finish_jobs<<<dim3((unsigned)std::max<int64_t>(1, std::min<int64_t>((max_q * max_q + 255) / 256, 4096)),
                            (unsigned)njobs), 256, 0, s>>>(jobs);
}


}  // namespace
}  // namespace iso
