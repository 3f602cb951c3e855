// OrthoMerge-G-TIES (App. F) for 2-D weight matrices with rows >= cols, in binary64 on the
// device, the matrices of a call in batches whose SVDs of each phase run as one Jacobi job set:
//   1. W_0 and W_i = W_0 + tau_i as column-major binary64; M_i = W_0^T W_i (n x n);
//   2. the one-sided Procrustes rotation R_i = U V^T from the block-Jacobi SVD M_i = U S V^T
//      (a zero singular value makes R_i non-unique and is flagged);
//   3. the inverse Cayley map A_i = (R_i + I)^{-1} (R_i - I).  For orthogonal R both factors are
//      functions of R and commute, and (R + I)^T (R + I) = 2I + R + R^T, so
//      A_i = (2I + R_i + R_i^T)^{-1} (R_i - R_i^T): the inverse of a symmetric positive definite
//      matrix (singular exactly when R_i has the eigenvalue -1, flagged), taken from its Jacobi
//      SVD as V S^{-1} U^T;
//   4. A = (mean_i |A_i|_F) sum_i A_i / |sum_i A_i|_F, zero when the sum cancels to 1e-12 of
//      sum_i |A_i|_F;
//   5. the forward map R = (I - A)^{-1} (I + A) = (I + A)^2 (I - A^2)^{-1} (again commuting
//      factors; I - A^2 = I + A^T A is symmetric positive definite), W_rot = W_0 R;
//   6. residuals delta_i = W_i - W_0 R_i rounded to binary32 and merged by the TIES path of the
//      library (iso_topk_mask with the tensor's k, iso_merge TIES with lambda: u = lambda * t
//      rounded to binary32);
//   7. out = W_rot + u, rounded once to the storage type.
#include <vector>

#include "iso_dense.h"
#include "iso_device.h"
#include "iso_ortho.h"

namespace iso {
namespace {

constexpr double kCancelRel = 1e-12;
constexpr int kNormChunks = 512;

// dst (m x n col-major) = W (+ D) from row-major storage
__global__ void k_om_load(double* __restrict__ dst, const void* __restrict__ w, const void* __restrict__ d, int64_t m,
                          int64_t n, int dt) {
  const int64_t total = m * n;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / n, c = e - r * n;
    double v = load_f64(w, e, dt);
    if (d != nullptr) v = v + load_f64(d, e, dt);
    dst[c * m + r] = v;
  }
}

// s = 2I + R + R^T, d = R - R^T (n x n col-major)
__global__ void k_om_sym_skew(double* __restrict__ s, double* __restrict__ d, const double* __restrict__ r,
                              int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n * n; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e % n, j = e / n;
    const double a = r[i + j * n], b = r[j + i * n];
    s[e] = (i == j ? 2.0 : 0.0) + a + b;
    d[e] = a - b;
  }
}

// out(:, k) = x(:, k) / s(k) (r x q col-major); a nonpositive s(k) is flagged
__global__ void k_om_div_cols(double* __restrict__ out, const double* __restrict__ x, const double* __restrict__ s,
                              int64_t r, int64_t q, uint32_t* status) {
  bool bad = false;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < r * q; e += (int64_t)gridDim.x * blockDim.x) {
    const double v = s[e / r];
    bad |= !(v > 0.0);
    out[e] = x[e] / v;
  }
  if (bad) flag_status(status, kStatusInternal);
}

// the smallest of a nonincreasing spectrum must be positive
__global__ void k_om_check_min(const double* __restrict__ s, int64_t n, uint32_t* status) {
  if (threadIdx.x == 0 && !(s[n - 1] > 0.0)) flag_status(status, kStatusInternal);
}

// t = I - a2, p = I + a (n x n col-major)
__global__ void k_om_forward_parts(double* __restrict__ t, double* __restrict__ p, const double* __restrict__ a2,
                                   const double* __restrict__ a, int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n * n; e += (int64_t)gridDim.x * blockDim.x) {
    const double id = ((e % n) == (e / n)) ? 1.0 : 0.0;
    t[e] = id - a2[e];
    p[e] = id + a[e];
  }
}

// part[y * kNormChunks + x] = sum of squares over chunk x of vector y
__global__ void __launch_bounds__(256) k_om_sq_part(const double* __restrict__ x0, int64_t stride, int64_t len,
                                                    double* __restrict__ part) {
  __shared__ double red[4];
  const double* x = x0 + (int64_t)blockIdx.y * stride;
  const int64_t per = (len + kNormChunks - 1) / kNormChunks;
  const int64_t e0 = (int64_t)blockIdx.x * per, e1 = min(len, e0 + per);
  double acc = 0.0;
  for (int64_t e = e0 + threadIdx.x; e < e1; e += blockDim.x) acc += x[e] * x[e];
  acc = wave_sum_f64(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0)
    part[(int64_t)blockIdx.y * kNormChunks + blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// norm[y] = sqrt(sum of the chunks of y, in order); one wave per vector
__global__ void __launch_bounds__(64) k_om_sq_sum(const double* __restrict__ part, double* __restrict__ norm) {
  const int y = blockIdx.x;
  double acc = 0.0;
  for (int z = threadIdx.x; z < kNormChunks; z += 64) acc += part[(int64_t)y * kNormChunks + z];
  acc = wave_sum_f64(acc);
  if (threadIdx.x == 0) norm[y] = sqrt(acc);
}

// coef = (mean of norm[0..K)) / norm[K], or 0 when norm[K] <= kCancelRel * sum norm[0..K)
__global__ void k_om_coef(const double* __restrict__ norm, int K, double* __restrict__ coef) {
  if (threadIdx.x != 0) return;
  double s = 0.0;
  for (int i = 0; i < K; ++i) s += norm[i];
  coef[0] = (norm[K] <= kCancelRel * s) ? 0.0 : (s / (double)K) / norm[K];
}

__global__ void k_om_scale(double* __restrict__ x, const double* __restrict__ coef, int64_t len) {
  const double c = coef[0];
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < len; e += (int64_t)gridDim.x * blockDim.x)
    x[e] = c * x[e];
}

// dst (m x n row-major binary32) = src (m x n col-major binary64), rounded to nearest
__global__ void k_om_to_f32(float* __restrict__ dst, const double* __restrict__ src, int64_t m, int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < m * n; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / n, c = e - r * n;
    dst[e] = (float)src[c * m + r];
  }
}

// out (row-major storage) = round(W_rot + u) with W_rot col-major binary64, u row-major binary32
__global__ void k_om_out(void* __restrict__ out, const double* __restrict__ wrot, const float* __restrict__ u,
                         int64_t m, int64_t n, int dt, uint32_t* status) {
  bool bad = false;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < m * n; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / n, c = e - r * n;
    const double v = wrot[c * m + r] + (double)u[e];
    bad |= !(fabs(v) <= 1.7976931348623157e308);
    if (dt == ISO_BF16) ((uint16_t*)out)[e] = (uint16_t)f64_to_bf16_rne(v);
    else ((float*)out)[e] = (float)v;
  }
  if (bad) flag_status(status, kStatusNonFinite);
}

__global__ void k_om_or_status(uint32_t* __restrict__ dst, const uint32_t* __restrict__ src) {
  if (threadIdx.x == 0 && src[0] != 0u) flag_status(dst, src[0]);
}

struct OmBump {
  uint8_t* p;
  size_t off = 0;
  template <typename T = double>
  T* take(int64_t n) {
    T* r = (T*)(p + off);
    off = align_up(off + sizeof(T) * (size_t)std::max<int64_t>(n, 1), 256);
    return r;
  }
};

// Device blocks of one matrix (the same take() sequence sizes the workspace).
struct OmBufs {
  iso_select_desc* desc;               // K descriptors of the residual TopKMask
  double *w0, *wrot;                   // m x n col-major
  double* wi[ISO_MAX_K];               // W_i, then delta_i (m x n col-major)
  double *ja[ISO_MAX_K], *jv[ISO_MAX_K], *U[ISO_MAX_K], *V[ISO_MAX_K], *S[ISO_MAX_K];
  double *R[ISO_MAX_K], *A[ISO_MAX_K];  // n x n
  double *T, *P, *PP, *Rm, *asum;      // n x n
  double *part, *norm, *coef;
  float* delta[ISO_MAX_K];             // m x n row-major binary32
  float* u;                            // m x n row-major binary32
  uint8_t* sub;                        // workspace of the residual TIES calls
  size_t sub_bytes;
};

size_t ties_sub_bytes(int64_t m, int64_t n, int K, int64_t k) {
  iso_tensor tt{};
  tt.rows = m;
  tt.cols = n;
  tt.k = k;
  const size_t a = iso_workspace_size(ISO_OP_TOPK, &tt, 1, K, ISO_F32);
  const size_t b = iso_workspace_size(ISO_OP_MERGE, &tt, 1, K, ISO_F32);
  return std::max(a, b);
}

OmBufs om_carve(OmBump& bp, int64_t m, int64_t n, int K, int64_t k) {
  OmBufs b{};
  b.desc = bp.take<iso_select_desc>(K);
  b.w0 = bp.take(m * n);
  b.wrot = bp.take(m * n);
  for (int i = 0; i < K; ++i) {
    b.wi[i] = bp.take(m * n);
    b.ja[i] = bp.take(n * n);
    b.jv[i] = bp.take(n * n);
    b.U[i] = bp.take(n * n);
    b.V[i] = bp.take(n * n);
    b.S[i] = bp.take(n);
    b.R[i] = bp.take(n * n);
    b.A[i] = bp.take(n * n);
    b.delta[i] = bp.take<float>(m * n);
  }
  b.T = bp.take(n * n);
  b.P = bp.take(n * n);
  b.PP = bp.take(n * n);
  b.Rm = bp.take(n * n);
  b.asum = bp.take(n * n);
  b.part = bp.take((int64_t)(K + 1) * kNormChunks);
  b.norm = bp.take(K + 1);
  b.coef = bp.take(1);
  b.u = bp.take<float>(m * n);
  b.sub_bytes = ties_sub_bytes(m, n, K, k);
  b.sub = bp.take<uint8_t>((int64_t)b.sub_bytes);
  return b;
}

// Frobenius norms of nv vectors of len entries, stride apart, into norm[0..nv)
void om_norms(const double* x, int64_t stride, int64_t len, int nv, double* part, double* norm, hipStream_t s) {
  k_om_sq_part<<<dim3(kNormChunks, (unsigned)nv), 256, 0, s>>>(x, stride, len, part);
  k_om_sq_sum<<<nv, 64, 0, s>>>(part, norm);
}

// C = A B^T for n x n col-major matrices
void gemm_abt(int64_t n, const double* A, const double* B, double* C, hipStream_t s) {
  gemm(n, n, n, 1.0, A, 1, n, B, n, 1, 0.0, C, 1, n, s);
}

// C = A B for n x n col-major matrices
void gemm_ab(int64_t n, const double* A, const double* B, double* C, hipStream_t s) {
  gemm(n, n, n, 1.0, A, 1, n, B, 1, n, 0.0, C, 1, n, s);
}

// Job tables of a batch of nm matrices: the nm K jobs of the Procrustes and inverse-Cayley job
// sets (job e K + i: matrix e, expert i, on its ja[i]) and the nm jobs of the forward-Cayley set
// (job e: matrix e's ja[0]), each with its states and finalize pointers; the split-step scratch.
struct OmTables {
  JacobiJob *jobs, *jobs1;
  JacobiState *jst, *jst1;
  double **ptrs, **ptrs1;               // left[], right[], sv[] of each set
  void* split;
};

OmTables om_tables(OmBump& bp, int nm, int K, int64_t max_n) {
  OmTables tb{};
  tb.jobs = bp.take<JacobiJob>((int64_t)nm * K);
  tb.jst = bp.take<JacobiState>((int64_t)nm * K);
  tb.ptrs = bp.take<double*>(3 * (int64_t)nm * K);
  tb.jobs1 = bp.take<JacobiJob>(nm);
  tb.jst1 = bp.take<JacobiState>(nm);
  tb.ptrs1 = bp.take<double*>(3 * (int64_t)nm);
  tb.split = bp.take<uint8_t>((int64_t)gram_split_bytes(nm * K, max_n, max_n));
  return tb;
}

constexpr size_t kOrthoBatchBytes = 48ull << 30;   // device blocks of the matrices of one batch
constexpr int kOrthoBatch = 16;

size_t om_matrix_bytes(const iso_tensor& x, int K) {
  OmBump bp{nullptr};
  om_carve(bp, x.rows, x.cols, K, x.k);
  return bp.off;
}

// Consecutive non-empty matrices of the table, at most kOrthoBatch and kOrthoBatchBytes a batch.
std::vector<std::vector<int>> om_batches(const iso_tensor* t, int n_t, int K) {
  std::vector<std::vector<int>> out;
  std::vector<int> cur;
  size_t bytes = 0;
  for (int j = 0; j < n_t; ++j) {
    if (t[j].rows == 0 || t[j].cols == 0) continue;
    const size_t mb = om_matrix_bytes(t[j], K);
    if (!cur.empty() && ((int)cur.size() == kOrthoBatch || bytes + mb > kOrthoBatchBytes)) {
      out.push_back(cur);
      cur.clear();
      bytes = 0;
    }
    cur.push_back(j);
    bytes += mb;
  }
  if (!cur.empty()) out.push_back(cur);
  return out;
}

size_t om_batch_bytes(const iso_tensor* t, const std::vector<int>& ids, int K) {
  int64_t max_n = 1;
  for (int j : ids) max_n = std::max(max_n, t[j].cols);
  OmBump bp{nullptr};
  om_tables(bp, (int)ids.size(), K, max_n);
  for (int j : ids) om_carve(bp, t[j].rows, t[j].cols, K, t[j].k);
  return bp.off;
}

}  // namespace

size_t ortho_workspace_bytes(const iso_tensor* t, int n_t, int K) {
  size_t most = 0;
  for (const auto& ids : om_batches(t, n_t, K)) most = std::max(most, om_batch_bytes(t, ids, K));
  return most;
}

iso_status run_ortho(const iso_tensor* t, int n_t, int K, iso_dtype dt, double lambda, uint8_t* ws,
                     uint32_t* status, hipStream_t s) {
#define OM_TRY(x)                                \
  do {                                           \
    if ((x) != hipSuccess) return ISO_ERR_HIP;   \
  } while (0)
  std::vector<uint8_t> host;
  for (const auto& ids : om_batches(t, n_t, K)) {
    const int nm = (int)ids.size(), nj = nm * K;
    int64_t max_n = 1;
    for (int j : ids) max_n = std::max(max_n, t[j].cols);
    OmBump bp{ws};
    const OmTables tb = om_tables(bp, nm, K, max_n);
    const size_t tab_bytes = bp.off;
    std::vector<OmBufs> bs(nm);
    for (int e = 0; e < nm; ++e) bs[e] = om_carve(bp, t[ids[e]].rows, t[ids[e]].cols, K, t[ids[e]].k);
    // job tables (host image, same layout as on the device)
    host.assign(tab_bytes, 0);
    const auto at = [&](const void* dev) { return host.data() + ((const uint8_t*)dev - ws); };
    JacobiJob* hj = (JacobiJob*)at(tb.jobs);
    JacobiJob* hj1 = (JacobiJob*)at(tb.jobs1);
    double** hp = (double**)at(tb.ptrs);
    double** hp1 = (double**)at(tb.ptrs1);
    for (int e = 0; e < nm; ++e) {
      const OmBufs& b = bs[e];
      const int64_t n = t[ids[e]].cols;
      for (int i = 0; i < K; ++i) {
        const int q = e * K + i;
        hj[q] = JacobiJob{b.ja[i], b.jv[i], n, n};
        hp[q] = b.U[i];
        hp[nj + q] = b.V[i];
        hp[2 * nj + q] = b.S[i];
      }
      hj1[e] = JacobiJob{b.ja[0], b.jv[0], n, n};
      hp1[e] = b.U[0];
      hp1[nm + e] = b.V[0];
      hp1[2 * nm + e] = b.S[0];
    }
    OM_TRY(hipMemcpyAsync(ws, host.data(), tab_bytes, hipMemcpyHostToDevice, s));
    // 1. W_0, W_i (col-major binary64); M_i = W_0^T W_i into the Jacobi matrices
    for (int e = 0; e < nm; ++e) {
      const iso_tensor& x = t[ids[e]];
      const OmBufs& b = bs[e];
      const int64_t m = x.rows, n = x.cols;
      const unsigned gmn = grid_for(m * n);
      k_om_load<<<gmn, 256, 0, s>>>(b.w0, x.base, nullptr, m, n, dt);
      for (int i = 0; i < K; ++i) {
        k_om_load<<<gmn, 256, 0, s>>>(b.wi[i], x.base, x.deltas[i], m, n, dt);
        gemm(n, n, m, 1.0, b.w0, m, 1, b.wi[i], 1, m, 0.0, b.ja[i], 1, n, s);
      }
    }
    // 2. R_i = U V^T from the SVDs of M_i, every matrix's K SVDs as one job set
    OM_TRY(jacobi_block(tb.jobs, nj, max_n, max_n, tb.jst, status, s, false, tb.split));
    svd_finalize(tb.jobs, tb.ptrs, tb.ptrs + nj, tb.ptrs + 2 * nj, nj, max_n, s);
    for (int e = 0; e < nm; ++e) {
      const OmBufs& b = bs[e];
      const int64_t n = t[ids[e]].cols;
      for (int i = 0; i < K; ++i) {
        k_om_check_min<<<1, 64, 0, s>>>(b.S[i], n, status);
        gemm_abt(n, b.U[i], b.V[i], b.R[i], s);
        // 3. the SPD matrix 2I + R + R^T into the Jacobi matrix, R - R^T into A_i
        k_om_sym_skew<<<grid_for(n * n), 256, 0, s>>>(b.ja[i], b.A[i], b.R[i], n);
      }
    }
    // 3. A_i = (2I + R_i + R_i^T)^{-1} (R_i - R_i^T), the inverse as V S^{-1} U^T of its SVD
    OM_TRY(jacobi_block(tb.jobs, nj, max_n, max_n, tb.jst, status, s, false, tb.split));
    svd_finalize(tb.jobs, tb.ptrs, tb.ptrs + nj, tb.ptrs + 2 * nj, nj, max_n, s);
    for (int e = 0; e < nm; ++e) {
      const OmBufs& b = bs[e];
      const int64_t n = t[ids[e]].cols;
      const unsigned gnn = grid_for(n * n);
      for (int i = 0; i < K; ++i) {
        gemm(n, n, n, 1.0, b.U[i], n, 1, b.A[i], 1, n, 0.0, b.T, 1, n, s);     // T = U^T D
        k_om_div_cols<<<gnn, 256, 0, s>>>(b.V[i], b.V[i], b.S[i], n, n, status);
        gemm_ab(n, b.V[i], b.T, b.A[i], s);                                      // A_i = V S^{-1} T
      }
      // 4. A = (mean |A_i|) sum A_i / |sum A_i|
      for (int i = 0; i < K; ++i) om_norms(b.A[i], 0, n * n, 1, b.part, b.norm + i, s);
      k_copy<<<gnn, 256, 0, s>>>(b.asum, b.A[0], n * n);
      for (int i = 1; i < K; ++i) k_add<<<gnn, 256, 0, s>>>(b.asum, b.asum, b.A[i], n * n);
      om_norms(b.asum, 0, n * n, 1, b.part, b.norm + K, s);
      k_om_coef<<<1, 64, 0, s>>>(b.norm, K, b.coef);
      k_om_scale<<<gnn, 256, 0, s>>>(b.asum, b.coef, n * n);
      // 5. I - A^2 into the Jacobi matrix, I + A into P
      gemm_ab(n, b.asum, b.asum, b.T, s);
      k_om_forward_parts<<<gnn, 256, 0, s>>>(b.ja[0], b.P, b.T, b.asum, n);
    }
    // 5. R = (I + A)^2 (I - A^2)^{-1}, W_rot = W_0 R
    OM_TRY(jacobi_block(tb.jobs1, nm, max_n, max_n, tb.jst1, status, s, false, tb.split));
    svd_finalize(tb.jobs1, tb.ptrs1, tb.ptrs1 + nm, tb.ptrs1 + 2 * nm, nm, max_n, s);
    for (int e = 0; e < nm; ++e) {
      const iso_tensor& x = t[ids[e]];
      const OmBufs& b = bs[e];
      const int64_t m = x.rows, n = x.cols;
      k_om_div_cols<<<grid_for(n * n), 256, 0, s>>>(b.V[0], b.V[0], b.S[0], n, n, status);
      gemm_abt(n, b.V[0], b.U[0], b.T, s);                                     // (I - A^2)^{-1}
      gemm_ab(n, b.P, b.P, b.PP, s);
      gemm_ab(n, b.PP, b.T, b.Rm, s);
      gemm(m, n, n, 1.0, b.w0, 1, m, b.Rm, 1, n, 0.0, b.wrot, 1, m, s);
      // 6. residuals delta_i = W_i - W_0 R_i (binary32, row-major) and their TIES merge
      for (int i = 0; i < K; ++i) {
        gemm(m, n, n, -1.0, b.w0, 1, m, b.R[i], 1, n, 1.0, b.wi[i], 1, m, s);
        k_om_to_f32<<<grid_for(m * n), 256, 0, s>>>(b.delta[i], b.wi[i], m, n);
      }
      OM_TRY(hipGetLastError());
      iso_tensor tt{};
      tt.base = b.delta[0];
      for (int i = 0; i < K; ++i) tt.deltas[i] = b.delta[i];
      tt.rows = m;
      tt.cols = n;
      tt.k = x.k;
      iso_status st = iso_topk_mask(&tt, 1, K, ISO_F32, b.desc, nullptr, b.sub, b.sub_bytes, s);
      if (st != ISO_OK) return st;
      float* uptr[1] = {b.u};
      st = iso_merge(&tt, 1, K, ISO_F32, ISO_MERGE_TIES, b.desc, lambda, 0.0, uptr, b.sub, b.sub_bytes, s);
      if (st != ISO_OK) return st;
      k_om_or_status<<<1, 64, 0, s>>>(status, (const uint32_t*)b.sub);
      // 7. out = round(W_rot + u)
      k_om_out<<<grid_for(m * n), 256, 0, s>>>(x.out, b.wrot, b.u, m, n, dt, status);
    }
    OM_TRY(hipGetLastError());
    // the next batch reuses the workspace and the host staging
    OM_TRY(hipStreamSynchronize(s));
  }
  return ISO_OK;
#undef OM_TRY
}

}  // namespace iso
