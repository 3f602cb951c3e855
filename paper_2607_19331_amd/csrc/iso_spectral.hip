// ISO-Merger (Sec. 4.2, App. E, Algorithm 1) on the GPU, binary64 throughout (the paper
// runs every SVD of ISO in FP64).  Per 2-D matrix W_0 (m x n, q = min(m, n)) and experts
// W_i = W_0 + tau_i:
//   1. thin SVDs of W_0 and every W_i: one-sided Jacobi (Hestenes 1958; Demmel & Veselic
//      1992, "Jacobi's method is more accurate than QR"), one workgroup per matrix, columns
//      paired in round-robin order, rotations accumulated into V; singular values sorted
//      nonincreasing;
//   2. joint sign canonicalisation s_ik = sign(<u_0k, u_ik>), sign(0) = 1, on u and v;
//   3. tangent projections xi = D - U_0 sym(U_0^T D) of D = U_i - U_0 (and V), then the
//      trailing modes k > k_keep = round(rho_keep q) are zeroed;
//   4. effect proxies g_i = xi_U Sigma_0 V_0^T + U_0 Sigma_0 xi_V^T and their Gram matrix;
//   5. ridge solve (Gamma + lambda I) c = diag Gamma over the nonzero proxies (Cholesky),
//      clip to [c_min, c_max];
//   6. xi_* = Pi(sum_i c_i xi_i), U_* = polar(U_0 + xi_U*), V_* = polar(V_0 + xi_V*) with
//      polar(X) = P Q^T from the SVD of X (one-sided Jacobi again);
//   7. W_* = U_* Sigma_0 V_*^T, rounded once to the storage type.
// Matrices are held column-major in the workspace; small dense products use a tiled
// binary64 GEMM.  Sizes up to ISO_SPECTRAL_MAX_DIM per side.
#include <vector>

#include "iso_dense.h"
#include "iso_device.h"
#include "iso_spectral.h"

namespace iso {

namespace {


// ---- conversions --------------------------------------------------------------------------------

// dst (col-major, rows x cols of the logical matrix) from row-major storage src (m x n):
// trans = 0: dst = W (m x n);  trans = 1: dst = W^T (n x m), i.e. the storage order itself.
__global__ void k_load_f64(double* __restrict__ dst, const void* __restrict__ w, const void* __restrict__ d, int64_t m,
                           int64_t n, int trans, int dt) {
  const int64_t total = m * n;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    // e indexes the storage (row-major): r = e / n, c = e % n
    const int64_t r = e / n, c = e - r * n;
    double v = load_f64(w, e, dt);
    if (d != nullptr) v = v + load_f64(d, e, dt);
    if (trans) dst[e] = v;              // (c, r) of W^T in col-major n x m
    else dst[c * m + r] = v;            // (r, c) of W in col-major m x n
  }
}

__global__ void k_store_w(void* __restrict__ out, const double* __restrict__ src, int64_t m, int64_t n, int dt,
                          uint32_t* status) {
  const int64_t total = m * n;
  bool bad = false;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / n, c = e - r * n;
    const double v = src[c * m + r];
    bad |= !(fabs(v) <= 1.7976931348623157e308);
    if (dt == ISO_BF16) ((uint16_t*)out)[e] = (uint16_t)f64_to_bf16_rne(v);
    else ((float*)out)[e] = (float)v;
  }
  if (bad) flag_status(status, kStatusNonFinite);
}

// Column signs s_k = sign(<u0_k, u_k>) (sign(0) = 1) applied to the columns of U and V.
__global__ void k_canonicalize(const double* __restrict__ u0, double* __restrict__ u, double* __restrict__ v, int64_t m,
                               int64_t n, int64_t q) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int64_t k = (int64_t)blockIdx.x * nw + wid; k < q; k += (int64_t)gridDim.x * nw) {
    double s = 0.0;
    for (int64_t t = lane; t < m; t += 64) s += u0[k * m + t] * u[k * m + t];
    s = wave_sum_f64(s);
    if (s < 0.0) {
      for (int64_t t = lane; t < m; t += 64) u[k * m + t] = -u[k * m + t];
      for (int64_t t = lane; t < n; t += 64) v[k * n + t] = -v[k * n + t];
    }
  }
}

// S = sym(P) for a q x q col-major P (in place into S)
__global__ void k_sym(double* __restrict__ s, const double* __restrict__ p, int64_t q) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < q * q; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e % q, j = e / q;
    s[e] = 0.5 * (p[i + j * q] + p[j + i * q]);
  }
}

// zero the columns k >= keep of an r x q col-major matrix
__global__ void k_mask_cols(double* __restrict__ x, int64_t r, int64_t q, int64_t keep) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < r * q; e += (int64_t)gridDim.x * blockDim.x)
    if (e / r >= keep) x[e] = 0.0;
}

// out(:, k) = x(:, k) * s(k)
__global__ void k_scale_cols(double* __restrict__ out, const double* __restrict__ x, const double* __restrict__ s,
                             int64_t r, int64_t q) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < r * q; e += (int64_t)gridDim.x * blockDim.x)
    out[e] = x[e] * s[e / r];
}

// Gram of K vectors of length len: G[i*K + j] = <g_i, g_j>.  One block per (i, j >= i).
__global__ void __launch_bounds__(1024) k_gram(const double* __restrict__ g, int64_t len, int K, double* __restrict__ G) {
  __shared__ double red[16];
  const int pr = blockIdx.x;
  int i = 0, j = 0, t = pr;
  for (i = 0; i < K; ++i) {
    if (t < K - i) { j = i + t; break; }
    t -= K - i;
  }
  const double* a = g + (int64_t)i * len;
  const double* b = g + (int64_t)j * len;
  double s = 0.0;
  for (int64_t e = threadIdx.x; e < len; e += blockDim.x) s += a[e] * b[e];
  s = wave_sum_f64(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) tot += red[w];
    G[i * K + j] = tot;
    G[j * K + i] = tot;
  }
}

// Unit-retention ridge solve over the nonzero proxies, then clip.  One thread.
__global__ void k_solve(const double* __restrict__ G, int K, double ridge, double cmin, double cmax,
                        double* __restrict__ c, double* __restrict__ coef_out, uint32_t* status) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  int idx[ISO_MAX_K];
  int m = 0;
  for (int i = 0; i < K; ++i) {
    c[i] = 0.0;
    if (G[i * K + i] > 0.0) idx[m++] = i;
  }
  double L[ISO_MAX_K][ISO_MAX_K];
  double b[ISO_MAX_K], y[ISO_MAX_K], x[ISO_MAX_K];
  bool ok = true;
  for (int a = 0; a < m; ++a) {
    b[a] = G[idx[a] * K + idx[a]];
    for (int bb = 0; bb <= a; ++bb) {
      double s = G[idx[a] * K + idx[bb]] + ((a == bb) ? ridge : 0.0);
      for (int t = 0; t < bb; ++t) s -= L[a][t] * L[bb][t];
      if (a == bb) {
        if (!(s > 0.0)) { ok = false; s = 1.0; }
        L[a][a] = sqrt(s);
      } else {
        L[a][bb] = s / L[bb][bb];
      }
    }
  }
  for (int a = 0; a < m; ++a) {
    double s = b[a];
    for (int t = 0; t < a; ++t) s -= L[a][t] * y[t];
    y[a] = s / L[a][a];
  }
  for (int a = m - 1; a >= 0; --a) {
    double s = y[a];
    for (int t = a + 1; t < m; ++t) s -= L[t][a] * x[t];
    x[a] = s / L[a][a];
  }
  for (int a = 0; a < m; ++a) c[idx[a]] = fmin(fmax(x[a], cmin), cmax);
  if (coef_out != nullptr)
    for (int i = 0; i < K; ++i) coef_out[i] = c[i];
  if (!ok) flag_status(status, kStatusInternal);
}

// out = sum_i c[i] * x_i  (K vectors of length len)
__global__ void k_combine(double* __restrict__ out, const double* __restrict__ x, const double* __restrict__ c, int K,
                          int64_t len) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < len; e += (int64_t)gridDim.x * blockDim.x) {
    double s = 0.0;
    for (int i = 0; i < K; ++i) s = s + c[i] * x[(int64_t)i * len + e];
    out[e] = s;
  }
}

// ---- host orchestration --------------------------------------------------------------------------

struct Bump {
  uint8_t* p;
  size_t off = 0;
  template <typename T = double>
  T* take(int64_t n) {
    T* r = (T*)(p + off);
    off = align_up(off + sizeof(T) * (size_t)std::max<int64_t>(n, 1), 256);
    return r;
  }
};

// Device blocks of one matrix; the same sequence of take() calls sizes the workspace.
struct Bufs {
  JacobiJob* jobs;          // K+1 SVD jobs, then the two polar jobs
  JacobiState* jst;         // K+3 convergence states
  double** ptrs;            // 3*(K+1) finalize outputs
  double *ja[ISO_MAX_K + 1], *jv[ISO_MAX_K + 1], *U[ISO_MAX_K + 1], *V[ISO_MAX_K + 1], *S[ISO_MAX_K + 1];
  double *XU, *XV, *P, *Sq, *FU, *FV, *G, *gram, *coef, *AU, *AV, *PA, *PV, *PL, *Wst;
};

Bufs carve(uint8_t* base, int64_t m, int64_t n, int K, size_t* used) {
  const int64_t q = std::min(m, n), r = std::max(m, n);
  Bump bp{base};
  Bufs b;
  b.jobs = bp.take<JacobiJob>(K + 3);
  b.jst = bp.take<JacobiState>(K + 3);
  b.ptrs = bp.take<double*>(3 * (K + 1));
  for (int i = 0; i <= K; ++i) {
    b.ja[i] = bp.take(r * q);
    b.jv[i] = bp.take(q * q);
    b.U[i] = bp.take(m * q);
    b.V[i] = bp.take(n * q);
    b.S[i] = bp.take(q);
  }
  b.XU = bp.take((int64_t)K * m * q);
  b.XV = bp.take((int64_t)K * n * q);
  b.P = bp.take(q * q);
  b.Sq = bp.take(q * q);
  b.FU = bp.take(m * q);
  b.FV = bp.take(n * q);
  b.G = bp.take((int64_t)K * m * n);
  b.gram = bp.take(K * K);
  b.coef = bp.take(K);
  b.AU = bp.take(m * q);
  b.AV = bp.take(n * q);
  b.PA = bp.take(r * q);    // polar: Jacobi copy
  b.PV = bp.take(q * q);    // polar: rotations
  b.PL = bp.take(r * q);    // polar: normalised columns
  b.Wst = bp.take(m * n);
  if (used) *used = bp.off;
  return b;
}

// xi = D - U0 sym(U0^T D) in place on D (r x q col-major), using P, S (q x q) as scratch
void tangent_project(double* d, const double* u0, int64_t r, int64_t q, double* P, double* S, hipStream_t s) {
  gemm(q, q, r, 1.0, u0, r, 1, d, 1, r, 0.0, P, 1, q, s);           // P = U0^T D
  k_sym<<<grid_for(q * q), 256, 0, s>>>(S, P, q);
  gemm(r, q, q, -1.0, u0, 1, r, S, 1, q, 1.0, d, 1, r, s);          // D -= U0 S
}

// X <- polar(X) = P Q^T for X (r x q col-major, r >= q).  Jacobi gives X Q = P diag(s);
// P Q^T does not depend on the column order, so no sort is needed.
hipError_t polar(double* X, int64_t r, int64_t q, const Bufs& b, const JacobiJob* job_dev, uint32_t* status,
                 hipStream_t s) {
  k_copy<<<grid_for(r * q), 256, 0, s>>>(b.PA, X, r * q);
  const hipError_t e = jacobi_block(job_dev, 1, r, q, b.jst, status, s);
  if (e != hipSuccess) return e;
  k_normalize_cols<<<(unsigned)std::max<int64_t>(1, std::min<int64_t>((q + 15) / 16, 1024)), 1024, 0, s>>>(b.PL, b.PA, r,
                                                                                                        q);
  gemm(r, q, q, 1.0, b.PL, 1, r, b.PV, q, 1, 0.0, X, 1, r, s);     // X = P Q^T
  return hipGetLastError();
}

}  // namespace

size_t spectral_workspace_bytes(const iso_tensor* t, int n_t, int K) {
  size_t b = 0;
  for (int j = 0; j < n_t; ++j) {
    size_t u = 0;
    carve(nullptr, std::max<int64_t>(t[j].rows, 1), std::max<int64_t>(t[j].cols, 1), K, &u);
    b = std::max(b, u);
  }
  return b;
}

iso_status run_spectral(const iso_tensor* t, int n_t, int K, iso_dtype dt, const SpectralArgs& a, uint8_t* ws,
                        uint32_t* status, hipStream_t s) {
#define SP_TRY(x)                                \
  do {                                           \
    if ((x) != hipSuccess) return ISO_ERR_HIP;   \
  } while (0)
  // host staging for the job tables; kept until the stream has consumed them
  std::vector<uint8_t> host;
  for (int jt = 0; jt < n_t; ++jt) {
    const int64_t m = t[jt].rows, n = t[jt].cols;
    if (m == 0 || n == 0) continue;
    const int64_t q = std::min(m, n), r = std::max(m, n);
    const bool wide = m < n;
    const Bufs b = carve(ws, m, n, K, nullptr);
    // job table: K+1 SVDs, polar of U_0 + xi_U (m x q), polar of V_0 + xi_V (n x q); finalize pointers
    const size_t jb = sizeof(JacobiJob) * (K + 3), pb = sizeof(double*) * 3 * (K + 1);
    host.assign(jb + pb, 0);
    JacobiJob* hj = (JacobiJob*)host.data();
    double** hp = (double**)(host.data() + jb);
    for (int i = 0; i <= K; ++i) {
      hj[i] = JacobiJob{b.ja[i], b.jv[i], r, q};
      hp[i] = wide ? b.V[i] : b.U[i];                 // left factor of the Jacobi matrix
      hp[(K + 1) + i] = wide ? b.U[i] : b.V[i];       // right factor
      hp[2 * (K + 1) + i] = b.S[i];
    }
    hj[K + 1] = JacobiJob{b.PA, b.PV, m, q};
    hj[K + 2] = JacobiJob{b.PA, b.PV, n, q};
    SP_TRY(hipMemcpyAsync(b.jobs, hj, jb, hipMemcpyHostToDevice, s));
    SP_TRY(hipMemcpyAsync(b.ptrs, hp, pb, hipMemcpyHostToDevice, s));
    // 1. W_0 and W_i = W_0 + tau_i as A = W (tall) or W^T (wide), r x q col-major; SVDs
    for (int i = 0; i <= K; ++i)
      k_load_f64<<<grid_for(m * n), 256, 0, s>>>(b.ja[i], t[jt].base, i ? t[jt].deltas[i - 1] : nullptr, m, n,
                                                  wide ? 1 : 0, dt);
    SP_TRY(jacobi_block(b.jobs, K + 1, r, q, b.jst, status, s));
    k_svd_finalize<<<K + 1, 1024, (sizeof(double) + sizeof(int)) * q, s>>>(b.jobs, b.ptrs, b.ptrs + (K + 1),
                                                                          b.ptrs + 2 * (K + 1));
    const int64_t keep = std::min<int64_t>(q, (int64_t)std::floor(a.rho_keep * (double)q + 0.5));
    for (int i = 1; i <= K; ++i) {
      double* xu = b.XU + (int64_t)(i - 1) * m * q;
      double* xv = b.XV + (int64_t)(i - 1) * n * q;
      // 2. sign canonicalisation against the base
      k_canonicalize<<<grid_for(q * 64), 256, 0, s>>>(b.U[0], b.U[i], b.V[i], m, n, q);
      // 3. displacements, tangent projection, D_keep
      k_sub<<<grid_for(m * q), 256, 0, s>>>(xu, b.U[i], b.U[0], m * q);
      k_sub<<<grid_for(n * q), 256, 0, s>>>(xv, b.V[i], b.V[0], n * q);
      tangent_project(xu, b.U[0], m, q, b.P, b.Sq, s);
      tangent_project(xv, b.V[0], n, q, b.P, b.Sq, s);
      k_mask_cols<<<grid_for(m * q), 256, 0, s>>>(xu, m, q, keep);
      k_mask_cols<<<grid_for(n * q), 256, 0, s>>>(xv, n, q, keep);
      // 4. g_i = xi_U Sigma_0 V_0^T + U_0 Sigma_0 xi_V^T  (m x n col-major)
      double* g = b.G + (int64_t)(i - 1) * m * n;
      k_scale_cols<<<grid_for(m * q), 256, 0, s>>>(b.FU, xu, b.S[0], m, q);
      gemm(m, n, q, 1.0, b.FU, 1, m, b.V[0], n, 1, 0.0, g, 1, m, s);
      k_scale_cols<<<grid_for(m * q), 256, 0, s>>>(b.FU, b.U[0], b.S[0], m, q);
      gemm(m, n, q, 1.0, b.FU, 1, m, xv, n, 1, 1.0, g, 1, m, s);
    }
    // 5. Gram, ridge solve, clip
    k_gram<<<K * (K + 1) / 2, 1024, 0, s>>>(b.G, m * n, K, b.gram);
    k_solve<<<1, 64, 0, s>>>(b.gram, K, a.ridge, a.c_min, a.c_max, b.coef,
                             a.coef_out ? a.coef_out + (int64_t)jt * K : nullptr, status);
    // 6. aggregate, project, retract
    k_combine<<<grid_for(m * q), 256, 0, s>>>(b.AU, b.XU, b.coef, K, m * q);
    k_combine<<<grid_for(n * q), 256, 0, s>>>(b.AV, b.XV, b.coef, K, n * q);
    tangent_project(b.AU, b.U[0], m, q, b.P, b.Sq, s);
    tangent_project(b.AV, b.V[0], n, q, b.P, b.Sq, s);
    k_add<<<grid_for(m * q), 256, 0, s>>>(b.AU, b.AU, b.U[0], m * q);
    k_add<<<grid_for(n * q), 256, 0, s>>>(b.AV, b.AV, b.V[0], n * q);
    SP_TRY(polar(b.AU, m, q, b, b.jobs + (K + 1), status, s));
    SP_TRY(polar(b.AV, n, q, b, b.jobs + (K + 2), status, s));
    // 7. W_* = U_* Sigma_0 V_*^T
    k_scale_cols<<<grid_for(m * q), 256, 0, s>>>(b.FU, b.AU, b.S[0], m, q);
    gemm(m, n, q, 1.0, b.FU, 1, m, b.AV, n, 1, 0.0, b.Wst, 1, m, s);
    k_store_w<<<grid_for(m * n), 256, 0, s>>>(t[jt].out, b.Wst, m, n, dt, status);
    SP_TRY(hipGetLastError());
    // the next tensor reuses the workspace and the host staging: let this one finish first
    SP_TRY(hipStreamSynchronize(s));
  }
  return ISO_OK;
#undef SP_TRY
}

}  // namespace iso
