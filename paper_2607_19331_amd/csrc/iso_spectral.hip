// ISO-Merger (Sec. 4.2, App. E, Algorithm 1) on the GPU, binary64 throughout (the paper
// runs every SVD of ISO in FP64).  Per 2-D matrix W_0 (m x n, q = min(m, n)) and experts
// W_i = W_0 + tau_i:
//   1. thin SVDs of W_0 and every W_i: one-sided Jacobi (Hestenes 1958; Demmel & Veselic
//      1992, on its accuracy), by column blocks paired round-robin over many workgroups,
//      rotations accumulated into V; singular values sorted nonincreasing;
//   2. joint sign canonicalisation s_ik = sign(<u_0k, u_ik>), sign(0) = 1, on u and v;
//   3. tangent projections xi = D - U_0 sym(U_0^T D) of D = U_i - U_0 (and V), then the
//      trailing modes k > k_keep = round(rho_keep q) are zeroed;
//   4. effect proxies g_i = xi_U Sigma_0 V_0^T + U_0 Sigma_0 xi_V^T and their Gram matrix;
//   5. ridge solve (Gamma + lambda I) c = diag Gamma over the nonzero proxies (Cholesky),
//      clip to [c_min, c_max];
//   6. xi_* = Pi(sum_i c_i xi_i), U_* = polar(U_0 + xi_U*), V_* = polar(V_0 + xi_V*) with
//      polar(X) = P Q^T from the SVD of X (one-sided Jacobi again);
//   7. W_* = U_* Sigma_0 V_*^T, rounded once to the storage type.
// Matrices are held column-major in the workspace; dense products use a tiled binary64 GEMM on
// MFMA.  The matrices of one call go in batches whose SVDs (and then whose polar retractions)
// run as one Jacobi job set.  The shorter side is at most ISO_SPECTRAL_MAX_DIM (the column norms
// of the SVD finalize sit in LDS); the longer side is unbounded but for the workspace.
#include <cmath>
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

// X[:, j] /= s[j] (a zero s gives a zero column), X r x q col-major.
__global__ void k_unit_cols(double* __restrict__ x, const double* __restrict__ s, int64_t r, int64_t q) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < r * q; e += (int64_t)gridDim.x * blockDim.x) {
    const double d = s[e / r];
    x[e] = (d > 0.0) ? x[e] / d : 0.0;
  }
}

// Tall matrices whose SVDs came from R: singular values from the Gram carry a relative error of
// about eps (s_max / s_j)^2 / 2, so a matrix with any factor that failed, or with a condition
// number above kQrMaxCond (error bound ~6e-11), is marked for plain Jacobi on A.
constexpr double kQrMaxCond = 1e3;

__global__ void k_qr_guard(const JacobiJob* __restrict__ jobs, double* const* sv, const int* __restrict__ fail,
                           const int* __restrict__ jmat, int njobs, int* __restrict__ bad) {
  for (int j = threadIdx.x; j < njobs; j += blockDim.x) {
    if (jmat[j] < 0) continue;
    const double* S = sv[j];
    const int64_t q = jobs[j].c;
    const bool ok = fail[j] == 0 && S[q - 1] > 0.0 && S[0] <= kQrMaxCond * S[q - 1];
    if (!ok) atomicOr(&bad[jmat[j]], 1);
  }
}

// ---- long reductions: many workgroups, fixed summation order ---------------------------------------
// Slot y of a DotSet sums f(a_y[e], b_y[e]) over len entries, f = a b (diff = 0) or (a - b)^2
// (diff = 1): kRedChunks workgroups per slot each sum one contiguous chunk into part, then one wave
// per slot adds the chunks in order and writes the total to out[o1[y]] and out[o2[y]].
constexpr int kRedChunks = 512;
constexpr int kRedSlots = ISO_MAX_K * (ISO_MAX_K + 1) / 2;

struct DotSet {
  const double* a[kRedSlots];
  const double* b[kRedSlots];
  int o1[kRedSlots], o2[kRedSlots];
};

__global__ void __launch_bounds__(256) k_dot_part(DotSet d, int64_t len, int diff, double* __restrict__ part) {
  __shared__ double red[4];
  const double* a = d.a[blockIdx.y];
  const double* b = d.b[blockIdx.y];
  const int64_t per = (len + kRedChunks - 1) / kRedChunks;
  const int64_t e0 = (int64_t)blockIdx.x * per, e1 = min(len, e0 + per);
  double x = 0.0;
  for (int64_t e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
    const double u = a[e], v = b[e];
    x += diff ? (u - v) * (u - v) : u * v;
  }
  x = wave_sum_f64(x);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) part[(int64_t)blockIdx.y * kRedChunks + blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ void __launch_bounds__(64) k_dot_sum(DotSet d, const double* __restrict__ part, double* __restrict__ out) {
  const int y = blockIdx.x, lane = threadIdx.x;
  double x = 0.0;
  for (int z = lane; z < kRedChunks; z += 64) x += part[(int64_t)y * kRedChunks + z];
  x = wave_sum_f64(x);
  if (lane == 0) {
    out[d.o1[y]] = x;
    out[d.o2[y]] = x;
  }
}

// part: kRedSlots * kRedChunks doubles
void dots(const DotSet& d, int nslots, int64_t len, bool diff, double* part, double* out, hipStream_t s) {
  k_dot_part<<<dim3(kRedChunks, (unsigned)nslots), 256, 0, s>>>(d, len, diff ? 1 : 0, part);
  k_dot_sum<<<nslots, 64, 0, s>>>(d, part, out);
}

// one slot: out[0] = sum over len entries of a b, or of (a - b)^2
void dot1(const double* a, const double* b, int64_t len, bool diff, double* part, double* out, hipStream_t s) {
  DotSet d{};
  d.a[0] = a;
  d.b[0] = b;
  dots(d, 1, len, diff, part, out, s);
}

// Gram of K vectors of length len: G[i*K + j] = <g_i, g_j>, one slot per pair j >= i.
void gram_of(const double* g, int64_t len, int K, double* part, double* G, hipStream_t s) {
  DotSet d{};
  int y = 0;
  for (int i = 0; i < K; ++i)
    for (int j = i; j < K; ++j, ++y) {
      d.a[y] = g + (int64_t)i * len;
      d.b[y] = g + (int64_t)j * len;
      d.o1[y] = i * K + j;
      d.o2[y] = j * K + i;
    }
  dots(d, y, len, false, part, G, s);
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

// ---- polar retraction by Newton-Schulz ----------------------------------------------------------
// polar(X) = P_X Q_X^T equals X (X^T X)^{-1/2} when X has full column rank, which the retraction
// arguments have: U_0 + xi_U with xi_U tangent gives X^T X = I + xi^T xi (Sec. 4.2, App. E).
// The iteration X <- X (3 I - X^T X) / 2 maps each singular value s to s (3 - s^2) / 2 and
// converges quadratically to the polar factor for s in (0, sqrt 3).  The first step scales X by
// 1 / sqrt(c), c the largest absolute column sum of X^T X (at least its largest eigenvalue, by
// Gershgorin), so that every s lies in (0, 1] -- unless c <= 2: every s is then at most sqrt 2,
// already inside the basin, and X is left unscaled (a near-orthonormal retraction argument would
// otherwise be shrunk by up to sqrt c and take several extra steps to grow back).  A job stops
// once max |X^T X - I| <= kNsTol, after one more step.
//
// Scaled variant (for arguments far from orthonormal): Chen and Chow's scaling (SIAM J. Matrix
// Anal. Appl., 2014).  If every s lies in [l, 1], the step X <- a X (3 I - a^2 X^T X) / 2 with
// a^2 = 3 / (1 + l + l^2) maps both l and 1 to l' = a l (3 - a^2 l^2) / 2 and every s into
// [l', 1]; l' grows about 2.6-fold per step while l is small and goes to one quadratically.
// The schedule starts from kNsScaledL0 (a singular value below kNsScaledL0 times the largest
// still grows at least 1.5-fold per step); from the second step on, l is raised to the bound
// s_min^2 >= 1 - q max |X^T X - I| when that is larger, and the last step is a plain one.
// A matrix whose Gram X^T X is exactly zero maps to the zero matrix (one step with T = 0).
struct NsJob {
  double* g;        // q x q: X^T X, then the step matrix T in place
  int64_t q;
  double* t;        // q-space iteration (see polar_gram_batch): T goes here, G is kept; else null
  double* pp[2];    // q-space iteration: the accumulated P_k, ping-pong
  int gs;           // 1: a q-space job (the X-form batch skips it), 0: an X-form job
};

struct NsState {
  unsigned long long err;    // max |G - I| (bit pattern of a nonnegative double)
  unsigned long long csum;   // max absolute column sum of G (likewise)
  int done;                  // no further steps
  int last;                  // the step being taken is the last
  int steps;                 // steps taken: the result is in buffer (steps & 1)
  int pad;
  double lb;                 // scaled variant: lower bound l of the singular values, this step
  double lb_next;            // ... and after it
};

constexpr double kNsTol = 1e-10;
constexpr int kNsMaxSteps = 48;
constexpr int kNsCheckSteps = 4;   // steps queued between host reads of the done flags
constexpr double kNsScaledL0 = 1e-6;

// gs_run: the batch runs the jobs with NsJob::gs equal to it; the others start (and stay) done
__global__ void k_ns_begin(const NsJob* __restrict__ jobs, NsState* st, int njobs, int gs_run) {
  for (int j = threadIdx.x; j < njobs; j += blockDim.x)
    st[j] = NsState{0ull, 0ull, jobs[j].gs != gs_run ? 1 : 0, 0, 0, 0, kNsScaledL0, kNsScaledL0};
}

// q-space jobs: P_0 = I
__global__ void k_ns_eye(const NsJob* __restrict__ jobs, const NsState* st) {
  const int job = blockIdx.y;
  if (st[job].done) return;
  const NsJob J = jobs[job];
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < J.q * J.q; e += (int64_t)gridDim.x * blockDim.x)
    J.pp[0][e] = ((e % J.q) == (e / J.q)) ? 1.0 : 0.0;
}

__global__ void k_ns_reset(NsState* st, int njobs) {
  for (int j = threadIdx.x; j < njobs; j += blockDim.x)
    if (!st[j].done) {
      st[j].err = 0ull;
      st[j].csum = 0ull;
    }
}

// one wave per column of G: its absolute sum and its largest deviation from the identity
__global__ void __launch_bounds__(256) k_ns_stats(const NsJob* __restrict__ jobs, NsState* st) {
  const int job = blockIdx.y;
  if (st[job].done) return;
  const NsJob J = jobs[job];
  const int lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  for (int64_t j = (int64_t)blockIdx.x * nw + (threadIdx.x >> 6); j < J.q; j += (int64_t)gridDim.x * nw) {
    double cs = 0.0, dev = 0.0;
    for (int64_t i = lane; i < J.q; i += 64) {
      const double v = J.g[j * J.q + i];
      cs += fabs(v);
      dev = fmax(dev, fabs(v - (i == j ? 1.0 : 0.0)));
    }
    cs = wave_sum_f64(cs);
    for (int o = 32; o > 0; o >>= 1) dev = fmax(dev, __shfl_xor(dev, o, 64));
    if (lane == 0) {
      atomicMax(&st[job].csum, (unsigned long long)__double_as_longlong(cs));
      atomicMax(&st[job].err, (unsigned long long)__double_as_longlong(dev));
    }
  }
}

// G <- T = (3 I - G / c) / (2 sqrt c) (into J.t instead for a q-space job), c the scale on the first
// step and 1 after it; with
// `scaled`, T = a (3 I - a^2 G / c) / (2 sqrt c) with a from the job's lower bound (a = 1 on the
// last step).
__global__ void k_ns_form(const NsJob* __restrict__ jobs, NsState* st, int scaled) {
  const int job = blockIdx.y;
  if (st[job].done) return;
  const NsJob J = jobs[job];
  const bool first = st[job].steps == 0;
  const double err = __longlong_as_double((long long)st[job].err);
  const double cs = __longlong_as_double((long long)st[job].csum);
  // X^T X == 0 on entry (the zero matrix, or entries whose squares underflow): no polar factor;
  // the result is the zero matrix, taken in this one step with T = 0
  const bool zero = first && cs == 0.0;
  const bool last = err <= kNsTol || zero;
  // the scaled schedule assumes s <= 1 from the start; the plain one only needs s < sqrt 3
  const double c = (first && (scaled || cs > 2.0)) ? cs : 1.0;
  const double ic = (c > 0.0) ? 1.0 / c : 1.0, is = sqrt(ic);
  double a = 1.0, l = 1.0;
  if (scaled && !last) {
    l = st[job].lb;
    if (!first) l = fmax(l, sqrt(fmax(0.0, 1.0 - (double)J.q * err)));
    l = fmin(l, 1.0);
    a = sqrt(3.0 / (1.0 + l + l * l));
  }
  const double a2 = a * a;
  const int64_t n = J.q * J.q;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e % J.q, j = e / J.q;
    (J.t != nullptr ? J.t : J.g)[e] = zero ? 0.0 : ((i == j ? 3.0 : 0.0) - J.g[e] * (a2 * ic)) * (0.5 * a * is);
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st[job].last = last;
    st[job].lb_next = 0.5 * a * l * (3.0 - a2 * l * l);
  }
}

__global__ void k_ns_check(const NsState* st, int njobs, uint32_t* status) {
  for (int j = threadIdx.x; j < njobs; j += blockDim.x)
    if (!st[j].done) flag_status(status, kStatusInternal);
}

__global__ void k_ns_step_end(NsState* st, int njobs) {
  for (int j = threadIdx.x; j < njobs; j += blockDim.x)
    if (!st[j].done) {
      st[j].steps += 1;
      st[j].lb = st[j].lb_next;
      if (st[j].last) st[j].done = 1;
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
  double *ja[ISO_MAX_K + 1], *jv[ISO_MAX_K + 1], *U[ISO_MAX_K + 1], *V[ISO_MAX_K + 1], *S[ISO_MAX_K + 1];
  double* jr[ISO_MAX_K + 1];  // tall matrices: the q x q Cholesky factor R of A^T A (the Jacobi matrix)
  double *XU, *XV, *P, *Sq, *FU, *FV, *G, *gram, *coef, *AU, *AV, *Wst;
  double* red;                // partial sums of the long reductions (kRedSlots x kRedChunks)
  double *PX[2][2], *PG[2];   // polar of U_0 + xi_U (m x q) and of V_0 + xi_V (n x q): the two buffers
                              // of the iterate X, the q x q Gram / step matrix
  double *QT, *QH, *QP[2];    // the tall side's polar in q space (qr_pre matrices): T, G T, P_k
};

// A matrix whose Jacobi runs on the Cholesky factor of A^T A instead of on A: tall enough that the
// q x q factor moves far fewer bytes per round than the r x q A.
bool qr_pre(int64_t m, int64_t n) {
  const int64_t q = std::min(m, n), r = std::max(m, n);
  return r >= 2 * q && r >= 1024;
}

Bufs carve(Bump& bp, int64_t m, int64_t n, int K) {
  const int64_t q = std::min(m, n), r = std::max(m, n);
  Bufs b;
  for (int i = 0; i <= K; ++i) {
    b.jr[i] = qr_pre(m, n) ? bp.take(q * q) : nullptr;
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
  b.gram = bp.take(std::max(K * K, 2));      // also the two norms of the diagnostics
  b.coef = bp.take(K);
  b.red = bp.take((int64_t)kRedSlots * kRedChunks);
  b.AU = bp.take(m * q);
  b.AV = bp.take(n * q);
  for (int h = 0; h < 2; ++h) {
    const int64_t rows = h ? n : m;
    b.PX[h][0] = bp.take(rows * q);
    b.PX[h][1] = bp.take(rows * q);
    b.PG[h] = bp.take(q * q);
  }
  b.Wst = bp.take(m * n);
  b.QT = b.QH = b.QP[0] = b.QP[1] = nullptr;
  if (qr_pre(m, n)) {
    b.QT = bp.take(q * q);
    b.QH = bp.take(q * q);
    b.QP[0] = bp.take(q * q);
    b.QP[1] = bp.take(q * q);
  }
  return b;
}

// Job tables of a batch of nm matrices: K+1 SVD jobs per matrix with their convergence states
// and 3 finalize pointer arrays; two polar jobs per matrix (U side, V side) with their states and
// four GEMM tables (X^T X and X T for either buffer holding X); the K warm-start products per
// matrix.
struct Tables {
  JacobiJob* jobs;
  JacobiState* jst;
  double** ptrs;
  NsJob* ns;
  NsState* nst;
  GemmJob* ngj[4];   // [2 p]: G = X_p^T X_p, [2 p + 1]: X_{1-p} = X_p T
  GemmJob* wgj;      // warm start of the expert SVDs: A_i V_0
  GemmJob* qgj[5];   // q-space polar: G_0 = X_0^T X_0, H = G T, G = T H, P_1 = P_0 T, P_0 = P_1 T
  CholJob* qch;      // the Cholesky factors of the tall matrices' SVDs (first nch entries)
  GemmJob* qtrail;   // their trailing updates, one panel at a time
  int* qfail;        // per SVD: its Cholesky factor failed (tall matrices)
  int* qmat;         // per SVD: its matrix's index in the batch if the Jacobi ran on R, else -1
  int* qbad;         // per matrix: its SVDs go to plain Jacobi on A
};

Tables carve_tables(Bump& bp, int nm, int K) {
  Tables tb;
  tb.jobs = bp.take<JacobiJob>((int64_t)nm * (K + 1));
  tb.jst = bp.take<JacobiState>((int64_t)nm * (K + 1));
  tb.ptrs = bp.take<double*>((int64_t)3 * nm * (K + 1));
  tb.ns = bp.take<NsJob>(2 * nm);
  tb.nst = bp.take<NsState>(2 * nm);
  for (int k = 0; k < 4; ++k) tb.ngj[k] = bp.take<GemmJob>(2 * nm);
  tb.wgj = bp.take<GemmJob>((int64_t)nm * K);
  for (int k = 0; k < 5; ++k) tb.qgj[k] = bp.take<GemmJob>(2 * nm);
  tb.qch = bp.take<CholJob>((int64_t)nm * (K + 1));
  tb.qtrail = bp.take<GemmJob>((int64_t)nm * (K + 1));
  tb.qfail = bp.take<int>((int64_t)nm * (K + 1));
  tb.qmat = bp.take<int>((int64_t)nm * (K + 1));
  tb.qbad = bp.take<int>(nm);
  return tb;
}

// Matrices of one call are merged in batches: consecutive nonempty matrices, at most
// kSpectralBatch of them and at most kSpectralBatchBytes of workspace (a matrix larger than that
// forms a batch of its own).  A batch runs its SVDs as one set of Jacobi jobs, so that a few
// mid-sized matrices fill the chip together where each alone would occupy a fraction of it.
constexpr int kSpectralBatch = 8;
constexpr size_t kSpectralBatchBytes = size_t(32) << 30;

size_t matrix_bytes(int64_t m, int64_t n, int K) {
  Bump bp{nullptr};
  carve(bp, m, n, K);
  return bp.off;
}

size_t tables_bytes(int nm, int K) {
  Bump bp{nullptr};
  carve_tables(bp, nm, K);
  return bp.off;
}

std::vector<std::vector<int>> spectral_batches(const iso_tensor* t, int n_t, int K) {
  std::vector<std::vector<int>> out;
  std::vector<int> cur;
  size_t bytes = 0;
  for (int j = 0; j < n_t; ++j) {
    if (t[j].rows == 0 || t[j].cols == 0) continue;
    const size_t mb = matrix_bytes(t[j].rows, t[j].cols, K);
    if (!cur.empty() && ((int)cur.size() == kSpectralBatch || bytes + mb > kSpectralBatchBytes)) {
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

// xi = D - U0 sym(U0^T D) in place on D (r x q col-major), using P, S (q x q) as scratch
void tangent_project(double* d, const double* u0, int64_t r, int64_t q, double* P, double* S, hipStream_t s) {
  gemm(q, q, r, 1.0, u0, r, 1, d, 1, r, 0.0, P, 1, q, s);           // P = U0^T D
  k_sym<<<grid_for(q * q), 256, 0, s>>>(S, P, q);
  gemm(r, q, q, -1.0, u0, 1, r, S, 1, q, 1.0, d, 1, r, s);          // D -= U0 S
}

// Steps 2 - 6 up to the polar inputs for one matrix whose K+1 SVDs are final: canonicalisation,
// tangent projections, D_keep, effect proxies, Gram, ridge solve and clip, aggregate projection;
// leaves U_0 + xi_U* in AU and V_0 + xi_V* in AV.
void middle_steps(const Bufs& b, int64_t m, int64_t n, int K, const SpectralArgs& a, double* coef_out,
                  uint32_t* status, hipStream_t s) {
  const int64_t q = std::min(m, n);
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
  gram_of(b.G, m * n, K, b.red, b.gram, s);
  k_solve<<<1, 64, 0, s>>>(b.gram, K, a.ridge, a.c_min, a.c_max, b.coef, coef_out, status);
  // 6. aggregate, project, shift to the base factors
  k_combine<<<grid_for(m * q), 256, 0, s>>>(b.AU, b.XU, b.coef, K, m * q);
  k_combine<<<grid_for(n * q), 256, 0, s>>>(b.AV, b.XV, b.coef, K, n * q);
  tangent_project(b.AU, b.U[0], m, q, b.P, b.Sq, s);
  tangent_project(b.AV, b.V[0], n, q, b.P, b.Sq, s);
  k_add<<<grid_for(m * q), 256, 0, s>>>(b.AU, b.AU, b.U[0], m * q);
  k_add<<<grid_for(n * q), 256, 0, s>>>(b.AV, b.AV, b.V[0], n * q);
}

// Newton-Schulz polar over the batch's 2 nm jobs (X of job p in buffer 0 on entry); the host
// reads the done flags every kNsCheckSteps steps.  On return hst holds every job's state.
hipError_t polar_batch(const Tables& tb, int njobs, int64_t max_rows, int64_t max_q, std::vector<NsState>& hst,
                       uint32_t* status, hipStream_t s, bool scaled = false) {
  const unsigned cb = (unsigned)std::max<int64_t>(1, std::min<int64_t>((max_q + 3) / 4, 1024));
  const unsigned fb = (unsigned)std::max<int64_t>(1, std::min<int64_t>((max_q * max_q + 255) / 256, 2048));
  k_ns_begin<<<1, 256, 0, s>>>(tb.ns, tb.nst, njobs, 0);
  hst.assign(njobs, NsState{});
  for (int step = 0; step < kNsMaxSteps;) {
    for (int b = 0; b < kNsCheckSteps && step < kNsMaxSteps; ++b, ++step) {
      const int p = step & 1;
      k_ns_reset<<<1, 256, 0, s>>>(tb.nst, njobs);
      gemm_jobs(tb.ngj[2 * p], njobs, max_q, max_q, s);
      k_ns_stats<<<dim3(cb, (unsigned)njobs), 256, 0, s>>>(tb.ns, tb.nst);
      k_ns_form<<<dim3(fb, (unsigned)njobs), 256, 0, s>>>(tb.ns, tb.nst, scaled ? 1 : 0);
      gemm_jobs(tb.ngj[2 * p + 1], njobs, max_rows, max_q, s);
      k_ns_step_end<<<1, 256, 0, s>>>(tb.nst, njobs);
    }
    hipError_t e = hipMemcpyAsync(hst.data(), tb.nst, sizeof(NsState) * njobs, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return e;
    bool all = true;
    for (int j = 0; j < njobs; ++j) all = all && hst[j].done;
    if (all) return hipGetLastError();
  }
  k_ns_check<<<1, 256, 0, s>>>(tb.nst, njobs, status);
  return hipGetLastError();
}

// The same Newton-Schulz iteration for the jobs with NsJob::gs set, carried in q space: with
// X_k = X_0 P_k, the Gram G_k = X_k^T X_k and the step matrix T_k (a polynomial in G_k) give
// G_{k+1} = T_k G_k T_k and P_{k+1} = P_k T_k, three q x q products per step instead of two
// rows x q ones, then X = X_0 P once.  The same steps, statistics and stopping test as the X form;
// the Gram is not re-formed from an iterate, so rounding drifts by a few units of eps cond(G_0)
// per step, negligible for the near-orthonormal retraction arguments (X^T X = I + xi^T xi) it
// serves.  On return hst holds every job's state; the result is X_0 P in the job's P buffer
// (steps & 1), formed by the caller.
hipError_t polar_gram_batch(const Tables& tb, int njobs, int64_t max_q, std::vector<NsState>& hst, uint32_t* status,
                            hipStream_t s) {
  const unsigned cb = (unsigned)std::max<int64_t>(1, std::min<int64_t>((max_q + 3) / 4, 1024));
  const unsigned fb = (unsigned)std::max<int64_t>(1, std::min<int64_t>((max_q * max_q + 255) / 256, 2048));
  k_ns_begin<<<1, 256, 0, s>>>(tb.ns, tb.nst, njobs, 1);
  k_ns_eye<<<dim3(fb, (unsigned)njobs), 256, 0, s>>>(tb.ns, tb.nst);
  gemm_jobs(tb.qgj[0], njobs, max_q, max_q, s);
  hst.assign(njobs, NsState{});
  for (int step = 0; step < kNsMaxSteps;) {
    for (int b = 0; b < kNsCheckSteps && step < kNsMaxSteps; ++b, ++step) {
      const int p = step & 1;
      k_ns_reset<<<1, 256, 0, s>>>(tb.nst, njobs);
      k_ns_stats<<<dim3(cb, (unsigned)njobs), 256, 0, s>>>(tb.ns, tb.nst);
      k_ns_form<<<dim3(fb, (unsigned)njobs), 256, 0, s>>>(tb.ns, tb.nst, 0);
      gemm_jobs(tb.qgj[1], njobs, max_q, max_q, s);
      gemm_jobs(tb.qgj[2], njobs, max_q, max_q, s);
      gemm_jobs(tb.qgj[3 + p], njobs, max_q, max_q, s);
      k_ns_step_end<<<1, 256, 0, s>>>(tb.nst, njobs);
    }
    hipError_t e = hipMemcpyAsync(hst.data(), tb.nst, sizeof(NsState) * njobs, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return e;
    bool all = true;
    for (int j = 0; j < njobs; ++j) all = all && hst[j].done;
    if (all) return hipGetLastError();
  }
  k_ns_check<<<1, 256, 0, s>>>(tb.nst, njobs, status);
  return hipGetLastError();
}

// One batch: every SVD of its matrices as one Jacobi job set, the per-matrix middle steps, both
// polar retractions of every matrix as one Newton-Schulz job set, then W_*.
iso_status run_batch(const iso_tensor* t, const std::vector<int>& ids, int K, iso_dtype dt, const SpectralArgs& a,
                     uint8_t* ws, uint32_t* status, hipStream_t s, std::vector<uint8_t>& host) {
#define SP_TRY(x)                                \
  do {                                           \
    if ((x) != hipSuccess) return ISO_ERR_HIP;   \
  } while (0)
  const int nm = (int)ids.size(), nsvd = nm * (K + 1), npol = 2 * nm;
  Bump bp{ws};
  const Tables tb = carve_tables(bp, nm, K);
  const size_t tables_end = bp.off;
  std::vector<Bufs> bs(nm);
  for (int e = 0; e < nm; ++e) bs[e] = carve(bp, t[ids[e]].rows, t[ids[e]].cols, K);
  int64_t split_r = 1, split_q = 1;
  for (int e = 0; e < nm; ++e) {
    split_r = std::max(split_r, std::max(t[ids[e]].rows, t[ids[e]].cols));
    split_q = std::max(split_q, std::min(t[ids[e]].rows, t[ids[e]].cols));
  }
  void* split = bp.take<uint8_t>((int64_t)gram_split_bytes(nsvd, split_r, split_q));
  // host image of the tables (same layout as on the device): the nm (K+1) SVDs (matrix e's W_0 at
  // e, its W_i at nm + e K + i - 1) with their finalize pointers (left, right, singular values);
  // the polar jobs (matrix e's U side at 2 e, V side at 2 e + 1) with their GEMM tables
  host.assign(tables_end, 0);
  const auto at = [&](const void* dev) { return host.data() + ((const uint8_t*)dev - ws); };
  JacobiJob* hj = (JacobiJob*)at(tb.jobs);
  double** hp = (double**)at(tb.ptrs);
  NsJob* hn = (NsJob*)at(tb.ns);
  GemmJob* hg[4];
  for (int k = 0; k < 4; ++k) hg[k] = (GemmJob*)at(tb.ngj[k]);
  GemmJob* hw = (GemmJob*)at(tb.wgj);
  GemmJob* hq[5];
  for (int k = 0; k < 5; ++k) hq[k] = (GemmJob*)at(tb.qgj[k]);
  int* hqm = (int*)at(tb.qmat);
  CholJob* hch = (CholJob*)at(tb.qch);
  int nch = 0;
  int64_t ch_q = 1;
  int64_t svd_r = 1, svd_c = 1;
  std::vector<char> pre(nm);
  for (int e = 0; e < nm; ++e) {
    const int64_t m = t[ids[e]].rows, n = t[ids[e]].cols, q = std::min(m, n), r = std::max(m, n);
    const bool wide = m < n;
    const Bufs& b = bs[e];
    pre[e] = qr_pre(m, n);
    // a tall matrix's Jacobi runs on R (q x q, R^T R = A^T A): the same V and singular values, its
    // left factor formed afterwards as A V S^{-1}
    const int64_t jr_rows = pre[e] ? q : r;
    for (int i = 0; i <= K; ++i) {
      const int j = i ? nm + e * K + i - 1 : e;
      // on R the convergence test keeps A's scale (r u): R's columns have A's inner products
      hj[j] = JacobiJob{pre[e] ? b.jr[i] : b.ja[i], b.jv[i], jr_rows, q, pre[e] ? r : 0};
      hp[j] = pre[e] ? nullptr : (wide ? b.V[i] : b.U[i]);   // left factor of the Jacobi matrix
      hp[nsvd + j] = wide ? b.U[i] : b.V[i];                  // right factor
      hp[2 * nsvd + j] = b.S[i];
      hqm[j] = pre[e] ? e : -1;
      if (pre[e]) {
        hch[nch++] = CholJob{b.jr[i], q, tb.qfail + j};
        ch_q = std::max(ch_q, q);
      }
    }
    // A_i V_0 as (A_0 V_0) + T_i V_0 (r x q), the first term the base's converged Jacobi matrix,
    // T_i (tau_i or its transpose) staged in the proxy buffer; on R: R_0 V_0 + (R_i - R_0) V_0
    for (int i = 1; i <= K; ++i)
      hw[e * K + i - 1] = GemmJob{b.G + (int64_t)(i - 1) * (pre[e] ? q * q : m * n), b.jv[0],
                                  pre[e] ? b.jr[i] : b.ja[i], 1, jr_rows, 1, q, 1, jr_rows, jr_rows, q, q, 1.0, 1.0};
    for (int h = 0; h < 2; ++h) {
      const int pj = 2 * e + h;
      const int64_t rows = h ? n : m;
      const int* skip = &tb.nst[pj].done;
      // the tall side of a tall matrix iterates in q space
      const bool gs = pre[e] && rows > q;
      hn[pj] = gs ? NsJob{b.PG[h], q, b.QT, {b.QP[0], b.QP[1]}, 1} : NsJob{b.PG[h], q};
      if (gs) {
        hq[0][pj] = GemmJob{b.PX[h][0], b.PX[h][0], b.PG[h], rows, 1, 1, rows, 1, q, q, q, rows, 1.0, 0.0, 0, skip};
        hq[1][pj] = GemmJob{b.PG[h], b.QT, b.QH, 1, q, 1, q, 1, q, q, q, q, 1.0, 0.0, 0, skip};
        hq[2][pj] = GemmJob{b.QT, b.QH, b.PG[h], 1, q, 1, q, 1, q, q, q, q, 1.0, 0.0, 0, skip};
        hq[3][pj] = GemmJob{b.QP[0], b.QT, b.QP[1], 1, q, 1, q, 1, q, q, q, q, 1.0, 0.0, 0, skip};
        hq[4][pj] = GemmJob{b.QP[1], b.QT, b.QP[0], 1, q, 1, q, 1, q, q, q, q, 1.0, 0.0, 0, skip};
      }
      for (int p = 0; p < 2; ++p) {
        const double* X = b.PX[h][p];
        double* Y = b.PX[h][1 - p];
        // G = X^T X (q x q), X (rows x q) col-major
        hg[2 * p][pj] = GemmJob{X, X, b.PG[h], rows, 1, 1, rows, 1, q, q, q, rows, 1.0, 0.0, 0, skip};
        // Y = X T (rows x q)
        hg[2 * p + 1][pj] = GemmJob{X, b.PG[h], Y, 1, rows, 1, q, 1, rows, rows, q, q, 1.0, 0.0, 0, skip};
      }
    }
    svd_r = std::max(svd_r, jr_rows);
    svd_c = std::max(svd_c, q);
  }
  SP_TRY(hipMemcpyAsync(ws, host.data(), tables_end, hipMemcpyHostToDevice, s));
  // 1. W_0 and W_i = W_0 + tau_i as A = W (tall) or W^T (wide), r x q col-major; SVDs.  When the
  //    batch's Jacobi workgroups outnumber what the chip holds at once, the base goes first and
  //    each expert's Jacobi starts from the base's right factor V_0 (A_i V_0, rotations
  //    accumulated onto V_0): W_i is a small perturbation of W_0, so A_i V_0 has nearly
  //    orthogonal columns and needs fewer sweeps.  A_i V_0 is formed as the base's converged
  //    matrix plus T_i V_0, so that tau_i = 0 gives the base's SVD exactly.  Otherwise every SVD
  //    runs at once from the identity (the rounds then cost the same with or without the experts).
  int64_t width = 0, per_cu = 0, wgs = 0;
  jacobi_block_shape(svd_r, svd_c, &width, &per_cu);
  for (int e = 0; e < nm; ++e) {
    const int64_t q = std::min(t[ids[e]].rows, t[ids[e]].cols);
    const int64_t nb = (q + width - 1) / width;
    // the Gram step splits each block pair's rows over workgroups of gram_slice_rows rows
    const int64_t sl = gram_slice_rows(svd_r);
    const int64_t rows = pre[e] ? q : std::max(t[ids[e]].rows, t[ids[e]].cols);
    const int64_t slices = width == kGW ? (rows + sl - 1) / sl : 1;
    wgs += (int64_t)(K + 1) * ((nb + 1) / 2) * slices;
  }
  int dev = 0, cus = 0;
  SP_TRY(hipGetDevice(&dev));
  SP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  const bool warm = wgs > per_cu * (int64_t)cus;
  // the Jacobi matrices in binary64, and for the tall matrices the Grams A_i^T A_i (upper
  // triangles) whose Cholesky factors R_i they run on; each matrix's own buffers, so the matrices
  // are spread over the streams
  {
    Fan fan;
    SP_TRY(fan.begin(s, nm));
    for (int e = 0; e < nm; ++e) {
      const iso_tensor& x = t[ids[e]];
      hipStream_t se = fan.at(e);
      for (int i = 0; i <= ((warm && !pre[e]) ? 0 : K); ++i)
        k_load_f64<<<grid_for(x.rows * x.cols), 256, 0, se>>>(bs[e].ja[i], x.base, i ? x.deltas[i - 1] : nullptr,
                                                              x.rows, x.cols, x.rows < x.cols ? 1 : 0, dt);
      if (!pre[e]) continue;
      const int64_t q = std::min(x.rows, x.cols), r = std::max(x.rows, x.cols);
      const Bufs& b = bs[e];
      for (int i = 0; i <= K; ++i)
        gemm_job(GemmJob{b.ja[i], b.ja[i], b.jr[i], r, 1, 1, r, 1, q, q, q, r, 1.0, 0.0, 1, nullptr}, se);
    }
    SP_TRY(fan.end());
  }
  // then, for the warm start, R_i - R_0 in the proxy buffer
  if (nch > 0) cholesky_upper_jobs(tb.qch, nch, ch_q, tb.qtrail, s);
  for (int e = 0; e < nm; ++e) {
    if (!pre[e] || !warm) continue;
    const int64_t q = std::min(t[ids[e]].rows, t[ids[e]].cols);
    const Bufs& b = bs[e];
    for (int i = 1; i <= K; ++i)
      k_sub<<<grid_for(q * q), 256, 0, s>>>(b.G + (int64_t)(i - 1) * q * q, b.jr[i], b.jr[0], q * q);
  }
  if (!warm) {
    SP_TRY(jacobi_block(tb.jobs, nsvd, svd_r, svd_c, tb.jst, status, s, false, split));
  } else {
    SP_TRY(jacobi_block(tb.jobs, nm, svd_r, svd_c, tb.jst, status, s, false, split));
    for (int e = 0; e < nm; ++e) {
      const iso_tensor& x = t[ids[e]];
      const int64_t q = std::min(x.rows, x.cols);
      for (int i = 1; i <= K; ++i) {
        if (pre[e]) {
          k_copy<<<grid_for(q * q), 256, 0, s>>>(bs[e].jr[i], bs[e].jr[0], q * q);
        } else {
          k_load_f64<<<grid_for(x.rows * x.cols), 256, 0, s>>>(bs[e].G + (int64_t)(i - 1) * x.rows * x.cols,
                                                               x.deltas[i - 1], nullptr, x.rows, x.cols,
                                                               x.rows < x.cols ? 1 : 0, dt);
          k_copy<<<grid_for(x.rows * x.cols), 256, 0, s>>>(bs[e].ja[i], bs[e].ja[0], x.rows * x.cols);
        }
        k_copy<<<grid_for(q * q), 256, 0, s>>>(bs[e].jv[i], bs[e].jv[0], q * q);
      }
    }
    gemm_jobs(tb.wgj, nm * K, svd_r, svd_c, s);
    SP_TRY(jacobi_block(tb.jobs + nm, nm * K, svd_r, svd_c, tb.jst + nm, status, s, true, split));
  }
  svd_finalize(tb.jobs, tb.ptrs, tb.ptrs + nsvd, tb.ptrs + 2 * nsvd, nsvd, svd_c, s);
  // tall matrices: left factor A_i V_i S_i^{-1}; a matrix whose factors fail the guard goes to
  // plain Jacobi on A (its A_i are still in the Jacobi buffers)
  bool any_pre = false;
  {
    Fan fan;
    SP_TRY(fan.begin(s, nm));
    for (int e = 0; e < nm; ++e) {
      if (!pre[e]) continue;
      any_pre = true;
      const int64_t m = t[ids[e]].rows, n = t[ids[e]].cols, q = std::min(m, n), r = std::max(m, n);
      const bool wide = m < n;
      const Bufs& b = bs[e];
      hipStream_t se = fan.at(e);
      for (int i = 0; i <= K; ++i) {
        double* L = wide ? b.V[i] : b.U[i];
        const double* Vs = wide ? b.U[i] : b.V[i];
        gemm(r, q, q, 1.0, b.ja[i], 1, r, Vs, 1, q, 0.0, L, 1, r, se);
        k_unit_cols<<<grid_for(r * q), 256, 0, se>>>(L, b.S[i], r, q);
      }
    }
    SP_TRY(fan.end());
  }
  if (any_pre) {
    k_qr_guard<<<1, 256, 0, s>>>(tb.jobs, tb.ptrs + 2 * nsvd, tb.qfail, tb.qmat, nsvd, tb.qbad);
    std::vector<int> bad(nm, 0);
    SP_TRY(hipMemcpyAsync(bad.data(), tb.qbad, sizeof(int) * nm, hipMemcpyDeviceToHost, s));
    SP_TRY(hipStreamSynchronize(s));
    std::vector<int> redo;
    for (int e = 0; e < nm; ++e)
      if (bad[e]) redo.push_back(e);
    if (!redo.empty()) {
      // the Jacobi job table and pointers are free again (the stream has drained; the host image
      // still holds the polar and warm-start tables, which go up unchanged): the redone matrices'
      // SVDs as one plain job set on A from the identity
      const int nr = (int)redo.size() * (K + 1);
      int64_t rr = 1, rq = 1;
      for (int x = 0; x < (int)redo.size(); ++x) {
        const int e = redo[x];
        const int64_t m = t[ids[e]].rows, n = t[ids[e]].cols, q = std::min(m, n), r = std::max(m, n);
        const bool wide = m < n;
        const Bufs& b = bs[e];
        for (int i = 0; i <= K; ++i) {
          const int j = x * (K + 1) + i;
          hj[j] = JacobiJob{b.ja[i], b.jv[i], r, q};
          hp[j] = wide ? b.V[i] : b.U[i];
          hp[nr + j] = wide ? b.U[i] : b.V[i];
          hp[2 * nr + j] = b.S[i];
        }
        rr = std::max(rr, r);
        rq = std::max(rq, q);
      }
      SP_TRY(hipMemcpyAsync(ws, host.data(), tables_end, hipMemcpyHostToDevice, s));
      SP_TRY(jacobi_block(tb.jobs, nr, rr, rq, tb.jst, status, s, false, split));
      svd_finalize(tb.jobs, tb.ptrs, tb.ptrs + nr, tb.ptrs + 2 * nr, nr, rq, s);
    }
  }
  // 2 - 6 per matrix (each matrix's own buffers, so the matrices run on several streams); the
  // polar arguments go to the first iterate buffers
  {
    Fan fan;
    SP_TRY(fan.begin(s, nm));
    for (int e = 0; e < nm; ++e) {
      const int64_t m = t[ids[e]].rows, n = t[ids[e]].cols, q = std::min(m, n);
      const Bufs& b = bs[e];
      hipStream_t se = fan.at(e);
      middle_steps(b, m, n, K, a, a.coef_out ? a.coef_out + (int64_t)ids[e] * K : nullptr, status, se);
      k_copy<<<grid_for(m * q), 256, 0, se>>>(b.PX[0][0], b.AU, m * q);
      k_copy<<<grid_for(n * q), 256, 0, se>>>(b.PX[1][0], b.AV, n * q);
    }
    SP_TRY(fan.end());
  }
  // 6'. U_* = polar(U_0 + xi_U*), V_* = polar(V_0 + xi_V*)
  //     the tall side of a tall matrix in q space (then X_0 P into the second iterate buffer),
  //     the others in X form
  std::vector<NsState> hst, hsq;
  bool any_gs = false;
  for (int e = 0; e < nm; ++e) any_gs = any_gs || pre[e];
  // (the frames have max(rows, cols) rows: split_r, not the Jacobi matrices' svd_r)
  SP_TRY(polar_batch(tb, npol, split_r, svd_c, hst, status, s));
  if (any_gs) {
    SP_TRY(polar_gram_batch(tb, npol, svd_c, hsq, status, s));
    for (int e = 0; e < nm; ++e) {
      if (!pre[e]) continue;
      const int64_t m = t[ids[e]].rows, n = t[ids[e]].cols, q = std::min(m, n);
      const int h = m > n ? 0 : 1;
      const int64_t rows = h ? n : m;
      const Bufs& b = bs[e];
      gemm(rows, q, q, 1.0, b.PX[h][0], 1, rows, b.QP[hsq[2 * e + h].steps & 1], 1, q, 0.0, b.PX[h][1], 1, rows, s);
    }
  }
  {
    Fan fan;
    SP_TRY(fan.begin(s, nm));
    for (int e = 0; e < nm; ++e) {
      const iso_tensor& x = t[ids[e]];
      const int64_t m = x.rows, n = x.cols, q = std::min(m, n);
      const Bufs& b = bs[e];
      const bool gu = pre[e] && m > n, gv = pre[e] && n > m;
      const double* Us = b.PX[0][gu ? 1 : (hst[2 * e].steps & 1)];
      const double* Vs = b.PX[1][gv ? 1 : (hst[2 * e + 1].steps & 1)];
      hipStream_t se = fan.at(e);
      // 7. W_* = U_* Sigma_0 V_*^T
      k_scale_cols<<<grid_for(m * q), 256, 0, se>>>(b.FU, Us, b.S[0], m, q);
      gemm(m, n, q, 1.0, b.FU, 1, m, Vs, n, 1, 0.0, b.Wst, 1, m, se);
      k_store_w<<<grid_for(m * n), 256, 0, se>>>(x.out, b.Wst, m, n, dt, status);
    }
    SP_TRY(fan.end());
  }
  SP_TRY(hipGetLastError());
  // the next batch reuses the workspace and the host staging: let this one finish first
  SP_TRY(hipStreamSynchronize(s));
  return ISO_OK;
#undef SP_TRY
}

// ---- ISO-Optimizer step (ISO-AdamW) ------------------------------------------------------------

// AdamW on n entries of x with gradient g and moments m, v (decoupled weight decay), in the
// order written in the interface: m, v, then x - lr ((m / bc1) / (sqrt(v / bc2) + eps) + wd x).
__global__ void k_adamw(double* __restrict__ x, const double* __restrict__ g, double* __restrict__ m,
                        double* __restrict__ v, int64_t n, double lr, double b1, double b2, double eps, double wd,
                        double bc1, double bc2) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const double gi = g[e];
    const double mi = b1 * m[e] + (1.0 - b1) * gi;
    const double vi = b2 * v[e] + (1.0 - b2) * (gi * gi);
    m[e] = mi;
    v[e] = vi;
    const double xi = x[e];
    x[e] = xi - lr * ((mi / bc1) / (sqrt(vi / bc2) + eps) + wd * xi);
  }
}

// Muon's momentum on n entries: b <- mu b + g, then the direction d = g + mu b (Nesterov) or b.
__global__ void k_muon_momentum(double* __restrict__ d, const double* __restrict__ g, double* __restrict__ b,
                                int64_t n, double mu, int nesterov) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const double gi = g[e];
    const double bi = mu * b[e] + gi;
    b[e] = bi;
    d[e] = nesterov ? gi + mu * bi : bi;
  }
}

// Muon's step on n entries of x along the orthogonalised direction o: x - lr (scale o + wd x).
__global__ void k_muon_apply(double* __restrict__ x, const double* __restrict__ o, int64_t n, double lr, double scale,
                             double wd) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const double xi = x[e];
    x[e] = xi - lr * (scale * o[e] + wd * xi);
  }
}

struct OptBufs {
  double *G, *FU, *FV, *GU, *GV, *Wst;
  double *PX[2][2], *PG[2];
};

OptBufs carve_opt(Bump& bp, int64_t m, int64_t n, int64_t q) {
  OptBufs b;
  b.G = bp.take(m * n);
  b.FU = bp.take(m * q);
  b.FV = bp.take(n * q);
  b.GU = bp.take(m * q);
  b.GV = bp.take(n * q);
  b.Wst = bp.take(m * n);
  for (int h = 0; h < 2; ++h) {
    const int64_t rows = h ? n : m;
    b.PX[h][0] = bp.take(rows * q);
    b.PX[h][1] = bp.take(rows * q);
    b.PG[h] = bp.take(q * q);
  }
  return b;
}

Tables carve_opt_tables(Bump& bp, int n_f) {
  Tables tb{};
  tb.ns = bp.take<NsJob>(2 * n_f);
  tb.nst = bp.take<NsState>(2 * n_f);
  for (int k = 0; k < 4; ++k) tb.ngj[k] = bp.take<GemmJob>(2 * n_f);
  return tb;
}

// ---- spectral diagnostics and spectrum interpolation ----------------------------------------------

// x[k] = <u0_k, p_k>^2 for the q columns (m rows, col-major): one wave per column.
__global__ void __launch_bounds__(1024) k_col_dot_sq(const double* __restrict__ u0, const double* __restrict__ p,
                                                     int64_t m, int64_t q, double* __restrict__ x) {
  const int lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  for (int64_t k = (int64_t)blockIdx.x * nw + (threadIdx.x >> 6); k < q; k += (int64_t)gridDim.x * nw) {
    double v = 0.0;
    for (int64_t i = lane; i < m; i += 64) v += u0[k * m + i] * p[k * m + i];
    v = wave_sum_f64(v);
    if (lane == 0) x[k] = v * v;
  }
}

// One workgroup: {delta_Sigma, rho_Sigma, kappa_spec} from the sorted spectra s0, s1 (q), the squared
// diagonal entries dg2 (q) of U_0^T Delta W V_0 and sums = {|W_0|_F^2, |Delta W|_F^2}.
__global__ void __launch_bounds__(1024) k_diag_final(const double* __restrict__ s0, const double* __restrict__ s1,
                                                     int64_t q, const double* __restrict__ dg2,
                                                     const double* __restrict__ sums, int64_t m, int64_t n,
                                                     double* __restrict__ out) {
  __shared__ double red[2][16];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  double d2 = 0.0, dg = 0.0;
  for (int64_t k = threadIdx.x; k < q; k += blockDim.x) {
    d2 += (s1[k] - s0[k]) * (s1[k] - s0[k]);
    dg += dg2[k];
  }
  d2 = wave_sum_f64(d2);
  dg = wave_sum_f64(dg);
  if (lane == 0) {
    red[0][wid] = d2;
    red[1][wid] = dg;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double a[2] = {0.0, 0.0};
    for (int c = 0; c < 2; ++c)
      for (int w = 0; w < nw; ++w) a[c] += red[c][w];
    const double dist = sqrt(a[0]);
    out[0] = dist / sqrt(sums[0]);
    out[1] = dist / sqrt(sums[1]);
    out[2] = ((double)m * (double)n / (double)q) * a[1] / sums[1];
  }
}

// Mean squared spectral error (App. G): out[0] = (1/q) sum_k (s1_k - s0_k)^2 over the sorted spectra
// (one workgroup, fixed summation order).
__global__ void __launch_bounds__(1024) k_spectral_error(const double* __restrict__ s0, const double* __restrict__ s1,
                                                         int64_t q, double* __restrict__ out) {
  __shared__ double red[16];
  double x = 0.0;
  for (int64_t k = threadIdx.x; k < q; k += blockDim.x) x += (s1[k] - s0[k]) * (s1[k] - s0[k]);
  x = wave_sum_f64(x);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) t += red[w];
    out[0] = t / (double)q;
  }
}

// Unexplained-update ratios from the squared residuals held in out[0..3] (|W_i^(r) - W_j^(r)|^2,
// then those of the mix, L and R reconstructions) and the two spectra s0 (incoming W_j) and s1
// (endpoint W_i): out = {u_mix, u_L, u_R, u_iso, gap}.  u_iso takes the closed form of Prop. 3.1,
// |sigma_i^(r) - sigma_j^(r)| / |W_i^(r) - W_j^(r)|.  One thread.
__global__ void k_transport_final(const double* __restrict__ s0, const double* __restrict__ s1, int64_t q, int64_t r,
                                  double* __restrict__ out) {
  if (threadIdx.x != 0) return;
  double ds = 0.0;
  for (int64_t k = 0; k < r; ++k) ds += (s1[k] - s0[k]) * (s1[k] - s0[k]);
  const double den = sqrt(out[0]);
  const double nan = __builtin_nan("");
  const double e[4] = {sqrt(out[1]), sqrt(out[2]), sqrt(out[3]), sqrt(ds)};
  for (int h = 0; h < 4; ++h) out[h] = den > 0.0 ? e[h] / den : nan;
  const double g0 = s0[r - 1] - (r < q ? s0[r] : 0.0), g1 = s1[r - 1] - (r < q ? s1[r] : 0.0);
  out[4] = fmin(g0, g1);
}

// s = (1 - alpha) s0 + alpha s1
__global__ void k_mix(double* __restrict__ s, const double* __restrict__ s0, const double* __restrict__ s1, int64_t q,
                      double alpha) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < q; k += (int64_t)gridDim.x * blockDim.x)
    s[k] = (1.0 - alpha) * s0[k] + alpha * s1[k];
}

}  // namespace

size_t spectral_workspace_bytes(const iso_tensor* t, int n_t, int K) {
  size_t most = 0;
  for (const auto& ids : spectral_batches(t, n_t, K)) {
    size_t b = tables_bytes((int)ids.size(), K);
    int64_t r = 1, q = 1;
    for (int j : ids) {
      b += matrix_bytes(t[j].rows, t[j].cols, K);
      r = std::max(r, std::max(t[j].rows, t[j].cols));
      q = std::max(q, std::min(t[j].rows, t[j].cols));
    }
    b += align_up(gram_split_bytes((int)ids.size() * (K + 1), r, q), 256);
    most = std::max(most, b);
  }
  return most;
}

iso_status run_spectral(const iso_tensor* t, int n_t, int K, iso_dtype dt, const SpectralArgs& a, uint8_t* ws,
                        uint32_t* status, hipStream_t s) {
  std::vector<uint8_t> host;    // host staging for the job tables; kept until the stream has consumed them
  for (const auto& ids : spectral_batches(t, n_t, K)) {
    const iso_status r = run_batch(t, ids, K, dt, a, ws, status, s, host);
    if (r != ISO_OK) return r;
  }
  return ISO_OK;
}

// polar_batch over the frames' 2 n_f jobs (frame e's U side at 2 e, V side at 2 e + 1) inside a
// profiling region, counting the binary64 flops its steps performed: per job of m x q and step
// taken, 2 m q^2 for the Gram (formed whole) and 2 m q^2 for the product.
hipError_t timed_polar(const Tables& tb, const iso_frame* f, int n_f, int64_t max_rows, int64_t max_q,
                       std::vector<NsState>& hst, uint32_t* status, hipStream_t s, bool scaled) {
  hipEvent_t ev[2];
  profile_region(ev);
  hipError_t e = hipSuccess;
  if (ev[0] != nullptr && (e = hipEventRecord(ev[0], s)) != hipSuccess) return e;
  if ((e = polar_batch(tb, 2 * n_f, max_rows, max_q, hst, status, s, scaled)) != hipSuccess) return e;
  if (ev[1] != nullptr && (e = hipEventRecord(ev[1], s)) != hipSuccess) return e;
  if (ev[0] != nullptr) {
    double flops = 0.0;
    for (int j = 0; j < 2 * n_f; ++j) {
      const double m = (double)((j & 1) ? f[j / 2].cols : f[j / 2].rows), q = (double)f[j / 2].rank;
      flops += (double)hst[j].steps * (4.0 * m * q * q);
    }
    profile_add_flops(flops);
  }
  return hipSuccess;
}

size_t optimizer_workspace_bytes(const iso_frame* f, int n_f) {
  Bump bp{nullptr};
  carve_opt_tables(bp, n_f);
  for (int e = 0; e < n_f; ++e) carve_opt(bp, f[e].rows, f[e].cols, f[e].rank);
  return bp.off;
}

// All frames of the call at once: gradients, AdamW, both polar factors of every frame as one
// Newton-Schulz job set, then W+ = U+ Sigma_0 V+^T and the frames written back.
iso_status run_optimizer(const iso_frame* f, int n_f, iso_dtype dt, const iso_adamw* adam, const iso_muon* muon,
                         uint8_t* ws, uint32_t* status, hipStream_t s) {
#define OP_TRY(x)                                \
  do {                                           \
    if ((x) != hipSuccess) return ISO_ERR_HIP;   \
  } while (0)
  Bump bp{ws};
  const Tables tb = carve_opt_tables(bp, n_f);
  const size_t tables_end = bp.off;
  std::vector<OptBufs> bs(n_f);
  for (int e = 0; e < n_f; ++e) bs[e] = carve_opt(bp, f[e].rows, f[e].cols, f[e].rank);
  std::vector<uint8_t> host(tables_end, 0);
  const auto at = [&](const void* dev) { return host.data() + ((const uint8_t*)dev - ws); };
  NsJob* hn = (NsJob*)at(tb.ns);
  GemmJob* hg[4];
  for (int k = 0; k < 4; ++k) hg[k] = (GemmJob*)at(tb.ngj[k]);
  int64_t max_rows = 1, max_q = 1;
  for (int e = 0; e < n_f; ++e) {
    const int64_t m = f[e].rows, n = f[e].cols, q = f[e].rank;
    const OptBufs& b = bs[e];
    for (int h = 0; h < 2; ++h) {
      const int pj = 2 * e + h;
      const int64_t rows = h ? n : m;
      const int* skip = &tb.nst[pj].done;
      hn[pj] = NsJob{b.PG[h], q};
      for (int p = 0; p < 2; ++p) {
        const double* X = b.PX[h][p];
        double* Y = b.PX[h][1 - p];
        hg[2 * p][pj] = GemmJob{X, X, b.PG[h], rows, 1, 1, rows, 1, q, q, q, rows, 1.0, 0.0, 0, skip};
        hg[2 * p + 1][pj] = GemmJob{X, b.PG[h], Y, 1, rows, 1, q, 1, rows, rows, q, q, 1.0, 0.0, 0, skip};
      }
    }
    max_rows = std::max(max_rows, std::max(m, n));
    max_q = std::max(max_q, q);
  }
  OP_TRY(hipMemcpyAsync(ws, host.data(), tables_end, hipMemcpyHostToDevice, s));
  const double bc1 = adam ? 1.0 - std::pow(adam->beta1, (double)adam->step) : 1.0;
  const double bc2 = adam ? 1.0 - std::pow(adam->beta2, (double)adam->step) : 1.0;
  for (int e = 0; e < n_f; ++e) {
    const iso_frame& F = f[e];
    const int64_t m = F.rows, n = F.cols, q = F.rank;
    const OptBufs& b = bs[e];
    // G_U = G_W V Sigma_0 (m x q), G_V = G_W^T U Sigma_0 (n x q); G col-major m x n
    k_load_f64<<<grid_for(m * n), 256, 0, s>>>(b.G, F.grad, nullptr, m, n, 0, dt);
    k_scale_cols<<<grid_for(n * q), 256, 0, s>>>(b.FV, F.v, F.sigma, n, q);
    k_scale_cols<<<grid_for(m * q), 256, 0, s>>>(b.FU, F.u, F.sigma, m, q);
    gemm(m, q, n, 1.0, b.G, 1, m, b.FV, 1, n, 0.0, b.GU, 1, m, s);
    gemm(n, q, m, 1.0, b.G, m, 1, b.FU, 1, m, 0.0, b.GV, 1, n, s);
    if (adam) {
      // AdamW on the frames (in place), then the tentative frames go to the iterate buffers
      k_adamw<<<grid_for(m * q), 256, 0, s>>>(F.u, b.GU, F.m_u, F.v_u, m * q, adam->lr, adam->beta1, adam->beta2,
                                             adam->eps, adam->weight_decay, bc1, bc2);
      k_adamw<<<grid_for(n * q), 256, 0, s>>>(F.v, b.GV, F.m_v, F.v_v, n * q, adam->lr, adam->beta1, adam->beta2,
                                             adam->eps, adam->weight_decay, bc1, bc2);
      k_copy<<<grid_for(m * q), 256, 0, s>>>(b.PX[0][0], F.u, m * q);
      k_copy<<<grid_for(n * q), 256, 0, s>>>(b.PX[1][0], F.v, n * q);
    } else {
      // Muon: momentum and direction; the directions are orthogonalised below
      k_muon_momentum<<<grid_for(m * q), 256, 0, s>>>(b.PX[0][0], b.GU, F.m_u, m * q, muon->momentum, muon->nesterov);
      k_muon_momentum<<<grid_for(n * q), 256, 0, s>>>(b.PX[1][0], b.GV, F.m_v, n * q, muon->momentum, muon->nesterov);
    }
  }
  std::vector<NsState> hst;
  if (muon) {
    // o = polar(d) for every frame's two directions (far from orthonormal: the scaled iteration),
    // then the step and the tentative frames
    OP_TRY(timed_polar(tb, f, n_f, max_rows, max_q, hst, status, s, true));
    for (int e = 0; e < n_f; ++e) {
      const iso_frame& F = f[e];
      const int64_t m = F.rows, n = F.cols, q = F.rank;
      const OptBufs& b = bs[e];
      const double su = std::sqrt(std::max(1.0, (double)m / (double)q));
      const double sv = std::sqrt(std::max(1.0, (double)n / (double)q));
      k_muon_apply<<<grid_for(m * q), 256, 0, s>>>(F.u, b.PX[0][hst[2 * e].steps & 1], m * q, muon->lr, su,
                                                   muon->weight_decay);
      k_muon_apply<<<grid_for(n * q), 256, 0, s>>>(F.v, b.PX[1][hst[2 * e + 1].steps & 1], n * q, muon->lr, sv,
                                                   muon->weight_decay);
      k_copy<<<grid_for(m * q), 256, 0, s>>>(b.PX[0][0], F.u, m * q);
      k_copy<<<grid_for(n * q), 256, 0, s>>>(b.PX[1][0], F.v, n * q);
    }
  }
  // U+ = polar(U), V+ = polar(V)
  OP_TRY(timed_polar(tb, f, n_f, max_rows, max_q, hst, status, s, false));
  for (int e = 0; e < n_f; ++e) {
    const iso_frame& F = f[e];
    const int64_t m = F.rows, n = F.cols, q = F.rank;
    const OptBufs& b = bs[e];
    const double* Us = b.PX[0][hst[2 * e].steps & 1];
    const double* Vs = b.PX[1][hst[2 * e + 1].steps & 1];
    k_copy<<<grid_for(m * q), 256, 0, s>>>(F.u, Us, m * q);
    k_copy<<<grid_for(n * q), 256, 0, s>>>(F.v, Vs, n * q);
    k_scale_cols<<<grid_for(m * q), 256, 0, s>>>(b.FU, Us, F.sigma, m, q);
    gemm(m, n, q, 1.0, b.FU, 1, m, Vs, n, 1, 0.0, b.Wst, 1, m, s);
    k_store_w<<<grid_for(m * n), 256, 0, s>>>(F.w_out, b.Wst, m, n, dt, status);
  }
  OP_TRY(hipGetLastError());
  OP_TRY(hipStreamSynchronize(s));   // the host staging of the tables ends with this call
  return ISO_OK;
#undef OP_TRY
}

iso_status run_spectrum_ops(const iso_tensor* t, int n_t, iso_dtype dt, SpectrumOp op, double* out, double param,
                            const double* fracs, int n_frac, uint8_t* ws, uint32_t* status, hipStream_t s) {
#define SO_TRY(x)                                \
  do {                                           \
    if ((x) != hipSuccess) return ISO_ERR_HIP;   \
  } while (0)
  std::vector<uint8_t> host;
  for (int j = 0; j < n_t; ++j) {
    const int64_t m = t[j].rows, n = t[j].cols;
    if (m == 0 || n == 0) continue;
    const int64_t q = std::min(m, n), r = std::max(m, n);
    const bool wide = m < n;
    Bump bp{ws};
    const Tables tb = carve_tables(bp, 1, 1);
    const size_t tables_end = bp.off;
    const Bufs b = carve(bp, m, n, 1);
    void* split = bp.take<uint8_t>((int64_t)gram_split_bytes(2, r, q));
    host.assign(tables_end, 0);
    const auto at = [&](const void* dev) { return host.data() + ((const uint8_t*)dev - ws); };
    JacobiJob* hj = (JacobiJob*)at(tb.jobs);
    double** hp = (double**)at(tb.ptrs);
    for (int i = 0; i < 2; ++i) {
      hj[i] = JacobiJob{b.ja[i], b.jv[i], r, q};
      hp[i] = wide ? b.V[i] : b.U[i];
      hp[2 + i] = wide ? b.U[i] : b.V[i];
      hp[4 + i] = b.S[i];
    }
    SO_TRY(hipMemcpyAsync(ws, host.data(), tables_end, hipMemcpyHostToDevice, s));
    if (op == SpectrumOp::kSelfSpectralError) {
      // App. G: W_0 = L S R^T by the Jacobi SVD of the Jacobi matrix A (W_0 or W_0^T), then
      // A_rec = (L S) R^T in binary64 into the second job's matrix and its own SVD
      k_load_f64<<<grid_for(m * n), 256, 0, s>>>(b.ja[0], t[j].base, nullptr, m, n, wide ? 1 : 0, dt);
      SO_TRY(jacobi_block(tb.jobs, 1, r, q, tb.jst, status, s, false, split));
      svd_finalize(tb.jobs, tb.ptrs, tb.ptrs + 2, tb.ptrs + 4, 1, q, s);
      const double* lf = wide ? b.V[0] : b.U[0];     // r x q left factor of A
      const double* rf = wide ? b.U[0] : b.V[0];     // q x q right factor
      k_scale_cols<<<grid_for(r * q), 256, 0, s>>>(b.G, lf, b.S[0], r, q);
      gemm(r, q, q, 1.0, b.G, 1, r, rf, q, 1, 0.0, b.ja[1], 1, r, s);
      SO_TRY(jacobi_block(tb.jobs + 1, 1, r, q, tb.jst + 1, status, s, false, split));
      svd_finalize(tb.jobs + 1, tb.ptrs + 1, tb.ptrs + 3, tb.ptrs + 5, 1, q, s);
      k_spectral_error<<<1, 1024, 0, s>>>(b.S[0], b.S[1], q, out + j);
      SO_TRY(hipGetLastError());
      SO_TRY(hipStreamSynchronize(s));
      continue;
    }
    for (int i = 0; i < 2; ++i) {
      // the spectral error compares two whole matrices; the other ops take W_0 and W_0 + Delta W
      const bool whole = op == SpectrumOp::kSpectralError && i == 1;
      k_load_f64<<<grid_for(m * n), 256, 0, s>>>(b.ja[i], whole ? t[j].deltas[0] : t[j].base,
                                                  (i && !whole) ? t[j].deltas[0] : nullptr, m, n, wide ? 1 : 0, dt);
    }
    SO_TRY(jacobi_block(tb.jobs, 2, r, q, tb.jst, status, s, false, split));
    svd_finalize(tb.jobs, tb.ptrs, tb.ptrs + 2, tb.ptrs + 4, 2, q, s);
    if (op == SpectrumOp::kSpectralError) {
      k_spectral_error<<<1, 1024, 0, s>>>(b.S[0], b.S[1], q, out + j);
    } else if (op == SpectrumOp::kDiagnostics) {
      // Delta W and W_0 col-major, P = Delta W V_0
      k_load_f64<<<grid_for(m * n), 256, 0, s>>>(b.G, t[j].deltas[0], nullptr, m, n, 0, dt);
      k_load_f64<<<grid_for(m * n), 256, 0, s>>>(b.Wst, t[j].base, nullptr, m, n, 0, dt);
      gemm(m, q, n, 1.0, b.G, 1, m, b.V[0], 1, n, 0.0, b.FU, 1, m, s);
      k_col_dot_sq<<<(unsigned)std::min<int64_t>((q + 15) / 16, 4096), 1024, 0, s>>>(b.U[0], b.FU, m, q, b.P);
      dot1(b.Wst, b.Wst, m * n, false, b.red, b.gram, s);
      dot1(b.G, b.G, m * n, false, b.red, b.gram + 1, s);
      k_diag_final<<<1, 1024, 0, s>>>(b.S[0], b.S[1], q, b.P, b.gram, m, n, out + 3 * (int64_t)j);
    } else if (op == SpectrumOp::kInterpolate) {
      k_mix<<<grid_for(q), 256, 0, s>>>(b.P, b.S[0], b.S[1], q, param);
      k_scale_cols<<<grid_for(m * q), 256, 0, s>>>(b.FU, b.U[1], b.P, m, q);
      gemm(m, n, q, 1.0, b.FU, 1, m, b.V[1], n, 1, 0.0, b.Wst, 1, m, s);
      k_store_w<<<grid_for(m * n), 256, 0, s>>>(t[j].out, b.Wst, m, n, dt, status);
    } else {
      // Prop. 3.1 with W_j = base (factors 0) and W_i = base + delta (factors 1), all col-major, at
      // each rank.  The Jacobi matrices are free after the finalize: ja[0] = W_i^(r), ja[1] = W_j^(r).
      for (int fi = 0; fi < n_frac; ++fi) {
        const int64_t rk = transport_rank(q, fracs[fi]);
        double* o = out + 5 * ((int64_t)j * n_frac + fi);
        double* wi = b.ja[0];
        double* wj = b.ja[1];
        k_scale_cols<<<grid_for(m * rk), 256, 0, s>>>(b.FU, b.U[1], b.S[1], m, rk);
        gemm(m, n, rk, 1.0, b.FU, 1, m, b.V[1], n, 1, 0.0, wi, 1, m, s);
        k_scale_cols<<<grid_for(m * rk), 256, 0, s>>>(b.FU, b.U[0], b.S[0], m, rk);
        gemm(m, n, rk, 1.0, b.FU, 1, m, b.V[0], n, 1, 0.0, wj, 1, m, s);
        dot1(wi, wj, m * n, true, b.red, o, s);
        // T1 = U_j^T W_i^(r) (rk x n), W_L = U_j T1
        gemm(rk, n, m, 1.0, b.U[0], m, 1, wi, 1, m, 0.0, b.FV, 1, rk, s);
        gemm(m, n, rk, 1.0, b.U[0], 1, m, b.FV, 1, rk, 0.0, b.G, 1, m, s);
        dot1(wi, b.G, m * n, true, b.red, o + 2, s);
        // T2 = W_i^(r) V_j (m x rk), W_R = T2 V_j^T
        gemm(m, rk, n, 1.0, wi, 1, m, b.V[0], 1, n, 0.0, b.XU, 1, m, s);
        gemm(m, n, rk, 1.0, b.XU, 1, m, b.V[0], n, 1, 0.0, b.G, 1, m, s);
        dot1(wi, b.G, m * n, true, b.red, o + 3, s);
        // core B = T1 V_j (rk x rk), W_mix = (U_j B) V_j^T
        gemm(rk, rk, n, 1.0, b.FV, 1, rk, b.V[0], 1, n, 0.0, b.P, 1, rk, s);
        gemm(m, rk, rk, 1.0, b.U[0], 1, m, b.P, 1, rk, 0.0, b.AU, 1, m, s);
        gemm(m, n, rk, 1.0, b.AU, 1, m, b.V[0], n, 1, 0.0, b.G, 1, m, s);
        dot1(wi, b.G, m * n, true, b.red, o + 1, s);
        k_transport_final<<<1, 64, 0, s>>>(b.S[0], b.S[1], q, rk, o);
      }
    }
    SO_TRY(hipGetLastError());
    SO_TRY(hipStreamSynchronize(s));   // the next tensor reuses the workspace and the staging
  }
  return ISO_OK;
#undef SO_TRY
}

}  // namespace iso
