// TSV-Merge (App. F) for bf16 weight matrices, batched over every (matrix, delta) pair of
// a chunk of the tensor table:
//   1. truncated SVD of each delta: randomised range finder with subspace iteration
//      (Halko, Martinsson & Tropp, SIAM Review 2011, Alg. 4.4), sketch width L = r + p,
//      two power iterations, Cholesky-QR2 re-orthonormalisation (Fukaya et al. 2014) in
//      binary64; the products with the delta are MFMA bf16 (v_mfma_f32_16x16x32_bf16) with
//      the right operand split into two bf16 terms, binary32 accumulation; the final
//      L x L core is decomposed by one-sided Jacobi in binary64;
//   2. concatenation U = [U_1|...|U_K], V likewise, Sigma = blockdiag(Sigma_i);
//   3. Procrustes orthogonalisation U_perp = P_U Q_U^T = U (U^T U)^{-1/2}, the inverse square
//      root of the K r x K r Gram matrix by the coupled Newton-Schulz iteration (binary64);
//      it needs U and V of full column rank (generic experts), else the status reports it;
//   4. out = round(W_0 + alpha * U_perp Sigma V_perp^T): MFMA bf16 with both operands split
//      into two bf16 terms (three products), binary32 accumulation, the update fused into the
//      epilogue.
// The randomised sketch draws its test matrix from a counter-based hash (SplitMix64); the
// result does not depend on it to the accuracy of the truncation where the spectrum has a gap.
#include <algorithm>
#include <cstring>
#include <utility>
#include <vector>

#include "iso_dense.h"
#include "iso_device.h"
#include "iso_tsv.h"

namespace iso {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kPowerIters = 2;
// Ping-pong buffer of the last X-side factor: one Cholesky-QR pass per X-side sketch
constexpr int kXLast = (1 + kPowerIters) & 1;
constexpr size_t kTsvChunkBudget = 32ull << 30;  // workspace per chunk of matrices (all 84 MLP matrices of a 7B stack)
constexpr int kMaxNB = 8;                         // sketch width up to 128

int64_t rup(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// One (matrix, delta) problem.
struct Prob {
  const uint16_t* delta;   // R x C row-major bf16
  int64_t R, C, L, ldb;    // ldb: padded length of the split operand columns
  double* X[2];            // R x L row-major (ping-pong)
  double* Z[2];            // C x L row-major (ping-pong)
  uint16_t* bh;            // bf16 split of the current right operand: L columns of ldb
  uint16_t* bl;
  double* Gp;              // kSlabs x L x L Gram partials
  double* G;               // L x L
  double* Rf;              // L x L row-major upper factor of the last Cholesky
  double* Ri;              // L x L row-major inverse
  double* Ra;              // L x L first factor of the final QR
  double* R2;              // L x L product of the final QR factors
  double* Ja;              // L x L Jacobi matrix
  double* Jv;              // L x L Jacobi rotations
  double* Ut;              // L x L sorted left factors (col-major)
  double* Vt;              // L x L sorted right factors (col-major)
  double* St;              // L sorted singular values
  uint64_t seed;
  const double* fu;        // given factors (or null): R x r, r, C x r row-major
  const double* fs;
  const double* fv;
};

// One matrix.
struct Mat {
  const uint16_t* w0;      // R x C bf16
  uint16_t* out;           // R x C bf16
  float* dhat;             // optional R x C fp32
  int64_t R, C, Kr, ldk;   // ldk = rup(Kr, 32)
  double* U;               // R x ldk row-major
  double* V;               // C x ldk row-major
  double* Sig;             // ldk
  double* GUp;             // kSlabs x Kr x Kr
  double* GU;              // Kr x Kr
  double* GV;
  double* ns[2][5];         // per side (U, V): Newton-Schulz Y0, Z0, Y1, Z1, T (Kr x Kr each)
  double* eye;              // Kr x Kr identity
  double* cs;               // 2 scale factors
  struct NsFlags* nf;       // per side: convergence of the Newton-Schulz iteration
  double* MU;  double* MV;  // Kr x Kr inverse square roots
  double* Up;  double* Vp;                              // R x Kr, C x Kr
  uint16_t* ah; uint16_t* al;   // R x ldk split of U_perp Sigma
  uint16_t* bh; uint16_t* bl;   // C x ldk split of V_perp
  double alpha;
};

constexpr int kSlabs = 16;
constexpr int kNsIters = 18;     // coupled Newton-Schulz steps at most (quadratic convergence from |I - A| < 1)
constexpr int kNsCheck = 4;      // steps queued between host reads of the done flags
constexpr double kNsTol = 1e-10; // max |T - I| from which one more step reaches rounding level

// One side of one matrix: a job stops after the step whose T = (3 I - Z Y) / 2 is within kNsTol
// of I (Z Y then within 2 kNsTol of I, and one more quadratic step takes it to rounding level).
struct NsFlags {
  int done;      // no further steps
  int last;      // the step being taken is the last
  int steps;     // steps taken: Y, Z are in buffers 2 (steps & 1) and 2 (steps & 1) + 1
  int pad;
};

__device__ __forceinline__ uint16_t bf16_rne_f32(float f) {
  uint32_t b = __float_as_uint(f);
  return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float f32_of_bf16(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ bf16x8_t ld_bf16x8(const uint16_t* p) {
  return *gmem((const bf16x8_t*)p);
}

// Row `row` of a row-major bf16 matrix with `ncols` columns: 8 entries from column k (zero
// outside the matrix).
__device__ __forceinline__ bf16x8_t ld_row8(const uint16_t* base, int64_t nrows, int64_t ncols, int64_t row, int64_t k,
                                            bool vec) {
  if (row < nrows) {
    const uint16_t* p = base + row * ncols + k;
    if (vec && k + 8 <= ncols) return ld_bf16x8(p);
    uint16_t t[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) t[e] = (k + e < ncols) ? gmem(p)[e] : (uint16_t)0;
    return __builtin_bit_cast(bf16x8_t, *(uint4*)t);
  }
  return __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0));
}

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

// ---- sketch operands -----------------------------------------------------------------------------

// Test matrix Omega (C x L): entries j/64, j uniform in [-64, 63] (exact in bf16), low part 0.
__global__ void k_omega(const Prob* __restrict__ probs) {
  const Prob& P = probs[blockIdx.y];
  const int64_t total = P.L * P.ldb;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = e % P.ldb;
    float v = 0.0f;
    if (k < P.C) v = (float)((int)(splitmix64(P.seed ^ (uint64_t)e) >> 57) - 64) * 0.015625f;
    P.bh[e] = bf16_rne_f32(v);
    P.bl[e] = 0;
  }
}

// ---- MFMA products with the delta -----------------------------------------------------------------
//
// Both products stream the delta once per call and keep the skinny right operand B (hi and,
// when LO, lo bf16 parts; L columns of ldb entries, ldb a multiple of 64 and zero beyond the
// operand's rows) in LDS, one k-step at a time, double-buffered: the next step's delta and B
// pieces are loaded into registers before the current step's MFMAs and written to LDS after
// them, with one workgroup barrier per step.  Each wave owns 64 output rows (four 16-row
// blocks), so every B fragment read from LDS feeds four MFMAs per part.
//
// Workgroups are renumbered so that the consecutive row blocks of one problem run on the same
// XCD (the hardware deals workgroups to the eight XCDs round-robin): the B window of a problem
// is then fetched from HBM into one XCD's L2, not into all eight.

constexpr int kSkRows = 256;   // output rows per workgroup: 4 waves x 64
constexpr int kXcds = 8;

// Linear workgroup id -> logical id, a bijection on [0, G) that gives each XCD a contiguous
// range of logical ids.
__device__ __forceinline__ int64_t xcd_logical_block(int64_t b, int64_t G) {
  const int64_t q = G / kXcds, rem = G % kXcds;
  const int64_t x = b % kXcds, i = b / kXcds;
  return (x < rem) ? x * (q + 1) + i : rem * (q + 1) + (x - rem) * q + i;
}

// B pieces of one k-step: H parts x NB*16 columns x KG 16-byte groups of 8 k.
template <int NB, int H, int KG>
struct SkB {
  static constexpr int kPieces = H * NB * 16 * KG;
  static constexpr int kPerThread = (kPieces + 255) / 256;
  bf16x8_t q[kPerThread];
  __device__ __forceinline__ void load(const Prob& P, int64_t k0) {
#pragma unroll
    for (int j = 0; j < kPerThread; ++j) {
      const int t = threadIdx.x + 256 * j;
      if (kPieces % 256 == 0 || t < kPieces) {
        const int h = t / (NB * 16 * KG), rem = t % (NB * 16 * KG), col = rem / KG, kg = rem % KG;
        q[j] = ld_bf16x8((h ? P.bl : P.bh) + (int64_t)col * P.ldb + k0 + 8 * kg);
      }
    }
  }
  __device__ __forceinline__ void store(bf16x8_t (*sh)[NB * 16][KG + 1]) const {
#pragma unroll
    for (int j = 0; j < kPerThread; ++j) {
      const int t = threadIdx.x + 256 * j;
      if (kPieces % 256 == 0 || t < kPieces) {
        const int h = t / (NB * 16 * KG), rem = t % (NB * 16 * KG), col = rem / KG, kg = rem % KG;
        sh[h][col][kg] = q[j];
      }
    }
  }
};

// X[out] (R x L) = Delta (R x C) * bh (C x L), hi part only (every product of this kind feeds a
// QR of the range finder).  64 k per step: each delta row is read 128 bytes at a time, straight
// into MFMA A fragments (lane (ln, g) holds row ln, k = 8g..8g+7 of each 32-k half).  Rows past R are clamped to R - 1 and not stored; with C % 8 == 0, k groups past
// C are clamped into the row (B is zero there), otherwise entries are loaded one by one and
// zero-filled.
template <int NB>
__global__ void __launch_bounds__(256) k_sk_nn(const Prob* __restrict__ probs, const int* __restrict__ order, int out,
                                               int64_t nbx) {
  constexpr int KS = 64, KG = KS / 8, H = 1;
  __shared__ bf16x8_t bsh[2][H][NB * 16][KG + 1];
  const int64_t lb = xcd_logical_block(blockIdx.x + (int64_t)gridDim.x * blockIdx.z, (int64_t)gridDim.x * gridDim.z);
  const Prob& P = probs[order[lb / nbx]];
  const int64_t R = P.R, C = P.C;
  const int64_t m0 = (lb % nbx) * kSkRows;
  if (m0 >= R) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  const int64_t wrow = m0 + 64 * w;
  const bool vec = (C % 8) == 0;
  const uint16_t* arow[4];
  int64_t rr[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    rr[rb] = min(R - 1, wrow + 16 * rb + ln);
    arow[rb] = P.delta + rr[rb] * C;
  }
  auto load_a = [&](int64_t k0, bf16x8_t (&a)[4][2]) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int64_t k = k0 + 32 * kb + 8 * g;
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        if (vec) a[rb][kb] = ld_bf16x8(arow[rb] + min(k, C - 8));
        else a[rb][kb] = ld_row8(P.delta, R, C, rr[rb], k, false);
      }
    }
  };
  f32x4_t acc[4][NB];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int64_t steps = (C + KS - 1) / KS;
  bf16x8_t a[4][2], an[4][2];
  SkB<NB, H, KG> bq;
  load_a(0, a);
  bq.load(P, 0);
  bq.store(bsh[0]);
  __syncthreads();
  for (int64_t s = 0; s < steps; ++s) {
    const bool more = s + 1 < steps;
    if (more) {
      bq.load(P, (s + 1) * KS);
      load_a((s + 1) * KS, an);
    }
    const int buf = (int)(s & 1);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const bf16x8_t bh = bsh[buf][0][cb * 16 + ln][4 * kb + g];
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rb][kb], bh, acc[rb][cb], 0, 0, 0);
      }
    if (more) bq.store(bsh[buf ^ 1]);
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) a[rb][kb] = an[rb][kb];
  }
  double* X = P.X[out];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t r = wrow + 16 * rb + 4 * g + e;
        if (r < R) gmem(X)[r * P.L + cb * 16 + ln] = (double)acc[rb][cb][e];
      }
}

// Swizzle of the delta tile in LDS (32 rows x 256 columns, row-major, no padding): the 8-byte
// chunk c of row r is stored at chunk c ^ 4*s(r).  s takes eight distinct values over the
// rows {0..3, 8..11} (and {4..7, 12..15}, ...), so each transposed read of 16 rows x 32 bytes
// below touches every LDS bank exactly twice.
__device__ __forceinline__ int sk_swz(int r) { return ((r & 3) | (((r >> 3) & 1) << 2)) << 2; }

typedef __bf16 bf16x4v_t __attribute__((__vector_size__(4 * sizeof(__bf16))));

// Z[out] (C x L) = Delta^T (C x R) * B (R x L).  Each workgroup owns 256 delta columns and walks
// the delta rows 32 at a time: the 32 x 256 tile (row segments of 512 bytes) goes through LDS and
// the A fragments of Delta^T are read from it with ds_read_b64_tr_b16.  Within a 16-lane group
// that instruction hands lane i, element m, the (i & 3)-th value of the 8 bytes that lane
// 4m + (i >> 2) addressed; with lane 4m + q pointing at columns 4q..4q+3 of row m, lane i
// receives column i of four consecutive rows.  Two such reads (rows 8g..8g+3, 8g+4..8g+7) form
// the fragment lane (ln, g) needs: column ln, k = 8g..8g+7.  Rows past R are clamped (B is zero
// there); columns past C are clamped and not stored.  Requires C % 8 == 0 (the host routes other
// shapes to k_sk_tn_any).
template <int NB, bool LO>
__global__ void __launch_bounds__(256) k_sk_tn(const Prob* __restrict__ probs, const int* __restrict__ order, int out,
                                               int64_t nbx) {
  constexpr int KS = 32, KG = KS / 8, H = LO ? 2 : 1;
  __shared__ __align__(16) uint16_t atile[2][KS][kSkRows];
  __shared__ bf16x8_t bsh[2][H][NB * 16][KG + 1];
  const int64_t lb = xcd_logical_block(blockIdx.x + (int64_t)gridDim.x * blockIdx.z, (int64_t)gridDim.x * gridDim.z);
  const Prob& P = probs[order[lb / nbx]];
  const int64_t R = P.R, C = P.C;
  const int64_t i0 = (lb % nbx) * kSkRows;
  if (i0 >= C) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  // tile pieces: 32 rows x 32 pieces of 16 bytes, four per thread
  bf16x8_t pa[4];
  auto load_a = [&](int64_t k0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = threadIdx.x + 256 * j, row = t >> 5, pc = t & 31;
      const int64_t gr = min(R - 1, k0 + row), gc = min(C - 8, i0 + 8 * pc);
      pa[j] = ld_bf16x8(P.delta + gr * C + gc);
    }
  };
  auto store_a = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = threadIdx.x + 256 * j, row = t >> 5, pc = t & 31;
      *(bf16x8_t*)&atile[buf][row][(8 * pc) ^ (4 * sk_swz(row))] = pa[j];
    }
  };
  // transposed-read addresses: lane 16G + 4m + q reads row 8G + 4h + m, logical chunk 16w + 4rb + q
  const int G = lane >> 4, m = (lane >> 2) & 3, q = lane & 3;
  f32x4_t acc[4][NB];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int64_t steps = (R + KS - 1) / KS;
  SkB<NB, H, KG> bq;
  load_a(0);
  bq.load(P, 0);
  store_a(0);
  bq.store(bsh[0]);
  __syncthreads();
  for (int64_t s = 0; s < steps; ++s) {
    const bool more = s + 1 < steps;
    if (more) {
      bq.load(P, (s + 1) * KS);
      load_a((s + 1) * KS);
    }
    const int buf = (int)(s & 1);
    bf16x8_t a[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      bf16x4v_t h2[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int row = 8 * G + 4 * h + m;
        const int chunk = (16 * w + 4 * rb + q) ^ sk_swz(row);
        h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (__attribute__((address_space(3))) bf16x4v_t*)&atile[buf][row][4 * chunk]);
      }
      const uint2 u0 = __builtin_bit_cast(uint2, h2[0]), u1 = __builtin_bit_cast(uint2, h2[1]);
      a[rb] = __builtin_bit_cast(bf16x8_t, make_uint4(u0.x, u0.y, u1.x, u1.y));
    }
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const bf16x8_t bh = bsh[buf][0][cb * 16 + ln][g];
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
        acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rb], bh, acc[rb][cb], 0, 0, 0);
      if (LO) {
        const bf16x8_t bl = bsh[buf][H - 1][cb * 16 + ln][g];
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rb], bl, acc[rb][cb], 0, 0, 0);
      }
    }
    if (more) {
      store_a(buf ^ 1);
      bq.store(bsh[buf ^ 1]);
    }
    __syncthreads();
  }
  double* Z = P.Z[out];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t r = i0 + 64 * w + 16 * rb + 4 * g + e;
        if (r < C) gmem(Z)[r * P.L + cb * 16 + ln] = (double)acc[rb][cb][e];
      }
}

// Z[out] (C x L) = Delta^T (C x R) * (bh + bl) for any C (rows not 16-byte aligned): a 32 x 256
// tile of the delta is staged in LDS and read transposed one entry at a time; B is read from
// global memory.  Each wave owns 64 output rows.
template <int NB>
__global__ void __launch_bounds__(256) k_sk_tn_any(const Prob* __restrict__ probs, int out) {
  __shared__ uint16_t tile[32][kSkRows + 2];
  const Prob& P = probs[blockIdx.z];
  const int64_t R = P.R, C = P.C;
  const int64_t i0 = (int64_t)blockIdx.x * kSkRows;
  if (i0 >= C) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  const bool vec = (C % 8) == 0;
  f32x4_t acc[4][NB];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // the next 32 x 256 delta tile is loaded into registers while the current one is used
  bf16x8_t pre[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int piece = threadIdx.x + 256 * q;
    pre[q] = ld_row8(P.delta, R, C, piece >> 5, i0 + (piece & 31) * 8, vec);
  }
  for (int64_t k0 = 0; k0 < R; k0 += 32) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int piece = threadIdx.x + 256 * q;
      const int tr = piece >> 5, tc = (piece & 31) * 8;
      const uint4 u = __builtin_bit_cast(uint4, pre[q]);
      const uint32_t ws[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        tile[tr][tc + 2 * e] = (uint16_t)(ws[e] & 0xFFFFu);
        tile[tr][tc + 2 * e + 1] = (uint16_t)(ws[e] >> 16);
      }
    }
    __syncthreads();
    if (k0 + 32 < R) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int piece = threadIdx.x + 256 * q;
        pre[q] = ld_row8(P.delta, R, C, k0 + 32 + (piece >> 5), i0 + (piece & 31) * 8, vec);
      }
    }
    bf16x8_t a[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      uint16_t t8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) t8[e] = tile[8 * g + e][64 * w + 16 * rb + ln];
      a[rb] = __builtin_bit_cast(bf16x8_t, *(uint4*)t8);
    }
    const int64_t k = k0 + 8 * g;
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const int64_t col = cb * 16 + ln;
      const bf16x8_t bh = ld_bf16x8(P.bh + col * P.ldb + k);
      const bf16x8_t bl = ld_bf16x8(P.bl + col * P.ldb + k);
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rb], bh, acc[rb][cb], 0, 0, 0);
        acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rb], bl, acc[rb][cb], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  double* Z = P.Z[out];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t r = i0 + 64 * w + 16 * rb + 4 * g + e;
        if (r < C) gmem(Z)[r * P.L + cb * 16 + ln] = (double)acc[rb][cb][e];
      }
}

// ---- Cholesky-QR pieces ------------------------------------------------------------------------------
//
// Binary64 throughout, on v_mfma_f64_16x16x4_f64: lane (ln, g) supplies A[ln][g] and B[g][ln] and
// receives D[g + 4v][ln] in its v-th register pair, v = 0..3 (probed on the device).

typedef double f64x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f64x4_t mfma64(double a, double b, f64x4_t c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// Tile pair p of the upper triangle (rb <= cb) of an nb x nb grid of 16 x 16 tiles, row by row.
constexpr int pair_rb(int p, int nb) {
  int rb = 0;
  while (p >= nb - rb) { p -= nb - rb; ++rb; }
  return rb;
}
constexpr int pair_cb(int p, int nb) {
  int rb = 0;
  while (p >= nb - rb) { p -= nb - rb; ++rb; }
  return rb + p;
}

template <int NB, int P>
struct TilePair {
  static constexpr int rb = pair_rb(P, NB), cb = pair_cb(P, NB);
};

// acc[i] += x[rb] x[cb]^T for the pairs W + 4i (compile-time indices throughout)
template <int NB, int W, int... I>
__device__ __forceinline__ void gram_mfmas(f64x4_t* acc, const double* x, std::integer_sequence<int, I...>) {
  ((acc[I] = mfma64(x[TilePair<NB, W + 4 * I>::rb], x[TilePair<NB, W + 4 * I>::cb], acc[I])), ...);
}
template <int NB, int W, int... I>
__device__ __forceinline__ void gram_store(const f64x4_t* acc, double* __restrict__ Gz, int g, int ln,
                                           std::integer_sequence<int, I...>) {
  constexpr int L = 16 * NB;
  (
      [&] {
        constexpr int rb = TilePair<NB, W + 4 * I>::rb, cb = TilePair<NB, W + 4 * I>::cb;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          Gz[(16 * rb + g + 4 * v) * L + 16 * cb + ln] = acc[I][v];
          if (rb != cb) Gz[(16 * cb + ln) * L + 16 * rb + g + 4 * v] = acc[I][v];
        }
      }(),
      ...);
}

// One wave's share of a Gram partial: pairs W, W + 4, ... of the upper triangle, over rows
// [r0, r1) of X (row-major, L = 16 NB columns), eight rows per step.  Writes both triangles.
template <int NB, int W>
__device__ __forceinline__ void gram_wave(const double* __restrict__ X, int64_t r0, int64_t r1, double* __restrict__ Gz,
                                          int lane) {
  constexpr int L = 16 * NB, NP = NB * (NB + 1) / 2, PW = (NP - W + 3) / 4;
  if constexpr (PW > 0) {
    using Seq = std::make_integer_sequence<int, PW>;
    const int g = lane >> 4, ln = lane & 15;
    f64x4_t acc[PW];
#pragma unroll
    for (int i = 0; i < PW; ++i) acc[i] = f64x4_t{0.0, 0.0, 0.0, 0.0};
    for (int64_t k0 = r0; k0 < r1; k0 += 8) {
      double x0[NB], x1[NB];
      const int64_t ra = k0 + g, rc = k0 + 4 + g;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        x0[j] = (ra < r1) ? gmem(X)[ra * L + 16 * j + ln] : 0.0;
        x1[j] = (rc < r1) ? gmem(X)[rc * L + 16 * j + ln] : 0.0;
      }
      gram_mfmas<NB, W>(acc, x0, Seq{});
      gram_mfmas<NB, W>(acc, x1, Seq{});
    }
    gram_store<NB, W>(acc, Gz, g, ln, Seq{});
  }
}

// Gram partials of the current tall factor: Gp[z] = sum over the rows of slab z of x x^T.
template <int NB>
__global__ void __launch_bounds__(256) k_gram_mf(const Prob* __restrict__ probs, int which, int cur) {
  const Prob& P = probs[blockIdx.y];
  const int64_t M = which ? P.C : P.R;
  const double* X = which ? P.Z[cur] : P.X[cur];
  const int64_t per = (M + kSlabs - 1) / kSlabs;
  const int64_t r0 = min(M, (int64_t)blockIdx.x * per), r1 = min(M, r0 + per);
  double* Gz = P.Gp + (int64_t)blockIdx.x * P.L * P.L;
  const int lane = threadIdx.x & 63;
  switch (threadIdx.x >> 6) {
    case 0: gram_wave<NB, 0>(X, r0, r1, Gz, lane); break;
    case 1: gram_wave<NB, 1>(X, r0, r1, Gz, lane); break;
    case 2: gram_wave<NB, 2>(X, r0, r1, Gz, lane); break;
    default: gram_wave<NB, 3>(X, r0, r1, Gz, lane); break;
  }
}

// G = sum of the partials, then G = R^T R (R upper, row-major in Rf) and Ri = R^{-1}.  With
// `acc`: R2 = Rf * Ra (second factor times the saved first), and `save`: Ra = Rf.  Both the
// factorisation and the inverse run pivot by pivot with the work of a pivot spread over the
// workgroup.  The inverse X = R^{-1} is formed column-oriented from X = I: for i = L-1 down to 0,
// row i of X is divided by R[i][i], then X[t][c] -= R[t][i] X[i][c] for t < i <= c.  X is upper
// triangular and is kept transposed in the unused lower triangle of g (X[t][c] at g[c][t]), its
// diagonal in di.
__global__ void __launch_bounds__(256) k_chol(const Prob* __restrict__ probs, int save, int accum, uint32_t* status) {
  extern __shared__ double g[];                  // L x L, then L diagonal entries of the inverse
  const Prob& P = probs[blockIdx.x];
  const int L = (int)P.L;
  const double* __restrict__ Gp = P.Gp;
  double* di = g + L * L;
  for (int e0 = threadIdx.x; e0 < L * L; e0 += 4 * blockDim.x) {
    double s[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int z = 0; z < kSlabs; ++z)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = e0 + u * blockDim.x;
        if (e < L * L) s[u] = s[u] + Gp[(int64_t)z * L * L + e];
      }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (e0 + u * (int)blockDim.x < L * L) g[e0 + u * blockDim.x] = s[u];
  }
  __syncthreads();
  double tr = 0.0;
  for (int j = 0; j < L; ++j) tr += g[j * L + j];
  const double shift = 1e-15 * tr / (double)L + 1e-300;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  for (int j = 0; j < L; ++j) {
    // every thread forms the pivot itself and row j is scaled; the pivot is stored once every
    // thread has read the old diagonal, then the trailing triangle is updated
    __syncthreads();
    const double d = g[j * L + j];
    const double piv = sqrt(d > shift ? d : shift);
    for (int k = j + 1 + threadIdx.x; k < L; k += blockDim.x) g[j * L + k] /= piv;
    __syncthreads();
    if (threadIdx.x == 0) g[j * L + j] = piv;
    for (int i = j + 1 + ty; i < L; i += 16) {
      const double a = g[j * L + i];
#pragma unroll 4
      for (int k = i + tx; k < L; k += 16) g[i * L + k] -= a * g[j * L + k];
    }
  }
  // inverse: X = I, then pivots from the last
  for (int e = threadIdx.x; e < L; e += blockDim.x) di[e] = 1.0;
  for (int c = ty; c < L; c += 16)
    for (int t = tx; t < c; t += 16) g[c * L + t] = 0.0;
  for (int i = L - 1; i >= 0; --i) {
    __syncthreads();
    const double rii = g[i * L + i];
    for (int c = i + threadIdx.x; c < L; c += blockDim.x) {
      if (c == i) di[i] = 1.0 / rii;
      else g[c * L + i] /= rii;
    }
    __syncthreads();
    for (int c = i + ty; c < L; c += 16) {
      const double xic = (c == i) ? di[i] : g[c * L + i];
#pragma unroll 4
      for (int t = tx; t < i; t += 16) g[c * L + t] -= g[t * L + i] * xic;
    }
  }
  __syncthreads();
  for (int i = ty; i < L; i += 16)
    for (int k = tx; k < L; k += 16) {
      const int e = i * L + k;
      P.Rf[e] = (k >= i) ? g[e] : 0.0;
      P.Ri[e] = (k > i) ? g[k * L + i] : ((k == i) ? di[i] : 0.0);
      if (save) P.Ra[e] = (k >= i) ? g[e] : 0.0;
    }
  if (accum) {
    // R2 = Rf * Ra  (both upper; Rf read from LDS, Ra saved by an earlier launch)
    const double* __restrict__ Ra = P.Ra;
    double* __restrict__ R2 = P.R2;
    for (int i = ty; i < L; i += 16)
      for (int k = tx; k < L; k += 16) {
        double s = 0.0;
#pragma unroll 8
        for (int t = i; t <= k; ++t) s = s + g[i * L + t] * Ra[t * L + k];
        R2[i * L + k] = (k >= i) ? s : 0.0;
      }
  }
  if (threadIdx.x == 0 && !(g[0] > 0.0)) flag_status(status, kStatusInternal);
}

// Y = X Ri (tall factor times the upper-triangular inverse factor), X and Y row-major M x L.
// Ri sits in LDS; each wave takes 16 rows per 64-row chunk, its A fragments straight from X
// (the next chunk's in flight), and the triangle is skipped at 16-column granularity.  Lane ln
// feeds row 4(ln % 4) + ln / 4 of the wave's 16, so that result register v of lane (ln, g),
// D row g + 4v, is row 4g + v: four consecutive rows per lane.  With
// `split`, the rows are also written as the bf16 hi/lo parts of the next product's operand
// (L columns of ldb, rows past M zero up to the next multiple of 64).
template <int NB>
__global__ void __launch_bounds__(256) k_apply_mf(const Prob* __restrict__ probs, int which, int src, int dst,
                                                  int split) {
  constexpr int L = 16 * NB;
  __shared__ double ri[L][L + 1];
  const Prob& P = probs[blockIdx.y];
  const int64_t M = which ? P.C : P.R;
  const double* X = which ? P.Z[src] : P.X[src];
  double* Y = which ? P.Z[dst] : P.X[dst];
  for (int e = threadIdx.x; e < L * L; e += blockDim.x) ri[e / L][e % L] = P.Ri[e];
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  const int64_t nchunks = (M + 63) / 64;
  double xa[4 * NB];
  const int lrow = 4 * (ln & 3) + (ln >> 2);
  auto load = [&](int64_t chunk, double (&x)[4 * NB]) {
    const int64_t r = chunk * 64 + 16 * w + lrow;
    const bool ok = chunk < nchunks && r < M;
#pragma unroll
    for (int s = 0; s < 4 * NB; ++s) x[s] = ok ? gmem(X)[r * L + 4 * s + g] : 0.0;
  };
  int64_t chunk = blockIdx.x;
  load(chunk, xa);
  for (; chunk < nchunks; chunk += gridDim.x) {
    // keeps the Ri fragments in LDS (read per chunk) instead of hoisted into registers
    asm volatile("" ::: "memory");
    const int64_t rn = (chunk + gridDim.x) * 64 + 16 * w + lrow;
    const bool nok = chunk + gridDim.x < nchunks && rn < M;
    f64x4_t acc[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) acc[cb] = f64x4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int s = 0; s < 4 * NB; ++s) {
      const double a = xa[s];
      xa[s] = nok ? gmem(X)[rn * L + 4 * s + g] : 0.0;      // the next chunk's fragment, one chunk ahead
#pragma unroll
      for (int cb = s / 4; cb < NB; ++cb) acc[cb] = mfma64(a, ri[4 * s + g][16 * cb + ln], acc[cb]);
    }
    const int64_t row0 = chunk * 64 + 16 * w + 4 * g;
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (row0 + v < M) gmem(Y)[(row0 + v) * L + 16 * cb + ln] = acc[cb][v];
      if (split) {
        uint16_t h[4], l[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float f = (float)acc[cb][v];
          h[v] = bf16_rne_f32(f);
          l[v] = bf16_rne_f32(f - f32_of_bf16(h[v]));
        }
        const int64_t o = (int64_t)(16 * cb + ln) * P.ldb + row0;
        *gmem((u32x2_t*)(P.bh + o)) = u32x2_t{h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16)};
        *gmem((u32x2_t*)(P.bl + o)) = u32x2_t{l[0] | ((uint32_t)l[1] << 16), l[2] | ((uint32_t)l[3] << 16)};
      }
    }
  }
}

// The one-sided Jacobi sweeps of k_jacobi with A (r x c) and V (c x c) held in LDS, for cores
// small enough to fit; A and V are written back at the end.
constexpr size_t kJacobiLdsMax = 150 * 1024;
__global__ void __launch_bounds__(kJacobiThreads) k_jacobi_lds(const JacobiJob* __restrict__ jobs, uint32_t* status) {
  extern __shared__ double jsh[];
  __shared__ int s_rot;
  const JacobiJob J = jobs[blockIdx.x];
  const int r = (int)J.r, c = (int)J.c;
  double* A = jsh;
  double* V = jsh + r * c;
  for (int e = threadIdx.x; e < r * c; e += blockDim.x) A[e] = J.a[e];
  for (int e = threadIdx.x; e < c * c; e += blockDim.x) V[e] = ((e % c) == (e / c)) ? 1.0 : 0.0;
  __syncthreads();
  const bool converged = (r <= 128) ? jacobi_sweeps<8>(A, V, r, c, &s_rot) : jacobi_sweeps<0>(A, V, r, c, &s_rot);
  for (int e = threadIdx.x; e < r * c; e += blockDim.x) J.a[e] = A[e];
  for (int e = threadIdx.x; e < c * c; e += blockDim.x) J.v[e] = V[e];
  if (!converged && threadIdx.x == 0) flag_status(status, kStatusInternal);
}

// Jacobi input: Ja = R2 read as column-major, i.e. R2^T.
__global__ void k_core_load(const Prob* __restrict__ probs, JacobiJob* jobs) {
  const Prob& P = probs[blockIdx.x];
  for (int64_t e = threadIdx.x; e < P.L * P.L; e += blockDim.x) P.Ja[e] = P.R2[e];
  if (threadIdx.x == 0) {
    jobs[blockIdx.x].a = P.Ja;
    jobs[blockIdx.x].v = P.Jv;
    jobs[blockIdx.x].r = P.L;
    jobs[blockIdx.x].c = P.L;
  }
}

// Sigma[i*r + c] = St[c] for c < r (Sig has ldk entries, the pad stays zero).
__global__ void k_sigma(const Prob* __restrict__ probs, Mat* mats, int K, int r) {
  const int p = blockIdx.x;
  const Prob& P = probs[p];
  Mat& M = mats[p / K];
  const int i = p % K;
  for (int c = threadIdx.x; c < r; c += blockDim.x) M.Sig[i * r + c] = P.St[c];
}

// Given factors: U_i and V_i into column block i of the concatenated U and V, s_i into Sig.
__global__ void k_load_factors(const Prob* __restrict__ probs, Mat* mats, int K, int r) {
  const int p = blockIdx.y;
  const Prob& P = probs[p];
  Mat& M = mats[p / K];
  const int i = p % K;
  const int64_t nu = P.R * r, nv = P.C * r;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nu + nv; e += (int64_t)gridDim.x * blockDim.x) {
    if (e < nu) {
      M.U[(e / r) * M.ldk + i * r + e % r] = P.fu[e];
    } else {
      const int64_t f = e - nu;
      M.V[(f / r) * M.ldk + i * r + f % r] = P.fv[f];
    }
  }
  if (blockIdx.x == 0)
    for (int c = threadIdx.x; c < r; c += blockDim.x) M.Sig[i * r + c] = P.fs[c];
}

// ---- orthogonalisation (Procrustes / Loewdin) ---------------------------------------------------

// bf16 hi/lo split of rows: dst (rows x ldk) = src (rows x Kr, row stride ldsrc) * (scale? s[col] : 1)
__global__ void k_split_rows(uint16_t* __restrict__ hi, uint16_t* __restrict__ lo, const double* __restrict__ src,
                             int64_t rows, int64_t Kr, int64_t ldsrc, int64_t ldk, const double* __restrict__ scale) {
  const int64_t total = rows * ldk;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / ldk, c = e - r * ldk;
    float v = 0.0f;
    if (c < Kr) v = (float)(src[r * ldsrc + c] * (scale ? scale[c] : 1.0));
    const uint16_t h = bf16_rne_f32(v);
    hi[e] = h;
    lo[e] = bf16_rne_f32(v - f32_of_bf16(h));
  }
}

// bf16 nearest-even of w + s (w a bf16 value, s binary32), rounded once: the binary32 sum and
// its exact error (TwoSum, Knuth) give w + s exactly as hi + lo; hi is replaced by its
// round-to-odd neighbour when lo != 0 (24 >= 8 + 2 bits, so the following nearest-even rounding
// to 8 bits is the correct rounding of w + s).
__device__ __forceinline__ uint32_t bf16_of_sum(float w, float s) {
  const float hi = w + s;
  const float bb = hi - w;
  const float lo = (w - (hi - bb)) + (s - bb);
  uint32_t b = __float_as_uint(hi);
  if (lo != 0.0f && (b & 1u) == 0u) b += ((__float_as_uint(lo) ^ b) >> 31) ? 0xFFFFFFFFu : 1u;
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// out = round(W0 + alpha * A B^T), A = ah + al (R x ldk), B = bh + bl (C x ldk); three MFMA
// products per step (hi*hi, hi*lo, lo*hi), binary32 accumulation.  128 x 128 output tile per
// workgroup, four waves as 2 x 2 of 64 x 64 (4 x 4 MFMA tiles); both operands go through LDS
// 32 k at a time, double-buffered, the next step's pieces loaded into registers while the
// current step's MFMAs run.  The MFMA computes the transposed tile (B fragments as its A operand)
// so that lane (ln, g) ends with four consecutive columns 4g..4g+3 of output row ln: W0 is read
// (before the last step) and the result written 8 bytes at a time (entry by entry when
// C % 4 != 0).  The update is W0 + fl32(alpha * acc) rounded once to bf16 (bf16_of_sum).
//
// The grid is one-dimensional, `tiles` slots per matrix.  Workgroups are renumbered so that each
// XCD takes a contiguous range, and within a matrix the tiles go column by column down groups of
// eight tile rows: the 64 tiles an XCD has in flight then share eight row panels of A and eight
// of B (2 MB of operands), which its L2 holds, instead of streaming 256 KB per tile from HBM.
constexpr int kRecT = 128, kRecK = 32, kRecKG = kRecK / 8, kRecGroup = 8;
__global__ void __launch_bounds__(256) k_mfma_recon(const Mat* __restrict__ mats, int64_t tiles) {
  __shared__ bf16x8_t ash[2][2][kRecT][kRecKG + 1];     // [buffer][hi, lo][row][k group]
  __shared__ bf16x8_t bsh[2][2][kRecT][kRecKG + 1];
  const int64_t lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const Mat& M = mats[lb / tiles];
  const int64_t R = M.R, C = M.C, ldk = M.ldk;
  const int64_t ntr = (R + kRecT - 1) / kRecT, ntc = (C + kRecT - 1) / kRecT;
  const int64_t t = lb % tiles;
  if (t >= ntr * ntc) return;
  const int64_t grp = t / (kRecGroup * ntc), r0 = grp * kRecGroup, gm = min<int64_t>(kRecGroup, ntr - r0);
  const int64_t loc = t - grp * kRecGroup * ntc;
  const int64_t m0 = (r0 + loc % gm) * kRecT, n0 = (loc / gm) * kRecT;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, ln = lane & 15;
  const int wm = w >> 1, wn = w & 1;
  // staging: 2 operands x 2 halves x 128 rows x 4 k groups = 2048 pieces, eight per thread
  bf16x8_t pq[8];
  auto load = [&](int64_t k0) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int t = threadIdx.x + 256 * j;
      const int op = t >> 10, h = (t >> 9) & 1, row = (t >> 2) & 127, kg = t & 3;
      const uint16_t* base = op ? (h ? M.bl : M.bh) : (h ? M.al : M.ah);
      const int64_t gr = op ? min(C - 1, n0 + row) : min(R - 1, m0 + row);
      pq[j] = ld_bf16x8(base + gr * ldk + k0 + 8 * kg);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int t = threadIdx.x + 256 * j;
      const int op = t >> 10, h = (t >> 9) & 1, row = (t >> 2) & 127, kg = t & 3;
      if (op) bsh[buf][h][row][kg] = pq[j];
      else ash[buf][h][row][kg] = pq[j];
    }
  };
  f32x4_t acc[4][4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) acc[rb][cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int64_t steps = ldk / kRecK;
  load(0);
  store(0);
  __syncthreads();
  const bool vec = (C % 4) == 0;
  u32x2_t wv[4][4];
  for (int64_t s = 0; s < steps; ++s) {
    const bool more = s + 1 < steps;
    if (more) load((s + 1) * kRecK);
    else if (vec) {
      // the epilogue's W0 values, in flight during the last step's MFMAs
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          const int64_t r = min(R - 1, m0 + 64 * wm + 16 * rb + ln), c0 = min(C - 4, n0 + 64 * wn + 16 * cb + 4 * g);
          wv[rb][cb] = *gmem((const u32x2_t*)(M.w0 + r * C + c0));
        }
    }
    const int buf = (int)(s & 1);
    bf16x8_t ah[4], al[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      ah[rb] = ash[buf][0][64 * wm + 16 * rb + ln][g];
      al[rb] = ash[buf][1][64 * wm + 16 * rb + ln][g];
    }
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const bf16x8_t bh = bsh[buf][0][64 * wn + 16 * cb + ln][g];
      const bf16x8_t bl = bsh[buf][1][64 * wn + 16 * cb + ln][g];
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh, ah[rb], acc[rb][cb], 0, 0, 0);
        acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bl, ah[rb], acc[rb][cb], 0, 0, 0);
        acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh, al[rb], acc[rb][cb], 0, 0, 0);
      }
    }
    if (more) store(buf ^ 1);
    __syncthreads();
  }
  const float alpha = (float)M.alpha;
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int64_t r = m0 + 64 * wm + 16 * rb + ln;
    if (r >= R) continue;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int64_t c0 = n0 + 64 * wn + 16 * cb + 4 * g;
      if (c0 >= C) continue;
      const int64_t idx = r * C + c0;
      if (vec) {
        const uint32_t wi[4] = {wv[rb][cb].x << 16, wv[rb][cb].x & 0xFFFF0000u, wv[rb][cb].y << 16,
                                wv[rb][cb].y & 0xFFFF0000u};
        uint32_t o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = bf16_of_sum(__uint_as_float(wi[e]), alpha * acc[rb][cb][e]);
        *gmem((u32x2_t*)(M.out + idx)) = u32x2_t{o[0] | (o[1] << 16), o[2] | (o[3] << 16)};
        if (M.dhat) *gmem((f32x4_t*)(M.dhat + idx)) = acc[rb][cb];
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (c0 + e < C) {
            gmem(M.out)[idx + e] = (uint16_t)bf16_of_sum(f32_of_bf16(gmem(M.w0)[idx + e]), alpha * acc[rb][cb][e]);
            if (M.dhat) gmem(M.dhat)[idx + e] = acc[rb][cb][e];
          }
      }
    }
  }
}

// ---- per-matrix helpers, batched over the matrices of a chunk (grid.y / grid.x = matrix) ----------

// G = sum of the Gram partials of one side for every matrix (the partials hold the tiles on
// and above the diagonal; the lower triangle is mirrored)
__global__ void k_sum_gram(const Mat* __restrict__ mats, int side) {
  const Mat& M = mats[blockIdx.y];
  const int64_t n = M.Kr * M.Kr;
  double* G = side ? M.GV : M.GU;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e / M.Kr, j = e - i * M.Kr;
    const int64_t src = (i > j) ? j * M.Kr + i : e;
    double acc = 0.0;
    for (int z = 0; z < kSlabs; ++z) acc = acc + M.GUp[(int64_t)z * n + src];
    G[e] = acc;
  }
}

// bf16 hi/lo split of U_perp Sigma (side 0) or V_perp (side 1) for every matrix
__global__ void k_split_mats(const Mat* __restrict__ mats, int side) {
  const Mat& M = mats[blockIdx.y];
  const int64_t rows = side ? M.C : M.R;
  const double* src = side ? M.Vp : M.Up;
  uint16_t* hi = side ? M.bh : M.ah;
  uint16_t* lo = side ? M.bl : M.al;
  const int64_t total = rows * M.ldk;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / M.ldk, c = e - r * M.ldk;
    float v = 0.0f;
    if (c < M.Kr) v = (float)(src[r * M.Kr + c] * (side ? 1.0 : M.Sig[c]));
    const uint16_t h = bf16_rne_f32(v);
    hi[e] = h;
    lo[e] = bf16_rne_f32(v - f32_of_bf16(h));
  }
}

// ---- inverse square root of the SPD Gram matrices (coupled Newton-Schulz) ------------------------
// Higham, "Functions of Matrices" (2008), Sec. 6.7: with A = G / c scaled so that its
// spectrum lies in (0, 1], Y_0 = A, Z_0 = I and T_k = (3I - Z_k Y_k) / 2, Y_{k+1} = Y_k T_k,
// Z_{k+1} = T_k Z_k converge quadratically to A^{1/2} and A^{-1/2}.

// c = max row sum of |G| (>= the largest eigenvalue); Y = G / c; Z = I; also writes I into `eye`.
__global__ void __launch_bounds__(256) k_ns_init(const Mat* __restrict__ mats, int side) {
  __shared__ double red[256];
  const Mat& M = mats[blockIdx.x];
  const int64_t n = M.Kr;
  const double* G = side ? M.GV : M.GU;
  double* Y = M.ns[side][0];
  double* Z = M.ns[side][1];
  double* eye = M.eye;
  double* cscale = M.cs + side;
  double m = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
    double s = 0.0;
    for (int64_t j = 0; j < n; ++j) s += fabs(G[i * n + j]);
    m = fmax(m, s);
  }
  red[threadIdx.x] = m;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + o]);
    __syncthreads();
  }
  const double c = (red[0] > 0.0) ? red[0] : 1.0;
  if (threadIdx.x == 0) {
    *cscale = c;
    M.nf[side] = NsFlags{0, 0, 0, 0};
  }
  for (int64_t e = threadIdx.x; e < n * n; e += blockDim.x) {
    const double id = ((e / n) == (e % n)) ? 1.0 : 0.0;
    Y[e] = G[e] / c;
    Z[e] = id;
    eye[e] = id;
  }
}

// T = 1.5 I - 0.5 (Z Y) is formed by a GEMM with beta on a copy of I; this copies I into T.
__global__ void k_copy_jobs(double* const* dst, const double* const* src, int64_t n) {
  const double* a = src[blockIdx.y];
  double* b = dst[blockIdx.y];
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
    b[e] = a[e];
}

// After the T products of a step: last = (max |T - I| <= kNsTol) for each job still running (job
// 2 m + side, one workgroup each).
__global__ void __launch_bounds__(256) k_ns_test(const Mat* __restrict__ mats) {
  __shared__ double red[256];
  const Mat& M = mats[blockIdx.x >> 1];
  const int side = blockIdx.x & 1;
  NsFlags& f = M.nf[side];
  if (f.done) return;
  const int64_t n = M.Kr;
  const double* T = M.ns[side][4];
  double d = 0.0;
  for (int64_t e = threadIdx.x; e < n * n; e += blockDim.x)
    d = fmax(d, fabs(T[e] - (((e / n) == (e % n)) ? 1.0 : 0.0)));
  red[threadIdx.x] = d;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + o]);
    __syncthreads();
  }
  // a NaN never passes the test: the job then runs to the step limit and is flagged
  if (threadIdx.x == 0) f.last = red[0] <= kNsTol ? 1 : 0;
}

__global__ void k_ns_step_end(const Mat* __restrict__ mats, int njobs) {
  for (int j = threadIdx.x; j < njobs; j += blockDim.x) {
    NsFlags& f = mats[j >> 1].nf[j & 1];
    if (!f.done) {
      f.steps += 1;
      if (f.last) f.done = 1;
    }
  }
}

// M = Z / sqrt(c) from the buffer the job's last step wrote; a job that did not converge within
// kNsIters steps is flagged.
__global__ void __launch_bounds__(256) k_ns_finish(const Mat* __restrict__ mats, uint32_t* status) {
  const Mat& M = mats[blockIdx.x];
  const int side = blockIdx.y;
  const int64_t n = M.Kr;
  const NsFlags f = M.nf[side];
  double* Mout = side ? M.MV : M.MU;
  const double* Z = M.ns[side][2 * (f.steps & 1) + 1];
  const double inv = 1.0 / sqrt(M.cs[side]);
  for (int64_t e = threadIdx.x; e < n * n; e += blockDim.x) Mout[e] = Z[e] * inv;
  if (threadIdx.x == 0 && !f.done) flag_status(status, kStatusInternal);
}

// ---- host side ----------------------------------------------------------------------------------

struct Sizes {
  int64_t R, C, L, ldb, Kr, ldk;
};

Sizes sizes_of(const iso_tensor& t, int K, int r) {
  Sizes z;
  z.R = t.rows;
  z.C = t.cols;
  z.L = tsv_sketch_width(t.rows, t.cols, r);
  z.ldb = rup(std::max(z.R, z.C), 64);
  z.Kr = (int64_t)K * r;
  z.ldk = rup(z.Kr, 32);
  return z;
}

// bytes carved for one problem / one matrix (same sequence as carve_* below)
struct Carver {
  uint8_t* base;
  size_t off = 0;
  template <typename T>
  T* take(int64_t n) {
    T* r = (T*)(base + off);
    off = align_up(off + sizeof(T) * (size_t)std::max<int64_t>(n, 1), 256);
    return r;
  }
};

void carve_prob(Carver& cv, Prob& P, const Sizes& z) {
  for (int b = 0; b < 2; ++b) P.X[b] = cv.take<double>(z.R * z.L);
  for (int b = 0; b < 2; ++b) P.Z[b] = cv.take<double>(z.C * z.L);
  P.bh = cv.take<uint16_t>(z.L * z.ldb);
  P.bl = cv.take<uint16_t>(z.L * z.ldb);
  P.Gp = cv.take<double>((int64_t)kSlabs * z.L * z.L);
  P.G = cv.take<double>(z.L * z.L);
  P.Rf = cv.take<double>(z.L * z.L);
  P.Ri = cv.take<double>(z.L * z.L);
  P.Ra = cv.take<double>(z.L * z.L);
  P.R2 = cv.take<double>(z.L * z.L);
  P.Ja = cv.take<double>(z.L * z.L);
  P.Jv = cv.take<double>(z.L * z.L);
  P.Ut = cv.take<double>(z.L * z.L);
  P.Vt = cv.take<double>(z.L * z.L);
  P.St = cv.take<double>(z.L);
}

void carve_mat(Carver& cv, Mat& M, const Sizes& z) {
  M.U = cv.take<double>(z.R * z.ldk);
  M.V = cv.take<double>(z.C * z.ldk);
  M.Sig = cv.take<double>(z.ldk);
  M.GUp = cv.take<double>((int64_t)kSlabs * z.Kr * z.Kr);
  M.GU = cv.take<double>(z.Kr * z.Kr);
  M.GV = cv.take<double>(z.Kr * z.Kr);
  for (int sd = 0; sd < 2; ++sd)
    for (int q = 0; q < 5; ++q) M.ns[sd][q] = cv.take<double>(z.Kr * z.Kr);
  M.eye = cv.take<double>(z.Kr * z.Kr);
  M.cs = cv.take<double>(2);
  M.MU = cv.take<double>(z.Kr * z.Kr);
  M.MV = cv.take<double>(z.Kr * z.Kr);
  M.Up = cv.take<double>(z.R * z.Kr);
  M.Vp = cv.take<double>(z.C * z.Kr);
  M.ah = cv.take<uint16_t>(z.R * z.ldk);
  M.al = cv.take<uint16_t>(z.R * z.ldk);
  M.bh = cv.take<uint16_t>(z.C * z.ldk);
  M.bl = cv.take<uint16_t>(z.C * z.ldk);
}

size_t bytes_per_matrix(const Sizes& z, int K) {
  Carver cv{nullptr};
  Prob P;
  for (int i = 0; i < K; ++i) carve_prob(cv, P, z);
  Mat M;
  carve_mat(cv, M, z);
  return cv.off;
}

int chunk_matrices(const iso_tensor* t, int n_t, int K, int r) {
  size_t per = 0;
  for (int j = 0; j < n_t; ++j) per = std::max(per, bytes_per_matrix(sizes_of(t[j], K, r), K));
  if (per == 0) return std::max(n_t, 1);
  return (int)std::max<size_t>(1, std::min<size_t>((size_t)n_t, kTsvChunkBudget / per));
}

// tables uploaded per chunk
size_t table_bytes(int nm, int K) {
  const int np = nm * K;
  size_t b = 0;
  b += align_up(sizeof(Prob) * np, 256);
  b += align_up(sizeof(Mat) * nm, 256);
  b += align_up(sizeof(JacobiJob) * std::max(np, 2 * nm), 256);
  b += align_up(sizeof(double*) * 3 * np, 256);
  b += 12 * align_up(sizeof(GemmJob) * (size_t)std::max(np, kSlabs * nm * 2), 256);
  b += 2 * align_up(sizeof(double*) * 2 * nm, 256);
  b += align_up(sizeof(NsFlags) * 2 * nm, 256);
  b += align_up(sizeof(int) * 2 * (size_t)np, 256);
  return b;
}

template <int NB>
void launch_nn(const Prob* d, const int* order, int np, int64_t maxR, int out, hipStream_t s) {
  const int64_t nbx = (maxR + kSkRows - 1) / kSkRows;
  k_sk_nn<NB><<<dim3((unsigned)nbx, 1, (unsigned)np), 256, 0, s>>>(d, order, out, nbx);
}
// lo: include the lo part of B (the last product, whose values form the result)
// aligned: every delta of the chunk has C % 8 == 0 (rows start 16-byte aligned)
template <int NB>
void launch_tn(const Prob* d, const int* order, int np, int64_t maxC, int out, bool lo, bool aligned, hipStream_t s) {
  const int64_t nbx = (maxC + kSkRows - 1) / kSkRows;
  const dim3 grid((unsigned)nbx, 1, (unsigned)np);
  if (!aligned) k_sk_tn_any<NB><<<grid, 256, 0, s>>>(d, out);
  else if (lo) k_sk_tn<NB, true><<<grid, 256, 0, s>>>(d, order, out, nbx);
  else k_sk_tn<NB, false><<<grid, 256, 0, s>>>(d, order, out, nbx);
}
template <int NB>
void launch_gram(const Prob* d, int np, int which, int cur, hipStream_t s) {
  k_gram_mf<NB><<<dim3(kSlabs, (unsigned)np), 256, 0, s>>>(d, which, cur);
}
template <int NB>
void launch_apply(const Prob* d, int np, int64_t maxM, int which, int src, int dst, int split, hipStream_t s) {
  const unsigned gx = (unsigned)std::max<int64_t>(1, std::min<int64_t>((maxM + 63) / 64, 16));
  k_apply_mf<NB><<<dim3(gx, (unsigned)np), 256, 0, s>>>(d, which, src, dst, split);
}

#define DISPATCH_NB(nb, F, ...)                 \
  switch (nb) {                                 \
    case 1: F<1>(__VA_ARGS__); break;           \
    case 2: F<2>(__VA_ARGS__); break;           \
    case 3: F<3>(__VA_ARGS__); break;           \
    case 4: F<4>(__VA_ARGS__); break;           \
    case 5: F<5>(__VA_ARGS__); break;           \
    case 6: F<6>(__VA_ARGS__); break;           \
    case 7: F<7>(__VA_ARGS__); break;           \
    default: F<8>(__VA_ARGS__); break;          \
  }

}  // namespace

int tsv_sketch_width(int64_t R, int64_t C, int r) {
  const int64_t q = std::min(R, C);
  int64_t L = rup((int64_t)r + std::max<int64_t>(8, r / 2), 16);
  L = std::min<int64_t>(L, 16 * kMaxNB);
  L = std::min<int64_t>(L, q / 16 * 16);
  if (L < r || L < 16) return 0;
  return (int)L;
}

size_t tsv_workspace_bytes(const iso_tensor* t, int n_t, int K, int rank) {
  if (n_t <= 0) return 0;
  const int nm = chunk_matrices(t, n_t, K, rank);
  size_t per = 0;
  for (int j = 0; j < n_t; ++j) per = std::max(per, bytes_per_matrix(sizes_of(t[j], K, rank), K));
  return table_bytes(nm, K) + per * (size_t)nm;
}

iso_status run_tsv(const iso_tensor* t, int n_t, int K, const TsvArgs& a, uint8_t* ws, size_t ws_bytes,
                   uint32_t* status, hipStream_t s) {
#define TS_TRY(x)                                \
  do {                                           \
    if ((x) != hipSuccess) return ISO_ERR_HIP;   \
  } while (0)
  (void)ws_bytes;
  const int r = a.rank;
  const int nm_max = chunk_matrices(t, n_t, K, r);
  std::vector<uint8_t> host;
  for (int j0 = 0; j0 < n_t; j0 += nm_max) {
    const int nm = std::min(nm_max, n_t - j0);
    const int np = nm * K;
    // ---- device layout of this chunk
    Carver cv{ws};
    Prob* d_prob = cv.take<Prob>(np);
    Mat* d_mat = cv.take<Mat>(nm);
    JacobiJob* d_jobs = cv.take<JacobiJob>(std::max(np, 2 * nm));
    double** d_ptrs = cv.take<double*>(3 * np);
    GemmJob* d_gj[12];
    for (int q = 0; q < 12; ++q) d_gj[q] = cv.take<GemmJob>(std::max(np, kSlabs * nm * 2));
    const double** d_nsrc = cv.take<const double*>(2 * nm);
    double** d_ndst = cv.take<double*>(2 * nm);
    NsFlags* d_nf = cv.take<NsFlags>(2 * nm);
    int* d_ord = cv.take<int>(2 * np);
    cv.off = table_bytes(nm, K);
    std::vector<Prob> hp(np);
    std::vector<Mat> hm(nm);
    int64_t maxR = 0, maxC = 0, L = 0, Kr = (int64_t)K * r;
    for (int m = 0; m < nm; ++m) {
      const iso_tensor& tt = t[j0 + m];
      const Sizes z = sizes_of(tt, K, r);
      maxR = std::max(maxR, z.R);
      maxC = std::max(maxC, z.C);
      L = std::max(L, z.L);
      for (int i = 0; i < K; ++i) {
        Prob& P = hp[m * K + i];
        std::memset(&P, 0, sizeof P);
        carve_prob(cv, P, z);
        P.delta = (const uint16_t*)tt.deltas[i];
        P.R = z.R;
        P.C = z.C;
        P.L = z.L;
        P.ldb = z.ldb;
        P.seed = 0x5EED0000ull + ((uint64_t)(j0 + m) << 8) + (uint64_t)i;
        if (a.factors != nullptr) {
          const iso_factors& f = a.factors[(size_t)(j0 + m) * K + i];
          P.fu = f.u;
          P.fs = f.s;
          P.fv = f.v;
        }
      }
      Mat& M = hm[m];
      std::memset(&M, 0, sizeof M);
      carve_mat(cv, M, z);
      M.w0 = (const uint16_t*)tt.base;
      M.out = (uint16_t*)tt.out;
      M.dhat = a.delta_hat ? a.delta_hat[j0 + m] : nullptr;
      M.R = z.R;
      M.C = z.C;
      M.Kr = z.Kr;
      M.ldk = z.ldk;
      M.alpha = a.alpha;
      M.nf = d_nf + 2 * m;
    }
    // all problems of a chunk share L (matrices of one chunk must give the same sketch width)
    for (int p = 0; p < np; ++p)
      if (hp[p].L != L) return ISO_ERR_UNSUPPORTED;
    const int NB = (int)(L / 16);
    bool aligned = true;
    for (int p = 0; p < np; ++p) aligned = aligned && hp[p].C % 8 == 0;
    const int64_t maxM = std::max(maxR, maxC);
    // gemm job tables: 0 U_i = X Ut[:, :r]; 1 V_i = Z Vt[:, :r]; 2 GU slabs; 3 GV slabs;
    // 5 U_perp = U M_U, V_perp = V M_V; 6..11 Newton-Schulz steps (T, Y, Z) for parities 0, 1
    std::vector<GemmJob> gj[12];
    std::vector<const double*> ns_src;
    std::vector<double*> ns_dst;
    for (int p = 0; p < np; ++p) {
      const Prob& P = hp[p];
      const Mat& M = hm[p / K];
      const int i = p % K;
      gj[0].push_back(GemmJob{P.X[kXLast], P.Ut, M.U + i * r, P.L, 1, 1, P.L, M.ldk, 1, P.R, r, P.L, 1.0, 0.0});
      gj[1].push_back(GemmJob{P.Z[0], P.Vt, M.V + i * r, P.L, 1, 1, P.L, M.ldk, 1, P.C, r, P.L, 1.0, 0.0});
    }
    for (int m = 0; m < nm; ++m) {
      const Mat& M = hm[m];
      for (int z = 0; z < kSlabs; ++z) {
        const int64_t perU = (M.R + kSlabs - 1) / kSlabs, perV = (M.C + kSlabs - 1) / kSlabs;
        const int64_t u0 = std::min<int64_t>(M.R, z * perU), u1 = std::min<int64_t>(M.R, u0 + perU);
        const int64_t v0 = std::min<int64_t>(M.C, z * perV), v1 = std::min<int64_t>(M.C, v0 + perV);
        // G_z = U[u0:u1]^T U[u0:u1]: A(i,k) = U(u0+k, i)
        gj[2].push_back(GemmJob{M.U + u0 * M.ldk, M.U + u0 * M.ldk, M.GUp + (int64_t)z * M.Kr * M.Kr, 1, M.ldk,
                                M.ldk, 1, M.Kr, 1, M.Kr, M.Kr, u1 - u0, 1.0, 0.0, 1});
        gj[3].push_back(GemmJob{M.V + v0 * M.ldk, M.V + v0 * M.ldk, M.GUp + (int64_t)z * M.Kr * M.Kr, 1, M.ldk,
                                M.ldk, 1, M.Kr, 1, M.Kr, M.Kr, v1 - v0, 1.0, 0.0, 1});
      }
      // Newton-Schulz on both sides: parity a uses (Y_a, Z_a) -> (Y_b, Z_b), b = 1 - a
      const int64_t n = M.Kr;
      for (int sd = 0; sd < 2; ++sd) {
        double* const* q = M.ns[sd];
        for (int a = 0; a < 2; ++a) {
          double* Ya = q[2 * a];
          double* Za = q[2 * a + 1];
          double* Yb = q[2 * (1 - a)];
          double* Zb = q[2 * (1 - a) + 1];
          double* T = q[4];
          const int* skip = &M.nf[sd].done;
          // T = 1.5 I - Z Y / 2, Y' = Y T, Z' = T Z
          gj[6 + 3 * a].push_back(GemmJob{Za, Ya, T, n, 1, n, 1, n, 1, n, n, n, -0.5, 1.5, 0, skip});
          gj[7 + 3 * a].push_back(GemmJob{Ya, T, Yb, n, 1, n, 1, n, 1, n, n, n, 1.0, 0.0, 0, skip});
          gj[8 + 3 * a].push_back(GemmJob{T, Za, Zb, n, 1, n, 1, n, 1, n, n, n, 1.0, 0.0, 0, skip});
        }
        ns_src.push_back(M.eye);
        ns_dst.push_back(q[4]);
      }
      gj[5].push_back(GemmJob{M.U, M.MU, M.Up, M.ldk, 1, M.Kr, 1, M.Kr, 1, M.R, M.Kr, M.Kr, 1.0, 0.0});
      gj[5].push_back(GemmJob{M.V, M.MV, M.Vp, M.ldk, 1, M.Kr, 1, M.Kr, 1, M.C, M.Kr, M.Kr, 1.0, 0.0});
    }
    // upload tables (one staging buffer, kept until the chunk is done)
    const size_t tb = table_bytes(nm, K);
    host.assign(tb, 0);
    {
      Carver hc{host.data()};
      Prob* h_prob = hc.take<Prob>(np);
      Mat* h_mat = hc.take<Mat>(nm);
      hc.take<JacobiJob>(std::max(np, 2 * nm));
      double** h_ptrs = hc.take<double*>(3 * np);
      GemmJob* h_gj[12];
      for (int q = 0; q < 12; ++q) h_gj[q] = hc.take<GemmJob>(std::max(np, kSlabs * nm * 2));
      const double** h_nsrc = hc.take<const double*>(2 * nm);
      double** h_ndst = hc.take<double*>(2 * nm);
      hc.take<NsFlags>(2 * nm);
      int* h_ord = hc.take<int>(2 * np);
      // launch order of the skinny products.  Each XCD works through its own contiguous range of
      // the order; the problems, sorted by the walk of one workgroup (k = C for Delta B, k = R for
      // Delta^T B), are dealt round-robin to the eight ranges, so that each XCD gets the same mix,
      // longest first, and the short ones fill the tail.
      auto deal = [&](int* o, bool by_c) {
        std::vector<int> srt(np);
        for (int p = 0; p < np; ++p) srt[p] = p;
        std::stable_sort(srt.begin(), srt.end(), [&](int x, int y) { return by_c ? hp[x].C > hp[y].C : hp[x].R > hp[y].R; });
        int n = 0;
        for (int x = 0; x < kXcds; ++x)
          for (int j = x; j < np; j += kXcds) o[n++] = srt[j];
      };
      deal(h_ord, true);
      deal(h_ord + np, false);
      std::memcpy(h_prob, hp.data(), sizeof(Prob) * np);
      std::memcpy(h_mat, hm.data(), sizeof(Mat) * nm);
      for (int p = 0; p < np; ++p) {
        h_ptrs[p] = hp[p].Ut;
        h_ptrs[np + p] = hp[p].Vt;
        h_ptrs[2 * np + p] = hp[p].St;
      }
      for (int q = 0; q < 12; ++q)
        if (!gj[q].empty()) std::memcpy(h_gj[q], gj[q].data(), sizeof(GemmJob) * gj[q].size());
      std::memcpy(h_nsrc, ns_src.data(), sizeof(double*) * ns_src.size());
      std::memcpy(h_ndst, ns_dst.data(), sizeof(double*) * ns_dst.size());
    }
    TS_TRY(hipMemcpyAsync(ws, host.data(), tb, hipMemcpyHostToDevice, s));
    const unsigned gx = grid_for(L * rup(maxM, 64));
    // split: the last pass also writes the bf16 hi/lo operand of the next product
    auto cholqr = [&](int which, int& cur, int save_first, int accum_second, int passes, int split) {
      const int64_t mm = which ? maxC : maxR;
      for (int pass = 0; pass < passes; ++pass) {
        DISPATCH_NB(NB, launch_gram, d_prob, np, which, cur, s);
        const size_t shb = sizeof(double) * (L * L + L);
        k_chol<<<np, 256, shb, s>>>(d_prob, (pass == 0) ? save_first : 0, (pass == 1) ? accum_second : 0, status);
        DISPATCH_NB(NB, launch_apply, d_prob, np, mm, which, cur, 1 - cur, (pass == passes - 1) ? split : 0, s);
        cur = 1 - cur;
      }
    };
    if (a.factors != nullptr) {
      k_load_factors<<<dim3(grid_for(maxM * r), (unsigned)np), 256, 0, s>>>(d_prob, d_mat, K, r);
    } else {
    // 1. range finder with subspace iteration
    int cx = 0, cz = 0;
    k_omega<<<dim3(gx, np), 256, 0, s>>>(d_prob);
    // One Cholesky-QR pass for every sketch of the range finder (its next product and QR absorb
    // the rounding), Cholesky-QR2 for the factor of the last product, whose R forms the core.
    // The sketches of the range finder only have to span the dominant subspace: rounding their
    // right operand to bf16 (relative 2^-9) tilts the next iterate by about 2^-9 sigma_{r+1} /
    // sigma_r, which the following QR and product absorb; the last product, whose values form
    // the result, takes both parts (relative 2^-17).
    DISPATCH_NB(NB, launch_nn, d_prob, d_ord, np, maxR, cx, s);
    cholqr(0, cx, 0, 0, 1, 1);
    for (int it = 0; it < kPowerIters; ++it) {
      DISPATCH_NB(NB, launch_tn, d_prob, d_ord + np, np, maxC, cz, false, aligned, s);
      cholqr(1, cz, 0, 0, 1, 1);
      DISPATCH_NB(NB, launch_nn, d_prob, d_ord, np, maxR, cx, s);
      cholqr(0, cx, 0, 0, 1, 1);
    }
    // 2. B^T = Delta^T Q, its QR (R2 accumulated), SVD of the L x L core R2^T
    DISPATCH_NB(NB, launch_tn, d_prob, d_ord + np, np, maxC, cz, true, aligned, s);
    cholqr(1, cz, 1, 1, 2, 0);
    k_core_load<<<np, 256, 0, s>>>(d_prob, d_jobs);
    const size_t jlds = sizeof(double) * 2 * (size_t)L * L;
    if (jlds <= kJacobiLdsMax) k_jacobi_lds<<<np, kJacobiThreads, jlds, s>>>(d_jobs, status);
    else k_jacobi<<<np, kJacobiThreads, 0, s>>>(d_jobs, status);
    svd_finalize(d_jobs, d_ptrs, d_ptrs + np, d_ptrs + 2 * np, np, L, s);
    // U_i = Q Ut[:, :r], V_i = Q2 Vt[:, :r]: Q ends in buffer kXLast (1 + kPowerIters QR passes),
    // Q2 in buffer 0 (kPowerIters + 2 passes)
    static_assert(kPowerIters % 2 == 0, "ping-pong parity");
    if (cx != kXLast || cz != 0) return ISO_ERR_INTERNAL;
    gemm_jobs(d_gj[0], np, maxR, r, s);
    gemm_jobs(d_gj[1], np, maxC, r, s);
    k_sigma<<<np, 64, 0, s>>>(d_prob, d_mat, K, r);
    }
    // 3. Procrustes orthogonalisation of U and V: U_perp = U (U^T U)^{-1/2}
    for (int side = 0; side < 2; ++side) {
      gemm_jobs(d_gj[2 + side], kSlabs * nm, Kr, Kr, s);
      k_sum_gram<<<dim3(grid_for(Kr * Kr), (unsigned)nm), 256, 0, s>>>(d_mat, side);
      k_ns_init<<<nm, 256, 0, s>>>(d_mat, side);
    }
    // every job takes its steps in the same parity order; a converged job's products are skipped
    // and the host stops queueing steps once every job is done
    std::vector<NsFlags> hf(2 * nm);
    for (int it = 0, par = 0; it < kNsIters;) {
      for (int b = 0; b < kNsCheck && it < kNsIters; ++b, ++it, par = 1 - par) {
        k_copy_jobs<<<dim3(grid_for(Kr * Kr), (unsigned)(2 * nm)), 256, 0, s>>>(d_ndst, d_nsrc, Kr * Kr);
        gemm_jobs(d_gj[6 + 3 * par], 2 * nm, Kr, Kr, s);
        k_ns_test<<<(unsigned)(2 * nm), 256, 0, s>>>(d_mat);
        gemm_jobs(d_gj[7 + 3 * par], 2 * nm, Kr, Kr, s);
        gemm_jobs(d_gj[8 + 3 * par], 2 * nm, Kr, Kr, s);
        k_ns_step_end<<<1, 256, 0, s>>>(d_mat, 2 * nm);
      }
      bool all = true;
      TS_TRY(hipMemcpyAsync(hf.data(), d_nf, sizeof(NsFlags) * 2 * nm, hipMemcpyDeviceToHost, s));
      TS_TRY(hipStreamSynchronize(s));
      for (int j = 0; j < 2 * nm; ++j) all = all && hf[j].done;
      if (all) break;
    }
    k_ns_finish<<<dim3((unsigned)nm, 2), 256, 0, s>>>(d_mat, status);
    gemm_jobs(d_gj[5], 2 * nm, maxM, Kr, s);
    // 4. reconstruction with the update fused
    k_split_mats<<<dim3(grid_for(maxR * rup(Kr, 32)), (unsigned)nm), 256, 0, s>>>(d_mat, 0);
    k_split_mats<<<dim3(grid_for(maxC * rup(Kr, 32)), (unsigned)nm), 256, 0, s>>>(d_mat, 1);
    int64_t rtiles = 0;
    for (int m = 0; m < nm; ++m) rtiles = std::max(rtiles, ((hm[m].R + kRecT - 1) / kRecT) * ((hm[m].C + kRecT - 1) / kRecT));
    k_mfma_recon<<<(unsigned)(rtiles * nm), 256, 0, s>>>(d_mat, rtiles);
    TS_TRY(hipGetLastError());
    TS_TRY(hipStreamSynchronize(s));
  }
  return ISO_OK;
#undef TS_TRY
}

}  // namespace iso
