// Single-read TIES (App. F: TopKMask trim, sign election, disjoint mean) fused with the
// update theta_0 + lambda*tau, for bf16 tensors.
//
// TopKMask needs the k-th largest magnitude of a whole delta before any of its coordinates
// can be merged.  The two-pass path reads every delta twice (histogram, then merge); this
// path reads each delta and the base once:
//   1. sample (one workgroup per delta): the exact key histogram of the whole delta when it
//      holds at most 2^20 entries, else of 4096 evenly spaced 256-entry blocks (2^20 entries).  From it a bracket [lo, hi]
//      of keys that holds the threshold with a binomial margin (5 standard deviations of
//      the sample rank, plus 2) and a provisional threshold prov;
//   2. main pass: a key above hi is kept, a key below lo is not; a nonzero key inside the
//      bracket is kept provisionally if key >= prov and its coordinate is logged as a
//      record (index, tensor, delta and base bits).  Every coordinate is merged and written
//      once.  Per tile and delta: the count of keys above hi and of each bracket code;
//   3. reduce + resolve: the exact threshold code, the count above it and the tie quota;
//      the tie cutoff (lowest flat indices first) from the per-tile counts and the records,
//      which hold every entry with the threshold code;
//   4. fix-up: records whose final mask differs from the provisional one are merged again
//      and rewritten where the result changes.
// A threshold outside its bracket (a misleading sample), a bracket wider than kFusedMaxW
// codes or a full record region sends the tensor to the exact two-pass path (histogram
// select, then merge) on the same stream; the result is identical either way.  Zero keys
// need no decision: a kept zero adds nothing to the election or to the mean.
#include <algorithm>

#include "iso_device.h"
#include "iso_fused.h"
#include "iso_kernels.h"
#include "iso_merge_math.h"

namespace iso {

namespace {

constexpr int kThreads = 256;
constexpr int kVPT = 2;                          // 16-byte vectors per thread per array in one tile
constexpr int64_t kTileElems = (int64_t)kThreads * kVPT * 8;
constexpr int kSampleSpan = 256;                 // entries per sampled block
constexpr int kSampleBlocks = 4096;              // sampled blocks per delta (1M entries)
constexpr int64_t kExactMax = 1ll << 20;         // deltas up to this size (the sample's) are histogrammed whole
constexpr double kMarginSd = 5.0;
constexpr int kBins = 1 << 15;

constexpr int kFlagWide = 1, kFlagFull = 2, kFlagMiss = 4;   // reasons, OR-ed into tflag

__device__ __forceinline__ uint32_t bkey(uint32_t b) { return b & 0x7FFFu; }

template <int K>
constexpr int kTileCapK = (K <= 4) ? (int)(kTileElems / 16) : (int)(kTileElems / 8);   // records per tile

template <int K>
constexpr int rec_words() {
  return ((2 * (K + 4) + 15) / 16) * 4;          // u32 index, u16 tensor, K+1 bf16 values; 16-byte units
}

__device__ __forceinline__ uint32_t lane_half(const uint4& v, int e) {
  const uint32_t w = (e < 2) ? v.x : (e < 4) ? v.y : (e < 6) ? v.z : v.w;
  return (e & 1) ? (w >> 16) : (w & 0xFFFFu);
}

// Inclusive prefix sum over the block (blockDim.x multiple of 64, at most 1024); sh[16]
// receives the block total.
__device__ int64_t block_scan(int64_t v, int64_t* sh /* >= 17 */) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int64_t x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  __syncthreads();                               // sh may still be read from the previous call
  if (lane == 63) sh[wid] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t run = 0;
    for (int w = 0; w < nw; ++w) { const int64_t t = sh[w]; sh[w] = run; run += t; }
    sh[16] = run;
  }
  __syncthreads();
  return x + sh[wid];
}

// ---- 0. per-call state -------------------------------------------------------------------------

__global__ void k_fs_init(const DevTensor* __restrict__ tab, int n_t, int K, FusedUnit* __restrict__ fu,
                          int* __restrict__ tflag) {
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u < n_t) tflag[u] = 0;
  if (u >= n_t * K) return;
  const DevTensor& T = tab[u / K];
  FusedUnit f;
  f.flags = (T.k == 0) ? kFusedNone : ((T.k == T.n) ? kFusedAll : 0u);
  if (f.flags & kFusedNone) f.lo = f.hi = f.prov = 0x8000u;   // above every key: nothing kept
  else f.lo = f.hi = f.prov = 0u;                            // k == n: every nonzero key is above
  f.t_key = 0;
  f.pad = 0;
  f.k = T.k;
  f.kept = 0;
  f.n_above = f.quota = f.count_t = 0;
  f.cutoff = T.n;
  for (int c = 0; c < kFusedMaxW; ++c) f.h[c] = 0;
  fu[u] = f;
}

// ---- 1. sample and bracket (one workgroup per delta) -------------------------------------------

__global__ void __launch_bounds__(1024) k_fs_sample(const DevTensor* __restrict__ tab, int K,
                                                    FusedUnit* __restrict__ fu, int* __restrict__ tflag) {
  __shared__ uint32_t bins[kBins];
  __shared__ int64_t sh[17];
  __shared__ int32_t found[3];
  const int u = blockIdx.x;
  const int j = u / K, i = u % K;
  const DevTensor& T = tab[j];
  if (fu[u].flags & (kFusedNone | kFusedAll)) return;
  for (int b = threadIdx.x; b < kBins; b += blockDim.x) bins[b] = 0;
  if (threadIdx.x < 3) found[threadIdx.x] = -1;
  __syncthreads();
  const int64_t n = T.n;
  const uint4* pv = (const uint4*)T.deltas[i];
  const bool exact = n <= kExactMax;
  auto count8 = [&](const uint4& a) {
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const uint32_t k0 = w[h] & 0x7FFFu, k1 = (w[h] >> 16) & 0x7FFFu;
      if (k0) atomicAdd(&bins[k0], 1u);
      if (k1) atomicAdd(&bins[k1], 1u);
    }
  };
  // kInFlight 16-byte loads per thread before any is counted: one workgroup per CU (the
  // histogram takes 128 KB of LDS), so the loads in flight set the rate
  constexpr int kInFlight = 16;
  int64_t ns;
  if (exact) {
    const int64_t nvec = n / 8;
    for (int64_t v = threadIdx.x; v < nvec; v += kInFlight * (int64_t)blockDim.x) {
      uint4 a[kInFlight];
#pragma unroll
      for (int q = 0; q < kInFlight; ++q) {
        const int64_t vv = v + q * (int64_t)blockDim.x;
        a[q] = (vv < nvec) ? ld_stream(pv + vv) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int q = 0; q < kInFlight; ++q) count8(a[q]);   // the zero fill adds nothing
    }
    const uint16_t* p = (const uint16_t*)T.deltas[i];
    for (int64_t e = nvec * 8 + threadIdx.x; e < n; e += blockDim.x) {
      const uint32_t k = bkey(p[e]);
      if (k) atomicAdd(&bins[k], 1u);
    }
    ns = n;
  } else {
    // block b starts at entry floor(b * nb / kSampleBlocks) * kSampleSpan, nb = n / kSampleSpan
    // (n > kExactMax, so the blocks are distinct); 32 threads, one 16-byte vector each, per block
    const int64_t nb = n / kSampleSpan;
    constexpr int kVecPerBlock = kSampleSpan / 8;
    const int per_iter = blockDim.x / kVecPerBlock;
    const int lb = threadIdx.x / kVecPerBlock, lv = threadIdx.x % kVecPerBlock;
    for (int b0 = 0; b0 < kSampleBlocks; b0 += kInFlight * per_iter) {
      uint4 a[kInFlight];
#pragma unroll
      for (int q = 0; q < kInFlight; ++q) {
        const int b = b0 + q * per_iter + lb;
        if (b < kSampleBlocks) {
          const int64_t blk = (int64_t)b * nb / kSampleBlocks;
          a[q] = ld_stream(pv + blk * kVecPerBlock + lv);
        } else {
          a[q] = make_uint4(0, 0, 0, 0);
        }
      }
#pragma unroll
      for (int q = 0; q < kInFlight; ++q) count8(a[q]);
    }
    ns = (int64_t)kSampleBlocks * kSampleSpan;
  }
  __syncthreads();
  // thread t owns bins [32t, 32t + 32); sample keys above its range = total - inclusive prefix
  constexpr int kPer = kBins / 1024;
  int64_t mine = 0;
  if (threadIdx.x < kBins / kPer)
    for (int q = 0; q < kPer; ++q) mine += bins[threadIdx.x * kPer + q];
  const int64_t incl = block_scan(mine, sh);
  const int64_t total = sh[16];
  // sample ranks (1-based, from the largest key) of the bracket ends and of the estimate
  const int64_t k = fu[u].k;
  int64_t want[3];
  bool top_open = false;
  if (exact) {
    want[0] = want[1] = want[2] = k;
  } else {
    const double p = (double)k / (double)n;
    const double rhat = p * (double)ns;
    const double sd = sqrt((double)ns * p * (1.0 - p));
    const double r_hi = floor(rhat - kMarginSd * sd) - 2.0;
    const double r_lo = ceil(rhat + kMarginSd * sd) + 2.0;
    top_open = r_hi < 1.0;                        // the sample cannot bound the threshold from above
    want[0] = top_open ? 1 : (int64_t)r_hi;
    want[1] = (int64_t)fmin(r_lo, (double)ns);
    want[2] = max<int64_t>(1, (int64_t)llround(rhat));
  }
  if (threadIdx.x < kBins / kPer) {
    int64_t run = total - incl;
    for (int q = kPer - 1; q >= 0; --q) {
      const int code = threadIdx.x * kPer + q;
      const int64_t c = bins[code];
#pragma unroll
      for (int r = 0; r < 3; ++r)
        if (c > 0 && run < want[r] && run + c >= want[r]) found[r] = code;
      run += c;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    // a rank past the sample's nonzero keys falls among the zeros: code 0
    const uint32_t hi = top_open ? 0x7FFFu : (uint32_t)max(found[0], 0);
    const uint32_t lo = (uint32_t)max(found[1], 0);
    const uint32_t est = (uint32_t)max(found[2], 0);
    FusedUnit& F = fu[u];
    F.lo = lo;
    F.hi = max(hi, lo);
    F.prov = max(lo, min(F.hi, est));
    if (F.hi - lo + 1u > (uint32_t)kFusedMaxW) atomicOr(&tflag[j], kFlagWide);
  }
}

// ---- 2. main pass --------------------------------------------------------------------------------
//
// The pass is bound by vector ALU issue more than by HBM, so the per-delta work runs on pairs
// of bf16 coordinates in packed 16-bit integer lanes: kept flag, kept value, counts of kept
// and of negative kept entries, bracket membership and key maxima, two coordinates per
// instruction.  The kept values are summed in binary32 (S = sum x, A = sum |x|); that is
// exact for a coordinate whenever A < 2^(E + 17), E the exponent of the smallest key that
// can be kept here (all partial sums are then multiples of 2^(E - 7) below 2^(E + 17)), and
// a thread with any coordinate outside that bound redoes its coordinates in the general
// binary64 form.  The mean t = RN64(ts / n) of the agreeing sum ts over n entries is formed
// branch-free from D = 2 ts as q = D * r, rem = fma(-q, 2n, D), t = fma(rem, r, q) with
// r = RN64(1/n) / 2: the remainder is exact and the correction gives the correctly rounded
// quotient (Markstein, IBM J. Res. Dev. 34(1), 1990); for n a power of two q is already
// exact.  Halving r and doubling the divisor scale every step by exactly 1/2.

typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
typedef int16_t i16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u16x2 as_u2(uint32_t w) { return __builtin_bit_cast(u16x2, w); }
__device__ __forceinline__ uint32_t as_w(u16x2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ uint32_t pk_add(uint32_t a, uint32_t b) { return as_w(as_u2(a) + as_u2(b)); }
__device__ __forceinline__ uint32_t pk_sub(uint32_t a, uint32_t b) { return as_w(as_u2(a) - as_u2(b)); }
__device__ __forceinline__ uint32_t pk_sign_fill(uint32_t a) {   // 0xFFFF in each half whose bit 15 is set
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(i16x2, a) >> (i16x2){15, 15});
}
__device__ __forceinline__ uint32_t pk_bit15(uint32_t a) { return as_w(as_u2(a) >> (u16x2){15, 15}); }
__device__ __forceinline__ uint32_t pk_min(uint32_t a, uint32_t b) {
  return as_w(__builtin_elementwise_min(as_u2(a), as_u2(b)));
}
__device__ __forceinline__ uint32_t pk_max(uint32_t a, uint32_t b) {
  return as_w(__builtin_elementwise_max(as_u2(a), as_u2(b)));
}
__device__ __forceinline__ uint32_t pk_subsat(uint32_t a, uint32_t b) {
  return as_w(__builtin_elementwise_sub_sat(as_u2(a), as_u2(b)));
}
__device__ __forceinline__ int lo_s16(uint32_t w) { return (int)(int16_t)(w & 0xFFFFu); }
__device__ __forceinline__ int hi_s16(uint32_t w) { return (int)(int16_t)(w >> 16); }
__device__ __forceinline__ uint32_t word_of(const uint4& v, int h) {
  return (h == 0) ? v.x : (h == 1) ? v.y : (h == 2) ? v.z : v.w;
}

// Workgroup barrier that orders LDS only: outstanding global loads and stores stay in flight
// (the main pass never reads global data another thread of the block wrote).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Inclusive prefix sum over a wave64 with DPP row shifts and row broadcasts (no LDS).
__device__ __forceinline__ uint32_t wave_scan_u32(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, true);   // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, true);   // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, true);   // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, true);   // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15 -> rows 1, 3
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31 -> rows 2, 3
  return x;
}

// Provisional threshold of a delta in the main pass: kept iff key >= prov_key.
__device__ __forceinline__ uint32_t prov_key(const FusedUnit& F) {
  return (F.flags & kFusedNone) ? 0x8000u : max(F.prov, 1u);
}

// One pair of coordinates (word h of the K deltas' vectors w and of the base wb): provisional
// TopKMask (ms: 0xFFFF where not kept), elected sign, disjoint mean and theta_0 + lambda t;
// Sv, Av: the binary32 sums S and A; o32: each result as binary32 bits, which round-to-nearest-
// even to bf16 turns into the output.  The reference value is v = RN64(w0 + t) with
// t = RN64(lambda RN64(D / 2cnt)).
//   EXACT: that binary64 sequence, rounded to binary32 with round-to-odd, after which the bf16
//   rounding is the correct one of v.
//   Otherwise round-to-nearest-even to binary32, which gives the same bf16 unless the binary32
//   result has low half 0x8000: bf16 values and the midpoints between them are binary32 values,
//   and rounding is monotone, so a result that is not such a midpoint lies strictly on the same
//   side of every midpoint as v.  With lambda = 1 and cnt a power of two, D / 2cnt is exact and
//   one binary32 fma gives RN32(w0 + t) from the exact sum (the same midpoint argument covers
//   v, which is within half a binary64 ulp of that sum); other counts (3, 5, 6, 7) read NaN from
//   the table and go to EXACT.
// Returns true when the pair is to be redone with EXACT (rare).
template <int K, bool LAM1, bool EXACT>
__device__ __forceinline__ bool merge_pair(const uint32_t (&w)[K], uint32_t wb, const uint32_t (&p1x2)[K],
                                           const double2* rtab, const float* rtab32, double lambda,
                                           uint32_t (&ms)[K], float (&Sv)[2], float (&Av)[2], uint32_t (&o32)[2]) {
  uint32_t nk = 0, nn = 0;
  float S0 = 0.0f, S1 = 0.0f, A0 = 0.0f, A1 = 0.0f;
#pragma unroll
  for (int i = 0; i < K; ++i) {
    const uint32_t key = w[i] & 0x7FFF7FFFu;
    ms[i] = pk_sign_fill(pk_sub(key, p1x2[i]));   // 0xFFFF: not kept
    const uint32_t wk = w[i] & ~ms[i];
    nk = pk_add(nk, ms[i]);
    nn = pk_add(nn, pk_bit15(wk));
    const float x0 = __uint_as_float(wk << 16), x1 = __uint_as_float(wk & 0xFFFF0000u);
    if (i == 0) {
      S0 = x0; S1 = x1; A0 = fabsf(x0); A1 = fabsf(x1);
    } else {
      S0 = S0 + x0; S1 = S1 + x1; A0 = A0 + fabsf(x0); A1 = A1 + fabsf(x1);
    }
  }
  // agreeing count if the elected sign is +: kept (K + nk) less negative, both halves
  const uint32_t npos = pk_sub(pk_add(nk, (uint32_t)K | ((uint32_t)K << 16)), nn);
  Sv[0] = S0; Sv[1] = S1; Av[0] = A0; Av[1] = A1;
  bool redo = false;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const float S = c ? S1 : S0, A = c ? A1 : A0;
    uint32_t cnt = (S < 0.0f) ? (c ? (nn >> 16) : (nn & 0xFFFFu)) : (c ? (npos >> 16) : (npos & 0xFFFFu));
    // D = S + gamma * A is twice the agreeing sum (exact).  With S = 0 no sign is elected:
    // entry 0 of the tables (zeros) gives t = +0 for any finite D
    cnt = (S != 0.0f) ? cnt : 0u;
    const float D = S + copysignf(A, S);
    const float w0 = __uint_as_float(c ? (wb & 0xFFFF0000u) : (wb << 16));
    if (EXACT || !LAM1) {
      const double d64 = (double)D;
      const double2 rn = rtab[cnt];
      const double qd = d64 * rn.x;
      const double rem = fma(-qd, rn.y, d64);
      double t = fma(rem, rn.x, qd);
      if (!LAM1) t = lambda * t;
      const double v = (double)w0 + t;
      o32[c] = EXACT ? f64_to_f32_odd_bits(v) : __float_as_uint((float)v);
    } else {
      const float sv = fmaf(D, rtab32[cnt], w0);
      o32[c] = __float_as_uint(sv);
      redo |= !(sv == sv);
    }
    if (!EXACT) redo |= (uint16_t)o32[c] == 0x8000u;
  }
  return redo;
}

struct MainArgs {
  const DevTensor* tab;
  const int* tmap;
  int n_t;
  const FusedUnit* fu;
  int* tflag;
  uint16_t* tstat;
  uint32_t one2;           // 0x00010001, passed in so that min(d, 1) stays one packed min
  uint2* tinfo;
  uint32_t* rec;
  int64_t tile_cap;
  double lambda;
  uint32_t* status;
};

// Up to K = 4 the pass fits 96 VGPRs without spilling: five waves per SIMD instead of four,
// which is what keeps enough loads in flight (the waves' lifetimes are latency-bound).
// LAM1: lambda = 1 (no product); SIGN: the elected signs are written too.
template <int K, bool LAM1, bool SIGN>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(K <= 4 ? 5 : 1)))
k_fs_main(MainArgs a) {
  constexpr int RW = rec_words<K>();
  __shared__ uint32_t hcnt[K][kFusedMaxW];
  __shared__ uint32_t s_kept[K][kThreads / 64];
  __shared__ uint32_t s_wtot[kThreads / 64];
  __shared__ double2 rtab[K + 1];                   // {RN(1/n) / 2, 2n}
  __shared__ float rtab32[K + 1];                   // 1 / 2n for n a power of two, else NaN; 0 for n = 0
  // the tile's deferred coordinates as staged, one array per word: the K delta words and the
  // base word of the coordinate's pair, then its offset in the tile (bit 0: which half).  Word
  // arrays (not one record per slot) so that every word is stored from the register it is in.
  __shared__ uint32_t s_raw[K + 2][kTileCapK<K> + 1];
  __shared__ int s_skip, s_redo;
  const int64_t tile = blockIdx.x;
  const int j = find_tensor_mapped(a.tab, a.tmap, a.n_t, tile);
  const DevTensor& T = a.tab[j];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  // the stream loads first: nothing below delays their issue
  const int64_t n = T.n, nvec = n / 8;
  const int64_t vbeg = (tile - T.tile0) * (int64_t)(kThreads * kVPT);
  // every vector of the tile whole (all tiles but a tensor's last): the addresses are a uniform
  // tile base plus the thread's 32-bit offset
  const bool full = vbeg + kThreads * kVPT <= nvec;
  uint4 dv[kVPT][K], wv[kVPT];
  int nv[kVPT];                                    // valid elements in this thread's vector q
  if (full) {
#pragma unroll
    for (int q = 0; q < kVPT; ++q) {
      nv[q] = 8;
      const int64_t v0 = vbeg + (int64_t)q * kThreads;
#pragma unroll
      for (int i = 0; i < K; ++i) dv[q][i] = ld_stream(((const uint4*)T.deltas[i] + v0) + threadIdx.x);
      wv[q] = ld_stream(((const uint4*)T.base + v0) + threadIdx.x);
    }
  } else {
#pragma unroll
  for (int q = 0; q < kVPT; ++q) {
    const int64_t vi = vbeg + (int64_t)q * kThreads + threadIdx.x;
    nv[q] = (vi < nvec) ? 8 : (int)max<int64_t>(0, min<int64_t>(8, n - vi * 8));
    if (vi < nvec) {
#pragma unroll
      for (int i = 0; i < K; ++i) dv[q][i] = ld_stream((const uint4*)T.deltas[i] + vi);
      wv[q] = ld_stream((const uint4*)T.base + vi);
    } else {
      uint32_t tmp[K + 1][4];
#pragma unroll
      for (int i = 0; i <= K; ++i)
        for (int h = 0; h < 4; ++h) tmp[i][h] = 0;
      for (int e = 0; e < nv[q]; ++e) {
        const int64_t idx = vi * 8 + e;
#pragma unroll
        for (int i = 0; i < K; ++i) tmp[i][e >> 1] |= (uint32_t)((const uint16_t*)T.deltas[i])[idx] << (16 * (e & 1));
        tmp[K][e >> 1] |= (uint32_t)((const uint16_t*)T.base)[idx] << (16 * (e & 1));
      }
#pragma unroll
      for (int i = 0; i < K; ++i) dv[q][i] = make_uint4(tmp[i][0], tmp[i][1], tmp[i][2], tmp[i][3]);
      wv[q] = make_uint4(tmp[K][0], tmp[K][1], tmp[K][2], tmp[K][3]);
    }
  }
  }
  // another block may flag this tensor while this one runs: one read, shared by the block
  if (threadIdx.x == 0) {
    s_skip = a.tflag[j];
    s_redo = 0;
  }
  if (threadIdx.x <= K) {
    const unsigned n1 = threadIdx.x;
    const double nn = (double)n1;
    rtab[n1] = (n1 == 0) ? make_double2(0.0, 0.0) : make_double2(0.5 / nn, 2.0 * nn);
    rtab32[n1] = (n1 == 0) ? 0.0f : ((n1 & (n1 - 1)) == 0 ? 0.5f / (float)n1 : __uint_as_float(0x7FC00000u));
  }
  for (int e = threadIdx.x; e < K * kFusedMaxW; e += kThreads) hcnt[e / kFusedMaxW][e % kFusedMaxW] = 0;
  // per-delta constants (two 16-bit copies): provisional key, bracket start and width - 1
  uint32_t p1x2[K], lo1x2[K], wm1x2[K], lo1[K], hi1[K], lo0[K];
  uint32_t emin = 0xFFu;
#pragma unroll
  for (int i = 0; i < K; ++i) {
    const FusedUnit& F = a.fu[j * K + i];
    const uint32_t p1 = prov_key(F);
    p1x2[i] = p1 | (p1 << 16);
    const uint32_t l1 = max(F.lo, 1u);
    const bool br = !(F.flags & (kFusedNone | kFusedAll)) && F.hi >= l1;
    lo0[i] = F.lo;
    lo1[i] = br ? l1 : 0x8000u;                    // 0x8000: no key is inside
    hi1[i] = br ? F.hi : 0u;
    lo1x2[i] = lo1[i] | (lo1[i] << 16);
    wm1x2[i] = br ? ((F.hi - l1) | ((F.hi - l1) << 16)) : 0u;
    if (!(F.flags & kFusedNone)) emin = min(emin, p1 >> 7);
  }
  const int ebound = (int)max(emin, 1u) - 127 + 17;             // A < 2^ebound: binary32 sums exact
  const uint32_t abound = (ebound >= 128) ? 0x7F800000u : ((uint32_t)(ebound + 127) << 23);
  // deferred coordinates: some nonzero key inside its delta's bracket (a zero half of dm)
  uint32_t dm[kVPT][4];
  uint32_t ndef[kVPT];
#pragma unroll
  for (int q = 0; q < kVPT; ++q) {
    uint32_t nd = 0;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      uint32_t d = 0xFFFFFFFFu;
#pragma unroll
      for (int i = 0; i < K; ++i) {
        const uint32_t key = word_of(dv[q][i], h) & 0x7FFF7FFFu;
        d = pk_min(d, pk_subsat(pk_sub(key, lo1x2[i]), wm1x2[i]));
      }
      dm[q][h] = d;
      nd = __builtin_amdgcn_sad_u16(pk_min(d, a.one2), 0u, nd);   // + nonzero halves
    }
    ndef[q] = 8u - nd;
  }
  // record slots: flat index order inside the tile (vector q, then thread, then element)
  static_assert(kVPT == 2, "the record scan packs two vector counts");
  const uint32_t packed = ndef[0] | (ndef[1] << 16);
  const uint32_t inc = wave_scan_u32(packed);
  if (lane == 63) s_wtot[wid] = inc;
  lds_barrier();                                 // s_skip, rtab, hcnt, s_wtot
  if (s_skip) {                                    // the whole tensor takes the two-pass path
    if (threadIdx.x == 0) a.tinfo[tile] = make_uint2(0u, 0u);
    return;
  }
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) {
    const uint32_t t = s_wtot[w];
    if (w < wid) before += t;
    tot += t;
  }
  const uint32_t tot0 = tot & 0xFFFFu, total = tot0 + (tot >> 16);
  const uint32_t excl = inc - packed + before;
  const bool rec_ok = total <= (uint32_t)a.tile_cap;
  if (threadIdx.x == 0) {
    a.tinfo[tile].x = rec_ok ? total : 0u;
    if (!rec_ok) atomicOr(&a.tflag[j], kFlagFull);
  }
  if (rec_ok) {
    // stage each deferred coordinate: the raw words of its pair (no VALU work on them) and its
    // offset; the record itself is built when the staged slots are written out, by the few
    // lanes that cover the tile's records
#pragma unroll
    for (int q = 0; q < kVPT; ++q) {
      uint32_t slot = (q == 0) ? (excl & 0xFFFFu) : tot0 + (excl >> 16);
      const uint32_t lofs = (uint32_t)(q * kThreads + threadIdx.x) * 8u;
#pragma unroll
      for (int h = 0; h < 4; ++h) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const bool def = ((dm[q][h] >> (16 * c)) & 0xFFFFu) == 0u;
          if (def) {                               // rare per lane: waves with no such lane skip the site
#pragma unroll
            for (int i = 0; i < K; ++i) s_raw[i][slot] = word_of(dv[q][i], h);
            s_raw[K][slot] = word_of(wv[q], h);
            s_raw[K + 1][slot] = lofs + (uint32_t)(2 * h + c);
            ++slot;
          }
        }
      }
    }
  }
  // merge every coordinate with the provisional masks
  const double lambda = a.lambda;
  uint32_t kc[K];                                  // per delta: minus the entries not kept (packed)
#pragma unroll
  for (int i = 0; i < K; ++i) kc[i] = 0;
  uint32_t bmax = 0, amax = 0;
#pragma unroll
  for (int q = 0; q < kVPT; ++q) {
    uint32_t ob[4];
    uint32_t sg[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      uint32_t w[K], ms[K], o32[2];
      float Sv[2], Av[2];
#pragma unroll
      for (int i = 0; i < K; ++i) w[i] = word_of(dv[q][i], h);
      const uint32_t wb = word_of(wv[q], h);
      if (merge_pair<K, LAM1, false>(w, wb, p1x2, rtab, rtab32, lambda, ms, Sv, Av, o32))   // rare
        merge_pair<K, LAM1, true>(w, wb, p1x2, rtab, rtab32, lambda, ms, Sv, Av, o32);
#pragma unroll
      for (int i = 0; i < K; ++i) kc[i] = pk_add(kc[i], ms[i]);
      bmax = pk_max(bmax, wb & 0x7FFF7FFFu);
      amax = max(amax, max(__float_as_uint(Av[0]), __float_as_uint(Av[1])));
      ob[h] = pack_bf16_rne(o32[0], o32[1]);
      if (SIGN) {
        uint32_t s2 = 0;
#pragma unroll
        for (int c = 0; c < 2; ++c) s2 |= (Sv[c] > 0.0f ? 0x01u : (Sv[c] < 0.0f ? 0xFFu : 0x00u)) << (8 * c);
        sg[h] = s2;
      }
    }
    const int64_t vi = vbeg + (int64_t)q * kThreads + threadIdx.x;
    if (full) {
      st_stream(make_uint4(ob[0], ob[1], ob[2], ob[3]), ((uint4*)T.out + (vbeg + (int64_t)q * kThreads)) + threadIdx.x);
      if (SIGN) *((uint2*)T.aux2 + vi) = make_uint2(sg[0] | (sg[1] << 16), sg[2] | (sg[3] << 16));
    } else if (nv[q] == 8) {
      st_stream(make_uint4(ob[0], ob[1], ob[2], ob[3]), (uint4*)T.out + vi);
      if (SIGN) *((uint2*)T.aux2 + vi) = make_uint2(sg[0] | (sg[1] << 16), sg[2] | (sg[3] << 16));
    } else {
      for (int e = 0; e < nv[q]; ++e) {
        const uint32_t ow = (e < 2) ? ob[0] : (e < 4) ? ob[1] : (e < 6) ? ob[2] : ob[3];
        const uint32_t sw = (e < 2) ? sg[0] : (e < 4) ? sg[1] : (e < 6) ? sg[2] : sg[3];
        ((uint16_t*)T.out)[vi * 8 + e] = (uint16_t)((e & 1) ? (ow >> 16) : ow);
        if (SIGN) ((int8_t*)T.aux2)[vi * 8 + e] = (int8_t)((e & 1) ? (sw >> 8) : sw);
      }
    }
  }
  if ((bmax & 0xFFFFu) >= 0x7F80u || (bmax >> 16) >= 0x7F80u) flag_status(a.status, kStatusNonFinite);
  // binary32 sums that may have rounded, or a non-finite kept delta (every non-finite key lies
  // above a finite threshold): the fix-up redoes the tile in binary64 and checks its inputs
  if (amax >= abound) s_redo = 1;
  // tile statistics: provisionally kept entries and bracket counts per delta
#pragma unroll
  for (int i = 0; i < K; i += 2) {                 // two deltas per reduction (16-bit halves, <= 1024 each)
    uint32_t x = (uint32_t)(16 + lo_s16(kc[i]) + hi_s16(kc[i]));
    if (i + 1 < K) x |= (uint32_t)(16 + lo_s16(kc[i + 1 < K ? i + 1 : i]) + hi_s16(kc[i + 1 < K ? i + 1 : i])) << 16;
    x = wave_scan_u32(x);                          // lane 63 holds the wave total
    if (lane == 63) {
      s_kept[i][wid] = x & 0xFFFFu;
      if (i + 1 < K) s_kept[i + 1 < K ? i + 1 : i][wid] = x >> 16;
    }
  }
  lds_barrier();                                 // staged records, s_kept, s_redo
  if (threadIdx.x == 0) a.tinfo[tile].y = (uint32_t)s_redo;
  if (rec_ok) {
    uint4* dst = (uint4*)(a.rec + (size_t)tile * a.tile_cap * RW);
    const uint32_t ibase = (uint32_t)(vbeg * 8);
    for (uint32_t r = threadIdx.x; r < total; r += kThreads) {
      // the record: halfwords 0-1 index, 2 tensor, 3 + x value x (deltas, then the base), each
      // value taken from half c of its pair word with one byte permute
      uint32_t v[K + 1];
#pragma unroll
      for (int x = 0; x <= K; ++x) v[x] = s_raw[x][r];
      const uint32_t off = s_raw[K + 1][r], c = off & 1u;
      const uint32_t sel_lo = c ? 0x07060100u : 0x05040100u;   // half c of word 0 over the tensor id
      const uint32_t sel_pr = c ? 0x07060302u : 0x05040100u;   // half c of two words
      uint32_t wds[RW];
#pragma unroll
      for (int z = 0; z < RW; ++z) wds[z] = 0;
      wds[0] = ibase + off;
      wds[1] = __builtin_amdgcn_perm(v[0], (uint32_t)j, sel_lo);
#pragma unroll
      for (int z = 2; z < RW; ++z) {
        const int x0 = 2 * z - 3, x1 = 2 * z - 2;
        if (x1 <= K)
          wds[z] = __builtin_amdgcn_perm(v[x1], v[x0], sel_pr);
        else if (x0 <= K)
          wds[z] = c ? (v[x0] >> 16) : (v[x0] & 0xFFFFu);
      }
#pragma unroll
      for (int z = 0; z < RW / 4; ++z)
        dst[r * (RW / 4) + z] = make_uint4(wds[4 * z], wds[4 * z + 1], wds[4 * z + 2], wds[4 * z + 3]);
#pragma unroll
      for (int i = 0; i < K; ++i) {
        const uint32_t key = (wds[(3 + i) >> 1] >> (16 * ((3 + i) & 1))) & 0x7FFFu;
        if (key >= lo1[i] && key <= hi1[i])
          atomicAdd(&hcnt[i][min(key - lo0[i], (uint32_t)kFusedMaxW - 1u)], 1u);   // bracket <= kFusedMaxW codes
      }
    }
    lds_barrier();                               // hcnt complete
  }
  for (int e = threadIdx.x; e < K * kFusedStat; e += kThreads) {
    const int i = e / kFusedStat, c = e % kFusedStat;
    uint32_t v;
    if (c == 0) {
      v = 0;
      for (int w = 0; w < kThreads / 64; ++w) v += s_kept[i][w];
    } else {
      v = hcnt[i][c - 1];
    }
    a.tstat[(size_t)tile * fused_stat_words(K) + e] = (uint16_t)v;
  }
}

// record halfword h: 0-1 index, 2 tensor, 3..3+K-1 deltas, 3+K base
__device__ __forceinline__ uint32_t rec_half(const uint32_t* r, int h) {
  return (r[h >> 1] >> (16 * (h & 1))) & 0xFFFFu;
}

// ---- 3. reduce, resolve, tie cutoff ---------------------------------------------------------------

__device__ __forceinline__ int64_t tensor_tiles(const DevTensor& T) { return (T.n + kTileElems - 1) / kTileElems; }

// One workgroup per (tensor, run of kFusedReduceTiles tiles), all K deltas at once: every
// tile's block of K * kFusedStat counts is read once, as whole contiguous lines.  Thread
// (g, s) adds count s of the tiles g, g + G, ...; the G partial sums meet in LDS.  The run's
// sums go to csum (delta-major per tensor, as the tie search reads them) and onto the units'
// totals.
template <int K>
__global__ void __launch_bounds__(1024) k_fs_reduce(const DevTensor* __restrict__ tab, int n_t,
                                                    const int64_t* __restrict__ ritem0, const int* __restrict__ tflag,
                                                    const uint16_t* __restrict__ tstat, uint32_t* __restrict__ csum,
                                                    FusedUnit* __restrict__ fu) {
  constexpr int NS = K * kFusedStat, SW = fused_stat_words(K), G = 1024 / NS;
  __shared__ uint32_t red[G][NS];
  const int64_t item = blockIdx.x;                 // counts runs over all tensors: ritem0 / K
  int lo = 0, hi = n_t - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (ritem0[mid] / K <= item) lo = mid; else hi = mid - 1;
  }
  const int j = lo;
  if (tflag[j]) return;
  const DevTensor& T = tab[j];
  const int64_t nt = tensor_tiles(T);
  const int64_t nrc = (nt + kFusedReduceTiles - 1) / kFusedReduceTiles;
  const int64_t r = item - ritem0[j] / K;
  const int64_t t0 = T.tile0 + r * kFusedReduceTiles, t1 = T.tile0 + min(nt, (r + 1) * kFusedReduceTiles);
  const int g = threadIdx.x / NS, sidx = threadIdx.x % NS;
  if (g < G) {
    uint32_t acc = 0;
#pragma unroll 8
    for (int64_t t = t0 + g; t < t1; t += G) acc += tstat[(size_t)t * SW + sidx];
    red[g][sidx] = acc;
  }
  __syncthreads();
  if (threadIdx.x < NS) {
    uint32_t v = 0;
#pragma unroll
    for (int q = 0; q < G; ++q) v += red[q][threadIdx.x];
    const int i = threadIdx.x / kFusedStat, c = threadIdx.x % kFusedStat;
    csum[(size_t)(ritem0[j] + (int64_t)i * nrc + r) * kFusedStat + c] = v;
    FusedUnit& F = fu[j * K + i];
    if (v) {
      if (c == 0) atomicAdd((unsigned long long*)&F.kept, (unsigned long long)v);
      else atomicAdd(&F.h[c - 1], v);
    }
  }
}

// Exact threshold per delta from the bracket counts (one thread per delta).  The main pass
// counts the entries it kept provisionally (key >= prov_key); those above the bracket are
// that count less the bracket codes at or above prov_key.
__global__ void k_fs_resolve(const DevTensor* __restrict__ tab, int n_t, int K, FusedUnit* __restrict__ fu,
                             int* __restrict__ tflag, uint32_t* status) {
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= n_t * K) return;
  const int j = u / K;
  if (tflag[j]) return;
  FusedUnit& F = fu[u];
  const int64_t n = tab[j].n;
  if (F.flags & kFusedNone) {
    F.t_key = kNoSelectKey;
    F.cutoff = 0;
    return;
  }
  const int64_t k = F.k;
  const int W = (int)(F.hi - F.lo + 1u);
  const uint32_t p1 = prov_key(F);
  int64_t cum = (int64_t)F.kept;
  if (!(F.flags & kFusedAll))
    for (int c = 0; c < W; ++c)
      if (F.lo + (uint32_t)c >= p1) cum -= F.h[c];
  if (F.flags & kFusedAll) {
    F.t_key = 0;
    F.n_above = cum;
    F.quota = k - cum;
    F.count_t = n - cum;
    F.cutoff = n;
    return;
  }
  if (k <= cum) {                                   // threshold above the bracket
    atomicOr(&tflag[j], kFlagMiss);
    return;
  }
  for (int c = W - 1; c >= 0; --c) {
    const uint32_t code = F.lo + (uint32_t)c;
    if (code == 0u) break;                          // zeros are not counted
    const int64_t h = F.h[c];
    if (cum + h >= k) {
      F.t_key = code;
      F.n_above = cum;
      F.quota = k - cum;
      F.count_t = h;
      F.cutoff = (F.quota == h) ? n : -1;           // -1: found from the records
      if (code >= 0x7F80u) flag_status(status, kStatusNonFinite);
      return;
    }
    cum += h;
  }
  if (F.lo == 0u) {                                 // every nonzero key is kept; the rest are zeros
    F.t_key = 0;
    F.n_above = cum;
    F.quota = k - cum;
    F.count_t = n - cum;
    F.cutoff = n;
    return;
  }
  atomicOr(&tflag[j], kFlagMiss);                   // threshold below the bracket
}

struct TieArgs {
  const DevTensor* tab;
  FusedUnit* fu;
  const int* tflag;
  const int64_t* ritem0;
  const uint32_t* csum;
  const uint16_t* tstat;
  const uint2* tinfo;
  const uint32_t* rec;
  int64_t tile_cap;
  uint32_t* status;
};

// One workgroup per delta whose threshold code is only partly kept: the reduction chunk,
// then the tile, then the record holding the quota-th entry of that code in flat order.
template <int K>
__global__ void __launch_bounds__(1024) k_fs_tiefind(TieArgs a) {
  constexpr int RW = rec_words<K>();
  __shared__ int64_t sh[17];
  __shared__ int64_t s_pos, s_before;
  const int u = blockIdx.x;
  const int j = u / K, i = u % K;
  if (a.tflag[j] || a.fu[u].cutoff >= 0) return;
  const DevTensor& T = a.tab[j];
  const int64_t quota = a.fu[u].quota;
  const uint32_t tk = a.fu[u].t_key;
  const int ct = 1 + (int)(tk - a.fu[u].lo);
  const int64_t nt = tensor_tiles(T);
  const int64_t nrc = (nt + kFusedReduceTiles - 1) / kFusedReduceTiles;
  const int64_t item0 = a.ritem0[j] + (int64_t)i * nrc;
  // 1) reduction chunk
  if (threadIdx.x == 0) { s_pos = -1; s_before = 0; }
  int64_t base = 0;
  for (int64_t c0 = 0; c0 < nrc; c0 += blockDim.x) {
    const int64_t c = c0 + threadIdx.x;
    const int64_t v = (c < nrc) ? (int64_t)a.csum[(size_t)(item0 + c) * kFusedStat + ct] : 0;
    const int64_t incl = base + block_scan(v, sh);
    if (c < nrc && incl - v < quota && incl >= quota) { s_pos = c; s_before = incl - v; }
    base += sh[16];
    __syncthreads();
    if (s_pos >= 0) break;
  }
  __syncthreads();
  const int64_t rc = s_pos;
  const int64_t before_chunk = s_before;
  __syncthreads();
  if (rc < 0) {
    if (threadIdx.x == 0) { flag_status(a.status, kStatusInternal); a.fu[u].cutoff = T.n; }
    return;
  }
  // 2) tile inside the chunk (at most 1024 tiles: one per thread)
  if (threadIdx.x == 0) s_pos = -1;
  const int64_t t0 = T.tile0 + rc * kFusedReduceTiles;
  const int64_t tn = min<int64_t>(kFusedReduceTiles, nt - rc * kFusedReduceTiles);
  {
    const int64_t t = t0 + threadIdx.x;
    const int64_t v =
        (threadIdx.x < tn) ? (int64_t)a.tstat[(size_t)t * fused_stat_words(K) + i * kFusedStat + ct] : 0;
    const int64_t incl = before_chunk + block_scan(v, sh);
    if (threadIdx.x < tn && incl - v < quota && incl >= quota) { s_pos = t; s_before = incl - v; }
  }
  __syncthreads();
  const int64_t tile = s_pos;
  const int64_t before_tile = s_before;
  __syncthreads();
  if (tile < 0) {
    if (threadIdx.x == 0) { flag_status(a.status, kStatusInternal); a.fu[u].cutoff = T.n; }
    return;
  }
  // 3) records of that tile, in flat order
  const uint32_t nrec = a.tinfo[tile].x;
  const uint32_t* region = a.rec + (size_t)tile * a.tile_cap * RW;
  if (threadIdx.x == 0) s_pos = -1;
  int64_t seen = before_tile;
  for (uint32_t r0 = 0; r0 < nrec; r0 += blockDim.x) {
    const uint32_t r = r0 + threadIdx.x;
    const uint32_t* w = region + (size_t)r * RW;
    const int64_t tie = (r < nrec) ? (int64_t)(bkey(rec_half(w, 3 + i)) == tk) : 0;
    const int64_t incl = seen + block_scan(tie, sh);
    if (tie && incl == quota) s_pos = (int64_t)w[0];
    seen += sh[16];
    __syncthreads();
    if (s_pos >= 0) break;
  }
  if (threadIdx.x == 0) {
    if (s_pos < 0) flag_status(a.status, kStatusInternal);
    a.fu[u].cutoff = (s_pos < 0) ? T.n : s_pos + 1;
  }
}

// ---- 4. fix-up -----------------------------------------------------------------------------------

struct FixArgs {
  const DevTensor* tab;
  int n_t;
  const FusedUnit* fu;
  const int* tflag;
  const uint2* tinfo;
  const uint32_t* rec;
  int64_t tile_cap;
  double lambda;
  int want_sign;
  uint32_t* status;
};

// Final TopKMask of one coordinate's deltas (threshold key, then the tie cutoff).
template <int K>
__device__ __forceinline__ uint32_t final_mask(const uint32_t (&b)[K], int64_t idx, const uint32_t* tk,
                                               const int64_t* cut) {
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < K; ++i) {
    const uint32_t key = bkey(b[i]);
    const bool kept = tk[i] != kNoSelectKey && key != 0u && (key > tk[i] || (key == tk[i] && idx < cut[i]));
    m |= (uint32_t)kept << i;
  }
  return m;
}

template <int K>
__device__ __forceinline__ void store_final(const DevTensor& T, int64_t idx, const uint32_t (&b)[K], uint32_t m,
                                            uint32_t wb, double lambda, int want_sign) {
  int gam;
  const double t = ties_general<ISO_BF16, K>(b, m, gam);
  ((uint16_t*)T.out)[idx] = (uint16_t)f64_to_bf16_rne(bits_to_f64<ISO_BF16>(wb) + lambda * t);
  if (want_sign) ((int8_t*)T.aux2)[idx] = (int8_t)gam;
}

// One workgroup per run of up to 64 tiles of one tensor.  Records whose final mask differs
// from the provisional one are merged again; a tile whose binary32 sums may have rounded is
// merged again whole, in binary64, from the inputs.  The records are read in batches of
// 256 NB; each batch first only decides which records changed (a few integer tests per
// record) and queues those in LDS, so that the binary64 merge runs on the changed records
// alone, one per lane, instead of once per record position of any lane that needs it.  A
// coordinate is rewritten only when its output (or elected sign) differs from the value the
// main pass stored for the provisional mask: a delta that joins or leaves the mean often
// moves the result by less than the base's bf16 spacing, and the scattered 2-byte writes are
// the costly part of this kernel.
template <int K>
__global__ void __launch_bounds__(256) k_fs_fixup(FixArgs a) {
  constexpr int RW = rec_words<K>();
  constexpr int NB = 4;                            // records in flight per thread
  __shared__ uint32_t s_pre[kFusedGroupTiles + 1];
  __shared__ uint32_t s_p1[K], s_tk[K];
  __shared__ int64_t s_cut[K];
  __shared__ int s_anyredo;
  __shared__ uint4 s_q[NB * 256 * (RW / 4)];      // changed records of the batch
  __shared__ uint32_t s_qn;
  const int64_t g = blockIdx.x;
  int lo = 0, hi = a.n_t - 1;                      // tensor owning run g (group0 ascending)
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.tab[mid].group0 <= g) lo = mid; else hi = mid - 1;
  }
  const int j = lo;
  if (a.tflag[j]) return;
  const DevTensor& T = a.tab[j];
  const int64_t nt = tensor_tiles(T);
  const int64_t t0 = T.tile0 + (g - T.group0) * kFusedGroupTiles;
  const int ntl = (int)min<int64_t>(kFusedGroupTiles, T.tile0 + nt - t0);
  if (threadIdx.x == 0) { s_anyredo = 0; s_qn = 0; }
  __syncthreads();
  if (threadIdx.x < 64) {                          // inclusive scan of the record counts (one wave)
    const int l = threadIdx.x;
    const uint2 ti = (l < ntl) ? a.tinfo[t0 + l] : make_uint2(0u, 0u);
    if (ti.y) s_anyredo = 1;
    uint32_t x = ti.x;
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = (uint32_t)__shfl_up((int)x, o, 64);
      if (l >= o) x += y;
    }
    s_pre[l + 1] = x;
    if (l == 0) s_pre[0] = 0;
  }
  if (threadIdx.x < K) {
    const FusedUnit& F = a.fu[j * K + threadIdx.x];
    s_p1[threadIdx.x] = prov_key(F);
    s_tk[threadIdx.x] = F.t_key;
    s_cut[threadIdx.x] = F.cutoff;
  }
  __syncthreads();
  uint32_t tk[K];
  int64_t cut[K];
  // When every delta's provisional key is its final threshold key, the two masks differ only
  // at threshold entries at or past the tie cutoff: no coordinate below the smallest cutoff
  // changes, and the records of tiles that end there need not be read.
  int64_t unchanged_below = INT64_MAX;
#pragma unroll
  for (int i = 0; i < K; ++i) {
    tk[i] = s_tk[i];
    cut[i] = s_cut[i];
    unchanged_below = (s_p1[i] == tk[i]) ? min(unchanged_below, cut[i]) : (int64_t)0;
  }
  int l0 = 0;                                      // first tile of the run with records to read
  while (l0 < ntl && (t0 + l0 - T.tile0 + 1) * kTileElems <= unchanged_below) ++l0;
  const uint32_t first = s_pre[l0];
  const uint32_t total = s_pre[kFusedGroupTiles];
  const uint32_t* __restrict__ rec = a.rec;
  uint16_t* __restrict__ out = (uint16_t*)T.out;
  const int lane = threadIdx.x & 63;
  int l = l0;                                      // tile of the thread's current record (advances monotonically)
  for (uint32_t r0 = first; r0 < total; r0 += NB * 256u) {
    uint4 wv[NB][RW / 4];
#pragma unroll
    for (int m = 0; m < NB; ++m) {
      const uint32_t r = r0 + (uint32_t)m * 256u + threadIdx.x;
      if (r < total) {
        while (s_pre[l + 1] <= r) ++l;
        const uint4* w = (const uint4*)(rec + ((size_t)(t0 + l) * a.tile_cap + (r - s_pre[l])) * RW);
#pragma unroll
        for (int z = 0; z < RW / 4; ++z) wv[m][z] = w[z];
      }
    }
#pragma unroll
    for (int m = 0; m < NB; ++m) {
      const uint32_t r = r0 + (uint32_t)m * 256u + threadIdx.x;
      bool changed = false;
      uint32_t kfin = 0, kprov = 0;
      if (r < total) {
        uint32_t w[RW];
#pragma unroll
        for (int z = 0; z < RW / 4; ++z) {
          w[4 * z] = wv[m][z].x; w[4 * z + 1] = wv[m][z].y; w[4 * z + 2] = wv[m][z].z; w[4 * z + 3] = wv[m][z].w;
        }
        uint32_t b[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
          b[i] = rec_half(w, 3 + i);
          kprov |= (uint32_t)(bkey(b[i]) >= s_p1[i]) << i;
        }
        kfin = final_mask<K>(b, (int64_t)w[0], tk, cut);
        changed = kprov != kfin;
      }
      // queue slot: one LDS atomic per wave, then the lane's rank among the changed lanes
      const uint64_t mask = __ballot(changed);
      uint32_t qbase = 0;
      if (lane == 0 && mask) qbase = atomicAdd(&s_qn, (uint32_t)__popcll(mask));
      qbase = (uint32_t)__shfl((int)qbase, 0, 64);
      if (changed) {
        const uint32_t slot = qbase + (uint32_t)__popcll(mask & ((1ull << lane) - 1ull));
        uint4 v0 = wv[m][0];
        // halfword 2 (the tensor id) carries the final mask and, above it, the provisional one
        v0.y = (v0.y & 0xFFFF0000u) | kfin | (kprov << 8);
        s_q[slot * (RW / 4)] = v0;
#pragma unroll
        for (int z = 1; z < RW / 4; ++z) s_q[slot * (RW / 4) + z] = wv[m][z];
      }
    }
    __syncthreads();
    const uint32_t nq = s_qn;
    for (uint32_t qi = threadIdx.x; qi < nq; qi += 256u) {
      uint32_t w[RW];
#pragma unroll
      for (int z = 0; z < RW / 4; ++z) {
        const uint4 v = s_q[qi * (RW / 4) + z];
        w[4 * z] = v.x; w[4 * z + 1] = v.y; w[4 * z + 2] = v.z; w[4 * z + 3] = v.w;
      }
      uint32_t b[K];
#pragma unroll
      for (int i = 0; i < K; ++i) b[i] = rec_half(w, 3 + i);
      const int64_t idx = w[0];
      const uint32_t masks = rec_half(w, 2);
      const double w0 = bits_to_f64<ISO_BF16>(rec_half(w, 3 + K));
      // the main pass wrote the value of the provisional mask (its binary32 forms give the
      // binary64 sequence bit for bit): rewrite only what the final mask changes
      int gam, gam_p;
      const double t = ties_general<ISO_BF16, K>(b, masks & 0xFFu, gam);
      const double tp = ties_general<ISO_BF16, K>(b, masks >> 8, gam_p);
      const uint32_t o = f64_to_bf16_rne(w0 + a.lambda * t);
      if (o != f64_to_bf16_rne(w0 + a.lambda * tp)) out[idx] = (uint16_t)o;
      if (a.want_sign && gam != gam_p) ((int8_t*)T.aux2)[idx] = (int8_t)gam;
    }
    __syncthreads();
    if (threadIdx.x == 0) s_qn = 0;
    __syncthreads();
  }
  if (!s_anyredo) return;
  uint32_t kmax = 0;
  for (int l = 0; l < ntl; ++l) {
    if (!a.tinfo[t0 + l].y) continue;
    const int64_t e0 = (t0 + l - T.tile0) * kTileElems, e1 = min(T.n, e0 + kTileElems);
    for (int64_t idx = e0 + threadIdx.x; idx < e1; idx += blockDim.x) {
      uint32_t b[K];
#pragma unroll
      for (int i = 0; i < K; ++i) {
        b[i] = ((const uint16_t*)T.deltas[i])[idx];
        kmax = max(kmax, bkey(b[i]));
      }
      store_final<K>(T, idx, b, final_mask<K>(b, idx, tk, cut), ((const uint16_t*)T.base)[idx], a.lambda,
                     a.want_sign);
    }
  }
  if (kmax >= 0x7F80u) flag_status(a.status, kStatusNonFinite);
}

__global__ void k_fs_count(const int* __restrict__ tflag, int n_t, uint32_t* __restrict__ count) {
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j < n_t; j += gridDim.x * blockDim.x)
    if (tflag[j]) atomicAdd(count, 1u);
}

template <int K>
hipError_t launch_k(const FusedPlan& pl, hipStream_t s) {
  const int nu = pl.n_t * K;
  k_fs_init<<<(std::max(nu, pl.n_t) + 255) / 256, 256, 0, s>>>(pl.tab, pl.n_t, K, pl.fu, pl.tflag);
  k_fs_sample<<<nu, 1024, 0, s>>>(pl.tab, K, pl.fu, pl.tflag);
  if (pl.tiles > 0) {
    MainArgs m;
    m.tab = pl.tab;
    m.tmap = pl.tmap;
    m.n_t = pl.n_t;
    m.fu = pl.fu;
    m.tflag = pl.tflag;
    m.tstat = pl.tstat;
    m.tinfo = pl.tinfo;
    m.rec = pl.rec;
    m.tile_cap = pl.tile_cap;
    m.lambda = pl.lambda;
    m.status = pl.status;
    m.one2 = 0x00010001u;
    if (pl.prof[0]) (void)hipEventRecord(pl.prof[0], s);
    if (pl.want_sign) k_fs_main<K, false, true><<<(unsigned)pl.tiles, kThreads, 0, s>>>(m);
    else if (pl.lambda == 1.0) k_fs_main<K, true, false><<<(unsigned)pl.tiles, kThreads, 0, s>>>(m);
    else k_fs_main<K, false, false><<<(unsigned)pl.tiles, kThreads, 0, s>>>(m);
    if (pl.prof[1]) (void)hipEventRecord(pl.prof[1], s);
  }
  if (pl.ritems > 0)
    k_fs_reduce<K><<<(unsigned)(pl.ritems / K), 1024, 0, s>>>(pl.tab, pl.n_t, pl.ritem0, pl.tflag, pl.tstat, pl.csum,
                                                               pl.fu);
  k_fs_resolve<<<(nu + 255) / 256, 256, 0, s>>>(pl.tab, pl.n_t, K, pl.fu, pl.tflag, pl.status);
  TieArgs ta;
  ta.tab = pl.tab;
  ta.fu = pl.fu;
  ta.tflag = pl.tflag;
  ta.ritem0 = pl.ritem0;
  ta.csum = pl.csum;
  ta.tstat = pl.tstat;
  ta.tinfo = pl.tinfo;
  ta.rec = pl.rec;
  ta.tile_cap = pl.tile_cap;
  ta.status = pl.status;
  k_fs_tiefind<K><<<nu, 1024, 0, s>>>(ta);
  if (pl.groups > 0) {
    FixArgs fa;
    fa.tab = pl.tab;
    fa.n_t = pl.n_t;
    fa.fu = pl.fu;
    fa.tflag = pl.tflag;
    fa.tinfo = pl.tinfo;
    fa.rec = pl.rec;
    fa.tile_cap = pl.tile_cap;
    fa.lambda = pl.lambda;
    fa.want_sign = pl.want_sign;
    fa.status = pl.status;
    k_fs_fixup<K><<<(unsigned)pl.groups, 256, 0, s>>>(fa);
  }
  k_fs_count<<<1, 256, 0, s>>>(pl.tflag, pl.n_t, pl.status + 1);
  // tensors the single read could not settle: the exact two-pass path, flagged tensors only
  SelectPlan sp = pl.sel;
  sp.filter = pl.tflag;
  hipError_t e = run_select(sp, ISO_BF16, s);
  if (e != hipSuccess) return e;
  MergePlan mp = pl.mrg;
  mp.filter = pl.tflag;
  mp.desc = sp.desc;
  mp.prof[0] = mp.prof[1] = nullptr;
  return run_merge(mp, ISO_BF16, s);
}

}  // namespace

int64_t fused_tile_elems() { return kTileElems; }

int64_t fused_groups(int64_t n) {
  const int64_t nt = (n + kTileElems - 1) / kTileElems;
  return (nt + kFusedGroupTiles - 1) / kFusedGroupTiles;
}

int64_t fused_reduce_items(int64_t n, int K) {
  const int64_t nt = (n + kTileElems - 1) / kTileElems;
  return (int64_t)K * ((nt + kFusedReduceTiles - 1) / kFusedReduceTiles);
}

size_t fused_record_bytes(int K) { return (size_t)((2 * (K + 4) + 15) / 16) * 16; }

int64_t fused_tile_cap(int K) {
  // record room per tile: 1/16 of its coordinates for K <= 4, 1/8 above
  switch (K) {
    case 1: return kTileCapK<1>;
    case 2: return kTileCapK<2>;
    case 3: return kTileCapK<3>;
    case 4: return kTileCapK<4>;
    default: return kTileCapK<8>;
  }
}

hipError_t run_fused(const FusedPlan& pl, hipStream_t s) {
  if (kTileElems != merge_tile_elems(ISO_BF16)) return hipErrorInvalidValue;   // shared tile numbering
  if (pl.n_t <= 0) return hipSuccess;
  if (pl.n_t > kFusedMaxTensors) return hipErrorInvalidValue;
  switch (pl.K) {
    case 1: return launch_k<1>(pl, s);
    case 2: return launch_k<2>(pl, s);
    case 3: return launch_k<3>(pl, s);
    case 4: return launch_k<4>(pl, s);
    case 5: return launch_k<5>(pl, s);
    case 6: return launch_k<6>(pl, s);
    case 7: return launch_k<7>(pl, s);
    case 8: return launch_k<8>(pl, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace iso
