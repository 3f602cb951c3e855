// Element-wise merges of App. F fused with the final update, one streaming pass:
//   TIES:  tilde tau_i = m_i (.) tau_i, gamma = sign(sum_i tilde tau_i) (exact),
//          tau = mean over A_p = {i : tilde tau_i != 0, sign(tilde tau_i) = gamma}, 0 if empty
//   TA:    tau = sum_i tau_i
//   RAM:   tau = mean over A_p = {i : |tau_i| > eps}, 0 if empty
// then u = lambda * tau and out = round(w0 + u).  Every delta and the base are read
// once with 16-byte vector loads; the weights (and optionally tau or gamma) are
// written once.
//
// Arithmetic follows the binary64 sequence fixed by the library: sums start at
// +0.0 and add terms in expert order; the mean divides by the count; u = lambda*t;
// v = w0 + u; v is rounded once.  Two implementations of the TIES coordinate:
//  - general: binary64 values; the sign of the binary64 sum is accepted when it
//    exceeds the recursive-summation error bound (|S| > K 2^-52 sum|x|, Higham,
//    "Accuracy and Stability of Numerical Algorithms", 2nd ed., eq. 4.4), else it
//    is decided exactly by Shewchuk's grow-expansion;
//  - fast (bf16 only, chosen per tensor): when every kept magnitude lies within
//    16 - ceil(log2 K) binades of the largest key of the tensor, all partial sums
//    of kept values are exact in binary32, so S, sum|x| and the agreeing-set sum
//    (S + gamma*sum|x|)/2 are exact real values and equal the binary64 sequence.
#include "iso_device.h"
#include "iso_kernels.h"
#include "iso_merge_math.h"

namespace iso {

constexpr int kMergeThreads = 256;
constexpr int kMergeVPT = 2;          // 16-byte vectors per thread per array in one tile
constexpr int64_t kMergeMaxGrid = 0;  // 0: one block per tile; else blocks loop over tiles

int64_t merge_tile_elems(int dt) {
  return (int64_t)kMergeThreads * kMergeVPT * (dt == ISO_BF16 ? Fmt<ISO_BF16>::kPerVec : Fmt<ISO_F32>::kPerVec);
}

template <int K>
struct TileThr {
  uint32_t teff[K];   // tile-uniform key threshold (kept iff key >= teff)
  uint32_t t[K];      // t_key
  uint32_t t1[K];     // t_key + 1 (saturating)
  int64_t cut[K];     // tie cutoff
};

template <int DT>
__device__ __forceinline__ uint32_t key_of(uint32_t b) {
  return b & Fmt<DT>::kKeyMask;
}

template <int DT, int K, bool STRADDLE>
__device__ __forceinline__ bool kept(const TileThr<K>& th, int i, uint32_t key, int64_t idx) {
  if constexpr (STRADDLE) return key >= ((idx < th.cut[i]) ? th.t[i] : th.t1[i]);
  else return key >= th.teff[i];
}

// One coordinate.  b[i]: storage bits of delta i; returns u (binary64) and gamma.
template <int DT, int K, int MODE, bool FAST, bool STRADDLE>
__device__ __forceinline__ double merge_coord(const uint32_t (&b)[K], int64_t idx, const TileThr<K>& th,
                                              double lambda, double eps, int& gamma, uint32_t& kacc) {
  double t;
  if constexpr (MODE == ISO_MERGE_TIES) {
    uint32_t km = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const uint32_t key = key_of<DT>(b[i]);
      if constexpr (!FAST) kacc = max(kacc, key);
      km |= (uint32_t)kept<DT, K, STRADDLE>(th, i, key, idx) << i;
    }
    if constexpr (FAST) t = ties_fast_bf16<K>(b, km, gamma);
    else t = ties_general<DT, K>(b, km, gamma);
  } else if constexpr (MODE == ISO_MERGE_TA) {
    t = 0.0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      kacc = max(kacc, key_of<DT>(b[i]));
      t = t + bits_to_f64<DT>(b[i]);
    }
    gamma = 0;
  } else {  // RAM
    double s = 0.0;
    int n = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      kacc = max(kacc, key_of<DT>(b[i]));
      double x = bits_to_f64<DT>(b[i]);
      bool act = fabs(x) > eps;
      s = s + (act ? x : 0.0);
      n += act;
    }
    gamma = 0;
    t = (n == 0) ? 0.0 : div_count(s, n);
  }
  return lambda * t;
}

template <int DT>
__device__ __forceinline__ uint32_t round_out(double v) {
  if constexpr (DT == ISO_BF16) return f64_to_bf16_rne(v);
  else return bits_from_f32((float)v);
}

template <int DT, int K, int MODE, int OUTS, int VPT, bool FAST, bool STRADDLE>
__device__ __forceinline__ void merge_body(const DevTensor& T, int64_t vbeg, const TileThr<K>& th, double lambda,
                                           double eps, uint32_t& kacc, uint32_t& wacc) {
  using F = Fmt<DT>;
  constexpr int E = F::kPerVec;
  const int64_t n = T.n;
  const int64_t nvec = n / E;
#pragma unroll
  for (int q = 0; q < VPT; ++q) {
    const int64_t vi = vbeg + (int64_t)q * kMergeThreads + threadIdx.x;
    if (vi < nvec) {
      uint4 dv[K];
#pragma unroll
      for (int i = 0; i < K; ++i) dv[i] = ld_stream((const uint4*)T.deltas[i] + vi);
      uint4 wv = make_uint4(0, 0, 0, 0);
      if constexpr ((OUTS & OUT_W) != 0) wv = ld_stream((const uint4*)T.base + vi);
      uint32_t ob[E];
      float tb[E];
      int gb[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        uint32_t b[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
          uint32_t w = (e / (E / 4) == 0) ? dv[i].x : (e / (E / 4) == 1) ? dv[i].y : (e / (E / 4) == 2) ? dv[i].z : dv[i].w;
          if constexpr (DT == ISO_BF16) b[i] = (e & 1) ? (w >> 16) : (w & 0xFFFFu);
          else b[i] = w;
        }
        int g;
        double u = merge_coord<DT, K, MODE, FAST, STRADDLE>(b, vi * E + e, th, lambda, eps, g, kacc);
        if constexpr ((OUTS & OUT_W) != 0) {
          uint32_t w = (e / (E / 4) == 0) ? wv.x : (e / (E / 4) == 1) ? wv.y : (e / (E / 4) == 2) ? wv.z : wv.w;
          uint32_t wb = (DT == ISO_BF16) ? ((e & 1) ? (w >> 16) : (w & 0xFFFFu)) : w;
          wacc = max(wacc, key_of<DT>(wb));
          ob[e] = round_out<DT>(bits_to_f64<DT>(wb) + u);
        }
        tb[e] = (float)u;
        gb[e] = g;
      }
      if constexpr ((OUTS & OUT_W) != 0) {
        uint4 o;
        if constexpr (DT == ISO_BF16) {
          o.x = ob[0] | (ob[1] << 16); o.y = ob[2] | (ob[3] << 16);
          o.z = ob[4] | (ob[5] << 16); o.w = ob[6] | (ob[7] << 16);
        } else {
          o.x = ob[0]; o.y = ob[1]; o.z = ob[2]; o.w = ob[3];
        }
        st_stream(o, (uint4*)T.out + vi);
      }
      if constexpr ((OUTS & OUT_TAU) != 0) {
        float4* tp = (float4*)T.aux + vi * (E / 4);
#pragma unroll
        for (int h = 0; h < E / 4; ++h)
          st_stream(make_float4(tb[4 * h], tb[4 * h + 1], tb[4 * h + 2], tb[4 * h + 3]), tp + h);
      }
      if constexpr ((OUTS & OUT_SIGN) != 0) {
        int8_t* sp = (int8_t*)(((OUTS & OUT_W) != 0) ? T.aux2 : T.aux) + vi * E;
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) lo |= ((uint32_t)gb[e] & 0xFFu) << (8 * e);
        if constexpr (E == 8) {
#pragma unroll
          for (int e = 0; e < 4; ++e) hi |= ((uint32_t)gb[4 + e] & 0xFFu) << (8 * e);
          *(uint2*)sp = make_uint2(lo, hi);
        } else {
          *(uint32_t*)sp = lo;
        }
      }
    } else if (vi == nvec && (n % E) != 0) {
      // ragged tail of the tensor: scalar elements
      for (int64_t idx = vi * E; idx < n; ++idx) {
        uint32_t b[K];
#pragma unroll
        for (int i = 0; i < K; ++i) b[i] = elem_bits<DT>(T.deltas[i], idx);
        int g;
        double u = merge_coord<DT, K, MODE, FAST, STRADDLE>(b, idx, th, lambda, eps, g, kacc);
        if constexpr ((OUTS & OUT_W) != 0) {
          uint32_t wb = elem_bits<DT>(T.base, idx);
          wacc = max(wacc, key_of<DT>(wb));
          uint32_t o = round_out<DT>(bits_to_f64<DT>(wb) + u);
          if constexpr (DT == ISO_BF16) ((uint16_t*)T.out)[idx] = (uint16_t)o;
          else ((uint32_t*)T.out)[idx] = o;
        }
        if constexpr ((OUTS & OUT_TAU) != 0) ((float*)T.aux)[idx] = (float)u;
        if constexpr ((OUTS & OUT_SIGN) != 0) ((int8_t*)(((OUTS & OUT_W) != 0) ? T.aux2 : T.aux))[idx] = (int8_t)g;
      }
    }
  }
}

template <int DT, int K, int MODE, int OUTS, int VPT>
__device__ __forceinline__ void merge_tile(const DevTensor* __restrict__ tab, int n_t,
                                           const iso_select_desc* __restrict__ desc, double lambda, double eps,
                                           uint32_t* status, int64_t tile) {
  using F = Fmt<DT>;
  constexpr int E = F::kPerVec;
  constexpr int64_t TV = (int64_t)kMergeThreads * VPT;    // vectors per tile
  const int j = find_tensor(tab, n_t, tile);
  const DevTensor& T = tab[j];
  const int64_t vbeg = (tile - T.tile0) * TV;
  const int64_t ebeg = vbeg * E;
  const int64_t eend = min(T.n, (vbeg + TV) * E);
  TileThr<K> th;
  bool straddle = false, fast = false;
  constexpr uint32_t expfield = (DT == ISO_BF16) ? 0x7F80u : 0x7F800000u;
  if constexpr (MODE == ISO_MERGE_TIES) {
    uint32_t fmax = 0, fmin = 0xFFFFFFFFu;
    bool all_ge1 = true, bad = false;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      uint32_t tk = 0, km = 0;
      int64_t cut = T.n;
      if (desc != nullptr) {
        const iso_select_desc d = desc[(int64_t)j * K + i];
        tk = d.t_key; km = d.key_max; cut = d.tie_cutoff;
      }
      th.t[i] = tk;
      th.t1[i] = (tk == 0xFFFFFFFFu) ? tk : tk + 1u;
      th.cut[i] = cut;
      if (eend <= cut) th.teff[i] = tk;
      else if (ebeg >= cut) th.teff[i] = th.t1[i];
      else { th.teff[i] = tk; straddle = true; }
      if (km >= expfield) bad = true;
      if (tk != kNoSelectKey) {
        if ((tk >> 7) < 1u) all_ge1 = false;
        fmax = max(fmax, km >> 7);
        fmin = min(fmin, tk >> 7);
      }
    }
    if (bad && threadIdx.x == 0 && (tile == T.tile0)) flag_status(status, kStatusNonFinite);
    constexpr int clog2k = (K <= 1) ? 0 : (K <= 2) ? 1 : (K <= 4) ? 2 : 3;
    if constexpr (DT == ISO_BF16) {
      fast = (desc != nullptr) && all_ge1 && !bad && (fmin == 0xFFFFFFFFu || fmax <= fmin + (uint32_t)(16 - clog2k));
    }
  } else {
#pragma unroll
    for (int i = 0; i < K; ++i) { th.t[i] = th.t1[i] = th.teff[i] = 0; th.cut[i] = 0; }
  }
  uint32_t kacc = 0, wacc = 0;
  constexpr bool kHasFast = (DT == ISO_BF16) && (MODE == ISO_MERGE_TIES);
  if (kHasFast && fast) {
    if constexpr (kHasFast) {
      if (straddle) merge_body<DT, K, MODE, OUTS, VPT, true, true>(T, vbeg, th, lambda, eps, kacc, wacc);
      else merge_body<DT, K, MODE, OUTS, VPT, true, false>(T, vbeg, th, lambda, eps, kacc, wacc);
    }
  } else {
    if (straddle) merge_body<DT, K, MODE, OUTS, VPT, false, true>(T, vbeg, th, lambda, eps, kacc, wacc);
    else merge_body<DT, K, MODE, OUTS, VPT, false, false>(T, vbeg, th, lambda, eps, kacc, wacc);
  }
  if (kacc >= expfield || wacc >= expfield) flag_status(status, kStatusNonFinite);
}

template <int DT, int K, int MODE, int OUTS, int VPT>
__global__ void __launch_bounds__(kMergeThreads) k_merge(const DevTensor* __restrict__ tab, int n_t,
                                                         const iso_select_desc* __restrict__ desc, double lambda,
                                                         double eps, uint32_t* status, int64_t tiles) {
  for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x)
    merge_tile<DT, K, MODE, OUTS, VPT>(tab, n_t, desc, lambda, eps, status, tile);
}

// Persistent form over the tiles of flagged tensors only.
template <int DT, int K, int MODE, int OUTS, int VPT>
__global__ void __launch_bounds__(kMergeThreads) k_merge_flagged(const DevTensor* __restrict__ tab, int n_t,
                                                                 const iso_select_desc* __restrict__ desc,
                                                                 double lambda, double eps, uint32_t* status,
                                                                 const int* __restrict__ filter) {
  __shared__ int sflag[1024];
  constexpr int64_t te = (int64_t)kMergeThreads * VPT * Fmt<DT>::kPerVec;
  for_flagged_items(
      filter, n_t, sflag, [&](int j) { return (tab[j].n + te - 1) / te; },
      [&](int j, int64_t it) {
        merge_tile<DT, K, MODE, OUTS, VPT>(tab, n_t, desc, lambda, eps, status, tab[j].tile0 + it);
      });
}

// ---- APPLY: out = round(w0 + lambda * tau_in) ----------------------------------------------------

template <int DT>
__global__ void __launch_bounds__(kMergeThreads) k_apply(const DevTensor* __restrict__ tab, int n_t, double lambda,
                                                         uint32_t* status) {
  using F = Fmt<DT>;
  constexpr int E = F::kPerVec;
  constexpr int64_t TV = (int64_t)kMergeThreads * kMergeVPT;
  const int64_t tile = blockIdx.x;
  const int j = find_tensor(tab, n_t, tile);
  const DevTensor& T = tab[j];
  const int64_t vbeg = (tile - T.tile0) * TV;
  const int64_t n = T.n, nvec = n / E;
  const float* tau = (const float*)T.aux;
  uint32_t wacc = 0, tacc = 0;
  for (int q = 0; q < kMergeVPT; ++q) {
    const int64_t vi = vbeg + (int64_t)q * kMergeThreads + threadIdx.x;
    if (vi < nvec) {
      uint4 wv = ld_stream((const uint4*)T.base + vi);
      uint32_t wbits[E];
      float tv[E];
      if constexpr (DT == ISO_BF16) {
        uint32_t w4[4] = {wv.x, wv.y, wv.z, wv.w};
        for (int h = 0; h < 4; ++h) { wbits[2 * h] = w4[h] & 0xFFFFu; wbits[2 * h + 1] = w4[h] >> 16; }
        float4 a = ld_stream((const float4*)tau + 2 * vi);
        float4 c = ld_stream((const float4*)tau + 2 * vi + 1);
        tv[0] = a.x; tv[1] = a.y; tv[2] = a.z; tv[3] = a.w; tv[4] = c.x; tv[5] = c.y; tv[6] = c.z; tv[7] = c.w;
      } else {
        wbits[0] = wv.x; wbits[1] = wv.y; wbits[2] = wv.z; wbits[3] = wv.w;
        float4 a = ld_stream((const float4*)tau + vi);
        tv[0] = a.x; tv[1] = a.y; tv[2] = a.z; tv[3] = a.w;
      }
      uint32_t ob[E];
      for (int e = 0; e < E; ++e) {
        wacc = max(wacc, key_of<DT>(wbits[e]));
        tacc = max(tacc, bits_from_f32(tv[e]) & 0x7FFFFFFFu);
        ob[e] = round_out<DT>(bits_to_f64<DT>(wbits[e]) + lambda * (double)tv[e]);
      }
      uint4 o;
      if constexpr (DT == ISO_BF16) {
        o.x = ob[0] | (ob[1] << 16); o.y = ob[2] | (ob[3] << 16);
        o.z = ob[4] | (ob[5] << 16); o.w = ob[6] | (ob[7] << 16);
      } else {
        o.x = ob[0]; o.y = ob[1]; o.z = ob[2]; o.w = ob[3];
      }
      st_stream(o, (uint4*)T.out + vi);
    } else if (vi == nvec && (n % E) != 0) {
      for (int64_t idx = vi * E; idx < n; ++idx) {
        uint32_t wb = elem_bits<DT>(T.base, idx);
        float tvv = tau[idx];
        wacc = max(wacc, key_of<DT>(wb));
        tacc = max(tacc, bits_from_f32(tvv) & 0x7FFFFFFFu);
        uint32_t o = round_out<DT>(bits_to_f64<DT>(wb) + lambda * (double)tvv);
        if constexpr (DT == ISO_BF16) ((uint16_t*)T.out)[idx] = (uint16_t)o;
        else ((uint32_t*)T.out)[idx] = o;
      }
    }
  }
  constexpr uint32_t expfield = (DT == ISO_BF16) ? 0x7F80u : 0x7F800000u;
  if (wacc >= expfield || tacc >= 0x7F800000u) flag_status(status, kStatusNonFinite);
}

// ---- dispatch -----------------------------------------------------------------------------------

template <int DT, int K, int MODE, int OUTS>
static void launch_merge(const MergePlan& pl, hipStream_t s) {
  if (pl.filter != nullptr) {
    k_merge_flagged<DT, K, MODE, OUTS, kMergeVPT><<<1024, kMergeThreads, 0, s>>>(pl.tab, pl.n_t, pl.desc, pl.lambda,
                                                                                 pl.eps, pl.status, pl.filter);
    return;
  }
  const int64_t grid = (kMergeMaxGrid > 0) ? std::min(pl.tiles, kMergeMaxGrid) : pl.tiles;
  if (pl.prof[0]) (void)hipEventRecord(pl.prof[0], s);
  k_merge<DT, K, MODE, OUTS, kMergeVPT><<<(unsigned)grid, kMergeThreads, 0, s>>>(pl.tab, pl.n_t, pl.desc, pl.lambda,
                                                                                 pl.eps, pl.status, pl.tiles);
  if (pl.prof[1]) (void)hipEventRecord(pl.prof[1], s);
}

template <int DT, int K, int MODE>
static bool dispatch_outs(const MergePlan& pl, hipStream_t s) {
  switch (pl.outs) {
    case OUT_W: launch_merge<DT, K, MODE, OUT_W>(pl, s); return true;
    case OUT_TAU: launch_merge<DT, K, MODE, OUT_TAU>(pl, s); return true;
    default: break;
  }
  if constexpr (MODE == ISO_MERGE_TIES) {
    switch (pl.outs) {
      case OUT_SIGN: launch_merge<DT, K, MODE, OUT_SIGN>(pl, s); return true;
      case OUT_W | OUT_SIGN: launch_merge<DT, K, MODE, OUT_W | OUT_SIGN>(pl, s); return true;
      default: break;
    }
  }
  return false;
}

template <int DT, int K>
static bool dispatch_mode(const MergePlan& pl, hipStream_t s) {
  switch (pl.mode) {
    case ISO_MERGE_TIES: return dispatch_outs<DT, K, ISO_MERGE_TIES>(pl, s);
    case ISO_MERGE_TA: return dispatch_outs<DT, K, ISO_MERGE_TA>(pl, s);
    case ISO_MERGE_RAM: return dispatch_outs<DT, K, ISO_MERGE_RAM>(pl, s);
    default: return false;
  }
}

template <int DT>
static bool dispatch_k(const MergePlan& pl, hipStream_t s) {
  switch (pl.K) {
    case 1: return dispatch_mode<DT, 1>(pl, s);
    case 2: return dispatch_mode<DT, 2>(pl, s);
    case 3: return dispatch_mode<DT, 3>(pl, s);
    case 4: return dispatch_mode<DT, 4>(pl, s);
    case 5: return dispatch_mode<DT, 5>(pl, s);
    case 6: return dispatch_mode<DT, 6>(pl, s);
    case 7: return dispatch_mode<DT, 7>(pl, s);
    case 8: return dispatch_mode<DT, 8>(pl, s);
    default: return false;
  }
}

hipError_t run_merge(const MergePlan& pl, int dt, hipStream_t s) {
  if (pl.tiles <= 0) return hipSuccess;
  bool ok = (dt == ISO_BF16) ? dispatch_k<ISO_BF16>(pl, s) : dispatch_k<ISO_F32>(pl, s);
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t run_apply(const DevTensor* tab, int n_t, int dt, double lambda, int64_t tiles, uint32_t* status,
                     hipStream_t s) {
  if (tiles <= 0) return hipSuccess;
  if (dt == ISO_BF16) k_apply<ISO_BF16><<<(unsigned)tiles, kMergeThreads, 0, s>>>(tab, n_t, lambda, status);
  else k_apply<ISO_F32><<<(unsigned)tiles, kMergeThreads, 0, s>>>(tab, n_t, lambda, status);
  return hipGetLastError();
}

}  // namespace iso
