// TopKMask selection (App. F, TIES "Trim"): exact k-largest-magnitude selection by
// radix select over the storage magnitude keys, ties at the threshold broken by
// flat index.  bf16 keys (15 bits) take one histogram pass; fp32 keys (31 bits)
// take three (15 + 8 + 8 bits).
//
// Per pass, every (tensor, delta) "unit" is cut into chunks; one 1024-thread
// workgroup per chunk builds a 2^bits-bin histogram in LDS (128 KB for 15 bits)
// and flushes its nonzero bins to the unit's global histogram with integer
// atomics (deterministic: counts only).  A resolve kernel (one workgroup per
// unit) then finds the digit holding the k-th largest key.  If only part of the
// threshold bucket is kept, a tie pass counts threshold keys per 64K-element
// chunk and a find kernel walks to the quota-th tie in flat order.
#include "iso_device.h"
#include "iso_kernels.h"

namespace iso {

constexpr int kHistThreads = 1024;
constexpr int kMaxBins = 1 << 15;

// ---- block helpers ------------------------------------------------------------------------------

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, 64));
  return v;
}

// Inclusive prefix sum over the block (blockDim.x <= 1024, multiple of 64).
__device__ int64_t block_inclusive_scan(int64_t v, int64_t* sh /* >= 16 */) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int64_t x = v;
  for (int o = 1; o < 64; o <<= 1) {
    int64_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wid] = x;
  __syncthreads();
  if (wid == 0) {
    int64_t t = (lane < nw) ? sh[lane] : 0;
    for (int o = 1; o < 16; o <<= 1) {
      int64_t y = __shfl_up(t, o, 64);
      if (lane >= o) t += y;
    }
    if (lane < nw) sh[lane] = t;
  }
  __syncthreads();
  int64_t add = (wid > 0) ? sh[wid - 1] : 0;
  __syncthreads();
  return x + add;
}

// ---- unit setup ---------------------------------------------------------------------------------

// With `filter` set, only units of flagged tensors take part; the others are finished
// (no key selected) before the first pass.
// A member of a joint selection starts with its group's count (so that it is histogrammed
// whenever the group keeps anything); k_group_assign sets its own share before the resolve.
__global__ void k_select_init(const DevTensor* tab, int n_t, int K, UnitState* st, const int* filter,
                              const int* gid, const int64_t* gk) {
  int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= n_t * K) return;
  const DevTensor& T = tab[u / K];
  const bool skip = (filter != nullptr) && !filter[u / K];
  const int g = (gid != nullptr) ? gid[u / K] : -1;
  const int64_t k = (g >= 0) ? gk[g] : T.k;
  UnitState s;
  s.prefix = 0;
  s.key_max = 0;
  s.k_rem = k;
  s.n_above = 0;
  s.bucket = T.n;
  s.cutoff = 0;
  s.done = (k == 0 || T.n == 0 || skip) ? 1 : 0;
  if (s.done) s.prefix = kNoSelectKey;
  s.pad[0] = s.pad[1] = s.pad[2] = 0;
  st[u] = s;
}

// Work item -> (tensor j, delta i, chunk c), items of tensor j laid out delta-major.
__device__ __forceinline__ void item_of(const int64_t* item0, int n_t, int K, int64_t chunk, const DevTensor* tab,
                                        int64_t item, int& j, int& i, int64_t& c) {
  int lo = 0, hi = n_t - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (item0[mid] <= item) lo = mid; else hi = mid - 1;
  }
  j = lo;
  int64_t nch = (tab[j].n + chunk - 1) / chunk;
  int64_t local = item - item0[j];
  i = (int)(local / nch);
  c = local - (int64_t)i * nch;
}

// ---- histogram pass -----------------------------------------------------------------------------
// With `dump` set (last pass only), the block also stores its chunk histogram (bin 0 =
// in-bucket entries whose digit is 0) so ties can later be located without another read.

struct HistLds {
  uint32_t bins[kMaxBins];
  uint32_t wmax[16];
  uint32_t wzero[16];
};

// One histogram work item: chunk c of delta i of tensor j; `item` numbers its dump slot.
template <int DT>
__device__ void hist_item(const DevTensor* __restrict__ tab, int K, int j, int i, int64_t c, int64_t item,
                          int64_t chunk, UnitState* __restrict__ st, uint32_t* __restrict__ hist, int shift,
                          int bits, int first, uint32_t* status, uint32_t* __restrict__ dump, HistLds& sm) {
  using F = Fmt<DT>;
  constexpr int U = 8;                         // 16-byte loads in flight per thread
  uint32_t* lds = sm.bins;
  uint32_t* wmax = sm.wmax;
  uint32_t* wzero = sm.wzero;
  const int u = j * K + i;
  const DevTensor& T = tab[j];
  const bool active = !st[u].done;             // k == 0 units only need key_max from the first pass
  if (!first && !active) return;               // uniform per block
  const uint32_t nb = 1u << bits;
  for (uint32_t b = threadIdx.x; b < nb; b += blockDim.x) lds[b] = 0;
  __syncthreads();

  const int hs = shift + bits;                 // bits above the digit must match the prefix
  const uint32_t want = (hs >= 32) ? 0u : (st[u].prefix >> hs);
  const uint32_t dmask = nb - 1u;
  const int64_t e0 = c * chunk;
  const int64_t e1 = min(T.n, e0 + chunk);
  const typename F::bits_t* p = (const typename F::bits_t*)T.deltas[i];
  uint32_t kmax = 0, nzero = 0;

  auto count = [&](uint32_t key) {
    if (first) kmax = max(kmax, key);
    bool match = active && (first || ((key >> hs) == want));
    uint32_t d = (key >> shift) & dmask;
    if (match && d != 0u) atomicAdd(&lds[d], 1u);
    nzero += (match && d == 0u);
  };

  const int64_t v0 = e0 / F::kPerVec;
  const int64_t v1 = e1 / F::kPerVec;         // full vectors only
  const uint4* pv = (const uint4*)p;
  for (int64_t v = v0 + threadIdx.x; v < v1; v += U * blockDim.x) {
    uint4 a[U];
#pragma unroll
    for (int q = 0; q < U; ++q) {
      int64_t vv = v + (int64_t)q * blockDim.x;
      a[q] = (vv < v1) ? ld_stream(pv + vv) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < U; ++q) {
      int64_t vv = v + (int64_t)q * blockDim.x;
      if (vv >= v1) break;
      uint32_t w[4] = {a[q].x, a[q].y, a[q].z, a[q].w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        if constexpr (DT == ISO_BF16) {
          count(w[h] & 0x7FFFu);
          count((w[h] >> 16) & 0x7FFFu);
        } else {
          count(w[h] & 0x7FFFFFFFu);
        }
      }
    }
  }
  // scalar tail (last chunk of a tensor whose size is not a multiple of the vector width)
  for (int64_t e = v1 * F::kPerVec + threadIdx.x; e < e1; e += blockDim.x)
    count(elem_bits<DT>(p, e) & F::kKeyMask);
  uint32_t zsum = 0;
  if (dump != nullptr) {
    uint32_t z = nzero;
    for (int o = 32; o > 0; o >>= 1) z += (uint32_t)__shfl_xor((int)z, o, 64);
    if ((threadIdx.x & 63) == 0) wzero[threadIdx.x >> 6] = z;
  }
  __syncthreads();
  if (dump != nullptr) {
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) zsum += wzero[w];
  }

  uint32_t* gh = hist + (size_t)u * kMaxBins;
  if (active) {
    uint32_t* dp = (dump != nullptr) ? dump + (size_t)item * nb : nullptr;
    for (uint32_t b = threadIdx.x; b < nb; b += blockDim.x) {
      uint32_t cnt = lds[b];
      if (cnt) atomicAdd(&gh[b], cnt);
      if (dp) dp[b] = (b == 0) ? zsum : cnt;
    }
  }
  if (first) {
    uint32_t m = wave_max_u32(kmax);
    if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t mm = 0;
      for (int w = 0; w < (int)(blockDim.x >> 6); ++w) mm = max(mm, wmax[w]);
      atomicMax(&st[u].key_max, mm);
      uint32_t expfield = (DT == ISO_BF16) ? 0x7F80u : 0x7F800000u;
      if (mm >= expfield) flag_status(status, kStatusNonFinite);
    }
  }
  __syncthreads();                             // LDS is reused by the block's next item
}

template <int DT>
__global__ void __launch_bounds__(kHistThreads) k_hist(const DevTensor* __restrict__ tab, int n_t, int K,
                                                       const int64_t* __restrict__ item0, int64_t chunk,
                                                       UnitState* __restrict__ st, uint32_t* __restrict__ hist,
                                                       int shift, int bits, int first, uint32_t* status,
                                                       uint32_t* __restrict__ dump) {
  __shared__ HistLds sm;
  int j, i;
  int64_t c;
  item_of(item0, n_t, K, chunk, tab, blockIdx.x, j, i, c);
  hist_item<DT>(tab, K, j, i, c, blockIdx.x, chunk, st, hist, shift, bits, first, status, dump, sm);
}

// Persistent form over the flagged tensors only (items numbered as in k_hist).
template <int DT>
__global__ void __launch_bounds__(kHistThreads) k_hist_flagged(const DevTensor* __restrict__ tab, int n_t, int K,
                                                               const int64_t* __restrict__ item0, int64_t chunk,
                                                               UnitState* __restrict__ st,
                                                               uint32_t* __restrict__ hist, int shift, int bits,
                                                               int first, uint32_t* status,
                                                               uint32_t* __restrict__ dump,
                                                               const int* __restrict__ filter) {
  __shared__ HistLds sm;
  __shared__ int sflag[1024];
  for_flagged_items(
      filter, n_t, sflag, [&](int j) { return (int64_t)K * ((tab[j].n + chunk - 1) / chunk); },
      [&](int j, int64_t it) {
        const int64_t nch = (tab[j].n + chunk - 1) / chunk;
        const int i = (int)(it / nch);
        const int64_t c = it - (int64_t)i * nch;
        hist_item<DT>(tab, K, j, i, c, item0[j] + it, chunk, st, hist, shift, bits, first, status, dump, sm);
      });
}

// Clears the global histograms of the flagged tensors' units.
__global__ void __launch_bounds__(1024) k_clear_hist_flagged(int n_t, int K, uint32_t* __restrict__ hist,
                                                             const int* __restrict__ filter) {
  __shared__ int sflag[1024];
  for_flagged_items(
      filter, n_t, sflag, [&](int) { return (int64_t)K * (kMaxBins / 1024); },
      [&](int j, int64_t it) { hist[(size_t)j * K * kMaxBins + (size_t)it * 1024 + threadIdx.x] = 0u; });
}

// ---- resolve: pick the digit holding the k_rem-th largest key ------------------------------------

__global__ void __launch_bounds__(kHistThreads) k_resolve(const DevTensor* __restrict__ tab, int K,
                                                          UnitState* __restrict__ st, uint32_t* __restrict__ hist,
                                                          int shift, int bits, int last, uint32_t* status) {
  __shared__ uint32_t sbin[kMaxBins];
  __shared__ int64_t sh[16];
  __shared__ int64_t found_d, found_above;
  __shared__ int64_t total_nonzero;
  const int u = blockIdx.x;
  UnitState s = st[u];
  if (s.done) return;
  const uint32_t nb = 1u << bits;
  uint32_t* gh = hist + (size_t)u * kMaxBins;
  // coalesced copy to LDS, clearing the global bins for the next pass / call
  for (uint32_t b = threadIdx.x; b < nb; b += blockDim.x) {
    sbin[b] = gh[b];
    gh[b] = 0;
  }
  if (threadIdx.x == 0) { found_d = -1; found_above = 0; }
  __syncthreads();
  const uint32_t per = (nb + blockDim.x - 1) / blockDim.x;   // consecutive bins per thread
  const uint32_t b0 = threadIdx.x * per;
  // thread sums of bins >= 1 (bin 0 is reconstructed from the bucket total)
  int64_t mine = 0;
  for (uint32_t q = 0; q < per; ++q) {
    uint32_t b = b0 + q;
    if (b < nb && b > 0) mine += sbin[b];
  }
  int64_t incl = block_inclusive_scan(mine, sh);
  if (threadIdx.x == blockDim.x - 1) total_nonzero = incl;
  __syncthreads();
  const int64_t zeros = s.bucket - total_nonzero;
  const int64_t above_me = total_nonzero - incl;       // entries in bins above this thread's range
  const int64_t need = s.k_rem;                        // 1 <= need <= bucket
  int64_t run = above_me;
  for (int q = (int)per - 1; q >= 0; --q) {
    uint32_t b = b0 + (uint32_t)q;
    if (b >= nb) continue;
    int64_t h = (b == 0) ? zeros : (int64_t)sbin[b];
    if (run < need && run + h >= need) { found_d = b; found_above = run; }
    run += h;
  }
  __syncthreads();
  // found_d < 0 would mean inconsistent counts (cannot happen for 1 <= k_rem <= bucket); never index with it
  const int64_t d = found_d < 0 ? 0 : found_d;
  if (threadIdx.x == 0) {
    if (found_d < 0) flag_status(status, kStatusInternal);
    const int64_t h_d = (d == 0) ? zeros : (int64_t)sbin[d];
    s.prefix |= (uint32_t)d << shift;
    s.n_above += found_above;
    s.k_rem = need - found_above;
    s.bucket = h_d;
    if (last) {
      const DevTensor& T = tab[u / K];
      if (s.k_rem == s.bucket) { s.cutoff = T.n; s.done = 1; }
    }
    st[u] = s;
  }
}

// ---- joint selection (bf16, one pass) -------------------------------------------------------------
// The group's histogram is the sum of its members'; its threshold key and the number of entries
// with that key it keeps follow from it as for one tensor.  Each member then keeps its entries
// above the threshold and the next share of the threshold entries in table order, which is
// exactly a TopKMask of the member with that count: the per-unit resolve and tie search then
// give its descriptor unchanged.

// Group bins are 64-bit: a group (a whole-model delta) can hold more than 2^32 entries even
// though each member's own counts fit 32 bits.
__global__ void __launch_bounds__(256) k_group_sum(int K, const int* __restrict__ gmem, const int* __restrict__ gmem0,
                                                   const uint32_t* __restrict__ hist, uint64_t* __restrict__ ghist) {
  const int gi = blockIdx.y, g = gi / K, i = gi % K;
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= kMaxBins) return;
  uint64_t sum = 0;
  for (int m = gmem0[g]; m < gmem0[g + 1]; ++m) sum += hist[((size_t)gmem[m] * K + i) * kMaxBins + b];
  ghist[(size_t)gi * kMaxBins + b] = sum;
}

// The group histogram (256 KB of 64-bit bins) does not fit LDS: each thread reads its run of
// consecutive bins from global memory twice (sum, then the walk from the top).
__global__ void __launch_bounds__(kHistThreads) k_group_resolve(const DevTensor* __restrict__ tab, int K,
                                                                const int* __restrict__ gmem,
                                                                const int* __restrict__ gmem0,
                                                                const int64_t* __restrict__ gk,
                                                                const uint64_t* __restrict__ ghist,
                                                                GroupState* __restrict__ gst, uint32_t* status) {
  __shared__ int64_t sh[16];
  __shared__ int64_t found_d, found_above, total_nonzero;
  const int gi = blockIdx.x, g = gi / K;
  const int64_t need = gk[g];
  if (need == 0) {
    if (threadIdx.x == 0) gst[gi] = GroupState{kNoSelectKey, 1, 0};
    return;
  }
  int64_t n_g = 0;
  for (int m = gmem0[g]; m < gmem0[g + 1]; ++m) n_g += tab[gmem[m]].n;
  const uint64_t* gh = ghist + (size_t)gi * kMaxBins;
  if (threadIdx.x == 0) { found_d = -1; found_above = 0; }
  __syncthreads();
  const uint32_t per = (kMaxBins + blockDim.x - 1) / blockDim.x;
  const uint32_t b0 = threadIdx.x * per;
  int64_t mine = 0;
  for (uint32_t q = 0; q < per; ++q) {
    const uint32_t b = b0 + q;
    if (b < kMaxBins && b > 0) mine += (int64_t)gh[b];
  }
  const int64_t incl = block_inclusive_scan(mine, sh);
  if (threadIdx.x == blockDim.x - 1) total_nonzero = incl;
  __syncthreads();
  const int64_t zeros = n_g - total_nonzero;
  int64_t run = total_nonzero - incl;
  for (int q = (int)per - 1; q >= 0; --q) {
    const uint32_t b = b0 + (uint32_t)q;
    if (b >= kMaxBins) continue;
    const int64_t h = (b == 0) ? zeros : (int64_t)gh[b];
    if (run < need && run + h >= need) { found_d = b; found_above = run; }
    run += h;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    if (found_d < 0) flag_status(status, kStatusInternal);
    gst[gi] = GroupState{(uint32_t)(found_d < 0 ? 0 : found_d), 0, need - found_above};
  }
}

// Per member unit: entries above the group's threshold key and entries equal to it.
__global__ void __launch_bounds__(1024) k_member_counts(const DevTensor* __restrict__ tab, int K,
                                                        const int* __restrict__ gid,
                                                        const GroupState* __restrict__ gst,
                                                        const uint32_t* __restrict__ hist, int64_t* __restrict__ mcnt) {
  __shared__ int64_t sh[16];
  const int u = blockIdx.x, j = u / K, i = u % K;
  const int g = gid[j];
  if (g < 0) return;
  const GroupState G = gst[g * K + i];
  if (G.none) return;
  const uint32_t* h = hist + (size_t)u * kMaxBins;
  int64_t above = 0, nonzero = 0;
  for (uint32_t b = threadIdx.x + 1; b < kMaxBins; b += blockDim.x) {
    const int64_t v = h[b];
    nonzero += v;
    if (b > G.t_key) above += v;
  }
  above = block_inclusive_scan(above, sh);
  __syncthreads();
  nonzero = block_inclusive_scan(nonzero, sh);
  if (threadIdx.x == blockDim.x - 1) {
    mcnt[2 * (size_t)u] = above;
    mcnt[2 * (size_t)u + 1] = (G.t_key == 0) ? tab[j].n - nonzero : (int64_t)h[G.t_key];
  }
}

// One thread per (group, delta): the threshold entries go to the members in table order.
__global__ void k_group_assign(int n_groups, int K, const int* __restrict__ gmem, const int* __restrict__ gmem0,
                               const GroupState* __restrict__ gst, const int64_t* __restrict__ mcnt,
                               UnitState* __restrict__ st) {
  const int gi = blockIdx.x * blockDim.x + threadIdx.x;
  if (gi >= n_groups * K) return;
  const int g = gi / K, i = gi % K;
  const GroupState G = gst[gi];
  if (G.none) return;
  int64_t rem = G.quota;
  for (int m = gmem0[g]; m < gmem0[g + 1]; ++m) {
    const int u = gmem[m] * K + i;
    if (st[u].done) continue;                       // an empty member
    const int64_t ties = mcnt[2 * (size_t)u + 1];
    const int64_t take = rem < ties ? rem : ties;
    rem -= take;
    const int64_t kk = mcnt[2 * (size_t)u] + take;
    st[u].k_rem = kk;
    if (kk == 0) {
      st[u].done = 1;
      st[u].prefix = kNoSelectKey;
    }
  }
}

// ---- ties from the chunk histograms: prefix over chunks, then one walk inside a chunk -----------

template <int DT>
__global__ void __launch_bounds__(kHistThreads) k_tie_find_dump(const DevTensor* __restrict__ tab, int K,
                                                                const int64_t* __restrict__ item0, int64_t chunk,
                                                                UnitState* __restrict__ st,
                                                                const uint32_t* __restrict__ dump, int bits,
                                                                uint32_t* status) {
  using F = Fmt<DT>;
  __shared__ int64_t sh[16];
  __shared__ int64_t s_chunk, s_before, s_seg, s_segbefore, s_idx, s_tot;
  const int u = blockIdx.x;
  if (st[u].done) return;
  const int j = u / K, i = u % K;
  const DevTensor& T = tab[j];
  const uint32_t nb = 1u << bits;
  const int64_t nch = (T.n + chunk - 1) / chunk;
  const int64_t first_item = item0[j] + (int64_t)i * nch;
  const int64_t quota = st[u].k_rem;
  const uint32_t tk = st[u].prefix;
  const uint32_t digit = tk & (nb - 1u);
  if (threadIdx.x == 0) { s_chunk = -1; s_before = 0; s_seg = -1; s_segbefore = 0; s_idx = -1; }
  __syncthreads();
  // 1) chunk holding the quota-th tie
  int64_t base = 0;
  for (int64_t c0 = 0; c0 < nch; c0 += blockDim.x) {
    const int64_t c = c0 + threadIdx.x;
    const int64_t v = (c < nch) ? (int64_t)dump[(size_t)(first_item + c) * nb + digit] : 0;
    const int64_t incl = block_inclusive_scan(v, sh);
    if (c < nch && base + incl - v < quota && base + incl >= quota) { s_chunk = c; s_before = base + incl - v; }
    if (threadIdx.x == blockDim.x - 1) s_tot = incl;
    __syncthreads();
    base += s_tot;
    __syncthreads();
    if (s_chunk >= 0) break;
  }
  __syncthreads();
  if (s_chunk < 0) {                                   // inconsistent counts: never walk out of range
    if (threadIdx.x == 0) { st[u].cutoff = T.n; st[u].done = 1; flag_status(status, kStatusInternal); }
    return;
  }
  const int64_t e0 = s_chunk * chunk, e1 = min(T.n, e0 + chunk);
  const int64_t want = quota - s_before;               // 1-based rank inside the chunk
  // 2) per-thread segments of whole vectors, in flat order
  const void* p = T.deltas[i];
  const int64_t len = e1 - e0;
  int64_t seg = (len + blockDim.x - 1) / blockDim.x;
  seg = (seg + F::kPerVec - 1) / F::kPerVec * F::kPerVec;
  const int64_t a0 = min(e1, e0 + (int64_t)threadIdx.x * seg), a1 = min(e1, a0 + seg);
  int64_t m = 0;
  {
    int64_t e = a0;
    for (; e + F::kPerVec <= a1; e += F::kPerVec) {
      uint4 q = *((const uint4*)p + e / F::kPerVec);
      uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        if constexpr (DT == ISO_BF16) m += ((w[h] & 0x7FFFu) == tk) + (((w[h] >> 16) & 0x7FFFu) == tk);
        else m += ((w[h] & 0x7FFFFFFFu) == tk);
      }
    }
    for (; e < a1; ++e) m += ((elem_bits<DT>(p, e) & F::kKeyMask) == tk);
  }
  const int64_t incl = block_inclusive_scan(m, sh);
  if (m > 0 && incl - m < want && incl >= want) { s_seg = threadIdx.x; s_segbefore = incl - m; }
  __syncthreads();
  if (s_seg < 0) {
    if (threadIdx.x == 0) { st[u].cutoff = T.n; st[u].done = 1; flag_status(status, kStatusInternal); }
    return;
  }
  // 3) the block walks that one segment (seg <= blockDim.x entries)
  const int64_t g0 = min(e1, e0 + s_seg * seg);
  const int64_t e = g0 + threadIdx.x;
  const int64_t tie = (threadIdx.x < seg && e < e1) ? ((elem_bits<DT>(p, e) & F::kKeyMask) == tk) : 0;
  const int64_t r = block_inclusive_scan(tie, sh);
  if (tie && s_segbefore + r == want) s_idx = e;
  __syncthreads();
  if (threadIdx.x == 0) {
    if (s_idx < 0) flag_status(status, kStatusInternal);
    st[u].cutoff = (s_idx < 0) ? T.n : s_idx + 1;
    st[u].done = 1;
  }
}

// ---- ties: count threshold keys per chunk, then walk to the quota-th one -------------------------

template <int DT>
__device__ void tie_count_item(const DevTensor* __restrict__ tab, int K, int j, int i, int64_t c, int64_t item,
                               int64_t chunk, const UnitState* __restrict__ st, int32_t* __restrict__ cnt,
                               int64_t* sh) {
  using F = Fmt<DT>;
  const int u = j * K + i;
  if (st[u].done) return;
  const uint32_t tk = st[u].prefix;
  const DevTensor& T = tab[j];
  const int64_t e0 = c * chunk, e1 = min(T.n, e0 + chunk);
  const void* p = T.deltas[i];
  int64_t m = 0;
  const int64_t v0 = e0 / F::kPerVec, v1 = e1 / F::kPerVec;
  for (int64_t v = v0 + threadIdx.x; v < v1; v += blockDim.x) {
    uint4 a = ld_stream((const uint4*)p + v);
    uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      if constexpr (DT == ISO_BF16) {
        m += ((w[h] & 0x7FFFu) == tk) + (((w[h] >> 16) & 0x7FFFu) == tk);
      } else {
        m += ((w[h] & 0x7FFFFFFFu) == tk);
      }
    }
  }
  for (int64_t e = v1 * F::kPerVec + threadIdx.x; e < e1; e += blockDim.x)
    m += ((elem_bits<DT>(p, e) & F::kKeyMask) == tk);
  m = wave_sum_i64(m);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) cnt[item] = (int32_t)(sh[0] + sh[1] + sh[2] + sh[3]);
  __syncthreads();
}

template <int DT>
__global__ void __launch_bounds__(256) k_tie_count(const DevTensor* __restrict__ tab, int n_t, int K,
                                                   const int64_t* __restrict__ item0, int64_t chunk,
                                                   const UnitState* __restrict__ st, int32_t* __restrict__ cnt) {
  __shared__ int64_t sh[4];
  int j, i;
  int64_t c;
  item_of(item0, n_t, K, chunk, tab, blockIdx.x, j, i, c);
  tie_count_item<DT>(tab, K, j, i, c, blockIdx.x, chunk, st, cnt, sh);
}

template <int DT>
__global__ void __launch_bounds__(256) k_tie_count_flagged(const DevTensor* __restrict__ tab, int n_t, int K,
                                                           const int64_t* __restrict__ item0, int64_t chunk,
                                                           const UnitState* __restrict__ st,
                                                           int32_t* __restrict__ cnt, const int* __restrict__ filter) {
  __shared__ int64_t sh[4];
  __shared__ int sflag[1024];
  for_flagged_items(
      filter, n_t, sflag, [&](int j) { return (int64_t)K * ((tab[j].n + chunk - 1) / chunk); },
      [&](int j, int64_t it) {
        const int64_t nch = (tab[j].n + chunk - 1) / chunk;
        const int i = (int)(it / nch);
        tie_count_item<DT>(tab, K, j, i, it - (int64_t)i * nch, item0[j] + it, chunk, st, cnt, sh);
      });
}

template <int DT>
__global__ void __launch_bounds__(kHistThreads) k_tie_find(const DevTensor* __restrict__ tab, int K,
                                                           const int64_t* __restrict__ item0, int64_t chunk,
                                                           UnitState* __restrict__ st,
                                                           const int32_t* __restrict__ cnt, uint32_t* cnt_status) {
  using F = Fmt<DT>;
  __shared__ int64_t sh[16];
  __shared__ int64_t s_chunk, s_before;
  __shared__ int64_t s_idx;
  const int u = blockIdx.x;
  if (st[u].done) return;
  const int j = u / K, i = u % K;
  const DevTensor& T = tab[j];
  const int64_t nch = (T.n + chunk - 1) / chunk;
  const int32_t* cu = cnt + item0[j] + (int64_t)i * nch;
  const int64_t quota = st[u].k_rem;
  const uint32_t tk = st[u].prefix;
  if (threadIdx.x == 0) { s_chunk = -1; s_before = 0; s_idx = -1; }
  __syncthreads();
  // 1) chunk that holds the quota-th tie
  int64_t base = 0;
  for (int64_t c0 = 0; c0 < nch; c0 += blockDim.x) {
    int64_t c = c0 + threadIdx.x;
    int64_t v = (c < nch) ? cu[c] : 0;
    int64_t incl = block_inclusive_scan(v, sh);
    int64_t excl = incl - v;
    if (c < nch && base + excl < quota && base + incl >= quota) { s_chunk = c; s_before = base + excl; }
    __shared__ int64_t s_tot;
    if (threadIdx.x == blockDim.x - 1) s_tot = incl;
    __syncthreads();
    base += s_tot;
    __syncthreads();
    if (s_chunk >= 0) break;
  }
  __syncthreads();
  if (s_chunk < 0) {                                  // inconsistent tie counts: never walk out of range
    if (threadIdx.x == 0) { st[u].cutoff = T.n; st[u].done = 1; flag_status(cnt_status, kStatusInternal); }
    return;
  }
  const int64_t c = s_chunk;
  int64_t want = quota - s_before;                    // 1-based rank inside the chunk
  // 2) walk the chunk in flat order
  const void* p = T.deltas[i];
  const int64_t e0 = c * chunk, e1 = min(T.n, e0 + chunk);
  int64_t seen = 0;
  for (int64_t b = e0; b < e1; b += blockDim.x) {
    int64_t e = b + threadIdx.x;
    int64_t tie = (e < e1) ? ((elem_bits<DT>(p, e) & F::kKeyMask) == tk) : 0;
    int64_t incl = block_inclusive_scan(tie, sh);
    if (tie && seen + incl == want) s_idx = e;
    __shared__ int64_t s_tot2;
    if (threadIdx.x == blockDim.x - 1) s_tot2 = incl;
    __syncthreads();
    seen += s_tot2;
    __syncthreads();
    if (s_idx >= 0) break;
  }
  if (threadIdx.x == 0) {
    if (s_idx < 0) flag_status(cnt_status, kStatusInternal);
    st[u].cutoff = (s_idx < 0) ? T.n : s_idx + 1;
    st[u].done = 1;
  }
}

__global__ void k_emit_desc(const UnitState* __restrict__ st, int n_units, iso_select_desc* __restrict__ desc) {
  int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= n_units) return;
  UnitState s = st[u];
  iso_select_desc d;
  d.t_key = s.prefix;
  d.key_max = s.key_max;
  if (s.prefix == kNoSelectKey) {
    d.n_above = 0; d.tie_quota = 0; d.tie_cutoff = 0;
  } else {
    d.n_above = s.n_above; d.tie_quota = s.k_rem; d.tie_cutoff = s.cutoff;
  }
  desc[u] = d;
}

// ---- optional bitset output ---------------------------------------------------------------------

template <int DT>
__global__ void __launch_bounds__(256) k_mask_bits(const DevTensor* __restrict__ tab, int n_t, int K,
                                                   const iso_select_desc* __restrict__ desc,
                                                   uint32_t* const* __restrict__ bits_out, int64_t words_per_block) {
  using F = Fmt<DT>;
  const int u = blockIdx.y;
  const int j = u / K, i = u % K;
  const DevTensor& T = tab[j];
  const iso_select_desc d = desc[u];
  const int64_t nw = (T.n + 31) / 32;
  uint32_t* out = bits_out[u];
  const void* p = T.deltas[i];
  for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < nw; w += (int64_t)gridDim.x * blockDim.x) {
    uint32_t m = 0;
    for (int b = 0; b < 32; ++b) {
      int64_t e = w * 32 + b;
      if (e >= T.n) break;
      uint32_t key = elem_bits<DT>(p, e) & F::kKeyMask;
      bool sel = (d.t_key != kNoSelectKey) && (key > d.t_key || (key == d.t_key && e < d.tie_cutoff));
      m |= (uint32_t)sel << b;
    }
    out[w] = m;
  }
  (void)n_t;
  (void)words_per_block;
}

__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// ---- host-side launch sequence ------------------------------------------------------------------

int64_t hist_chunk_for(int64_t total_elems_times_k) {
  int64_t c = 1 << 16;
  while (c < (1 << 20) && total_elems_times_k / c > 2048) c <<= 1;
  return c;
}

hipError_t fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
  k_fill_u32<<<(unsigned)blocks, 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

template <int DT>
static hipError_t run_select_t(const SelectPlan& pl, hipStream_t s) {
  const int nu = pl.n_t * pl.K;
  const bool flt = pl.filter != nullptr;
  constexpr unsigned kFlaggedGrid = 256;
  if (flt) k_clear_hist_flagged<<<kFlaggedGrid, 1024, 0, s>>>(pl.n_t, pl.K, pl.hist, pl.filter);
  if (pl.n_groups > 0 && DT != ISO_BF16) return hipErrorInvalidValue;   // the entry points reject these
  k_select_init<<<(nu + 255) / 256, 256, 0, s>>>(pl.tab, pl.n_t, pl.K, pl.states, pl.filter,
                                                 pl.n_groups > 0 ? pl.gid : nullptr, pl.gk);
  struct Pass { int shift, bits; };
  const Pass bf[1] = {{0, 15}};
  const Pass f32[3] = {{16, 15}, {8, 8}, {0, 8}};
  const Pass* ps = (DT == ISO_BF16) ? bf : f32;
  const int np = (DT == ISO_BF16) ? 1 : 3;
  for (int q = 0; q < np; ++q) {
    uint32_t* dump = (q == np - 1) ? pl.chunk_hist : nullptr;
    if (pl.hist_items > 0 && flt)
      k_hist_flagged<DT><<<kFlaggedGrid, kHistThreads, 0, s>>>(pl.tab, pl.n_t, pl.K, pl.hist_item0, pl.hist_chunk,
                                                               pl.states, pl.hist, ps[q].shift, ps[q].bits, q == 0,
                                                               pl.status, dump, pl.filter);
    else if (pl.hist_items > 0)
      k_hist<DT><<<(unsigned)pl.hist_items, kHistThreads, 0, s>>>(pl.tab, pl.n_t, pl.K, pl.hist_item0, pl.hist_chunk,
                                                                  pl.states, pl.hist, ps[q].shift, ps[q].bits,
                                                                  q == 0, pl.status, dump);
    if (pl.n_groups > 0) {
      const int ngk = pl.n_groups * pl.K;
      k_group_sum<<<dim3(kMaxBins / 256, (unsigned)ngk), 256, 0, s>>>(pl.K, pl.gmem, pl.gmem0, pl.hist, pl.ghist);
      k_group_resolve<<<ngk, kHistThreads, 0, s>>>(pl.tab, pl.K, pl.gmem, pl.gmem0, pl.gk, pl.ghist, pl.gstate,
                                                   pl.status);
      k_member_counts<<<nu, 1024, 0, s>>>(pl.tab, pl.K, pl.gid, pl.gstate, pl.hist, pl.mcnt);
      k_group_assign<<<(ngk + 63) / 64, 64, 0, s>>>(pl.n_groups, pl.K, pl.gmem, pl.gmem0, pl.gstate, pl.mcnt,
                                                    pl.states);
    }
    k_resolve<<<nu, kHistThreads, 0, s>>>(pl.tab, pl.K, pl.states, pl.hist, ps[q].shift, ps[q].bits, q == np - 1,
                                          pl.status);
  }
  if (pl.chunk_hist != nullptr) {
    k_tie_find_dump<DT><<<nu, kHistThreads, 0, s>>>(pl.tab, pl.K, pl.hist_item0, pl.hist_chunk, pl.states,
                                                    pl.chunk_hist, ps[np - 1].bits, pl.status);
  } else {
    if (pl.tie_items > 0 && flt)
      k_tie_count_flagged<DT><<<kFlaggedGrid * 4, 256, 0, s>>>(pl.tab, pl.n_t, pl.K, pl.tie_item0, pl.tie_chunk,
                                                               pl.states, pl.tie_cnt, pl.filter);
    else if (pl.tie_items > 0)
      k_tie_count<DT><<<(unsigned)pl.tie_items, 256, 0, s>>>(pl.tab, pl.n_t, pl.K, pl.tie_item0, pl.tie_chunk,
                                                             pl.states, pl.tie_cnt);
    k_tie_find<DT><<<nu, kHistThreads, 0, s>>>(pl.tab, pl.K, pl.tie_item0, pl.tie_chunk, pl.states, pl.tie_cnt,
                                                pl.status);
  }
  k_emit_desc<<<(nu + 255) / 256, 256, 0, s>>>(pl.states, nu, pl.desc);
  return hipGetLastError();
}

int select_last_bits(int dt) { return dt == ISO_BF16 ? 15 : 8; }

hipError_t run_select(const SelectPlan& pl, int dt, hipStream_t s) {
  return dt == ISO_BF16 ? run_select_t<ISO_BF16>(pl, s) : run_select_t<ISO_F32>(pl, s);
}

hipError_t run_mask_bits(const DevTensor* tab, int n_t, int K, int dt, const iso_select_desc* desc,
                         uint32_t* const* bits_dev, int64_t max_n, hipStream_t s) {
  const int nu = n_t * K;
  int64_t nw = (max_n + 31) / 32;
  unsigned gx = (unsigned)std::max<int64_t>(1, std::min<int64_t>((nw + 255) / 256, 2048));
  dim3 grid(gx, nu);
  if (dt == ISO_BF16) k_mask_bits<ISO_BF16><<<grid, 256, 0, s>>>(tab, n_t, K, desc, bits_dev, 0);
  else k_mask_bits<ISO_F32><<<grid, 256, 0, s>>>(tab, n_t, K, desc, bits_dev, 0);
  return hipGetLastError();
}

}  // namespace iso
