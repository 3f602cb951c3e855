// Internal device-side definitions shared by the libiso kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "iso.h"

namespace iso {

// ---- workspace layout ----------------------------------------------------------------------------
// [0, 256)            status block (u32 flags)
// [256, ...)          per-call tables and scratch, each region 256-byte aligned
constexpr size_t kStatusBytes = 256;
constexpr uint32_t kStatusNonFinite = 1u;
constexpr uint32_t kStatusInternal = 2u;   // a kernel found counts that cannot occur; results invalid

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Global-memory view of a generic pointer (one that points into device memory).  A pointer read
// from a job or problem table is generic, and accesses through it compile to flat instructions,
// which count against the LDS wait counter as well as the vector-memory one: every wait for an LDS
// read then also waits for the global loads in flight, so a prefetch issued before the LDS reads
// of the current step is drained by them.  Through this view they compile to global instructions.
template <typename T>
__device__ __forceinline__ const __attribute__((address_space(1))) T* gmem(const T* p) {
  return (const __attribute__((address_space(1))) T*)p;
}
template <typename T>
__device__ __forceinline__ __attribute__((address_space(1))) T* gmem(T* p) {
  return (__attribute__((address_space(1))) T*)p;
}

// Table entry as the kernels see it.
struct DevTensor {
  const void* base;
  const void* deltas[ISO_MAX_K];
  void* out;        // weight output (FUSED / APPLY) or nullptr
  void* aux;        // tau_out (float) / sign_out (int8) / tau_in (float), per entry point
  void* aux2;       // second optional output (FUSED TIES sign_out)
  int64_t n;        // elements
  int64_t k;        // TopKMask count
  int64_t tile0;    // first tile of this tensor in the launch's tile space
  int64_t group0;   // first record region of this tensor (single-read fused path)
};
static_assert(sizeof(DevTensor) % 16 == 0, "table entry alignment");

// Per (tensor, delta) select state, lives in the workspace.
struct UnitState {
  uint32_t prefix;     // key bits fixed so far (final: t_key)
  uint32_t key_max;    // largest key (atomicMax in the first histogram pass)
  int64_t k_rem;       // rank still to place inside the current prefix bucket
  int64_t n_above;     // elements with key strictly above the prefix bucket
  int64_t bucket;      // elements inside the current prefix bucket
  int64_t cutoff;      // final tie cutoff
  int32_t done;        // 1 when the descriptor is final before the tie search
  int32_t pad[3];
};
static_assert(sizeof(UnitState) == 56, "unit state size");

constexpr uint32_t kNoSelectKey = 0xFFFFFFFFu;

// ---- storage-format helpers ----------------------------------------------------------------------

template <int DT> struct Fmt;
template <> struct Fmt<ISO_BF16> {
  using bits_t = uint16_t;
  static constexpr int kPerVec = 8;           // elements per 16-byte vector
  static constexpr uint32_t kKeyMask = 0x7FFFu;
  static constexpr int kKeyBits = 15;
};
template <> struct Fmt<ISO_F32> {
  using bits_t = uint32_t;
  static constexpr int kPerVec = 4;
  static constexpr uint32_t kKeyMask = 0x7FFFFFFFu;
  static constexpr int kKeyBits = 31;
};

// Streaming (read-once / write-once) 16-byte accesses.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_stream(const uint4* p) {
  u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 ld_stream(const float4* p) {
  f32x4_t v = __builtin_nontemporal_load((const f32x4_t*)p);
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st_stream(uint4 v, uint4* p) {
  u32x4_t w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, (u32x4_t*)p);
}
__device__ __forceinline__ void st_stream(float4 v, float4* p) {
  f32x4_t w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, (f32x4_t*)p);
}

__device__ __forceinline__ float f32_from_bits(uint32_t b) { return __uint_as_float(b); }
__device__ __forceinline__ uint32_t bits_from_f32(float f) { return __float_as_uint(f); }

// bits of element e (0..7) of a 16-byte vector of bf16 held as uint4, widened to fp32 bits
__device__ __forceinline__ uint32_t bf16_word(const uint4& v, int e) {
  uint32_t w = (e < 2) ? v.x : (e < 4) ? v.y : (e < 6) ? v.z : v.w;
  return (e & 1) ? (w & 0xFFFF0000u) : (w << 16);
}

// binary64 -> bf16 with one round-to-nearest-even step: round to binary32 with
// round-to-odd (which keeps the information a second rounding needs), then
// round that to bf16 with round-to-nearest-even.  Round-to-odd to a format
// with at least two more significand bits than the target makes the double
// rounding innocuous (Boldo & Melquiond, "Emulation of FMA and correctly
// rounded sums: proved algorithms using rounding to odd", IEEE TC 2008).
__device__ __forceinline__ uint32_t f64_to_bf16_rne(double v) {
  float f = (float)v;                       // round to nearest even
  uint32_t b = bits_from_f32(f);
  double back = (double)f;
  if (back != v) {                          // inexact (NaN compares unequal: keep NaN bits)
    if (v == v) {
      if (fabs(back) > fabs(v)) b -= 1u;    // step the magnitude back toward zero: truncation
      b |= 1u;                              // sticky: odd
    }
  }
  if ((b & 0x7FFFFFFFu) > 0x7F800000u) return (b >> 16) | 0x40u;   // quiet NaN
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// The first half of that rounding for finite v: binary64 to binary32 with round-to-odd, as bits.
__device__ __forceinline__ uint32_t f64_to_f32_odd_bits(double v) {
  const float f = (float)v;
  uint32_t b = bits_from_f32(f);
  const double back = (double)f;
  if (back != v) {
    if (fabs(back) > fabs(v)) b -= 1u;
    b |= 1u;
  }
  return b;
}

typedef __bf16 iso_bf16x2_t __attribute__((ext_vector_type(2)));
typedef float iso_f32x2_t __attribute__((ext_vector_type(2)));

// The second half for two values at once: finite binary32 bit patterns to bf16 with
// round-to-nearest-even in one v_cvt_pk_bf16_f32 (lo in bits 0-15, hi in 16-31); the same
// result as the integer rounding below for every finite input, denormals included.
__device__ __forceinline__ uint32_t pack_bf16_rne(uint32_t lo, uint32_t hi) {
  const iso_f32x2_t v = {__uint_as_float(lo), __uint_as_float(hi)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, iso_bf16x2_t));
}

// The same rounding for finite v without the NaN case (callers that flag non-finite
// inputs elsewhere and leave such outputs unspecified).
__device__ __forceinline__ uint32_t f64_to_bf16_rne_finite(double v) {
  const float f = (float)v;
  uint32_t b = bits_from_f32(f);
  const double back = (double)f;
  if (back != v) {
    if (fabs(back) > fabs(v)) b -= 1u;
    b |= 1u;
  }
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ double load_f64(const void* p, int64_t i, int dt) {
  if (dt == ISO_BF16) return (double)f32_from_bits((uint32_t)((const uint16_t*)p)[i] << 16);
  return (double)((const float*)p)[i];
}

// Scalar access for tails.
template <int DT>
__device__ __forceinline__ uint32_t elem_bits(const void* p, int64_t i) {
  if constexpr (DT == ISO_BF16) return (uint32_t)((const uint16_t*)p)[i];
  else return ((const uint32_t*)p)[i];
}
template <int DT>
__device__ __forceinline__ double bits_to_f64(uint32_t b) {
  if constexpr (DT == ISO_BF16) return (double)f32_from_bits(b << 16);
  else return (double)f32_from_bits(b);
}
template <int DT>
__device__ __forceinline__ bool bits_nonfinite(uint32_t b) {
  if constexpr (DT == ISO_BF16) return (b & 0x7F80u) == 0x7F80u;
  else return (b & 0x7F800000u) == 0x7F800000u;
}

__device__ __forceinline__ void flag_status(uint32_t* status, uint32_t f) {
  __hip_atomic_fetch_or(status, f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Find the tensor owning global tile `tile` (tile0 ascending).
__device__ __forceinline__ int find_tensor(const DevTensor* tab, int n_t, int64_t tile) {
  int lo = 0, hi = n_t - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (tab[mid].tile0 <= tile) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Coarse tile map: entry m holds the tensor owning tile m << kTileMapShift, so a lookup is one
// read and a short forward walk (none at all when every tensor spans at least 2^kTileMapShift
// tiles and the tile is not in the first block of a tensor's range).
constexpr int kTileMapShift = 8;
inline int64_t tile_map_entries(int64_t tiles) { return (tiles >> kTileMapShift) + 1; }

__device__ __forceinline__ int find_tensor_mapped(const DevTensor* tab, const int* tmap, int n_t, int64_t tile) {
  int j = tmap[tile >> kTileMapShift];
  while (j + 1 < n_t && tab[j + 1].tile0 <= tile) ++j;
  return j;
}

// Persistent-grid walk over the work of flagged tensors only.  Every block scans the flags
// (through LDS, 1024 at a time) in tensor order and takes every gridDim.x-th work item of
// the flagged tensors; count(j) gives tensor j's item count.  With no flag set a block
// only reads the flags.  body(j, item) may synchronise the block: the loop is uniform.
template <class Count, class Body>
__device__ __forceinline__ void for_flagged_items(const int* __restrict__ flags, int n_t, int* sflag, Count count,
                                                  Body body) {
  const int64_t G = gridDim.x;
  int64_t run = 0;   // items of flagged tensors before tensor j
  for (int j0 = 0; j0 < n_t; j0 += 1024) {
    __syncthreads();
    for (int q = threadIdx.x; q < 1024; q += blockDim.x) sflag[q] = (j0 + q < n_t) ? flags[j0 + q] : 0;
    __syncthreads();
    const int nq = min(1024, n_t - j0);
    for (int q = 0; q < nq; ++q) {
      if (!sflag[q]) continue;
      const int j = j0 + q;
      const int64_t m = count(j);
      int64_t first = ((int64_t)blockIdx.x - run) % G;
      if (first < 0) first += G;
      for (int64_t it = first; it < m; it += G) body(j, it);
      run += m;
    }
  }
}

}  // namespace iso
