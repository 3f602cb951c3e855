// Single-read TIES select + merge + update for bf16 tensors: host-side launcher (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "iso_device.h"
#include "iso_kernels.h"

namespace iso {

constexpr int kFusedMaxW = 16;                 // codes in one delta's threshold bracket
constexpr int kFusedStat = 1 + kFusedMaxW;     // per (tile, delta): keys above the bracket, one count per code
constexpr int kFusedGroupTiles = 64;           // tiles per fix-up workgroup
constexpr int kFusedReduceTiles = 1024;        // tiles per reduction item
constexpr int kFusedMaxTensors = 65535;        // records carry a 16-bit tensor id

// Tile statistics: K * kFusedStat 16-bit counts per tile (a tile holds 4096 coordinates, so no
// count exceeds 4096), padded to a multiple of 8 so that each tile's block is 16-byte aligned.
constexpr int fused_stat_words(int K) { return (K * kFusedStat + 7) / 8 * 8; }

// Per (tensor, delta) state.
struct FusedUnit {
  uint32_t lo, hi, prov;   // bracket [lo, hi] of magnitude keys and the provisional threshold
  uint32_t flags;          // kFused* below
  uint32_t t_key;          // exact threshold key (kNoSelectKey: nothing kept)
  uint32_t pad;
  int64_t k;
  uint64_t kept;           // entries the main pass kept provisionally (key >= max(prov, 1))
  int64_t n_above, quota, count_t;
  int64_t cutoff;          // tie cutoff (-1: to be found from the records)
  uint32_t h[kFusedMaxW];  // keys equal to lo + c
};

constexpr uint32_t kFusedNone = 1u;   // k == 0
constexpr uint32_t kFusedAll = 2u;    // k == n

struct FusedPlan {
  const DevTensor* tab;
  const int* tmap;         // coarse tile -> tensor map (find_tensor_mapped)
  int n_t, K;
  int64_t tiles, groups;   // groups: runs of up to kFusedGroupTiles tiles of one tensor (fix-up work)
  FusedUnit* fu;           // n_t * K
  int* tflag;              // n_t: nonzero sends the tensor to the exact two-pass path
  uint16_t* tstat;         // tiles * fused_stat_words(K): per tile, delta-major counts
  uint2* tinfo;            // tiles: {records, 1 if the tile is to be merged again in binary64}
  uint32_t* rec;           // tiles * tile_cap records of fused_record_bytes(K)
  int64_t tile_cap;
  const int64_t* ritem0;   // n_t prefix of fused_reduce_items()
  int64_t ritems;
  uint32_t* csum;          // ritems * kFusedStat
  double lambda;
  int want_sign;           // .aux2 of the table holds the int8 sign output
  uint32_t* status;        // status block; word 1 receives the number of tensors that took the two-pass path
  SelectPlan sel;          // exact two-pass path (its filter is set to tflag by the launcher)
  MergePlan mrg;
  hipEvent_t prof[2] = {nullptr, nullptr};   // recorded around the main pass when set
};

int64_t fused_tile_elems();
int64_t fused_groups(int64_t n);   // fix-up runs of a tensor of n entries (tensors never share one)
int64_t fused_reduce_items(int64_t n, int K);
size_t fused_record_bytes(int K);
int64_t fused_tile_cap(int K);
hipError_t run_fused(const FusedPlan& pl, hipStream_t s);

}  // namespace iso
