// Host-side launchers of the libiso kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "iso.h"
#include "iso_device.h"

namespace iso {

// Per (group, delta) of a joint selection: threshold key and how many entries with that key
// the group keeps.
struct GroupState {
  uint32_t t_key;
  int32_t none;      // 1: the group keeps nothing
  int64_t quota;
};

struct SelectPlan {
  const DevTensor* tab;
  int n_t, K;
  UnitState* states;
  uint32_t* hist;               // n_t*K * 32768 u32, zero on entry
  const int64_t* hist_item0;    // n_t prefix of K*ceil(n/hist_chunk)
  int64_t hist_chunk, hist_items;
  const int64_t* tie_item0;     // n_t prefix of K*ceil(n/tie_chunk)
  int64_t tie_chunk, tie_items;
  int32_t* tie_cnt;             // tie_items (used when chunk_hist is null)
  uint32_t* chunk_hist;         // hist_items * 2^last_bits per-chunk histograms of the last pass, or null
  iso_select_desc* desc;        // n_t*K, device
  uint32_t* status;
  const int* filter = nullptr;  // n_t device flags: only flagged tensors are selected (others get
                                // t_key = none); null: every tensor.  Histograms of flagged units are
                                // cleared by the launch itself.
  // joint selection (bf16): n_groups groups of tensors selected together per delta
  int n_groups = 0;
  const int* gid = nullptr;         // n_t: dense group index or -1
  const int* gmem = nullptr;        // members of every group, in table order
  const int* gmem0 = nullptr;       // n_groups + 1 offsets into gmem
  const int64_t* gk = nullptr;      // n_groups: the group's count (sum of its members' k)
  uint64_t* ghist = nullptr;        // n_groups * K * 32768
  GroupState* gstate = nullptr;     // n_groups * K
  int64_t* mcnt = nullptr;          // 2 * n_t * K: per unit, entries above the group threshold and ties
};

int64_t hist_chunk_for(int64_t total_elems_times_k);
hipError_t fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s);
hipError_t run_select(const SelectPlan& pl, int dt, hipStream_t s);
int select_last_bits(int dt);
hipError_t run_mask_bits(const DevTensor* tab, int n_t, int K, int dt, const iso_select_desc* desc,
                         uint32_t* const* bits_dev, int64_t max_n, hipStream_t s);

// Outputs of the element-wise merge kernel.
enum : int { OUT_W = 1, OUT_TAU = 2, OUT_SIGN = 4 };

struct MergePlan {
  const DevTensor* tab;         // .out = weights (OUT_W), .aux = tau (OUT_TAU) or sign (OUT_SIGN alone),
                                // .aux2 = sign when OUT_W|OUT_SIGN
  int n_t, K;
  int mode;                     // iso_merge_mode
  int outs;                     // OUT_* bits
  const iso_select_desc* desc;  // TIES thresholds (n_t*K), or nullptr: every entry kept
  double lambda, eps;
  int64_t tiles;                // total tiles over the table
  uint32_t* status;
  const int* filter = nullptr;  // n_t device flags: only flagged tensors are merged; null: every tensor
  hipEvent_t prof[2] = {nullptr, nullptr};   // recorded around the merge kernel when set
};

int64_t merge_tile_elems(int dt);
hipError_t run_merge(const MergePlan& pl, int dt, hipStream_t s);
hipError_t run_apply(const DevTensor* tab, int n_t, int dt, double lambda, int64_t tiles, uint32_t* status,
                     hipStream_t s);

}  // namespace iso
