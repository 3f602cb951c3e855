// TSV-Merge block-diagonal/SVD projection on the GPU: host-side launcher (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "iso.h"

namespace iso {

struct TsvArgs {
  int rank;          // r: top singular triplets kept per delta
  double alpha;      // W = W_0 + alpha * Delta_hat
  float* const* delta_hat;   // optional: n_t device pointers, N floats each (row-major)
  const iso_factors* factors = nullptr;   // optional: n_t*K given truncated factors (skip the SVD)
};

// Sketch width used for rank r on an R x C matrix, or 0 if the shape is too small.
int tsv_sketch_width(int64_t R, int64_t C, int r);
size_t tsv_workspace_bytes(const iso_tensor* t, int n_t, int K, int rank);
iso_status run_tsv(const iso_tensor* t, int n_t, int K, const TsvArgs& a, uint8_t* ws, size_t ws_bytes,
                   uint32_t* status, hipStream_t s);

}  // namespace iso
