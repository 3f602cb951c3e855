// OrthoMerge-G-TIES (App. F) on the GPU: host-side launcher (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "iso.h"

namespace iso {

// Workspace of run_ortho after the status word: the largest batch's job tables and matrix blocks
// (consecutive matrices, at most 16 and 48 GiB of blocks a batch, each batch's SVDs of a phase
// as one Jacobi job set; batches run one after another).
size_t ortho_workspace_bytes(const iso_tensor* t, int n_t, int K);
// Every tensor: rows >= cols, k its residual TopKMask count; out = W_rot + lambda tau_TIES(delta).
iso_status run_ortho(const iso_tensor* t, int n_t, int K, iso_dtype dt, double lambda, uint8_t* ws,
                     uint32_t* status, hipStream_t s);

}  // namespace iso
