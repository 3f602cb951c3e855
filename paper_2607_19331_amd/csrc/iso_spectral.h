// ISO-Merger (Algorithm 1) on the GPU in binary64: host-side launcher (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "iso.h"

namespace iso {

struct SpectralArgs {
  double rho_keep, ridge, c_min, c_max;
  double* coef_out;   // n_t*K device doubles or nullptr
};

size_t spectral_workspace_bytes(const iso_tensor* t, int n_t, int K);
size_t optimizer_workspace_bytes(const iso_frame* f, int n_f);
// diagnostics (out != nullptr) or spectrum interpolation (alpha) of each tensor, one at a time
iso_status run_spectrum_ops(const iso_tensor* t, int n_t, iso_dtype dt, double* out, double alpha, uint8_t* ws,
                            uint32_t* status, hipStream_t s);
iso_status run_optimizer(const iso_frame* f, int n_f, iso_dtype dt, const iso_adamw& o, uint8_t* ws,
                         uint32_t* status, hipStream_t s);
iso_status run_spectral(const iso_tensor* t, int n_t, int K, iso_dtype dt, const SpectralArgs& a, uint8_t* ws,
                        uint32_t* status, hipStream_t s);

}  // namespace iso
