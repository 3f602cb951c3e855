// ISO-Merger (Algorithm 1) on the GPU in binary64: host-side launcher (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cmath>

#include "iso.h"

namespace iso {

struct SpectralArgs {
  double rho_keep, ridge, c_min, c_max;
  double* coef_out;   // n_t*K device doubles or nullptr
};

size_t spectral_workspace_bytes(const iso_tensor* t, int n_t, int K);
size_t optimizer_workspace_bytes(const iso_frame* f, int n_f);
enum class SpectrumOp { kDiagnostics, kInterpolate, kTransport, kSpectralError, kSelfSpectralError };

// Truncation rank r = max(1, floor(frac q)) of the unexplained-update ratios.
inline int64_t transport_rank(int64_t q, double frac) {
  const int64_t r = (int64_t)std::floor(frac * (double)q);
  return r < 1 ? 1 : r;
}

// Per tensor, one at a time: drift diagnostics (3 doubles of out), spectrum interpolation
// (param = alpha, writes the tensor's out), unexplained-update ratios (5 doubles of out for
// each of the n_frac host rank fractions) or the mean squared spectral error (1 double of out;
// W_rec = deltas[0], or the reconstruction from the library's own SVD of the base).
iso_status run_spectrum_ops(const iso_tensor* t, int n_t, iso_dtype dt, SpectrumOp op, double* out, double param,
                            const double* fracs, int n_frac, uint8_t* ws, uint32_t* status, hipStream_t s);
// Benchmark timing hooks of the library (defined with iso_profile_begin): the next event pair
// ({null, null} when profiling is off) and the flops performed inside a timed region.
void profile_region(hipEvent_t (&ev)[2]);
void profile_add_flops(double flops);
// One ISO-Optimizer step with AdamW (adam != nullptr) or Muon (muon != nullptr) as the base rule.
iso_status run_optimizer(const iso_frame* f, int n_f, iso_dtype dt, const iso_adamw* adam, const iso_muon* muon,
                         uint8_t* ws, uint32_t* status, hipStream_t s);
iso_status run_spectral(const iso_tensor* t, int n_t, int K, iso_dtype dt, const SpectralArgs& a, uint8_t* ws,
                        uint32_t* status, hipStream_t s);

}  // namespace iso
