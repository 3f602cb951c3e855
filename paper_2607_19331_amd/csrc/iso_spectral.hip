#include "iso_spectral.h"

namespace iso {

size_t spectral_workspace_bytes(const iso_tensor* t, int n_t, int K) {
  (void)t; (void)n_t; (void)K;
  return 0;
}

iso_status run_spectral(const iso_tensor* t, int n_t, int K, iso_dtype dt, const SpectralArgs& a, uint8_t* ws,
                        uint32_t* status, hipStream_t s) {
  (void)t; (void)n_t; (void)K; (void)dt; (void)a; (void)ws; (void)status; (void)s;
  return ISO_ERR_UNSUPPORTED;
}

}  // namespace iso
