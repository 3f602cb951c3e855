/* Host fill of synthetic tensors (gcc build of philox.h).  Test and benchmark
 * infrastructure: used to build inputs on the CPU for the oracle and for
 * uploads, and to regenerate sampled elements of device-generated tensors. */
#include "philox.h"
#include <stddef.h>

void synth_fill_host(void* out, int64_t n, int dtype, const synth_recipe* r, int64_t first) {
  if (dtype == SYNTH_BF16) {
    uint16_t* o = (uint16_t*)out;
    for (int64_t i = 0; i < n; ++i) o[i] = synth_bf16_from_f64(synth_value(r, (uint64_t)(first + i)));
  } else {
    float* o = (float*)out;
    for (int64_t i = 0; i < n; ++i) o[i] = synth_f32_from_f64(synth_value(r, (uint64_t)(first + i)));
  }
}

/* Values at an arbitrary list of flat indices. */
void synth_gather_host(void* out, const int64_t* idx, int64_t n, int dtype, const synth_recipe* r) {
  if (dtype == SYNTH_BF16) {
    uint16_t* o = (uint16_t*)out;
    for (int64_t i = 0; i < n; ++i) o[i] = synth_bf16_from_f64(synth_value(r, (uint64_t)idx[i]));
  } else {
    float* o = (float*)out;
    for (int64_t i = 0; i < n; ++i) o[i] = synth_f32_from_f64(synth_value(r, (uint64_t)idx[i]));
  }
}

void synth_philox_host(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  synth_u32x4 c;
  for (int i = 0; i < 4; ++i) c.v[i] = ctr[i];
  c = synth_philox4x32_10(c, key[0], key[1]);
  for (int i = 0; i < 4; ++i) out[i] = c.v[i];
}

double synth_log_host(double x) { return synth_log(x); }
