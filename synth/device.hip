// Device fill of synthetic tensors (hipcc build of philox.h).  Benchmark and
// test infrastructure: generates large inputs directly in HBM with the same
// bits as the host build.
#include <hip/hip_runtime.h>
#include "philox.h"

namespace {

template <typename T>
__global__ void __launch_bounds__(256) synth_fill_kernel(T* __restrict__ out, int64_t n, synth_recipe r,
                                                        int64_t first) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    double v = synth_value(&r, (uint64_t)(first + i));
    if constexpr (sizeof(T) == 2) out[i] = synth_bf16_from_f64(v);
    else out[i] = synth_f32_from_f64(v);
  }
}

}  // namespace

extern "C" int synth_fill_device(void* out, int64_t n, int dtype, const synth_recipe* r, int64_t first,
                                 hipStream_t s) {
  if (n <= 0) return 0;
  if (out == nullptr || r == nullptr) return 1;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 256 * 64) blocks = 256 * 64;
  if (dtype == SYNTH_BF16)
    synth_fill_kernel<uint16_t><<<(unsigned)blocks, 256, 0, s>>>((uint16_t*)out, n, *r, first);
  else
    synth_fill_kernel<float><<<(unsigned)blocks, 256, 0, s>>>((float*)out, n, *r, first);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
