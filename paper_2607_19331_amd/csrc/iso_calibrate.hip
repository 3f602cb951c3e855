// Streaming calibration for the roofline, declared in include/iso_calibrate.h (not part of the
// merge path): the traffic pattern of the fused single-read pass with trivial arithmetic.  n_in
// arrays of n_vec 16-byte vectors are read once with nontemporal loads, two vectors per thread in
// 256-thread workgroups as the main pass does, and their XOR is written once (or, with write == 0,
// only read).  One launch over the 7B stack's bytes gives the rate this chip sustains for the mix.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "iso_calibrate.h"

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

struct Inputs {
  const u32x4* p[8];
};

template <int NIN, bool WRITE>
__global__ void __launch_bounds__(256) k_stream(Inputs in, u32x4* out, int64_t n_vec) {
  const int64_t v0 = (int64_t)blockIdx.x * 512;
  u32x4 x[NIN][2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int64_t vi = v0 + q * 256 + threadIdx.x;
#pragma unroll
    for (int r = 0; r < NIN; ++r)
      x[r][q] = (vi < n_vec) ? __builtin_nontemporal_load(in.p[r] + vi) : u32x4{0u, 0u, 0u, 0u};
  }
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    u32x4 acc = x[0][q];
#pragma unroll
    for (int r = 1; r < NIN; ++r) acc ^= x[r][q];
    const int64_t vi = v0 + q * 256 + threadIdx.x;
    if (WRITE) {
      if (vi < n_vec) __builtin_nontemporal_store(acc, out + vi);
    } else if (acc.x == 0x9E3779B9u && acc.y == 0x7F4A7C15u && acc.z == 0u && acc.w == 1u) {
      out[0] = acc;        // never taken on the calibration data (all bytes equal per array); keeps the loads
    }
  }
}

template <int NIN>
hipError_t launch(const Inputs& in, u32x4* out, int64_t n_vec, bool write, hipStream_t s) {
  const unsigned grid = (unsigned)((n_vec + 511) / 512);
  if (write) k_stream<NIN, true><<<grid, 256, 0, s>>>(in, out, n_vec);
  else k_stream<NIN, false><<<grid, 256, 0, s>>>(in, out, n_vec);
  return hipGetLastError();
}

}  // namespace

extern "C" int iso_calibrate_stream(const void* const* in, int n_in, void* out, int64_t n_vec, int write,
                                    void* stream) {
  if (in == nullptr || n_in < 1 || n_in > 8 || out == nullptr || n_vec < 1) return 1;
  Inputs p{};
  for (int r = 0; r < n_in; ++r) {
    if (in[r] == nullptr) return 1;
    p.p[r] = (const u32x4*)in[r];
  }
  hipStream_t s = (hipStream_t)stream;
  u32x4* o = (u32x4*)out;
  hipError_t e;
  switch (n_in) {
    case 1: e = launch<1>(p, o, n_vec, write != 0, s); break;
    case 2: e = launch<2>(p, o, n_vec, write != 0, s); break;
    case 3: e = launch<3>(p, o, n_vec, write != 0, s); break;
    case 4: e = launch<4>(p, o, n_vec, write != 0, s); break;
    case 5: e = launch<5>(p, o, n_vec, write != 0, s); break;
    case 6: e = launch<6>(p, o, n_vec, write != 0, s); break;
    case 7: e = launch<7>(p, o, n_vec, write != 0, s); break;
    default: e = launch<8>(p, o, n_vec, write != 0, s); break;
  }
  return e == hipSuccess ? 0 : 2;
}
