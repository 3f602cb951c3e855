// Arithmetic of one merged TIES coordinate (App. F: elect + disjoint mean), shared by the
// two-pass merge kernel and the single-read fused kernel.  `kept` has bit i set when delta i
// survives TopKMask at this coordinate; the result is the disjoint mean t (before lambda),
// and gamma the elected sign.
#pragma once

#include "iso_device.h"

namespace iso {

__device__ __forceinline__ void two_sum(double a, double b, double& s, double& e) {
  s = a + b;
  double bb = s - a;
  e = (a - (s - bb)) + (b - bb);
}

// Exact sign of x[0] + ... + x[K-1] (Shewchuk 1997, Grow-Expansion).
template <int K>
__device__ __forceinline__ int exact_sign(const double (&x)[K]) {
  double e[K];
#pragma unroll
  for (int i = 0; i < K; ++i) {
    double q = x[i];
#pragma unroll
    for (int j = 0; j < i; ++j) {
      double s, h;
      two_sum(q, e[j], s, h);
      e[j] = h;
      q = s;
    }
    e[i] = q;
  }
  int sg = 0;
#pragma unroll
  for (int i = 0; i < K; ++i)
    if (e[i] != 0.0) sg = (e[i] > 0.0) ? 1 : -1;
  return sg;
}

// t / n for a count n >= 1: powers of two scale exactly, others divide (IEEE).
__device__ __forceinline__ double div_count(double t, int n) {
  if ((n & (n - 1)) == 0) {
    int s = __ffs(n) - 1;
    return t * __hiloint2double((1023 - s) << 20, 0);
  }
  return t / (double)n;
}

// General form: binary64 values; the sign of the binary64 sum is accepted when it exceeds
// the recursive-summation error bound (|S| > K 2^-52 sum|x|, Higham, "Accuracy and
// Stability of Numerical Algorithms", 2nd ed., eq. 4.4), else decided by grow-expansion.
template <int DT, int K>
__device__ __forceinline__ double ties_general(const uint32_t (&b)[K], uint32_t kept, int& gamma) {
  double x[K];
#pragma unroll
  for (int i = 0; i < K; ++i) x[i] = ((kept >> i) & 1u) ? bits_to_f64<DT>(b[i]) : 0.0;
  double S = x[0], A = fabs(x[0]);
#pragma unroll
  for (int i = 1; i < K; ++i) {
    S = S + x[i];
    A = A + fabs(x[i]);
  }
  int g;
  if (fabs(S) > A * ((double)K * 0x1p-52)) g = (S > 0.0) ? 1 : -1;
  else if (A == 0.0) g = 0;
  else g = exact_sign<K>(x);
  const double gd = (double)g;
  double M = 0.0;
  int n = 0;
#pragma unroll
  for (int i = 0; i < K; ++i) {
    const double y = gd * x[i];
    M = M + fmax(y, 0.0);
    n += y > 0.0;
  }
  gamma = g;
  return (n == 0) ? 0.0 : div_count(gd * M, n);
}

// bf16 form exact by construction when every kept magnitude lies within 16 - ceil(log2 K)
// binades of the largest kept key: then all partial sums of kept values are exact in
// binary32, so S, sum|x| and the agreeing-set sum (S + gamma sum|x|)/2 are the exact real
// values and equal the binary64 sequence of the general form.
template <int K>
__device__ __forceinline__ double ties_fast_bf16(const uint32_t (&b)[K], uint32_t kept, int& gamma) {
  float x[K];
#pragma unroll
  for (int i = 0; i < K; ++i) x[i] = ((kept >> i) & 1u) ? f32_from_bits(b[i] << 16) : 0.0f;
  float S = x[0], A = fabsf(x[0]);
  int np = x[0] > 0.0f, nn = x[0] < 0.0f;
#pragma unroll
  for (int i = 1; i < K; ++i) {
    S = S + x[i];
    A = A + fabsf(x[i]);
    np += x[i] > 0.0f;
    nn += x[i] < 0.0f;
  }
  const float g = (S > 0.0f) ? 1.0f : ((S < 0.0f) ? -1.0f : 0.0f);
  const float ts = (S + g * A) * 0.5f;
  const int n = (S > 0.0f) ? np : ((S < 0.0f) ? nn : 0);
  gamma = (int)g;
  return (n == 0) ? 0.0 : div_count((double)ts, n);
}

constexpr int clog2_of(int K) { return (K <= 1) ? 0 : (K <= 2) ? 1 : (K <= 4) ? 2 : 3; }

}  // namespace iso
