// Small exact integer helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace oz {

// Centred residue of an integer-valued double v (|v| <= 2^58) modulo M
// (odd M >= 197, or a power of two), in [-(M/2), (M-1)/2].  q = rint(v / M)
// is formed with one FP64 multiply by the rounded reciprocal, which errs by
// at most |v| 2^-52 / M < 1/3; so q is the nearest quotient or one off, the
// remainder v - q M (exact in one FMA) lies within 0.84 M of zero, and one
// correction each way brings it into the centred range.  For a power of two
// v / M is exact and the tie +M/2 maps to -M/2.
template <int M>
__device__ __forceinline__ int cmod_f64(double v) {
  constexpr double inv = 1.0 / M;
  constexpr int hi = (M - 1) / 2;
  constexpr int lo = hi - M + 1;
  const double q = __builtin_rint(v * inv);
  const int r = (int)__builtin_fma(-q, (double)M, v);
  const int r1 = r > hi ? r - M : r;
  return r1 < lo ? r1 + M : r1;
}

// Residue of an int32 x (|x| < 2^24) modulo M in [0, M).  The FP32 quotient
// may be one off near integers; the two corrections fix that.
template <int M>
__device__ __forceinline__ int pmod_small(int x) {
  constexpr float inv = 1.0f / M;
  const int q = (int)__builtin_floorf((float)x * inv);
  int r = x - q * M;
  r = r < 0 ? r + M : r;
  return r >= M ? r - M : r;
}

}  // namespace oz
