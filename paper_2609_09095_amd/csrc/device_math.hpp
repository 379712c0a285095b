// Small exact integer helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace oz {

// Centred residue of an integer-valued double v (|v| < 2^56) modulo M, in
// [-(M/2), (M-1)/2].  q = rint(v / M) is formed with one FP64 multiply by
// the rounded reciprocal; the remainder v - q M is exact in one FMA; the
// quotient can be one off only when v / M lies within 2^-6 of a half
// integer, which puts the remainder just outside the centred range on the
// other side, so one correction each way restores it.  The even modulus
// 1024 also lands here: v 2^-10 is exact, and the tie +512 maps to -512.
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
