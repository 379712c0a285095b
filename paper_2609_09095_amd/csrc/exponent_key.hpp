// The exponent scan's reduction key (Eq. (scale), the setup of Alg. 1),
// shared by the separate scans and the row deconstruction that scans its
// own rows.  The reduction runs on the magnitude's bit pattern (|x| as
// uint64 is monotone in |x|; NaN and infinity sort above every finite
// value), then on a 32-bit order-preserving key: 0 for zero, e + 2048 for
// finite nonzero values with frexp exponent e, all ones for non-finite.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace oz {

constexpr uint32_t kKeyNonfinite = 0xFFFFFFFFu;
constexpr uint64_t kAbsMask = 0x7FFFFFFFFFFFFFFFull;

__device__ __forceinline__ uint32_t exponent_key(uint64_t absbits) {
  if (absbits >= 0x7FF0000000000000ull) return kKeyNonfinite;
  if (absbits == 0) return 0;
  const int biased = (int)(absbits >> 52);
  // normal: |x| in [2^(b-1023), 2^(b-1022)); subnormal: mantissa bit p set,
  // |x| in [2^(p-1074), 2^(p-1073)).
  const int e = biased ? biased - 1022 : (63 - __builtin_clzll(absbits)) - 1073;
  return (uint32_t)(e + 2048);
}

__device__ __forceinline__ int32_t key_to_sigma(uint32_t key, int t) {
  if (key == kKeyNonfinite) return INT32_MIN;
  if (key == 0) return t;  // frexp(0) has exponent 0
  return t - ((int)key - 2048);
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = (uint32_t)__shfl_xor((int)v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}

}  // namespace oz
