// Reconstruction (Alg. 3): Garner's mixed-radix digits of the twelve centred
// residues (Eq. (garner)), Horner recombination to the integer X in [0, M)
// (Eq. (horner)), the symmetric lift to [-M/2, M/2), and one rounding of
// X 2^(-sigma_i - tau_j) to FP64.  One thread per output; the residue loads
// coalesce along the output row.  HBM-bound: 12 residues in, 8 bytes out.
#include <utility>

#include "device_math.hpp"
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

using u128 = unsigned __int128;
using i128 = __int128;

constexpr u128 product_of_moduli() {
  u128 p = 1;
  for (int i = 0; i < kR; ++i) p *= (u128)kModulus[i];
  return p;
}
constexpr u128 kM = product_of_moduli();

// Digit J of Garner's recurrence: v_J = (c_J - sum_{l<J} v_l (m_0..m_{l-1}))
// w_J mod m_J, with the weights reduced mod m_J at compile time.  The
// subtracted sum stays below 12 * 1089^2 < 2^24.
template <int J>
__device__ __forceinline__ void garner_digit(const int (&c)[kR], int (&v)[kR]) {
  constexpr int M = kModulus[J];
  int s = c[J];
  [&]<int... L>(std::integer_sequence<int, L...>) {
    ((s -= v[L] * radix_mod(L, J)), ...);
  }(std::make_integer_sequence<int, J>{});
  const int u = pmod_small<M>(s);
  v[J] = pmod_small<M>(u * garner_w(J));
}

// RN_even(X 2^e) for |X| < 2^112: keep the top 53 bits (fewer in the
// subnormal range, where the quantum is 2^-1074), round half to even on the
// dropped bits, and scale the integer significand by ldexp, which is exact
// here and overflows to infinity past the largest double.
__device__ __forceinline__ double round_scaled(i128 X, int e) {
  if (X == 0) return 0.0;
  const bool neg = X < 0;
  const u128 mag = neg ? (u128)(-X) : (u128)X;
  const uint64_t hi = (uint64_t)(mag >> 64), lo = (uint64_t)mag;
  const int p = hi ? 127 - __builtin_clzll(hi) : 63 - __builtin_clzll(lo);  // top bit
  const int E = p + e;                                                     // exponent of |X 2^e|
  const int qe = E - 52 > -1074 ? E - 52 : -1074;                          // quantum exponent
  const int sh = qe - e;                                                   // dropped bits
  uint64_t mant;
  if (sh <= 0) {
    mant = (uint64_t)mag << (-sh);  // at most 53 bits
  } else if (sh > 113) {
    mant = 0;  // below half the smallest subnormal
  } else {
    mant = (uint64_t)(mag >> sh);
    const u128 rem = mag & (((u128)1 << sh) - 1);
    const u128 half = (u128)1 << (sh - 1);
    mant += (rem > half || (rem == half && (mant & 1))) ? 1 : 0;
  }
  const double r = __builtin_ldexp((double)mant, qe);
  return neg ? -r : r;
}

template <typename RT>
__global__ __launch_bounds__(256) void reconstruct_kernel(int64_t m, int64_t n,
                                                          const RT* __restrict__ cres,
                                                          const int32_t* __restrict__ ea,
                                                          const int32_t* __restrict__ eb,
                                                          double* __restrict__ C, int64_t ldc,
                                                          int subtract) {
  const int64_t nb = (n + 255) / 256;
  const int64_t row = blockIdx.x / nb;
  const int64_t col = (int64_t)(blockIdx.x % nb) * 256 + threadIdx.x;
  if (row >= m || col >= n) return;
  const int64_t mn = m * n, e = row * n + col;
  int c[kR], v[kR];
#pragma unroll
  for (int q = 0; q < kR; ++q) c[q] = (int)cres[q * mn + e];
  const int sa = ea[row], sb = eb[col];
  double r;
  if (sa == INT32_MIN || sb == INT32_MIN) {
    r = __builtin_nan("");
  } else {
    [&]<int... J>(std::integer_sequence<int, J...>) {
      (garner_digit<J>(c, v), ...);
    }(std::make_integer_sequence<int, kR>{});
    // Horner: v_0 + m_0 (v_1 + m_1 (v_2 + ...)) in [0, M)
    u128 X = (u128)v[kR - 1];
#pragma unroll
    for (int j = kR - 2; j >= 0; --j) X = X * (u128)kModulus[j] + (u128)v[j];
    const i128 Xs = X >= kM / 2 ? (i128)X - (i128)kM : (i128)X;
    r = round_scaled(Xs, -sa - sb);
  }
  double* out = C + row * ldc + col;
  *out = subtract ? *out - r : r;
}

__global__ __launch_bounds__(256) void zero_c_kernel(int64_t m, int64_t n, double* C, int64_t ldc) {
  const int64_t nb = (n + 255) / 256;
  const int64_t row = blockIdx.x / nb;
  const int64_t col = (int64_t)(blockIdx.x % nb) * 256 + threadIdx.x;
  if (row < m && col < n) C[row * ldc + col] = 0.0;
}

template <typename RT>
hipError_t launch_rec(int64_t m, int64_t n, const RT* cres, const int32_t* ea, const int32_t* eb,
                      double* C, int64_t ldc, int subtract, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  const int64_t blocks = m * ((n + 255) / 256);
  hipLaunchKernelGGL(reconstruct_kernel<RT>, dim3((unsigned)blocks), dim3(256), 0, stream, m, n, cres,
                     ea, eb, C, ldc, subtract);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_reconstruct_i32(int64_t m, int64_t n, const int32_t* cres, const int32_t* ea,
                                  const int32_t* eb, double* C, int64_t ldc, int subtract,
                                  hipStream_t stream) {
  return launch_rec<int32_t>(m, n, cres, ea, eb, C, ldc, subtract, stream);
}

hipError_t launch_reconstruct_i16(int64_t m, int64_t n, const int16_t* cres, const int32_t* ea,
                                  const int32_t* eb, double* C, int64_t ldc, int subtract,
                                  hipStream_t stream) {
  return launch_rec<int16_t>(m, n, cres, ea, eb, C, ldc, subtract, stream);
}

hipError_t launch_zero_c(int64_t m, int64_t n, double* C, int64_t ldc, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  const int64_t blocks = m * ((n + 255) / 256);
  hipLaunchKernelGGL(zero_c_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, m, n, C, ldc);
  return hipGetLastError();
}

}  // namespace oz
