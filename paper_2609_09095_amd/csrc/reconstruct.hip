// Reconstruction (Alg. 3): Garner's mixed-radix digits of the twelve centred
// residues (Eq. (garner)), Horner recombination (Eq. (horner)), the symmetric
// lift to [-M/2, M/2), and one rounding of X 2^(-sigma_i - tau_j) to FP64.
// One thread per output; the residue loads coalesce along the output row.
// HBM-bound: 12 residues in, 8 bytes out.
//
// Integer work per output, all exact:
//  - digit j in one reduction: v_j = (c_j w_j - sum_{l<j} v_l R_lj) mod m_j
//    with R_lj = (m_0..m_{l-1}) w_j mod m_j folded at compile time; the
//    argument stays below 2^24 in magnitude, so an FP32 quotient is exact up
//    to one step that the corrections absorb.
//  - Horner in two 64-bit halves, X = Xh P + Xl with P = m_0..m_5 < 2^59,
//    Xl = v_0 + m_0 (v_1 + ... m_4 v_5) < P and Xh = v_6 + ... < M / P < 2^54.
//  - the lift X >= M/2 compares the halves (M/2 = ((Q-1)/2) P + P/2 with
//    Q = M / P odd); the magnitude is then H P + L with H < 2^54, L <= P,
//    formed as a 128-bit integer and rounded once.
#include <utility>

#include "device_math.hpp"
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

using u128 = unsigned __int128;

constexpr int kSplit = 6;  // digits 0..5 in the low half, 6..11 in the high half

constexpr uint64_t prod_range(int a, int b) {
  uint64_t p = 1;
  for (int i = a; i < b; ++i) p *= (uint64_t)kModulus[i];
  return p;
}
constexpr uint64_t kP = prod_range(0, kSplit);   // m_0 ... m_5
constexpr uint64_t kQ = prod_range(kSplit, kR);  // m_6 ... m_11
static_assert(kP < (1ull << 59) && kQ < (1ull << 54), "halves fit 64 bits");
static_assert(kQ % 2 == 1 && kP % 2 == 0, "lift rule assumes Q odd, P even");

// Weight of digit l in the equation of digit j, times w_j, mod m_j; as
// template variables so that they are compile-time immediates in the kernel.
constexpr int garner_weight(int l, int j) {
  return (int)((int64_t)radix_mod(l, j) * garner_w(j) % kModulus[j]);
}
template <int L, int J>
inline constexpr int kGarnerWeight = garner_weight(L, J);
template <int J>
inline constexpr int kGarnerW = garner_w(J);

template <int J>
__device__ __forceinline__ void garner_digit(const int (&c)[kR], int (&v)[kR]) {
  constexpr int M = kModulus[J];
  // every factor is below 2^11 in magnitude: 24-bit multiplies are exact
  int s = __mul24(c[J], kGarnerW<J>);
  [&]<int... L>(std::integer_sequence<int, L...>) {
    ((s -= __mul24(v[L], kGarnerWeight<L, J>)), ...);
  }(std::make_integer_sequence<int, J>{});
  v[J] = pmod_small<M>(s);
}

// X = sum_{j in [a, b)} v_j prod_{a <= l < j} m_l, Horner from the top.
template <int A, int B>
__device__ __forceinline__ uint64_t horner(const int (&v)[kR]) {
  uint64_t x = (uint64_t)v[B - 1];
#pragma unroll
  for (int j = B - 2; j >= A; --j) x = x * (uint64_t)kModulus[j] + (uint64_t)v[j];
  return x;
}

// RN_even(mag 2^e) for 0 < mag < 2^113: keep the top 53 bits (fewer in the
// subnormal range, where the quantum is 2^-1074), round half to even on the
// dropped bits, and scale the integer significand by ldexp, which is exact
// here and overflows to infinity past the largest double.
__device__ __forceinline__ double round_scaled(u128 mag, int e) {
  const uint64_t hi = (uint64_t)(mag >> 64), lo = (uint64_t)mag;
  const int p = hi ? 127 - __builtin_clzll(hi) : 63 - __builtin_clzll(lo);  // top bit
  const int E = p + e;                                                     // exponent of the value
  const int qe = E - 52 > -1074 ? E - 52 : -1074;                          // quantum exponent
  const int sh = qe - e;                                                   // dropped bits
  uint64_t mant;
  if (sh <= 0) {
    mant = lo << (-sh);  // at most 53 bits
  } else if (sh > 113) {
    mant = 0;  // below half the smallest subnormal
  } else {
    mant = (uint64_t)(mag >> sh);
    const u128 rem = mag & (((u128)1 << sh) - 1);
    const u128 half = (u128)1 << (sh - 1);
    mant += (rem > half || (rem == half && (mant & 1))) ? 1 : 0;
  }
  return __builtin_ldexp((double)mant, qe);
}

template <typename RT>
__device__ __forceinline__ double reconstruct_one(const RT* __restrict__ cres, int64_t mn, int64_t e,
                                                  int sa, int sb) {
  if (sa == INT32_MIN || sb == INT32_MIN) return __builtin_nan("");
  int c[kR], v[kR];
#pragma unroll
  for (int q = 0; q < kR; ++q) c[q] = (int)cres[q * mn + e];
  [&]<int... J>(std::integer_sequence<int, J...>) {
    (garner_digit<J>(c, v), ...);
  }(std::make_integer_sequence<int, kR>{});
  const uint64_t xl = horner<0, kSplit>(v);   // < P
  const uint64_t xh = horner<kSplit, kR>(v);  // < Q
  constexpr uint64_t kHalfQ = (kQ - 1) / 2, kHalfP = kP / 2;
  const bool neg = xh > kHalfQ || (xh == kHalfQ && xl >= kHalfP);
  // |X| = H P + L: for X - M = (xh - Q) P + xl < 0, H = Q - xh - 1, L = P - xl
  uint64_t H = neg ? kQ - xh - 1 : xh;
  uint64_t L = neg ? kP - xl : xl;
  if (L == kP) {  // only when xl == 0
    H += 1;
    L = 0;
  }
  const u128 mag = (u128)H * (u128)kP + (u128)L;
  if (mag == 0) return 0.0;
  const double r = round_scaled(mag, -sa - sb);
  return neg ? -r : r;
}

// Grid: x over 256-column strips, y over rows (strided by gridDim.y).
template <typename RT>
__global__ __launch_bounds__(256) void reconstruct_kernel(int64_t m, int64_t n,
                                                          const RT* __restrict__ cres,
                                                          const int32_t* __restrict__ ea,
                                                          const int32_t* __restrict__ eb,
                                                          double* __restrict__ C, int64_t ldc,
                                                          int subtract) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= n) return;
  const int64_t mn = m * n;
  const int sb = eb[col];
  for (int64_t row = blockIdx.y; row < m; row += gridDim.y) {
    const double r = reconstruct_one(cres, mn, row * n + col, ea[row], sb);
    double* out = C + row * ldc + col;
    *out = subtract ? *out - r : r;
  }
}

__global__ __launch_bounds__(256) void zero_c_kernel(int64_t m, int64_t n, double* C, int64_t ldc) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= n) return;
  for (int64_t row = blockIdx.y; row < m; row += gridDim.y) C[row * ldc + col] = 0.0;
}

dim3 grid_for(int64_t m, int64_t n) {
  return dim3((unsigned)((n + 255) / 256), (unsigned)(m < 65535 ? m : 65535));
}

template <typename RT>
hipError_t launch_rec(int64_t m, int64_t n, const RT* cres, const int32_t* ea, const int32_t* eb,
                      double* C, int64_t ldc, int subtract, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  hipLaunchKernelGGL(reconstruct_kernel<RT>, grid_for(m, n), dim3(256), 0, stream, m, n, cres, ea,
                     eb, C, ldc, subtract);
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
  hipLaunchKernelGGL(zero_c_kernel, grid_for(m, n), dim3(256), 0, stream, m, n, C, ldc);
  return hipGetLastError();
}

}  // namespace oz
