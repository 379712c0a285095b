// The last step of the reconstruction (Alg. 3): X, the balanced
// mixed-radix value of the centred Garner digits, times 2^e rounded once to
// FP64 (to nearest, ties to even, subnormal results included).  X is taken
// in two halves, X = xh P + xl; round_exact forms |X| as a 128-bit integer,
// round_fast evaluates the same rounding in FP64 with a proof that the
// result is the correct one and declines where the proof does not go
// through.  Plain arithmetic only (no target builtins beyond __mul24), so
// the functions also compile for the host.
#pragma once

#include <cstdint>

#include "moduli.hpp"

namespace oz {

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
static_assert(kModulus[1] == 1024, "the power-of-two modulus sits at index 1");

// Balanced half sum_{j in [A, A+6)} v_j prod_{A <= l < j} m_l: digit pairs in
// 24-bit arithmetic, then (g0 + b0 (g1 + b1 g2)) in 64 bits.
template <int A>
__device__ __forceinline__ int64_t half_value(const int (&v)[kR]) {
  constexpr int m0 = kModulus[A], m1 = kModulus[A + 1], m2 = kModulus[A + 2];
  constexpr int m3 = kModulus[A + 3], m4 = kModulus[A + 4];
  const int g0 = v[A] + __mul24(v[A + 1], m0);
  const int g1 = v[A + 2] + __mul24(v[A + 3], m2);
  const int g2 = v[A + 4] + __mul24(v[A + 5], m4);
  constexpr int64_t b0 = (int64_t)m0 * m1, b1 = (int64_t)m2 * m3;
  const int64_t t = (int64_t)g1 + b1 * (int64_t)g2;  // |t| < 2^40
  return (int64_t)g0 + b0 * t;
}

// The same half in FP64: the pairs and their 40-bit combination are exact,
// and the last fma rounds the half once (exact when it is below 2^53).
template <int A>
__device__ __forceinline__ double half_fp64(const int (&v)[kR]) {
  constexpr int m0 = kModulus[A], m2 = kModulus[A + 2], m4 = kModulus[A + 4];
  const int g0 = v[A] + __mul24(v[A + 1], m0);
  const int g1 = v[A + 2] + __mul24(v[A + 3], m2);
  const int g2 = v[A + 4] + __mul24(v[A + 5], m4);
  constexpr double b0 = (double)m0 * kModulus[A + 1], b1 = (double)m2 * kModulus[A + 3];
  const double t = __builtin_fma(b1, (double)g2, (double)g1);  // |t| < 2^40
  return __builtin_fma(b0, t, (double)g0);
}

// RN_even(mag 2^e) for 0 < mag < 2^MAXBITS (MAXBITS <= 127).
//  - normal (and overflowing) results: the top 64 bits of mag, with every
//    lower bit ORed into bit 0 as a sticky bit, convert to FP64 with the one
//    correct rounding (bit 0 lies ten places below the rounding point), and
//    ldexp scales exactly or overflows to infinity as rounding would.
//  - subnormal results (exponent below -1022): keep the bits down to 2^-1074
//    and round half to even on the dropped ones by hand.
template <int MAXBITS>
__device__ __forceinline__ double round_scaled(u128 mag, int e) {
  static_assert(MAXBITS <= 127, "shifts stay inside 128 bits");
  const uint64_t hi = (uint64_t)(mag >> 64), lo = (uint64_t)mag;
  const int c = hi ? __builtin_clzll(hi) : 64 + __builtin_clzll(lo);  // leading zeros of mag
  const int E = 127 - c + e;  // the value lies in [2^E, 2^(E+1))
  if (E >= -1022) {
    const u128 norm = mag << c;
    const uint64_t top = (uint64_t)(norm >> 64) | ((uint64_t)norm != 0 ? 1u : 0u);
    return __builtin_ldexp((double)top, E - 63);
  }
  const int sh = -1074 - e;  // dropped bits: the quantum is 2^-1074
  if (sh <= 0) return __builtin_ldexp((double)(lo << -sh), -1074);  // exact, below 2^53
  if (sh > MAXBITS) return 0.0;  // below half the smallest subnormal
  uint64_t mant = (uint64_t)(mag >> sh);
  const u128 rem = mag & (((u128)1 << sh) - 1);
  const u128 half = (u128)1 << (sh - 1);
  mant += (rem > half || (rem == half && (mant & 1))) ? 1 : 0;
  return __builtin_ldexp((double)mant, -1074);
}

// RN(X 2^e) from the digits in 128-bit integer arithmetic: every case.
__device__ __forceinline__ double round_exact(const int (&v)[kR], int e) {
  const int64_t xl = half_value<0>(v);       // |xl| < P
  int64_t xh = half_value<kSplit>(v);        // |xh| <= (Q - 1) / 2
  constexpr int64_t kHalfQ = (int64_t)(kQ - 1) / 2, kHalfP = (int64_t)(kP / 2);
  if (xh == -kHalfQ && xl < -kHalfP) xh += (int64_t)kQ;  // below -M/2: lift by M
  if (xh == 0 && xl == 0) return 0.0;
  const bool neg = xh < 0 || (xh == 0 && xl < 0);
  // |X| = |xh| P + (+-xl), the sign of the second term following X
  const uint64_t H = (uint64_t)(neg ? -xh : xh);
  const int64_t L = neg ? -xl : xl;
  const u128 mag = (u128)H * (u128)kP + (u128)(__int128)L;
  const double r = round_scaled<113>(mag, e);
  return neg ? -r : r;
}

// Fast evaluation of the same rounding in FP64, with a proof that it is the
// correctly rounded one:
//  - xh = X's high half is an integer below 2^53 (computed exactly), xl~ the
//    low half rounded once, |xl - xl~| <= 32 since |xl| < P < 2^59.
//  - P = m_0..m_5 is exact in FP64.  p = RN(xh P), ep = xh P - p (exact, by
//    fma), t = RN(ep + xl~), r = RN(p + t), and res = p + t - r exactly
//    (Fast2Sum: |p| >= |t| whenever xh != 0).
//  - So X - r = res + d, |d| <= 32 + ulp(t)/2 <= 32 + |t| 2^-53.  When
//    |res| + |d| < ulp(r)/2 (bounded with a factor-2 margin, so the rounding
//    of the test itself cannot flip it) and r is no power of two, r = RN(X);
//    with xh = 0, r = RN(xl) = RN(X) directly.  ldexp then scales exactly
//    while the result stays normal, and overflows as rounding would.
// Returns false where that proof does not go through (X within about 2^-44
// relative of a rounding boundary, a power-of-two r, the lift xh = -(Q-1)/2,
// or a subnormal result); those outputs take round_exact.
constexpr double kPd = (double)kP;
static_assert((uint64_t)kPd == kP, "P is exact in FP64");
static_assert((kQ - 1) / 2 < (1ull << 53), "the high half is exact in FP64");
__device__ __forceinline__ bool round_fast(const int (&v)[kR], int e, double& out) {
  const double xh = half_fp64<kSplit>(v), xl = half_fp64<0>(v);
  const double p = xh * kPd;
  const double ep = __builtin_fma(xh, kPd, -p);
  const double t = ep + xl;
  const double r = p + t;
  const double res = t - (r - p);
  const uint64_t rb = __builtin_bit_cast(uint64_t, r);
  const int eb = (int)(rb >> 52) & 0x7FF;  // biased exponent of r (r >= 2^57 when xh != 0)
  const double halfu = __builtin_bit_cast(double, (uint64_t)(eb - 53) << 52);
  const double bound = __builtin_fma(__builtin_fabs(t), 0x1p-51, 64.0) + __builtin_fabs(res);
  const bool rounded = xh == 0.0 || (bound < halfu && (rb << 12) != 0 &&
                                     xh != -(double)((kQ - 1) / 2));
  out = __builtin_ldexp(r, e);
  return rounded && (eb + e >= 1 || eb == 0);
}

// ---- all-byte set (Sec. 5.1, candidate A): halves over digits 0-6 and 7-14
constexpr int kSplitA = 7;
constexpr uint64_t prod_range_a(int a, int b) {
  uint64_t p = 1;
  for (int i = a; i < b; ++i) p *= (uint64_t)kModulusA[i];
  return p;
}
constexpr uint64_t kPA = prod_range_a(0, kSplitA);
constexpr uint64_t kQA = prod_range_a(kSplitA, kRA);
static_assert(kPA < (1ull << 56) && kQA < (1ull << 63), "halves fit 64 bits");
static_assert(kModulusA[0] == 256 && kQA % 2 == 1, "the one even modulus leads the low half");

// Balanced value of digits [A, B): digit pairs v_j + m_j v_{j+1} in 24-bit
// arithmetic (|pair| < 2^16), then Horner over the pairs in 64 bits.
template <int A, int B>
__device__ __forceinline__ int64_t half_value_a(const int (&v)[kRA]) {
  constexpr int np = (B - A + 1) / 2;
  int g[np];
#pragma unroll
  for (int i = 0; i < np; ++i) {
    const int j = A + 2 * i;
    g[i] = j + 1 < B ? v[j] + __mul24(v[j + 1], kModulusA[j]) : v[j];
  }
  int64_t x = g[np - 1];
#pragma unroll
  for (int i = np - 2; i >= 0; --i) {
    const int j = A + 2 * i;
    x = (int64_t)g[i] + (int64_t)kModulusA[j] * kModulusA[j + 1] * x;
  }
  return x;
}

// RN(X 2^e) from the halves in 128-bit integer arithmetic: every case.
__device__ __forceinline__ double round_exact_a(int64_t xl, int64_t xh, int e) {
  if (xh == 0 && xl == 0) return 0.0;
  const bool neg = xh < 0 || (xh == 0 && xl < 0);
  const uint64_t H = (uint64_t)(neg ? -xh : xh);
  const int64_t L = neg ? -xl : xl;
  const u128 mag = (u128)H * (u128)kPA + (u128)(__int128)L;
  const double r = round_scaled<117>(mag, e);
  return neg ? -r : r;
}

// The halves of the all-byte set in FP64 from digit pairs g = v_j + m_j
// v_{j+1} (|g| < 2^16).  Low half (digits 0-6): two exact fmas (below 2^40)
// and one that rounds, so lh = RN(xl).  High half (digits 7-14): exact
// fmas up to 2^47, then the last weight's product split exactly by fma
// (ph + pl), pl + g exact (integers below 2^16), and Fast2Sum of ph and that
// sum (|ph| is larger unless ph = 0, and then hl = 0), so hh = RN(xh) and
// hl = xh - hh exactly, |hl| <= 2^8.
__device__ __forceinline__ int digit_pair_a(const int (&v)[kRA], int j) {
  return v[j] + __mul24(v[j + 1], kModulusA[j]);
}
__device__ __forceinline__ double weight_a(int j) { return (double)kModulusA[j] * kModulusA[j + 1]; }
static_assert(kSplitA == 7 && kRA == 15, "three pairs and a digit low, four pairs high");
__device__ __forceinline__ void halves_fp64_a(const int (&v)[kRA], double& lh, double& hh, double& hl) {
  const double tl = __builtin_fma(weight_a(4), (double)v[6], (double)digit_pair_a(v, 4));
  const double tm = __builtin_fma(weight_a(2), tl, (double)digit_pair_a(v, 2));
  lh = __builtin_fma(weight_a(0), tm, (double)digit_pair_a(v, 0));
  const double u = __builtin_fma(weight_a(11), (double)digit_pair_a(v, 13), (double)digit_pair_a(v, 11));
  const double w = __builtin_fma(weight_a(9), u, (double)digit_pair_a(v, 9));
  const double ph = weight_a(7) * w;
  const double pl = __builtin_fma(weight_a(7), w, -ph);
  const double ee = pl + (double)digit_pair_a(v, 7);
  hh = ph + ee;
  hl = ee - (hh - ph);
}

// The same rounding in FP64 with a proof, as round_fast for the published
// set; here the high half reaches 2^61, so it enters as hh + hl (hl != 0
// only above 2^53, |hl| <= 2^8), P is exact in FP64, and the low half as
// RN(xl) (|xl| <= P/2 < 2^55: error <= 2):
//   p = RN(hh P), ep = hh P - p exactly, q = RN(hl P + RN(xl)) (|.| < 2^64,
//   error <= 2^10), t = RN(ep + q), r = RN(p + t), res = p + t - r exactly
//   (Fast2Sum: |p| >= |t| whenever xh != 0),
// so X - r = res + d with |d| <= 2^10 + 2 + ulp(t)/2, bounded below with a
// factor-2 margin.  With xh = 0, r = RN(xl) = RN(X).  Returns false where
// the proof does not go through (near a rounding boundary, a power-of-two
// r, a subnormal result); those outputs take round_exact_a.
constexpr double kPAd = (double)kPA;
static_assert((uint64_t)kPAd == kPA, "P is exact in FP64");
__device__ __forceinline__ bool round_fast_a(const int (&v)[kRA], int e, double& out) {
  double lh, hh, hl;
  halves_fp64_a(v, lh, hh, hl);
  const double p = hh * kPAd;
  const double ep = __builtin_fma(hh, kPAd, -p);
  const double q = __builtin_fma(hl, kPAd, lh);
  const double t = ep + q;
  const double r = p + t;
  const double res = t - (r - p);
  const uint64_t rb = __builtin_bit_cast(uint64_t, r);
  const int eb = (int)(rb >> 52) & 0x7FF;  // biased exponent of r (r >= 2^55 when xh != 0)
  const double halfu = __builtin_bit_cast(double, (uint64_t)(eb - 53) << 52);
  const double bound = __builtin_fma(__builtin_fabs(t), 0x1p-51, 0x1p13) + __builtin_fabs(res);
  const bool rounded = hh == 0.0 || (bound < halfu && (rb << 12) != 0);
  out = __builtin_ldexp(r, e);
  return rounded && (eb + e >= 1 || eb == 0);
}

}  // namespace oz
