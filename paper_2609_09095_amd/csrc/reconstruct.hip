// Reconstruction (Alg. 3): Garner's mixed-radix digits of the twelve (or,
// for the all-byte set, fifteen) centred residues (Eq. (garner)), Horner
// recombination (Eq. (horner)), the lift to [-M/2, M/2), and one rounding
// of X 2^(-sigma_i - tau_j) to FP64.
// One thread per output; the residue loads coalesce along the output row.
// 24 bytes in and 8 out per output (8 more in for C -= ...): the mix of
// reads and writes bounds it at the rate of a plain copy, with the VALU work
// (about 140 instructions per output) hidden under it.
//
// Integer work per output, all exact:
//  - centred digits in one reduction each: v_j = (c_j w_j - sum_{l<j} v_l
//    R_lj) mod m_j with w_j and R_lj = (m_0..m_{l-1}) w_j mod m_j centred
//    compile-time constants.  The residue GEMM's compact int16 residues c'_j
//    are the true ones divided by a per-modulus factor f_j and reduced to
//    |c'_j| <= 0.51 m_j: the term is then c'_j (f_j w_j mod m_j).  Every
//    term is below 567 * 545 in magnitude, the sum of at most twelve below
//    2^22, so for odd m_j the FP32 quotient
//    rint(s / m_j) errs by less than 1/(2 m_j), the least distance of s / m_j
//    from a half integer: one rint and one multiply-add give the centred
//    digit.  m_j = 1024 takes the low ten bits.
//  - centred digits make X = Xl + P Xh a balanced mixed-radix number with
//    P = m_0..m_5 (even) and halves Xl = v_0 + m_0 (v_1 + ... m_4 v_5),
//    |Xl| < P, and Xh likewise over m_6..m_11 with |Xh| <= (Q-1)/2, Q odd.
//    Its range is [-M/2 - 544, M/2 - 545]; the few values below -M/2 are
//    moved up by M (Xh += Q), which gives exactly the lift to [-M/2, M/2).
//  - Horner pairs digits with 24-bit multiply-adds (|pair| < 2^20) and joins
//    the three pairs of a half in 64-bit arithmetic.
//  - |X| = H P + L with H = |Xh| < 2^53 and |L| < P, formed as a 128-bit
//    integer and rounded once.
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
static_assert(kModulus[1] == 1024, "the power-of-two modulus sits at index 1");

constexpr int centred_const(int64_t x, int m) { return (int)(x > m / 2 ? x - m : x); }
// centred weight of digit l in the equation of digit j (times w_j), and w_j;
// as template variables so that they are compile-time immediates
template <int L, int J>
inline constexpr int kGarnerWeight =
    centred_const((int64_t)radix_mod(L, J) * garner_w(J) % kModulus[J], kModulus[J]);
template <int J>
inline constexpr int kGarnerW = centred_const(garner_w(J), kModulus[J]);
// the same for the residue GEMM's compact outputs, which leave out the
// factor compact_scale(j): w_j times it
template <int J>
inline constexpr int kGarnerWCompact =
    centred_const((int64_t)garner_w(J) * compact_scale(J) % kModulus[J], kModulus[J]);

constexpr bool garner_sums_fit() {
  // |c_j w_j| + sum_{l<j} |v_l R_lj| < 2^22 with |v| <= m/2 and |c| <= 0.51 m
  // (compact residues are reduced but not wrapped into the centred range)
  for (int j = 0; j < kR; ++j) {
    const int64_t mj = kModulus[j];
    int64_t s = (mj / 2 + mj / 50 + 1) * (mj / 2 + 1);
    for (int l = 0; l < j; ++l) s += (kModulus[l] / 2 + 1) * (mj / 2 + 1);
    if (s >= (int64_t)1 << 22) return false;
  }
  return true;
}
static_assert(garner_sums_fit(), "Garner sums stay below 2^22");

// The sum over earlier digits runs on v_dot2_i32_i16, two terms per
// instruction: digits and weights are centred residues, |.| <= 544, so they
// fit int16.  Word Q of the weights of digit J holds -R_lJ for l = 2Q, 2Q+1
// (0 for l >= J); word Q of the digits holds v_2Q (low half) and v_2Q+1.
constexpr uint32_t garner_pack(int q, int j) {
  uint32_t w = 0;
  for (int i = 0; i < 2; ++i) {
    const int l = 2 * q + i;
    if (l < j) {
      const int r = centred_const((int64_t)radix_mod(l, j) * garner_w(j) % kModulus[j], kModulus[j]);
      w |= (uint32_t)(-r & 0xffff) << (16 * i);
    }
  }
  return w;
}
template <int Q, int J>
inline constexpr int kGarnerPack = (int)garner_pack(Q, J);
static_assert(kModulus[0] / 2 < 32767, "centred weights and digits fit int16");

typedef short v2s __attribute__((ext_vector_type(2)));

// digit J from the residue c_J and the packed earlier digits
template <int J, bool COMPACT>
__device__ __forceinline__ void garner_digit(const int (&c)[kR], int (&v)[kR], uint32_t (&packed)[kR / 2]) {
  constexpr int M = kModulus[J];
  // every factor is below 2^11 in magnitude: 24-bit multiplies are exact
  int s = __mul24(c[J], COMPACT ? kGarnerWCompact<J> : kGarnerW<J>);
  [&]<int... Q>(std::integer_sequence<int, Q...>) {
    ((s = __builtin_amdgcn_sdot2(__builtin_bit_cast(v2s, packed[Q]),
                                 __builtin_bit_cast(v2s, kGarnerPack<Q, J>), s, false)),
     ...);
  }(std::make_integer_sequence<int, (J + 1) / 2>{});
  int d;
  if constexpr (M == 1024) {
    d = ((s + 512) & 1023) - 512;
  } else {
    const int q = (int)__builtin_rintf((float)s * (1.0f / M));
    d = s - __mul24(q, M);  // |q| < 2^13
  }
  v[J] = d;
  // an even digit opens its word (the high half's weight is 0 until the
  // odd digit fills it); an odd one completes it
  if constexpr (J % 2 == 0)
    packed[J / 2] = (uint32_t)d;
  else
    packed[J / 2] = (packed[J / 2] & 0xffffu) | ((uint32_t)d << 16);
}

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

// Residue q of output (row, col): a buffer load with the row's scalar base
// (row-uniform) and the column's 32-bit byte offset, shared by all twelve.
template <typename RT>
__device__ __forceinline__ int load_residue(const RT* rowbase, int n, int col) {
  // readfirstlane returns int: take both halves as uint32_t before widening
  // (a sign-extended low half would corrupt the high one)
  const uint64_t v = (uint64_t)rowbase;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  const void* base = (const void*)(((uint64_t)hi << 32) | lo);
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, n * (int)sizeof(RT), 0x00020000);
  if constexpr (sizeof(RT) == 1)
    return (int)(int8_t)__builtin_amdgcn_raw_buffer_load_b8(rs, col, 0, 0);
  else if constexpr (sizeof(RT) == 2)
    return (int)(int16_t)__builtin_amdgcn_raw_buffer_load_b16(rs, col * 2, 0, 0);
  else
    return (int)__builtin_amdgcn_raw_buffer_load_b32(rs, col * 4, 0, 0);
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

// rowq: residues of this output row for modulus 0 (row-uniform); the
// modulus-q row sits mn elements further per q.
template <typename RT>
__device__ __forceinline__ double reconstruct_one(const RT* rowq, int64_t mn, int n, int col, int sa,
                                                  int sb) {
  if (sa == INT32_MIN || sb == INT32_MIN) return __builtin_nan("");
  int c[kR], v[kR];
  uint32_t packed[kR / 2];
#pragma unroll
  for (int q = 0; q < kR; ++q) c[q] = load_residue(rowq + q * mn, n, col);
  [&]<int... J>(std::integer_sequence<int, J...>) {
    (garner_digit<J, sizeof(RT) == 2>(c, v, packed), ...);
  }(std::make_integer_sequence<int, kR>{});
  const int e = -sa - sb;
  double out;
  if (!round_fast(v, e, out)) out = round_exact(v, e);
  return out;
}

// ---- all-byte set (Sec. 5.1, candidate A) ---------------------------------
// Fifteen centred residues, |c| <= 128.  Garner sums stay below 15 * 2^14 <
// 2^18, so the FP32 quotient of a digit errs by less than 2^-5 / m_j and
// rint gives the centred digit for odd m_j; m_0 = 256 takes the low eight
// bits.  The sums run four terms at a time on the int8 dot product.  With
// 256 first and every other modulus odd, the balanced halves
// Xl (digits 0-6, |Xl| <= P/2) and Xh (digits 7-14, |Xh| <= (Q-1)/2, Q odd)
// give X = Xl + P Xh in exactly [-M/2, M/2): no lift is needed.  |X| < 2^117.
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

template <int J>
inline constexpr int kGarnerWA = centred_const(garner_w_a(J), kModulusA[J]);

// Digits and Garner weights of the all-byte set are centred residues of
// byte moduli, so they fit int8 and the sum over earlier digits runs on
// v_dot4_i32_i8, four terms per instruction: word Q of the weights of digit
// J holds -R_lJ for l = 4Q..4Q+3 (0 for l >= J; |R_lJ| <= 127 for the odd
// m_J, so the negation fits).
constexpr uint32_t garner_pack_a(int q, int j) {
  uint32_t w = 0;
  for (int i = 0; i < 4; ++i) {
    const int l = 4 * q + i;
    if (l < j) {
      const int r = centred_const((int64_t)radix_mod_a(l, j) * garner_w_a(j) % kModulusA[j], kModulusA[j]);
      w |= (uint32_t)(-r & 0xff) << (8 * i);
    }
  }
  return w;
}
template <int Q, int J>
inline constexpr int kGarnerPackA = (int)garner_pack_a(Q, J);
constexpr bool garner_weights_fit_int8() {
  for (int j = 1; j < kRA; ++j)
    for (int l = 0; l < j; ++l) {
      const int r = centred_const((int64_t)radix_mod_a(l, j) * garner_w_a(j) % kModulusA[j], kModulusA[j]);
      if (r < -127 || r > 127) return false;
    }
  return true;
}
static_assert(garner_weights_fit_int8(), "negated weights fit int8");

// digit J from the residue c_J and the packed earlier digits; appends v_J
template <int J>
__device__ __forceinline__ int garner_digit_a(const int (&c)[kRA], uint32_t (&packed)[4]) {
  constexpr int M = kModulusA[J];
  int s = __mul24(c[J], kGarnerWA<J>);
  [&]<int... Q>(std::integer_sequence<int, Q...>) {
    ((s = __builtin_amdgcn_sdot4((int)packed[Q], kGarnerPackA<Q, J>, s, false)), ...);
  }(std::make_integer_sequence<int, (J + 3) / 4>{});
  int v;
  if constexpr (M == 256) {
    v = ((s + 128) & 255) - 128;
  } else {
    const int q = (int)__builtin_rintf((float)s * (1.0f / M));
    v = s - __mul24(q, M);  // |q| < 2^11
  }
  packed[J / 4] |= (uint32_t)(v & 0xff) << (8 * (J % 4));
  return v;
}

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

// x = hi + lo exactly with hi = RN(x): the two 32-bit halves convert
// exactly and Fast2Sum splits their one rounded sum (the high term has the
// larger exponent unless it is 0, and then lo = 0).
__device__ __forceinline__ double split_i64(int64_t x, double& lo) {
  const double a = (double)(int32_t)(x >> 32) * 0x1p32, b = (double)(uint32_t)x;
  const double hi = a + b;
  lo = b - (hi - a);
  return hi;
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
__device__ __forceinline__ bool round_fast_a(int64_t xl, int64_t xh, int e, double& out) {
  double hl, ll;
  const double hh = split_i64(xh, hl), lh = split_i64(xl, ll);
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
  const bool rounded = xh == 0 || (bound < halfu && (rb << 12) != 0);
  out = __builtin_ldexp(r, e);
  return rounded && (eb + e >= 1 || eb == 0);
}

template <typename RT>
__device__ __forceinline__ double reconstruct_one_a(const RT* rowq, int64_t mn, int n, int col,
                                                    int sa, int sb) {
  if (sa == INT32_MIN || sb == INT32_MIN) return __builtin_nan("");
  int c[kRA], v[kRA];
#pragma unroll
  for (int q = 0; q < kRA; ++q) c[q] = load_residue(rowq + q * mn, n, col);
  uint32_t packed[4] = {0, 0, 0, 0};
  [&]<int... J>(std::integer_sequence<int, J...>) {
    ((v[J] = garner_digit_a<J>(c, packed)), ...);
  }(std::make_integer_sequence<int, kRA>{});
  const int64_t xl = half_value_a<0, kSplitA>(v);   // |xl| <= P/2
  const int64_t xh = half_value_a<kSplitA, kRA>(v);  // |xh| <= (Q - 1) / 2
  const int e = -sa - sb;
  double out;
  if (!round_fast_a(xl, xh, e, out)) out = round_exact_a(xl, xh, e);
  return out;
}

// Grid: x over 256-column strips, y over rows (strided by gridDim.y).
template <bool BYTES, typename RT>
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
    const double r = BYTES ? reconstruct_one_a(cres + row * n, mn, (int)n, (int)col, ea[row], sb)
                           : reconstruct_one(cres + row * n, mn, (int)n, (int)col, ea[row], sb);
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

template <bool BYTES, typename RT>
hipError_t launch_rec(int64_t m, int64_t n, const RT* cres, const int32_t* ea, const int32_t* eb,
                      double* C, int64_t ldc, int subtract, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  hipLaunchKernelGGL((reconstruct_kernel<BYTES, RT>), grid_for(m, n), dim3(256), 0, stream, m, n,
                     cres, ea, eb, C, ldc, subtract);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_reconstruct_i32(int64_t m, int64_t n, const int32_t* cres, const int32_t* ea,
                                  const int32_t* eb, double* C, int64_t ldc, int subtract,
                                  hipStream_t stream) {
  return launch_rec<false, int32_t>(m, n, cres, ea, eb, C, ldc, subtract, stream);
}

hipError_t launch_reconstruct_i16(int64_t m, int64_t n, const int16_t* cres, const int32_t* ea,
                                  const int32_t* eb, double* C, int64_t ldc, int subtract,
                                  hipStream_t stream) {
  return launch_rec<false, int16_t>(m, n, cres, ea, eb, C, ldc, subtract, stream);
}

hipError_t launch_reconstruct_bytes_i32(int64_t m, int64_t n, const int32_t* cres,
                                        const int32_t* ea, const int32_t* eb, double* C,
                                        int64_t ldc, int subtract, hipStream_t stream) {
  return launch_rec<true, int32_t>(m, n, cres, ea, eb, C, ldc, subtract, stream);
}

hipError_t launch_reconstruct_bytes_i8(int64_t m, int64_t n, const int8_t* cres, const int32_t* ea,
                                       const int32_t* eb, double* C, int64_t ldc, int subtract,
                                       hipStream_t stream) {
  return launch_rec<true, int8_t>(m, n, cres, ea, eb, C, ldc, subtract, stream);
}

hipError_t launch_zero_c(int64_t m, int64_t n, double* C, int64_t ldc, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_c_kernel, grid_for(m, n), dim3(256), 0, stream, m, n, C, ldc);
  return hipGetLastError();
}

}  // namespace oz
