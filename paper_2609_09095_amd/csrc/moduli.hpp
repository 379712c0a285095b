// Compile-time constants of the modulus sets and the tables derived from
// them.  The published set (Eq. (moduli)): limb layout (Eq. (pieces),
// Lemma 1), epilogue coefficients (square epilogue {1, s, s}, Eq. (karcarry))
// and Garner constants (Eq. (garner)).  The all-byte set (Sec. 5.1,
// candidate A): fifteen moduli <= 256 whose centred residues are int8
// operands as they stand.  Everything is constexpr, so kernels see the
// moduli as immediates and no table lives in memory.
#pragma once

#include <cstdint>

namespace oz {

constexpr int kR = 12;
constexpr int kPlanes = 30;
constexpr int kKAlign = 128;

// Published order: six squares, then the six nonsquares near 2^9.
constexpr int kModulus[kR] = {1089, 1024, 961, 841, 625, 529, 511, 509, 503, 499, 491, 487};

constexpr int exact_sqrt(int m) {
  for (int s = 1; s * s <= m; ++s)
    if (s * s == m) return s;
  return 0;
}

// Square root of a square modulus, 0 for the nonsquares.
constexpr int root_of(int i) { return exact_sqrt(kModulus[i]); }
constexpr int planes_of(int i) { return root_of(i) ? 2 : 3; }
constexpr int plane_base(int i) {
  int q = 0;
  for (int j = 0; j < i; ++j) q += planes_of(j);
  return q;
}
// Upper end of the centred range [-(m/2), (m-1)/2].
constexpr int centred_hi(int m) { return (m - 1) / 2; }

constexpr int64_t mod_pos(int64_t a, int64_t m) { return ((a % m) + m) % m; }
constexpr int64_t inverse_mod(int64_t a, int64_t m) {
  int64_t r0 = m, r1 = mod_pos(a, m), t0 = 0, t1 = 1;
  while (r1 != 0) {
    int64_t q = r0 / r1;
    int64_t r2 = r0 - q * r1;
    r0 = r1;
    r1 = r2;
    int64_t t2 = t0 - q * t1;
    t0 = t1;
    t1 = t2;
  }
  return mod_pos(t0, m);
}

// (m_0 ... m_{l-1}) mod m_j: weight of mixed-radix digit l seen modulo m_j.
constexpr int radix_mod(int l, int j) {
  int64_t p = 1;
  for (int q = 0; q < l; ++q) p = (p * kModulus[q]) % kModulus[j];
  return (int)p;
}
// Garner constant w_j = (m_0 ... m_{j-1})^{-1} mod m_j.
constexpr int garner_w(int j) { return (int)inverse_mod(radix_mod(j, j), kModulus[j]); }

// Limb-product coefficients of modulus i, one per product in issue order.
// Squares: P(d0,e0)*1 + P(d0,e1)*s + P(d1,e0)*s.  Nonsquares, Eq. (karcarry):
// P(d0,e0)*(-15) + P(d1,e1)*240 + P(d0+d1,e0+e1)*16.
constexpr int product_coef(int i, int p) {
  return root_of(i) ? (p == 0 ? 1 : root_of(i)) : (p == 0 ? -15 : (p == 1 ? 240 : 16));
}
// Plane index (relative to plane_base) of the A / B operand of product p.
constexpr int product_plane_a(int i, int p) { return root_of(i) ? (p == 2 ? 1 : 0) : p; }
constexpr int product_plane_b(int i, int p) { return root_of(i) ? (p == 1 ? 1 : 0) : p; }

// The residue GEMM's compact (int16) outputs leave out the weight of the
// last limb product it issues: a stored residue times compact_scale(i) is
// the true one, mod m_i.  Squares end on the weight-1 product, nonsquares on
// the weight-16 one.
constexpr int compact_scale(int i) { return root_of(i) ? 1 : 16; }

static_assert(plane_base(kR) == kPlanes, "30 stored planes for the published set");

// ---- all-byte set (Sec. 5.1, candidate A): 256 first, then fourteen odd
// moduli; log2 of the product 117.8
constexpr int kRA = 15;
constexpr int kModulusA[kRA] = {256, 255, 253, 251, 247, 241, 239, 233,
                                229, 227, 223, 217, 211, 199, 197};

// (m_0 ... m_{l-1}) mod m_j and the Garner constants of the all-byte set
constexpr int radix_mod_a(int l, int j) {
  int64_t p = 1;
  for (int q = 0; q < l; ++q) p = (p * kModulusA[q]) % kModulusA[j];
  return (int)p;
}
constexpr int garner_w_a(int j) { return (int)inverse_mod(radix_mod_a(j, j), kModulusA[j]); }

constexpr bool set_a_is_coprime_bytes() {
  for (int i = 0; i < kRA; ++i) {
    if (kModulusA[i] > 256 || kModulusA[i] < 2) return false;
    for (int j = i + 1; j < kRA; ++j) {
      int64_t a = kModulusA[i], b = kModulusA[j];
      while (b) {
        const int64_t t = a % b;
        a = b;
        b = t;
      }
      if (a != 1) return false;
    }
  }
  return true;
}
static_assert(set_a_is_coprime_bytes(), "pairwise coprime moduli of at most 256");
constexpr bool garner_constants_invert() {
  for (int j = 1; j < kR; ++j)
    if ((int64_t)radix_mod(j, j) * garner_w(j) % kModulus[j] != 1) return false;
  return true;
}
static_assert(garner_constants_invert(), "w_j (m_0 ... m_{j-1}) = 1 mod m_j");
constexpr bool garner_constants_invert_a() {
  for (int j = 1; j < kRA; ++j)
    if ((int64_t)radix_mod_a(j, j) * garner_w_a(j) % kModulusA[j] != 1) return false;
  return true;
}
static_assert(garner_constants_invert_a(), "w_j (m_0 ... m_{j-1}) = 1 mod m_j, all-byte set");

}  // namespace oz
