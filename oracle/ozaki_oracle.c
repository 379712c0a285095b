/*
 * CPU oracle for the Ozaki Scheme II emulated DGEMM (round-to-nearest variant,
 * published twelve-modulus set, and the all-byte candidate set A of Sec. 5.1
 * on the INT8 route).  TEST INFRASTRUCTURE ONLY: the tests, the
 * smoke check and the benchmark's CPU-baseline leg call it; the product path
 * never does.  It shares no code, header, table or constant generator with the
 * HIP library: every constant below is derived here from the moduli.
 *
 * Plain, slow, obviously correct: scalar loops, int64/__int128 exact integer
 * arithmetic and one IEEE rounding at the end.  Each function names the
 * passage of the paper it writes out.
 *
 *  - Eq. (scale): per-row (A) / per-column (B) power-of-two scaling and the
 *    integer quantiser (round to nearest, ties to even).
 *  - Eq. (moduli): the residue system, M > 2 mu with mu = k 2^{2t}.
 *  - Eq. (residueprod) and the centred residue convention [-x/2, x/2).
 *  - Eq. (pieces), the square-modulus two-plane split and Lemma 1 (the
 *    carry-corrected three-plane layout for the nonsquare moduli).
 *  - Eq. (garner) and Eq. (horner): mixed-radix reconstruction, symmetric
 *    lift, single rounding.
 *  - Sec. 5.1, candidate A: fifteen byte moduli whose centred residues fit an
 *    int8 operand directly, so on the INT8 route each residue is its own
 *    plane and each modulus needs one product (the oracle_set_* functions;
 *    set 0 is the published set, set 1 is candidate A).
 *
 * Pin status: every function here is checked in the CPU tests against the
 * paper's worked values, closed forms or brute force with Python integers /
 * fractions.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_R 12
#define OR_NPLANES 30
#define OR_NONFINITE INT32_MIN

typedef __int128 i128;
typedef unsigned __int128 u128;

/* Published set S in its published order (Eq. (moduli)): six squares
 * 33^2, 32^2, 31^2, 29^2, 25^2, 23^2, then six nonsquares. */
static const int64_t OR_MODULI[OR_R] = {1089, 1024, 961, 841, 625, 529,
                                        511,  509,  503, 499, 491, 487};

/* Candidate set A of Sec. 5.1 (all-byte): fifteen coprime moduli <= 256. */
#define OR_RA 15
static const int64_t OR_MODULI_A[OR_RA] = {256, 255, 253, 251, 247, 241, 239, 233,
                                           229, 227, 223, 217, 211, 199, 197};

/* Set 0: the published set; set 1: candidate A.  r and the moduli. */
static int or_set_r(int set) { return set == 1 ? OR_RA : OR_R; }
static const int64_t* or_set_m(int set) { return set == 1 ? OR_MODULI_A : OR_MODULI; }

int oracle_set_num_moduli(int set) { return or_set_r(set); }
int64_t oracle_set_modulus(int set, int i) { return or_set_m(set)[i]; }

/* Integer square root of m when m is a perfect square, else 0. */
static int64_t or_square_root(int64_t m) {
  for (int64_t s = 1; s * s <= m; ++s)
    if (s * s == m) return s;
  return 0;
}

int oracle_num_moduli(void) { return OR_R; }
int oracle_num_planes(void) { return OR_NPLANES; }
int64_t oracle_modulus(int i) { return OR_MODULI[i]; }
int oracle_planes_of(int i) { return or_square_root(OR_MODULI[i]) ? 2 : 3; }

/* M = prod m_i (Eq. (moduli)), returned as two 64-bit halves. */
void oracle_set_product_of_moduli(int set, uint64_t* hi, uint64_t* lo) {
  u128 M = 1;
  for (int i = 0; i < or_set_r(set); ++i) M *= (u128)or_set_m(set)[i];
  *hi = (uint64_t)(M >> 64);
  *lo = (uint64_t)M;
}
void oracle_product_of_moduli(uint64_t* hi, uint64_t* lo) { oracle_set_product_of_moduli(0, hi, lo); }

/* t(k): the largest t with k * 2^{2t} <= M/2 - 1, so that every entry of
 * A'B' (bounded by k 2^{2t}, Eq. (moduli)) lies strictly inside the symmetric
 * range [-M/2, M/2).  Returns -1 for k < 1. */
int oracle_set_scale_bits(int set, int64_t k) {
  if (k < 1) return -1;
  u128 M = 1;
  for (int i = 0; i < or_set_r(set); ++i) M *= (u128)or_set_m(set)[i];
  u128 q = (M / 2 - 1) / (u128)k; /* 2^{2t} <= q */
  int t = 0;
  while (((u128)1 << (2 * (t + 1))) <= q) ++t;
  return t;
}
int oracle_scale_bits(int64_t k) { return oracle_set_scale_bits(0, k); }

/* a1 (Eq. (scale) and the exponent scan of Alg. 1): for each of nvec vectors
 * of length k, element l of vector v at X[v*sv + l*sk], the exponent e of the
 * vector's largest magnitude in frexp form (max in [2^{e-1}, 2^e); e = 0 for
 * an all-zero vector) gives sigma = t - e.  A vector holding a NaN or an
 * infinity gets the sentinel INT32_MIN. */
void oracle_exponents(int64_t nvec, int64_t k, const double* X, int64_t sv,
                      int64_t sk, int t, int32_t* exps) {
  for (int64_t v = 0; v < nvec; ++v) {
    double mx = 0.0;
    int nonfinite = 0;
    for (int64_t l = 0; l < k; ++l) {
      double x = X[v * sv + l * sk];
      if (!isfinite(x)) nonfinite = 1;
      else if (fabs(x) > mx) mx = fabs(x);
    }
    if (nonfinite) {
      exps[v] = OR_NONFINITE;
    } else {
      int e = 0;
      (void)frexp(mx, &e);
      exps[v] = t - e;
    }
  }
}

/* a2 (Eq. (scale), round-to-nearest variant): z = RN_even(x * 2^sigma).  The
 * power-of-two scaling is exact here (|x 2^sigma| < 2^t), so rint is the only
 * rounding.  Rows flagged non-finite quantise to zero. */
int64_t oracle_quantise(double x, int32_t sigma) {
  if (sigma == OR_NONFINITE) return 0;
  return (int64_t)rint(ldexp(x, sigma));
}

/* a2, truncation variant (Ozaki-II-TZ of Table variants, the quantiser of
 * Eq. (scale) being truncation toward zero): z = trunc(x * 2^sigma), the
 * scaling again exact. */
int64_t oracle_quantise_tz(double x, int32_t sigma) {
  if (sigma == OR_NONFINITE) return 0;
  return (int64_t)trunc(ldexp(x, sigma));
}

/* quant 0: round to nearest (Ozaki-II-RN); 1: toward zero (Ozaki-II-TZ) */
void oracle_quantise_vectors_q(int quant, int64_t nvec, int64_t k, const double* X, int64_t sv,
                               int64_t sk, const int32_t* exps, int64_t* Z) {
  for (int64_t v = 0; v < nvec; ++v)
    for (int64_t l = 0; l < k; ++l)
      Z[v * k + l] = quant == 1 ? oracle_quantise_tz(X[v * sv + l * sk], exps[v])
                                : oracle_quantise(X[v * sv + l * sk], exps[v]);
}

void oracle_quantise_vectors(int64_t nvec, int64_t k, const double* X, int64_t sv,
                             int64_t sk, const int32_t* exps, int64_t* Z) {
  oracle_quantise_vectors_q(0, nvec, k, X, sv, sk, exps, Z);
}

/* The centred residue convention: z mod x in [-x/2, x/2), for even x the
 * endpoint -x/2 included and +x/2 excluded; for odd x the range
 * [-(x-1)/2, (x-1)/2]. */
int64_t oracle_centred_mod(int64_t z, int64_t x) {
  int64_t r = z % x;
  if (r < 0) r += x;           /* r in [0, x) */
  if (r > (x - 1) / 2) r -= x; /* upper half wraps to the negative side */
  return r;
}

/* a3 (Eq. (residueprod)): residues of quantised vectors, out[i][v][l]. */
void oracle_set_residues(int set, int64_t nvec, int64_t k, const int64_t* Z, int16_t* out) {
  for (int i = 0; i < or_set_r(set); ++i)
    for (int64_t v = 0; v < nvec; ++v)
      for (int64_t l = 0; l < k; ++l)
        out[(i * nvec + v) * k + l] = (int16_t)oracle_centred_mod(Z[v * k + l], or_set_m(set)[i]);
}
void oracle_residues(int64_t nvec, int64_t k, const int64_t* Z, int16_t* out) {
  oracle_set_residues(0, nvec, k, Z, out);
}

/* Candidate A on the INT8 route (Sec. 5.1): the centred residue of a byte
 * modulus lies in [-128, 127] and is itself the stored int8 plane, one per
 * modulus: planes[i][v][kp], kp >= k, zero padded. */
void oracle_set_a_planes(int64_t nvec, int64_t k, int64_t kp, const int64_t* Z, int8_t* planes) {
  memset(planes, 0, (size_t)OR_RA * (size_t)nvec * (size_t)kp);
  for (int i = 0; i < OR_RA; ++i)
    for (int64_t v = 0; v < nvec; ++v)
      for (int64_t l = 0; l < k; ++l)
        planes[((int64_t)i * nvec + v) * kp + l] =
            (int8_t)oracle_centred_mod(Z[v * k + l], OR_MODULI_A[i]);
}

/* Membership in the e4m3 integer set: integers M 2^e with |M| <= 15 and
 * magnitude at most 448 (Lemma 1's set).  Written as a direct search. */
int oracle_in_e4m3(int64_t v) {
  if (v < -448 || v > 448) return 0;
  for (int64_t M = -15; M <= 15; ++M)
    for (int e = 0; e <= 9; ++e)
      if (M * ((int64_t)1 << e) == v) return 1;
  return 0;
}

/* Lemma 1's rule on its own (it depends on d only, not on the modulus):
 * canonical balanced base-16 split, then the one carry when d0 + d1 is not
 * e4m3-exact.  out = (d0, d1, d0 + d1) as int64. */
void oracle_split16(int64_t d, int64_t* out) {
  int64_t d0 = oracle_centred_mod(d, 16);
  int64_t d1 = (d - d0) / 16;
  if (!oracle_in_e4m3(d0 + d1)) {
    int64_t sg = (d0 > 0) - (d0 < 0);
    d0 -= 16 * sg;
    d1 += sg;
  }
  out[0] = d0;
  out[1] = d1;
  out[2] = d0 + d1;
}

/* a4: the stored limbs of one centred residue d modulo the i-th modulus.
 *  - square m = s^2 (Eq. (pieces) with base s; d1 e1 vanishes mod s^2):
 *    d0 is the balanced base-s digit (the centred residue of d mod s) and
 *    d1 = (d - d0)/s; stored (d0, d1).
 *  - nonsquare (Lemma 1): canonical balanced base-16 digit d0 in [-8, 7],
 *    d1 = (d - d0)/16; if d0 + d1 is not e4m3-exact, move one unit of 16
 *    between the limbs against the sign of d0; stored (d0, d1, d0 + d1).
 * Returns the number of limbs written (2 or 3). */
int oracle_limbs(int i, int64_t d, int8_t* out) {
  int64_t m = OR_MODULI[i];
  int64_t s = or_square_root(m);
  if (s) {
    int64_t d0 = oracle_centred_mod(d, s);
    int64_t d1 = (d - d0) / s;
    out[0] = (int8_t)d0;
    out[1] = (int8_t)d1;
    return 2;
  }
  int64_t l[3];
  oracle_split16(d, l);
  out[0] = (int8_t)l[0];
  out[1] = (int8_t)l[1];
  out[2] = (int8_t)l[2];
  return 3;
}

/* Product of two residues from their limbs, following the epilogues the
 * paper gives: square moduli d e = d0 e0 + s (d0 e1 + d1 e0) + s^2 d1 e1,
 * whose last term vanishes mod s^2; nonsquare moduli Eq. (karcarry):
 * d e = (1-16) d0 e0 + 16 (d0+d1)(e0+e1) + (16^2-16) d1 e1.  Returns the
 * centred residue of the limb combination modulo m_i. */
int64_t oracle_limb_product(int i, const int8_t* dl, const int8_t* el) {
  int64_t m = OR_MODULI[i];
  int64_t s = or_square_root(m);
  int64_t v;
  if (s)
    v = (int64_t)dl[0] * el[0] + s * ((int64_t)dl[0] * el[1] + (int64_t)dl[1] * el[0]);
  else
    v = -15 * (int64_t)dl[0] * el[0] + 16 * (int64_t)dl[2] * el[2] + 240 * (int64_t)dl[1] * el[1];
  return oracle_centred_mod(v, m);
}

/* The limb-product epilogue over every ordered pair of centred residues of
 * modulus i: out[a * m + b] = oracle_limb_product(limbs(d_a), limbs(e_b))
 * with d_a = a - floor(m/2), e_b = b - floor(m/2). */
void oracle_limb_product_table(int i, int32_t* out) {
  int64_t m = OR_MODULI[i];
  int64_t lo = -(m / 2);
  for (int64_t a = 0; a < m; ++a) {
    int8_t dl[3] = {0, 0, 0};
    oracle_limbs(i, lo + a, dl);
    for (int64_t b = 0; b < m; ++b) {
      int8_t el[3] = {0, 0, 0};
      oracle_limbs(i, lo + b, el);
      out[a * m + b] = (int32_t)oracle_limb_product(i, dl, el);
    }
  }
}

/* Index of the first stored plane of modulus i (2 per square, 3 per
 * nonsquare, in the order of the set). */
int oracle_plane_base(int i) {
  int q = 0;
  for (int j = 0; j < i; ++j) q += oracle_planes_of(j);
  return q;
}

/* a2-a4 for whole vectors: planes[q][v][kp], kp >= k, zero padded. */
void oracle_planes(int64_t nvec, int64_t k, int64_t kp, const int64_t* Z, int8_t* planes) {
  memset(planes, 0, (size_t)OR_NPLANES * (size_t)nvec * (size_t)kp);
  for (int i = 0; i < OR_R; ++i) {
    int q0 = oracle_plane_base(i);
    for (int64_t v = 0; v < nvec; ++v)
      for (int64_t l = 0; l < k; ++l) {
        int8_t limbs[3];
        int np = oracle_limbs(i, oracle_centred_mod(Z[v * k + l], OR_MODULI[i]), limbs);
        for (int p = 0; p < np; ++p) planes[((int64_t)(q0 + p) * nvec + v) * kp + l] = limbs[p];
      }
  }
}

/* a5 (Eq. (residueprod)): C^(i) = centred(sum_l d_il e_lj mod m_i) from the
 * residues themselves (not the limbs), in plain int64 loops.  resA is
 * [12][m][k] (rows of A), resB is [12][n][k] (columns of B), C is [12][m][n]. */
void oracle_set_residue_gemm(int set, int64_t m, int64_t n, int64_t k, const int16_t* resA,
                             const int16_t* resB, int32_t* C) {
  for (int i = 0; i < or_set_r(set); ++i)
    for (int64_t r = 0; r < m; ++r)
      for (int64_t c = 0; c < n; ++c) {
        const int16_t* a = resA + (i * m + r) * k;
        const int16_t* b = resB + (i * n + c) * k;
        int64_t acc = 0;
        for (int64_t l = 0; l < k; ++l) acc += (int64_t)a[l] * b[l];
        C[(i * m + r) * n + c] = (int32_t)oracle_centred_mod(acc, or_set_m(set)[i]);
      }
}
void oracle_residue_gemm(int64_t m, int64_t n, int64_t k, const int16_t* resA,
                         const int16_t* resB, int32_t* C) {
  oracle_set_residue_gemm(0, m, n, k, resA, resB, C);
}

/* Modular inverse by the extended Euclidean algorithm (a, m coprime). */
static int64_t or_inverse(int64_t a, int64_t m) {
  int64_t r0 = m, r1 = ((a % m) + m) % m, t0 = 0, t1 = 1;
  while (r1 != 0) {
    int64_t q = r0 / r1, tmp;
    tmp = r0 - q * r1; r0 = r1; r1 = tmp;
    tmp = t0 - q * t1; t0 = t1; t1 = tmp;
  }
  return ((t0 % m) + m) % m;
}

/* Garner constants w_j = (m_1 ... m_{j-1})^{-1} mod m_j (Eq. (garner)). */
void oracle_set_garner_constants(int set, int64_t* w) {
  const int r = or_set_r(set);
  const int64_t* mod = or_set_m(set);
  w[0] = 1;
  for (int j = 1; j < r; ++j) {
    int64_t p = 1;
    for (int l = 0; l < j; ++l) p = (p * (mod[l] % mod[j])) % mod[j];
    w[j] = or_inverse(p, mod[j]);
  }
}
void oracle_garner_constants(int64_t* w) { oracle_set_garner_constants(0, w); }

/* a6 (Eq. (garner), Eq. (horner) and the symmetric lift): the integer X in
 * [-M/2, M/2) with X = c[i] (mod m_i) for all i.  Digits v_j in [0, m_j). */
static i128 or_garner(int set, const int64_t* c) {
  const int r = or_set_r(set);
  const int64_t* mod = or_set_m(set);
  int64_t w[OR_RA], v[OR_RA];
  oracle_set_garner_constants(set, w);
  u128 M = 1;
  for (int i = 0; i < r; ++i) M *= (u128)mod[i];
  for (int j = 0; j < r; ++j) {
    int64_t mj = mod[j];
    /* partial = v_1 + v_2 m_1 + ... + v_{j-1} m_1...m_{j-2} */
    u128 partial = 0, radix = 1;
    for (int l = 0; l < j; ++l) {
      partial += (u128)v[l] * radix;
      radix *= (u128)mod[l];
    }
    int64_t cj = ((c[j] % mj) + mj) % mj;
    int64_t pm = (int64_t)(partial % (u128)mj);
    int64_t diff = ((cj - pm) % mj + mj) % mj;
    v[j] = (diff * w[j]) % mj;
  }
  /* Horner: v_1 + m_1 (v_2 + m_2 (v_3 + ... + m_{r-1} v_r)) */
  u128 X = (u128)v[r - 1];
  for (int j = r - 2; j >= 0; --j) X = X * (u128)mod[j] + (u128)v[j];
  if (X >= M / 2) return (i128)X - (i128)M;
  return (i128)X;
}

/* Garner over a block of outputs: Cres [r][m][n] -> X as (hi, lo) words of
 * the two's-complement 128-bit value, X = hi * 2^64 + lo. */
void oracle_set_garner(int set, int64_t m, int64_t n, const int32_t* Cres, int64_t* Xhi,
                       uint64_t* Xlo) {
  for (int64_t e = 0; e < m * n; ++e) {
    int64_t c[OR_RA];
    for (int i = 0; i < or_set_r(set); ++i) c[i] = Cres[(int64_t)i * m * n + e];
    i128 X = or_garner(set, c);
    Xhi[e] = (int64_t)(X >> 64);
    Xlo[e] = (uint64_t)X;
  }
}
void oracle_garner(int64_t m, int64_t n, const int32_t* Cres, int64_t* Xhi, uint64_t* Xlo) {
  oracle_set_garner(0, m, n, Cres, Xhi, Xlo);
}

/* The exact integer product X = sum_l a'_il b'_lj directly (the quantity CRT
 * reconstruction must reproduce).  ZA is [m][k], ZB is [n][k]. */
void oracle_exact_product(int64_t m, int64_t n, int64_t k, const int64_t* ZA,
                          const int64_t* ZB, int64_t* Xhi, uint64_t* Xlo) {
  for (int64_t r = 0; r < m; ++r)
    for (int64_t c = 0; c < n; ++c) {
      i128 acc = 0;
      for (int64_t l = 0; l < k; ++l) acc += (i128)ZA[r * k + l] * (i128)ZB[c * k + l];
      Xhi[r * n + c] = (int64_t)(acc >> 64);
      Xlo[r * n + c] = (uint64_t)acc;
    }
}

/* Single rounding (Alg. 3, last step): RN_even(X * 2^e) for a signed integer
 * X (|X| < 2^127).  An X of at most 113 bits converts exactly to binary128
 * (113-bit significand); a longer one is first shifted right by s bits with
 * every dropped bit ORed into the lowest kept bit (exact for the rounding to
 * 53 bits: that bit lies far below the rounding point) and e grows by s.
 * The power-of-two scaling is exact in binary128's exponent range, and the
 * conversion to double rounds once, to nearest even, including the
 * subnormal and overflow ranges.  X = 0 gives +0.0. */
double oracle_round_scaled(int64_t Xhi, uint64_t Xlo, int e) {
  i128 X = (i128)(((u128)(uint64_t)Xhi << 64) | (u128)Xlo);
  if (X == 0) return 0.0;
  int neg = X < 0;
  u128 a = neg ? (u128)(-X) : (u128)X;
  int bits = 0;
  for (u128 t = a; t; t >>= 1) ++bits;
  if (bits > 113) {
    int sh = bits - 113;
    u128 dropped = a & (((u128)1 << sh) - 1);
    a = (a >> sh) | (dropped ? 1 : 0);
    e += sh;
  }
  __float128 q = neg ? -(__float128)a : (__float128)a;
  __float128 p = 1;
  for (int i = 0; i < e; ++i) p *= 2;
  for (int i = 0; i > e; --i) p /= 2;
  return (double)(q * p);
}

/* Output element: C_ij = RN(X 2^{-sigma_i - tau_j}); NaN when row i of A or
 * column j of B held a non-finite value.  With subtract, C_ij = C_ij - that
 * (two roundings: the product is rounded, then the IEEE subtraction). */
void oracle_reconstruct(int64_t m, int64_t n, const int64_t* Xhi, const uint64_t* Xlo,
                        const int32_t* expsA, const int32_t* expsB, int subtract,
                        double* C, int64_t ldc) {
  for (int64_t r = 0; r < m; ++r)
    for (int64_t c = 0; c < n; ++c) {
      double v;
      if (expsA[r] == OR_NONFINITE || expsB[c] == OR_NONFINITE)
        v = NAN;
      else
        v = oracle_round_scaled(Xhi[r * n + c], Xlo[r * n + c], -expsA[r] - expsB[c]);
      if (subtract) C[r * ldc + c] = C[r * ldc + c] - v;
      else C[r * ldc + c] = v;
    }
}

/* Alg. 1's last step and the range check that closes Alg. 3 (reading of this
 * build: the paper names the check and the native re-issue but does not
 * define the range): an output whose row of A or column of B holds a NaN or
 * an infinity is outside what the integer quantiser of Eq. (scale) can
 * represent, so it is re-issued on the native FP64 path -- the plain dot
 * product in index order l = 0..k-1 from +0, each product rounded, then
 * added (no fused multiply-add; the oracle is compiled with
 * -ffp-contract=off).  Every other output keeps the emulated value.  Such
 * outputs are always an infinity or a NaN, with the IEEE semantics of that
 * order of operations (Inf * 0, Inf - Inf and intermediate overflow
 * included).  With Cin, C_ij = Cin_ij - (that sum). */
void oracle_native_fallback(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                            const double* B, int64_t ldb, const int32_t* expsA,
                            const int32_t* expsB, const double* Cin, double* C, int64_t ldc) {
  for (int64_t r = 0; r < m; ++r)
    for (int64_t c = 0; c < n; ++c) {
      if (expsA[r] != OR_NONFINITE && expsB[c] != OR_NONFINITE) continue;
      double s = 0.0;
      for (int64_t l = 0; l < k; ++l) {
        double p = A[r * lda + l] * B[l * ldb + c];
        s = s + p;
      }
      C[r * ldc + c] = Cin ? Cin[r * ldc + c] - s : s;
    }
}


/* ---- accurate-mode scaling (reading of this build) ----------------------
 * Sec. 2 (Eq. (alpha), alpha = 3r + 1) says only that the accurate mode runs
 * one additional low-precision GEMM that estimates an input magnitude
 * bound.  This build reads it as follows:
 *  1. magnitude digits: alpha_il = ceil(16 |a_il| 2^{-e_i}) in {0..16}, e_i
 *     the frexp exponent of row i's largest magnitude, so that
 *     |a_il| <= alpha_il 2^{e_i - 4}; likewise beta_lj for the columns of B;
 *     0 on non-finite rows / columns (they take the native path);
 *  2. the bound GEMM: U_ij = sum_l alpha_il beta_lj (exact integers);
 *  3. shifts: for s_i >= 4, alpha_il 2^{s_i - 4} is an integer at least
 *     |a_il| 2^{s_i - e_i}, so RN (or truncation) of the scaled value cannot
 *     pass it: |a'_il| <= alpha_il 2^{s_i - 4}, and
 *     |sum_l a'_il b'_lj| <= 2^{s_i + u_j - 8} U_ij.  The admissible total
 *     L_ij is the largest L with 2^L U_ij <= 2^8 (M/2 - 1) (unbounded for
 *     U_ij = 0); u_j = min(58, floor(min_i L_ij / 2)) and
 *     s_i = min(58, min_j (L_ij - u_j)), so that s_i + u_j <= L_ij for every
 *     pair and every entry of A'B' stays below M/2, as Eq. (moduli) needs.
 *     58 is the largest t(k) of either modulus set (the all-byte set at
 *     k = 1): the scaled integers stay in the range the fast mode reaches;
 *  4. sigma_i = s_i - e_i, tau_j = u_j - f_j; the rest as in fast mode.
 * With U_ij <= 256 k, L_ij >= 2 t(k), so s_i, u_j >= t(k): never fewer bits
 * than the fast rule. */

#define OR_ACC_CAP 58
#define OR_ACC_INF 100000

/* Step 1 for one value: ceil(16 |x| 2^{-e}); |x| < 2^e, so the result is at
 * most 16.  The scaling by 2^{4-e} is exact unless it lands below the
 * normal range (x far below its vector's maximum), where the true value lies
 * in (0, 1) and its ceiling is 1. */
int oracle_mag_digit(double x, int e) {
  if (x == 0.0) return 0;
  const double d = ceil(ldexp(fabs(x), 4 - e));
  return d < 1.0 ? 1 : (int)d;
}

/* Step 1 for vectors: D[v][l] for vector v (element l at X[v*sv + l*sk]), with
 * the vector's frexp exponent e[v] (INT32_MIN: a non-finite vector, digits 0). */
void oracle_mag_digits(int64_t nvec, int64_t k, const double* X, int64_t sv, int64_t sk,
                       const int32_t* e, uint8_t* D) {
  for (int64_t v = 0; v < nvec; ++v)
    for (int64_t l = 0; l < k; ++l)
      D[v * k + l] = e[v] == OR_NONFINITE ? 0 : (uint8_t)oracle_mag_digit(X[v * sv + l * sk], e[v]);
}

/* Step 2: U[i][j] = sum_l DA[i][l] DB[j][l], plain int64 loops. */
void oracle_bound_gemm(int64_t m, int64_t n, int64_t k, const uint8_t* DA, const uint8_t* DB,
                       int64_t* U) {
  for (int64_t i = 0; i < m; ++i)
    for (int64_t j = 0; j < n; ++j) {
      int64_t acc = 0;
      for (int64_t l = 0; l < k; ++l) acc += (int64_t)DA[i * k + l] * DB[j * k + l];
      U[i * n + j] = acc;
    }
}

/* 2^8 (M/2 - 1) of a set. */
static u128 or_acc_limit(int set) {
  u128 M = 1;
  for (int i = 0; i < or_set_r(set); ++i) M *= (u128)or_set_m(set)[i];
  return (M / 2 - 1) << 8;
}

static int or_bitlen(u128 x) {
  int b = 0;
  while (x) {
    ++b;
    x >>= 1;
  }
  return b;
}

/* Step 3 for one entry: the largest L with 2^L U <= T = 2^8 (M/2 - 1),
 * searched upward from bitlen(T) - bitlen(U) - 1, which always qualifies
 * (2^L U < 2^(bitlen(T) - 1) <= T there). */
static int or_acc_total_T(u128 T, int64_t Uij) {
  if (Uij <= 0) return OR_ACC_INF;
  const u128 U = (u128)Uij;
  int L = or_bitlen(T) - or_bitlen(U) - 1;
  while ((U << (L + 1)) <= T) ++L;
  return L;
}

int oracle_acc_total(int set, int64_t Uij) { return or_acc_total_T(or_acc_limit(set), Uij); }

/* Step 3: the shifts s[m] and u[n] from U (flagA / flagB nonzero: a
 * non-finite row / column, left out of the minima -- its digits are zero,
 * so its L is unbounded anyway).  Returns 0, or -1 if a shift falls below 4
 * (outside the bound of step 3; needs k near 2^100). */
int oracle_acc_shifts(int set, int64_t m, int64_t n, const int64_t* U, const int32_t* flagA,
                      const int32_t* flagB, int32_t* s, int32_t* u) {
  const u128 T = or_acc_limit(set);
  int32_t* L = (int32_t*)malloc((size_t)(m * n > 0 ? m * n : 1) * sizeof(int32_t));
  if (!L) return -2; /* out of host memory */
  for (int64_t q = 0; q < m * n; ++q) L[q] = or_acc_total_T(T, U[q]);
  for (int64_t j = 0; j < n; ++j) {
    int mn = OR_ACC_INF;
    for (int64_t i = 0; i < m; ++i)
      if (!flagA[i] && L[i * n + j] < mn) mn = L[i * n + j];
    const int uj = mn / 2;
    u[j] = uj < OR_ACC_CAP ? uj : OR_ACC_CAP;
  }
  for (int64_t i = 0; i < m; ++i) {
    int mn = OR_ACC_INF;
    for (int64_t j = 0; j < n; ++j) {
      if (flagB[j]) continue;
      const int d = L[i * n + j] - u[j];
      if (d < mn) mn = d;
    }
    s[i] = mn < OR_ACC_CAP ? mn : OR_ACC_CAP;
  }
  free(L);
  for (int64_t i = 0; i < m; ++i)
    if (!flagA[i] && s[i] < 4) return -1;
  for (int64_t j = 0; j < n; ++j)
    if (!flagB[j] && u[j] < 4) return -1;
  return 0;
}
