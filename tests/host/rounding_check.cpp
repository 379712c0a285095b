// Host check of the reconstruction's last step (fp64_round.hpp), compiled
// with g++ by tests/test_host_rounding.py: wherever round_fast /
// round_fast_a claim a result, it equals round_exact / round_exact_a bit for
// bit.  Cases: random digit vectors; values at and next to FP64 rounding
// boundaries (powers of two, midpoints) at every magnitude, scaled onto the
// subnormal and overflow thresholds; small values (high half 0 or small);
// values below -M/2 that the published set's lift moves.  Also checked:
// exact midpoints above P (nonzero high half) never take the fast path,
// and random inputs almost always do.  Exit status 0 on success.
#include <cstdio>
#include <cstring>

#include "fp64_round.hpp"

using namespace oz;
typedef __int128 i128;

static uint64_t st = 0x9E3779B97F4A7C15ull;
static uint64_t rnd() {
  st ^= st << 13;
  st ^= st >> 7;
  st ^= st << 17;
  return st;
}
static bool same(double a, double b) {
  uint64_t x, y;
  memcpy(&x, &a, 8);
  memcpy(&y, &b, 8);
  return x == y;
}

template <int R>
struct Set {
  const int* mod;
  long fast = 0, slow = 0, bad = 0;
  i128 M() const {
    i128 p = 1;
    for (int j = 0; j < R; ++j) p *= mod[j];
    return p;
  }
  // centred mixed-radix digits of X in [-M/2, M/2)
  void digits(i128 X, int (&v)[R]) const {
    for (int j = 0; j < R; ++j) {
      int r = (int)(X % mod[j]);
      if (r < 0) r += mod[j];
      if (2 * r >= mod[j]) r -= mod[j];
      v[j] = r;
      X = (X - r) / mod[j];
    }
  }
  i128 value(const int (&v)[R]) const {
    i128 x = 0;
    for (int j = R - 1; j >= 0; --j) x = x * mod[j] + v[j];
    return x;
  }
};

static bool run_s12(Set<kR>& S, const int (&v)[kR], int e) {
  double f;
  const bool ok = round_fast(v, e, f);
  const double x = round_exact(v, e);
  if (ok) {
    ++S.fast;
    if (!same(f, x) && ++S.bad < 5) printf("S12 mismatch e=%d fast=%a exact=%a\n", e, f, x);
  } else {
    ++S.slow;
  }
  return ok;
}
static bool run_a15(Set<kRA>& S, const int (&v)[kRA], int e) {
  const int64_t xl = half_value_a<0, kSplitA>(v), xh = half_value_a<kSplitA, kRA>(v);
  // the FP64 halves: lh = RN(xl), hh = RN(xh), hh + hl = xh exactly (the
  // host's int64 -> double conversion rounds to nearest even)
  double lh, hh, hl;
  halves_fp64_a(v, lh, hh, hl);
  if (!same(lh, (double)xl) || !same(hh, (double)xh) || (i128)(int64_t)hh + (i128)(int64_t)hl != (i128)xh) {
    if (++S.bad < 5) printf("A15 halves differ: xl=%lld xh=%lld\n", (long long)xl, (long long)xh);
  }
  double f;
  const bool ok = round_fast_a(v, e, f);
  const double x = round_exact_a(xl, xh, e);
  if (ok) {
    ++S.fast;
    if (!same(f, x) && ++S.bad < 5) printf("A15 mismatch e=%d fast=%a exact=%a\n", e, f, x);
  } else {
    ++S.slow;
  }
  return ok;
}

// X at or next to a rounding boundary of magnitude 2^E; *tie set for exact midpoints
static i128 boundary(int E, bool* tie) {
  static const long ds[] = {0, 1, -1, 2, -2, 3, -3, 17, -17, 31, -31, 32, -32, 33, -33, 64, -64,
                            1023, -1024, 4096, -4096, 100000, -100000};
  const int kind = (int)(rnd() % 4);
  const uint64_t mt = (rnd() >> 12) | (1ull << 52);
  i128 X;
  bool mid = false;
  if (kind == 0) {
    X = (i128)1 << E;
  } else if (kind == 1) {
    X = (((i128)mt << 1) | 1) << (E - 53);
    mid = true;
  } else {
    X = (i128)mt << (E - 52);
  }
  const long d = ds[rnd() % (sizeof ds / sizeof ds[0])];
  i128 off = d;
  if (rnd() % 3 == 0) off = (i128)d << (E - 60 > 0 ? E - 60 : 0);
  *tie = mid && off == 0;
  X += off;
  return (rnd() & 1) ? -X : X;
}

static int scale_for(int E) {
  switch ((int)(rnd() % 8)) {
    case 0: return -1022 - E + (int)(rnd() % 5) - 2;  // normal / subnormal threshold
    case 1: return 1023 - E + (int)(rnd() % 5) - 2;   // overflow threshold
    case 2: return -1074 - E + (int)(rnd() % 60) - 30;
    default: return (int)(rnd() % 200) - 150;
  }
}

template <int R, typename Run>
static int check(Set<R>& S, const char* name, int top_bits, i128 P, Run run) {
  const i128 h = S.M() / 2;
  int v[R];
  int fails = 0;
  // random digits: the fast path should take practically all of them
  for (int it = 0; it < 1000000; ++it) {
    for (int j = 0; j < R; ++j) v[j] = (int)(rnd() % S.mod[j]) - S.mod[j] / 2;
    run(S, v, (int)(rnd() % 200) - 150);
  }
  if (S.slow > 2) {
    printf("%s: %ld random inputs declined\n", name, S.slow);
    ++fails;
  }
  long ties_fast = 0;
  for (int it = 0; it < 600000; ++it) {
    const int E = 54 + (int)(rnd() % (top_bits - 54));
    bool tie;
    const i128 X = boundary(E, &tie);
    if (X >= h || X < -h) continue;
    S.digits(X, v);
    if (S.value(v) != X) {
      printf("%s: digit error\n", name);
      return 1;
    }
    // with a nonzero high half (|X| > P) an exact midpoint must be declined;
    // below it, r is the one fma rounding of the low half, ties included
    if (run(S, v, scale_for(E)) && tie && (X > P || X < -P)) ++ties_fast;
  }
  if (ties_fast) {
    printf("%s: %ld exact midpoints took the fast path\n", name, ties_fast);
    ++fails;
  }
  // small values, values near small multiples of P, and the high half's range
  for (int it = 0; it < 600000; ++it) {
    i128 X;
    const int kind = (int)(rnd() % 3);
    if (kind == 0) X = (i128)(rnd() >> (rnd() % 64));
    else if (kind == 1) X = P * (i128)((int)(rnd() % 5) - 2) + (i128)(rnd() % (uint64_t)P) - P / 2;
    else X = ((i128)1 << (40 + rnd() % 20)) * P + (i128)(rnd() % (uint64_t)P) - P / 2;
    if (rnd() & 1) X = -X;
    if (X >= h || X < -h) continue;
    S.digits(X, v);
    run(S, v, (int)(rnd() % 2200) - 1100);
  }
  printf("%s: fast %ld slow %ld mismatches %ld\n", name, S.fast, S.slow, S.bad);
  return fails + (S.bad != 0);
}

int main() {
  Set<kR> s12{kModulus};
  Set<kRA> a15{kModulusA};
  int fails = check(s12, "S12", 111, (i128)kP, run_s12);
  fails += check(a15, "A15", 117, (i128)kPA, run_a15);
  // the lift: high digits at their minimum and low digits near theirs give
  // values below -M/2; the fast path must decline all of them
  long lifted = 0, lifted_fast = 0;
  const i128 h = s12.M() / 2;
  for (int it = 0; it < 200000; ++it) {
    int v[kR];
    for (int j = 0; j < kR; ++j) v[j] = -(kModulus[j] / 2);
    v[0] += (int)(rnd() % 1200);
    const bool below = s12.value(v) < -h;
    lifted += below;
    if (run_s12(s12, v, (int)(rnd() % 200) - 150) && below) ++lifted_fast;
  }
  printf("lift: %ld below -M/2, %ld on the fast path, mismatches %ld\n", lifted, lifted_fast, s12.bad);
  if (lifted == 0 || lifted_fast != 0 || s12.bad != 0) ++fails;
  return fails != 0;
}
