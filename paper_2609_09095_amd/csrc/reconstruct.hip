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
#include <hip/hip_runtime.h>

#include <utility>

#include "fp64_round.hpp"
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

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

// Residue q of output (row, col): a buffer load with the row's scalar base
// (row-uniform) and the column's 32-bit byte offset, shared by all twelve;
// streaming (nt), as every residue is read once.
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
    return (int)(int8_t)__builtin_amdgcn_raw_buffer_load_b8(rs, col, 0, 2);
  else if constexpr (sizeof(RT) == 2)
    return (int)(int16_t)__builtin_amdgcn_raw_buffer_load_b16(rs, col * 2, 0, 2);
  else
    return (int)__builtin_amdgcn_raw_buffer_load_b32(rs, col * 4, 0, 2);
}

// rowq: residues of this output row for modulus 0 (row-uniform); the
// modulus-q row sits mn elements further per q.
// fill: the value of an output on a row or column flagged non-finite (NaN,
// or +0 when the native re-issue supplies those outputs)
template <typename RT>
__device__ __forceinline__ double reconstruct_one(const RT* rowq, int64_t mn, int n, int col, int sa,
                                                  int sb, double fill) {
  if (sa == INT32_MIN || sb == INT32_MIN) return fill;
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

template <typename RT>
__device__ __forceinline__ double reconstruct_one_a(const RT* rowq, int64_t mn, int n, int col,
                                                    int sa, int sb, double fill) {
  if (sa == INT32_MIN || sb == INT32_MIN) return fill;
  int c[kRA], v[kRA];
#pragma unroll
  for (int q = 0; q < kRA; ++q) c[q] = load_residue(rowq + q * mn, n, col);
  uint32_t packed[4] = {0, 0, 0, 0};
  [&]<int... J>(std::integer_sequence<int, J...>) {
    ((v[J] = garner_digit_a<J>(c, packed)), ...);
  }(std::make_integer_sequence<int, kRA>{});
  const int e = -sa - sb;
  double out;
  if (!round_fast_a(v, e, out))  // |xl| <= P/2, |xh| <= (Q - 1) / 2
    out = round_exact_a(half_value_a<0, kSplitA>(v), half_value_a<kSplitA, kRA>(v), e);
  return out;
}

// Grid: x over 256-column strips, y over rows (strided by gridDim.y).
template <bool BYTES, typename RT>
__global__ __launch_bounds__(256) void reconstruct_kernel(int64_t m, int64_t n,
                                                          const RT* __restrict__ cres,
                                                          const int32_t* __restrict__ ea,
                                                          const int32_t* __restrict__ eb,
                                                          double* __restrict__ C, int64_t ldc,
                                                          int subtract, double fill) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= n) return;
  const int64_t mn = m * n;
  const int sb = eb[col];
  for (int64_t row = blockIdx.y; row < m; row += gridDim.y) {
    const double r = BYTES ? reconstruct_one_a(cres + row * n, mn, (int)n, (int)col, ea[row], sb, fill)
                           : reconstruct_one(cres + row * n, mn, (int)n, (int)col, ea[row], sb, fill);
    // C streams through once: non-temporal load and store (with the
    // residues' nt loads, the 32768^2 update 8.14 -> 7.74 ms; the all-byte
    // set and 8192^3 unchanged)
    double* out = C + row * ldc + col;
    __builtin_nontemporal_store(subtract ? __builtin_nontemporal_load(out) - r : r, out);
  }
}

// Alg. 1's last step, the native FP64 re-issue: an output whose row of A or
// column of B holds a NaN or an infinity (exponent INT32_MIN) has no
// emulated value, and becomes the dot product of that row and column in
// index order from +0, each product rounded and then added (the library is
// built with -ffp-contract=off; contraction is also switched off here).
// Such a value is always an infinity or a NaN.
__device__ __forceinline__ double native_dot(const double* __restrict__ a, const double* __restrict__ b,
                                             int64_t ldb, int64_t k) {
#pragma clang fp contract(off)
  double s = 0.0;
  for (int64_t l = 0; l < k; ++l) {
    const double p = a[l] * b[l * ldb];
    s = s + p;
  }
  return s;
}

// One block per 256 x 256 output tile (row tiles strided by gridDim.y):
// the flags of the tile's rows and columns are loaded coalesced and OR-ed
// across the block, so a tile with none -- every tile, on finite inputs --
// costs two loads and a barrier.  Otherwise each thread walks its column of
// the tile and re-issues the flagged outputs: C = dot, or C = C - dot.
// It runs apart from the reconstruction (whose loop it would slow), which
// then fills those outputs with +0: after it for C = AB, before it for
// C -= AB (C - (+0) leaves every value, NaN and infinities included, as it is).
__global__ __launch_bounds__(256) void native_reissue_kernel(int64_t m, int64_t n,
                                                             const int32_t* __restrict__ ea,
                                                             const int32_t* __restrict__ eb,
                                                             NativeOperands nat, double* C,
                                                             int64_t ldc, int subtract) {
  __shared__ int rowflag[256];
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const bool colflag = col < n && eb[col] == INT32_MIN;
  const int64_t tiles = (m + 255) / 256;
  for (int64_t t = blockIdx.y; t < tiles; t += gridDim.y) {
    const int64_t row0 = t * 256, r = row0 + threadIdx.x;
    const bool rf = r < m && ea[r] == INT32_MIN;
    rowflag[threadIdx.x] = rf;
    if (__syncthreads_or(rf || colflag) && col < n) {
      const int rows = m - row0 < 256 ? (int)(m - row0) : 256;
      for (int i = 0; i < rows; ++i) {
        if (!rowflag[i] && !colflag) continue;
        const int64_t row = row0 + i;
        const double d = native_dot(nat.A + row * nat.lda, nat.B + col, nat.ldb, nat.k);
        double* out = C + row * ldc + col;
        *out = subtract ? *out - d : d;
      }
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void zero_c_kernel(int64_t m, int64_t n, double* C, int64_t ldc) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= n) return;
  for (int64_t row = blockIdx.y; row < m; row += gridDim.y) C[row * ldc + col] = 0.0;
}

// Two rows per thread at least (rows y and y + gridDim.y): measured against
// one, the reconstruction of 8192^3 0.465 -> 0.397 ms (all-byte set 0.49 ->
// 0.43), of the 32768^2 x 1024 update 8.40 -> 8.08 ms (8.0 -> 7.5), same
// results; four, eight or sixteen rows, or two adjacent rows, are no better
// across shapes.
dim3 grid_for(int64_t m, int64_t n) {
  const int64_t y = (m + 1) / 2;
  return dim3((unsigned)((n + 255) / 256), (unsigned)(y < 65535 ? y : 65535));
}

template <bool BYTES, typename RT>
hipError_t launch_rec(int64_t m, int64_t n, const RT* cres, const int32_t* ea, const int32_t* eb,
                      double* C, int64_t ldc, int subtract, const NativeOperands& nat,
                      hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  const dim3 grid = grid_for(m, n);
  if (nat.A && subtract) {
    hipLaunchKernelGGL(native_reissue_kernel, dim3(grid.x, (unsigned)(m < 16776960 ? (m + 255) / 256 : 65535)),
                       dim3(256), 0, stream, m, n, ea, eb, nat, C, ldc, subtract);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((reconstruct_kernel<BYTES, RT>), grid, dim3(256), 0, stream, m, n, cres, ea, eb, C,
                     ldc, subtract, nat.A ? 0.0 : __builtin_nan(""));
  if (nat.A && !subtract) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(native_reissue_kernel, dim3(grid.x, (unsigned)(m < 16776960 ? (m + 255) / 256 : 65535)),
                       dim3(256), 0, stream, m, n, ea, eb, nat, C, ldc, subtract);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_reconstruct_i32(int64_t m, int64_t n, const int32_t* cres, const int32_t* ea,
                                  const int32_t* eb, double* C, int64_t ldc, int subtract,
                                  hipStream_t stream) {
  return launch_rec<false, int32_t>(m, n, cres, ea, eb, C, ldc, subtract, NativeOperands{}, stream);
}

hipError_t launch_reconstruct_i16(int64_t m, int64_t n, const int16_t* cres, const int32_t* ea,
                                  const int32_t* eb, double* C, int64_t ldc, int subtract,
                                  const NativeOperands& nat, hipStream_t stream) {
  return launch_rec<false, int16_t>(m, n, cres, ea, eb, C, ldc, subtract, nat, stream);
}

hipError_t launch_reconstruct_bytes_i32(int64_t m, int64_t n, const int32_t* cres,
                                        const int32_t* ea, const int32_t* eb, double* C,
                                        int64_t ldc, int subtract, hipStream_t stream) {
  return launch_rec<true, int32_t>(m, n, cres, ea, eb, C, ldc, subtract, NativeOperands{}, stream);
}

hipError_t launch_reconstruct_bytes_i8(int64_t m, int64_t n, const int8_t* cres, const int32_t* ea,
                                       const int32_t* eb, double* C, int64_t ldc, int subtract,
                                       const NativeOperands& nat, hipStream_t stream) {
  return launch_rec<true, int8_t>(m, n, cres, ea, eb, C, ldc, subtract, nat, stream);
}

hipError_t launch_zero_c(int64_t m, int64_t n, double* C, int64_t ldc, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_c_kernel, grid_for(m, n), dim3(256), 0, stream, m, n, C, ldc);
  return hipGetLastError();
}

}  // namespace oz
