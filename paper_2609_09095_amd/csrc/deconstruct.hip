// Deconstruction (Alg. 2): scale by 2^sigma, quantise (round to nearest even,
// or toward zero for the truncating variant), twelve
// centred residues, limb split, packed e4m3 plane stores (every limb is an
// e4m3-exact integer, Lemma 1, so the conversion is exact).  For the
// all-byte set (Sec. 5.1, candidate A) fifteen centred residues stored as
// int8, one plane per modulus.
//
// Each thread owns one vector (row of A / column of B) and 16 consecutive k,
// so every plane store is one 16-byte write.  VALU work and HBM traffic (8
// bytes read and 30 bytes written per element) are close: the nonsquare
// limb split comes from a small LDS table to keep the VALU side short.
// A wavefront covers 8 vectors x 128 k on both sides (group_of), so each of
// its plane stores is one contiguous KiB of the k-block-major layout:
//  - A (side 0): eight lanes read 1 KiB of one row;
//  - B (side 1): every FP64 load reads 64 contiguous bytes of 8 rows of B.
#include <utility>

#include "exponent_key.hpp"
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

constexpr int kElems = 16;  // k values per thread

// 16 plane bytes: a streaming store (the planes are read back by the
// residue GEMM long after, from HBM)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void put16(int8_t* p, uint4 w) {
  __builtin_nontemporal_store(u32x4{w.x, w.y, w.z, w.w}, reinterpret_cast<u32x4*>(p));
}

// four limbs as e4m3 bytes (OCP E4M3FN), the first in the low byte
__device__ __forceinline__ uint32_t pack4(float a, float b, float c, float d) {
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c, d, lo, true);
}

__device__ __forceinline__ void store16(int8_t* p, const float (&b)[kElems]) {
  uint4 w;
  w.x = pack4(b[0], b[1], b[2], b[3]);
  w.y = pack4(b[4], b[5], b[6], b[7]);
  w.z = pack4(b[8], b[9], b[10], b[11]);
  w.w = pack4(b[12], b[13], b[14], b[15]);
  put16(p, w);
}

// Integer-valued doubles y with |y| <= 2^51 sit in the low mantissa bits of
// y + kMagic (every such sum lies in [2^52, 2^53], where the spacing is 1),
// so the low word of that sum is y mod 2^32.
constexpr double kMagic = 6755399441055744.0;  // 1.5 * 2^52
__device__ __forceinline__ uint32_t low_word(double v) {
  return (uint32_t)__builtin_bit_cast(uint64_t, v);
}
constexpr int log2_exact(int m) { return m <= 1 ? 0 : 1 + log2_exact(m / 2); }

// Residue modes (the template parameter RM below), by the range of the
// scaled integers y = RN(x 2^sigma), |y| <= 2^t:
//  1: nearest quotient, ylo = y mod 2^32 from y + kMagic      (|y| <= 2^51)
//  2: nearest quotient, ylo split off by one exact FMA        (|y| <= 2^52,
//     the odd byte moduli only)
//  3: quotient within one of the nearest, ylo split off, one correction
//     each way                                                (|y| <= 2^58)
// 2^58 bounds every scale the library uses (t(k) <= 58 for both sets, and
// the accurate mode's shifts are capped there).
//
// y - q M modulo 2^24 for the FMA quotient q (ylo = y mod 2^32).  For odd M
// the FMA rounds y RN(1/M) + kMagic once, to kMagic + the integer nearest
// y RN(1/M) (|y / M| < 2^51, so the sum lies in [2^52, 2^53), where the
// spacing is 1); that product is within |y| ulp(1/M) / 2 of y / M.  For
// |y| <= 2^51 that is at most 1/(4M), while y / M is at least 1/(2M) away
// from a half integer, so the integer is the nearest quotient q and the low
// word of the sum is q mod 2^32.  For the odd byte moduli (M <= 255,
// ulp(1/M) / 2 = 2^-61) this holds up to |y| <= 2^52: the error is at most
// 2^-9 < 1/510.  Up to |y| <= 2^58 (every odd modulus here has
// ulp(1/M) / 2 <= 2^-61) the error is at most 1/8, so q is within 5/8 of
// y / M: |y - q M| <= 5 M / 8, one correction from the centred range.  The
// 24-bit multiply-add gives y - q M mod 2^24.  For a power of two M, y
// itself (mod 2^24) serves: its low log2(M) bits are the residue.
template <int M>
__device__ __forceinline__ int residue_low(double y, uint32_t ylo) {
  if constexpr ((M & (M - 1)) == 0) {
    return (int)ylo;
  } else {
    const double t = __builtin_fma(y, 1.0 / M, kMagic);
    // spelled out: left to itself the compiler widens this into a 64-bit
    // multiply-add once it sees that only the low bits are used
    int r;
    asm("v_mad_i32_i24 %0, %1, %2, %3" : "=v"(r) : "v"(low_word(t)), "s"(-M), "v"(ylo));
    return r;
  }
}

// Centred residue of the integer-valued y modulo M, in [-(M/2), (M-1)/2]
// (an int, |residue| <= 544): the low bits of residue_low, sign-extended --
// log2(M) bits for a power of two (the two's complement field is
// [-M/2, M/2) by itself), 24 bits for odd M, already centred when q is the
// nearest quotient (RM 1, 2) and after one correction otherwise (RM 3).
template <int M, int RM>
__device__ __forceinline__ int centred_residue(double y, uint32_t ylo) {
  if constexpr ((M & (M - 1)) == 0) {
    constexpr int sh = 32 - log2_exact(M);
    return (int)(ylo << sh) >> sh;
  } else {
    const int r = (int)((uint32_t)residue_low<M>(y, ylo) << 8) >> 8;
    if constexpr (RM == 3) {
      constexpr int hi = (M - 1) / 2, lo = hi - M + 1;
      const int r1 = r > hi ? r - M : r;
      return r1 < lo ? r1 + M : r1;
    } else {
      return r;
    }
  }
}

// Square modulus s^2 (Eq. (pieces) with base s): d0 = centred d mod s (the
// balanced digit, [-16, 15] for s = 32), d1 = (d - d0) / s.  |d| <= 544, so
// every step is exact in FP32 and the digits come out as the floats the
// e4m3 conversion takes.
template <int S>
__device__ __forceinline__ void split_square(float d, float& d0, float& d1) {
  // d1 = floor(d / s + 1/2): for even s exactly the balanced digit with d0 in
  // [-s/2, s/2); for odd s, d / s is never within 1/(2s) of a half integer,
  // far above the FP32 error of the FMA, so this is the nearest digit.  floor
  // never returns -0 here, so a zero digit gets the e4m3 code 0x00.
  d1 = __builtin_floorf(__builtin_fmaf(d, 1.0f / S, 0.5f));
  d0 = __builtin_fmaf(-(float)S, d1, d);
}

// Nonsquare modulus (Lemma 1): canonical balanced base-16 split (d0 in
// [-8, 7]), then one carry when d0 + d1 is odd with |d0 + d1| >= 17 --
// exactly the sums +-17, +-19, +-21, +-23 that e4m3 cannot hold.  d0 != 0
// whenever it fires.  All in FP32 on small integers, so exact; no -0 can
// arise (x - x and x + (-x) give +0 under round to nearest).
__device__ __forceinline__ void split_16(float d, float& d0, float& d1, float& d2) {
  float h = __builtin_floorf(__builtin_fmaf(d, 1.0f / 16, 0.5f));
  float l = __builtin_fmaf(-16.0f, h, d);
  const float s = l + h;
  const bool carry = __builtin_fabsf(s) > 16.0f && __builtin_amdgcn_fractf(s * 0.5f) != 0.0f;
  const float sg = l > 0.0f ? 1.0f : -1.0f;
  l = carry ? __builtin_fmaf(-16.0f, sg, l) : l;
  h = carry ? h + sg : h;
  d0 = l;
  d1 = h;
  d2 = l + h;
}

// The split depends on the residue alone, not on the modulus, and every
// nonsquare residue lies in [-255, 255]: a block tabulates it once in LDS
// as the three e4m3 codes (d0, d1, d0 + d1) in bytes 0-2 of entry d + 256.
constexpr int kSplitTable = 512;

__device__ __forceinline__ uint32_t split_16_codes(int d) {
  float d0, d1, d2;
  split_16((float)d, d0, d1, d2);
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(d0, d1, 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(d2, 0.0f, lo, true);
}

// Byte k of four table entries into one dword per plane (v_perm_b32 picks
// bytes of {hi, lo}: 0-3 from lo, 4-7 from hi, 12 gives 0).
__device__ __forceinline__ void gather_planes(uint32_t x0, uint32_t x1, uint32_t x2, uint32_t x3,
                                              uint32_t& p0, uint32_t& p1, uint32_t& p2) {
  const uint32_t t01 = __builtin_amdgcn_perm(x1, x0, 0x05010400u);  // x0.b0 x1.b0 x0.b1 x1.b1
  const uint32_t t23 = __builtin_amdgcn_perm(x3, x2, 0x05010400u);
  const uint32_t u01 = __builtin_amdgcn_perm(x1, x0, 0x0c0c0602u);  // x0.b2 x1.b2 0 0
  const uint32_t u23 = __builtin_amdgcn_perm(x3, x2, 0x0c0c0602u);
  p0 = __builtin_amdgcn_perm(t23, t01, 0x05040100u);
  p1 = __builtin_amdgcn_perm(t23, t01, 0x07060302u);
  p2 = __builtin_amdgcn_perm(u23, u01, 0x05040100u);
}

template <int I, int RM>
__device__ __forceinline__ void emit_modulus(const double (&y)[kElems], const uint32_t (&ylo)[kElems],
                                             int8_t* planes,
                                             int64_t plane_stride, int64_t off,
                                             const uint32_t* lut) {
  constexpr int M = kModulus[I];
  constexpr int S = root_of(I);
  constexpr int Q = plane_base(I);
  int8_t* base = planes + (int64_t)Q * plane_stride + off;
  if constexpr (S != 0) {
    float l0[kElems], l1[kElems];
#pragma unroll
    for (int c = 0; c < kElems; ++c)
      split_square<S>((float)centred_residue<M, RM>(y[c], ylo[c]), l0[c], l1[c]);
    store16(base, l0);
    store16(base + plane_stride, l1);
  } else {
    uint32_t x[kElems];
#pragma unroll
    for (int c = 0; c < kElems; ++c) x[c] = lut[centred_residue<M, RM>(y[c], ylo[c]) + 256];
    uint4 w0, w1, w2;
    gather_planes(x[0], x[1], x[2], x[3], w0.x, w1.x, w2.x);
    gather_planes(x[4], x[5], x[6], x[7], w0.y, w1.y, w2.y);
    gather_planes(x[8], x[9], x[10], x[11], w0.z, w1.z, w2.z);
    gather_planes(x[12], x[13], x[14], x[15], w0.w, w1.w, w2.w);
    put16(base, w0);
    put16(base + plane_stride, w1);
    put16(base + 2 * plane_stride, w2);
  }
}

template <int RM, int... I>
__device__ __forceinline__ void emit_all(std::integer_sequence<int, I...>, const double (&y)[kElems],
                                         const uint32_t (&ylo)[kElems], int8_t* planes,
                                         int64_t plane_stride, int64_t off, const uint32_t* lut) {
  (emit_modulus<I, RM>(y, ylo, planes, plane_stride, off, lut), ...);
}

// Thread -> (vector, 16-k group), both sides: a block covers 32 vectors x
// 128 k -- one k-block of the plane layout -- and a wavefront 8 vectors, so
// every plane store of a wavefront fills 1 KiB of contiguous plane bytes and
// consecutive blocks continue the same k-block: the stores sweep each plane
// region linearly.  Lane l takes vector l%8 and k group l/8 (for B, eight
// consecutive columns: each FP64 load reads 64 contiguous bytes of 8 rows).
__device__ __forceinline__ void group_of(int64_t vecs, int64_t& v, int64_t& g) {
  const int64_t vb = (vecs + 31) / 32;
  const int lane = threadIdx.x & 63;
  v = (int64_t)(blockIdx.x % vb) * 32 + (threadIdx.x >> 6) * 8 + (lane & 7);
  g = (int64_t)(blockIdx.x / vb) * 8 + (lane >> 3);
}

// Byte offset of a thread's 16 plane bytes within plane 0, in the layout
// [k_pad/128][planes][vecs][128]: plane q adds q * vecs * 128.
__device__ __forceinline__ int64_t plane_offset(int64_t vecs, int nplanes, int64_t v, int64_t g) {
  return ((g >> 3) * nplanes * vecs + v) * 128 + (g & 7) * 16;
}

// The 16 inputs of a group: unconditional loads from clamped (always valid)
// addresses, then the mask, so no branches sit around the loads; zeros past
// k, for inactive threads and for a non-finite vector.  Returns sigma (0 for
// a non-finite vector).
// keys_in: exps holds the column scan's exponent keys, turned into sigma here.
template <int SIDE>
__device__ __forceinline__ int load_group(int64_t vecs, int64_t k, const double* __restrict__ X,
                                          int64_t ldx, const int32_t* __restrict__ exps, bool keys_in,
                                          int t, int64_t v, int64_t k0, bool active, double (&x)[kElems]) {
  const int raw = active ? exps[v] : 0;
  int sigma = keys_in ? key_to_sigma((uint32_t)raw, t) : raw;
  const bool finite = sigma != INT32_MIN;
  sigma = finite ? sigma : 0;
  // lim = last valid c of this group
  const int64_t vc = v < vecs ? v : vecs - 1;
  const int64_t kc = k0 < k ? k0 : k - 1;
  const int lim = k0 < k ? (int)(k - k0 < kElems ? k - k0 : kElems) - 1 : 0;
  const double* first = SIDE == 0 ? X + vc * ldx + kc : X + kc * ldx + vc;
  const bool live = active && finite;
  if constexpr (SIDE == 0) {
    // a whole group of a row whose start is 16-byte aligned: eight 16-byte
    // loads (the vector memory path moves twice the bytes per request)
    if (k0 + kElems <= k && (((uintptr_t)X | (uintptr_t)(ldx * 8)) & 15) == 0) {
      const double2* p = reinterpret_cast<const double2*>(first);
#pragma unroll
      for (int c = 0; c < kElems / 2; ++c) {
        const double2 q = p[c];
        x[2 * c] = live ? q.x : 0.0;
        x[2 * c + 1] = live ? q.y : 0.0;
      }
      return sigma;
    }
  }
#pragma unroll
  for (int c = 0; c < kElems; ++c) {
    const int cc = c < lim ? c : lim;
    const double xv = SIDE == 0 ? first[cc] : first[(int64_t)cc * ldx];
    x[c] = (live && c <= lim && k0 + c < k) ? xv : 0.0;
  }
  return sigma;
}

// |x 2^sigma| < 2^t: the scaling is exact, and the quantiser of Eq. (scale)
// is the one rounding: to nearest even (RN), or toward zero (TZ).  Then
// ylo = y mod 2^32: from y + kMagic (RM 1, |y| <= 2^51), or (RM 2, 3: past
// 2^51 that sum is no longer exact) as y - h 2^32 with h = floor(y 2^-32),
// one exact FMA.
template <bool TZ, int RM>
__device__ __forceinline__ void scale_round(const double (&x)[kElems], int sigma,
                                            double (&y)[kElems], uint32_t (&ylo)[kElems]) {
#pragma unroll
  for (int c = 0; c < kElems; ++c) {
    const double v = __builtin_ldexp(x[c], sigma);
    y[c] = TZ ? __builtin_trunc(v) : __builtin_rint(v);
    if constexpr (RM == 1)
      ylo[c] = low_word(y[c] + kMagic);
    else
      ylo[c] = (uint32_t)__builtin_fma(-__builtin_floor(y[c] * 0x1p-32), 0x1p32, y[c]);
  }
}

template <int SIDE, int RM, bool TZ>
__global__ __launch_bounds__(256) void deconstruct_kernel(int64_t vecs, int64_t vstride, int64_t k,
                                                          int64_t kp, const double* __restrict__ X,
                                                          int64_t ldx, const int32_t* __restrict__ exps,
                                                          bool keys_in, int t,
                                                          int8_t* __restrict__ planes) {
  int64_t v, g;
  group_of(vecs, v, g);
  const bool active = v < vecs && g < kp / kElems;
  const int64_t k0 = g * kElems;
  double x[kElems];
  const int sigma = load_group<SIDE>(vecs, k, X, ldx, exps, keys_in, t, v, k0, active, x);
  // the split table, built while the loads are in flight
  __shared__ uint32_t lut[kSplitTable];
  for (int i = threadIdx.x; i < kSplitTable; i += 256) lut[i] = split_16_codes(i - 256);
  __syncthreads();
  if (!active) return;
  double y[kElems];
  uint32_t ylo[kElems];
  scale_round<TZ, RM>(x, sigma, y, ylo);
  emit_all<RM>(std::make_integer_sequence<int, kR>{}, y, ylo, planes, vstride * 128,
                  plane_offset(vstride, kPlanes, v, g), lut);
}

// ---- all-byte set (Sec. 5.1, candidate A) on the int8 route: the centred
// residue of a byte modulus lies in [-128, 127] and is stored as it stands,
// one int8 plane per modulus (8 bytes read, 15 written per element).

// four residues in [-128, 127] as bytes, the first in the low byte
// (v_perm_b32 selectors: 0-3 bytes of the second operand, 4-7 of the first,
// 12 gives 0)
__device__ __forceinline__ uint32_t pack_bytes(int a, int b, int c, int d) {
  const uint32_t ab = __builtin_amdgcn_perm((uint32_t)b, (uint32_t)a, 0x0c0c0400u);
  const uint32_t cd = __builtin_amdgcn_perm((uint32_t)d, (uint32_t)c, 0x0c0c0400u);
  return __builtin_amdgcn_perm(cd, ab, 0x05040100u);
}

// The byte of the centred residue: its low eight bits, which residue_low
// already holds when q is the nearest quotient (RM 1, 2).
template <int I, int RM>
__device__ __forceinline__ void emit_byte_modulus(const double (&y)[kElems],
                                                  const uint32_t (&ylo)[kElems], int8_t* planes,
                                                  int64_t plane_stride, int64_t off) {
  constexpr int M = kModulusA[I];
  int r[kElems];
#pragma unroll
  for (int c = 0; c < kElems; ++c)
    r[c] = RM == 3 ? centred_residue<M, 3>(y[c], ylo[c]) : residue_low<M>(y[c], ylo[c]);
  uint4 w;
  w.x = pack_bytes(r[0], r[1], r[2], r[3]);
  w.y = pack_bytes(r[4], r[5], r[6], r[7]);
  w.z = pack_bytes(r[8], r[9], r[10], r[11]);
  w.w = pack_bytes(r[12], r[13], r[14], r[15]);
  put16(planes + (int64_t)I * plane_stride + off, w);
}

template <int RM, int... I>
__device__ __forceinline__ void emit_all_bytes(std::integer_sequence<int, I...>,
                                               const double (&y)[kElems],
                                               const uint32_t (&ylo)[kElems], int8_t* planes,
                                               int64_t plane_stride, int64_t off) {
  (emit_byte_modulus<I, RM>(y, ylo, planes, plane_stride, off), ...);
}

// RM: the residue mode (1, 2 or 3, as for residue_low).
template <int SIDE, int RM, bool TZ>
__global__ __launch_bounds__(256) void deconstruct_bytes_kernel(int64_t vecs, int64_t vstride, int64_t k,
                                                                int64_t kp, const double* __restrict__ X,
                                                                int64_t ldx,
                                                                const int32_t* __restrict__ exps,
                                                                bool keys_in, int t,
                                                                int8_t* __restrict__ planes) {
  int64_t v, g;
  group_of(vecs, v, g);
  const bool active = v < vecs && g < kp / kElems;
  if (!active) return;
  const int64_t k0 = g * kElems;
  double x[kElems], y[kElems];
  uint32_t ylo[kElems];
  const int sigma = load_group<SIDE>(vecs, k, X, ldx, exps, keys_in, t, v, k0, true, x);
  scale_round<TZ, RM>(x, sigma, y, ylo);
  emit_all_bytes<RM>(std::make_integer_sequence<int, kRA>{}, y, ylo, planes, vstride * 128,
                            plane_offset(vstride, kRA, v, g));
}

// ---- accurate mode (Sec. 2, Eq. (alpha)): the magnitude digit of every
// element, ceil(16 |x| 2^-e) in {0..16} with e the vector's frexp exponent,
// as one int8 plane in the plane layout (the operand of the bound product).
// exps holds -e (the exponent scan at t = 0; with keys_in the column scan's
// keys).  16 |x| 2^-e is exact in FP64 unless it falls below the normal
// range, where its ceiling is 1; a non-finite vector gets zero digits.
template <int SIDE>
__global__ __launch_bounds__(256) void digits_kernel(int64_t vecs, int64_t k, int64_t kp,
                                                     const double* __restrict__ X, int64_t ldx,
                                                     const int32_t* __restrict__ exps, bool keys_in,
                                                     int8_t* __restrict__ digits) {
  int64_t v, g;
  group_of(vecs, v, g);
  if (v >= vecs || g >= kp / kElems) return;
  double x[kElems];
  const int ne = load_group<SIDE>(vecs, k, X, ldx, exps, keys_in, 0, v, g * kElems, true, x);
  int d[kElems];
#pragma unroll
  for (int c = 0; c < kElems; ++c) {
    const double a = __builtin_fabs(x[c]);
    const double u = __builtin_ceil(__builtin_ldexp(a, 4 + ne));
    d[c] = a == 0.0 ? 0 : (u < 1.0 ? 1 : (int)u);
  }
  uint4 w;
  w.x = pack_bytes(d[0], d[1], d[2], d[3]);
  w.y = pack_bytes(d[4], d[5], d[6], d[7]);
  w.z = pack_bytes(d[8], d[9], d[10], d[11]);
  w.w = pack_bytes(d[12], d[13], d[14], d[15]);
  put16(digits + plane_offset(vecs, 1, v, g), w);
}

struct DecArgs {
  int64_t blocks, vecs, vstride, k, kp;
  const double* X;
  int64_t ldx;
  const int32_t* exps;
  bool keys_in;
  int t;
  int8_t* planes;
};

template <int SIDE, bool BYTES, int RM, bool TZ>
void launch_one(const DecArgs& a, hipStream_t stream) {
  if constexpr (BYTES)
    hipLaunchKernelGGL((deconstruct_bytes_kernel<SIDE, RM, TZ>), dim3((unsigned)a.blocks), dim3(256), 0,
                       stream, a.vecs, a.vstride, a.k, a.kp, a.X, a.ldx, a.exps, a.keys_in, a.t, a.planes);
  else if constexpr (RM != 2)  // the nearest-quotient bound of RM 2 holds for byte moduli only
    hipLaunchKernelGGL((deconstruct_kernel<SIDE, RM, TZ>), dim3((unsigned)a.blocks), dim3(256), 0, stream,
                       a.vecs, a.vstride, a.k, a.kp, a.X, a.ldx, a.exps, a.keys_in, a.t, a.planes);
}

template <int SIDE, bool BYTES>
void launch_side(int rm, bool tz, const DecArgs& a, hipStream_t stream) {
  if (rm == 1) {
    if (tz) launch_one<SIDE, BYTES, 1, true>(a, stream);
    else launch_one<SIDE, BYTES, 1, false>(a, stream);
  } else if (rm == 2) {
    if (tz) launch_one<SIDE, BYTES, 2, true>(a, stream);
    else launch_one<SIDE, BYTES, 2, false>(a, stream);
  } else {
    if (tz) launch_one<SIDE, BYTES, 3, true>(a, stream);
    else launch_one<SIDE, BYTES, 3, false>(a, stream);
  }
}

}  // namespace

hipError_t launch_digits(int side, int64_t vecs, int64_t k, int64_t kp, const double* X, int64_t ldx,
                         const int32_t* exps, bool keys_in, int8_t* digits, hipStream_t stream) {
  if (vecs <= 0 || kp <= 0) return hipSuccess;
  const int64_t blocks = ((vecs + 31) / 32) * (kp / 128);
  if (blocks > (int64_t)UINT32_MAX) return hipErrorInvalidValue;
  if (side == 0)
    hipLaunchKernelGGL(digits_kernel<0>, dim3((unsigned)blocks), dim3(256), 0, stream, vecs, k, kp, X, ldx,
                       exps, keys_in, digits);
  else
    hipLaunchKernelGGL(digits_kernel<1>, dim3((unsigned)blocks), dim3(256), 0, stream, vecs, k, kp, X, ldx,
                       exps, keys_in, digits);
  return hipGetLastError();
}

hipError_t launch_deconstruct(int set, int quant, int side, int64_t vecs, int64_t vstride, int64_t k,
                              int64_t kp, int t, const double* X, int64_t ldx, const int32_t* exps,
                              bool keys_in, int8_t* planes, hipStream_t stream) {
  if (vstride < vecs || t > kMaxScaleBits) return hipErrorInvalidValue;
  if (vecs <= 0 || kp <= 0) return hipSuccess;
  const bool bytes = set == kSetBytes;
  const bool tz = quant == kQuantTZ;
  // |y| <= 2^t: the nearest quotient with ylo from kMagic, then (the byte
  // moduli at t = 52) with ylo split off, else one correction
  const int mode = t <= (bytes ? 51 : 50) ? 1 : (bytes && t == 52 ? 2 : 3);
  const DecArgs a{((vecs + 31) / 32) * (kp / 128), vecs, vstride, k, kp, X, ldx, exps, keys_in, t, planes};
  if (side == 0) {
    if (bytes) launch_side<0, true>(mode, tz, a, stream);
    else launch_side<0, false>(mode, tz, a, stream);
  } else {
    if (bytes) launch_side<1, true>(mode, tz, a, stream);
    else launch_side<1, false>(mode, tz, a, stream);
  }
  return hipGetLastError();
}

}  // namespace oz
