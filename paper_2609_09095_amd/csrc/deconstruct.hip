// Deconstruction (Alg. 2): scale by 2^sigma, round to nearest even, twelve
// centred residues, limb split, packed e4m3 plane stores (every limb is an
// e4m3-exact integer, Lemma 1, so the conversion is exact).
//
// Each thread owns one vector (row of A / column of B) and 16 consecutive k,
// so every plane store is one 16-byte write.  Bound by VALU work (about 300
// instructions per element) with HBM close behind: 8 bytes read and 30 bytes
// written per element.
//  - A (side 0): a wavefront covers 1 row x 1024 k, so each plane store of the
//    wavefront is 1 KiB contiguous.
//  - B (side 1): a wavefront covers 8 columns x 128 k, so each plane store of
//    the wavefront fills eight whole 128-byte lines; every FP64 load reads 64
//    contiguous bytes of 8 rows of B.
#include <utility>

#include "device_math.hpp"
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

constexpr int kElems = 16;  // k values per thread

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
  *reinterpret_cast<uint4*>(p) = w;
}

// Centred residue of the integer-valued y modulo M, in [-(M/2), (M-1)/2],
// as a float (exact: |residue| <= 544).  EXACT (|y| <= 2^50): the FP64
// quotient y * RN(1/M) is within |y| 2^-52 / M <= 1/(4M) of y / M, while for
// odd M y / M is at least 1/(2M) away from a half integer, so rint gives the
// nearest quotient and y - qM is already centred; for M = 1024 the quotient
// is exact and only the tie +512 needs mapping to -512.  Otherwise the
// general form with its two corrections.
template <int M, bool EXACT>
__device__ __forceinline__ float centred_residue(double y) {
  if constexpr (!EXACT) {
    return (float)cmod_f64<M>(y);
  } else {
    constexpr double inv = 1.0 / M;
    const double q = __builtin_rint(y * inv);
    // y - q M in one three-operand FMA (the two-operand form would first copy
    // y, which every modulus reuses)
    double t;
    asm("v_fma_f64 %0, %1, %2, %3" : "=v"(t) : "v"(q), "s"(-(double)M), "v"(y));
    const float r = (float)t;
    if constexpr ((M & 1) == 0)
      return r == (float)(M / 2) ? -(float)(M / 2) : r;
    else
      return r;
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

template <int I, bool EXACT>
__device__ __forceinline__ void emit_modulus(const double (&y)[kElems], int8_t* planes,
                                             int64_t plane_stride, int64_t off) {
  constexpr int M = kModulus[I];
  constexpr int S = root_of(I);
  constexpr int Q = plane_base(I);
  int8_t* base = planes + (int64_t)Q * plane_stride + off;
  float l0[kElems], l1[kElems], l2[kElems];
#pragma unroll
  for (int c = 0; c < kElems; ++c) {
    const float d = centred_residue<M, EXACT>(y[c]);
    if constexpr (S != 0)
      split_square<S>(d, l0[c], l1[c]);
    else
      split_16(d, l0[c], l1[c], l2[c]);
  }
  store16(base, l0);
  store16(base + plane_stride, l1);
  if constexpr (S == 0) store16(base + 2 * plane_stride, l2);
}

template <bool EXACT, int... I>
__device__ __forceinline__ void emit_all(std::integer_sequence<int, I...>, const double (&y)[kElems],
                                         int8_t* planes, int64_t plane_stride, int64_t off) {
  (emit_modulus<I, EXACT>(y, planes, plane_stride, off), ...);
}

template <int SIDE, bool EXACT>
__global__ __launch_bounds__(256) void deconstruct_kernel(int64_t vecs, int64_t k, int64_t kp,
                                                          const double* __restrict__ X, int64_t ldx,
                                                          const int32_t* __restrict__ exps,
                                                          int8_t* __restrict__ planes) {
  const int64_t ngroups = kp / kElems;
  int64_t v, g;
  if constexpr (SIDE == 0) {  // block: 4 rows x 64 groups, a wavefront per row
    const int64_t gb = (ngroups + 63) / 64;
    v = (int64_t)(blockIdx.x / gb) * 4 + (threadIdx.x >> 6);
    g = (int64_t)(blockIdx.x % gb) * 64 + (threadIdx.x & 63);
  } else {  // block: 32 columns x 8 groups, a wavefront per 8 columns
    const int64_t gb = (ngroups + 7) / 8;
    const int lane = threadIdx.x & 63;
    v = (int64_t)(blockIdx.x / gb) * 32 + (threadIdx.x >> 6) * 8 + (lane & 7);
    g = (int64_t)(blockIdx.x % gb) * 8 + (lane >> 3);
  }
  if (v >= vecs || g >= ngroups) return;
  int sigma = exps[v];
  const bool finite = sigma != INT32_MIN;
  sigma = finite ? sigma : 0;
  const int64_t k0 = g * kElems;
  double y[kElems];
#pragma unroll
  for (int c = 0; c < kElems; ++c) {
    const int64_t l = k0 + c;
    double x = 0.0;
    if (finite && l < k) x = SIDE == 0 ? X[v * ldx + l] : X[l * ldx + v];
    // |x 2^sigma| < 2^t: the scaling is exact, rint is the one rounding.
    y[c] = __builtin_rint(__builtin_ldexp(x, sigma));
  }
  emit_all<EXACT>(std::make_integer_sequence<int, kR>{}, y, planes, vecs * kp, v * kp + k0);
}

template <int SIDE>
void launch_side(int64_t blocks, bool exact, int64_t vecs, int64_t k, int64_t kp, const double* X,
                 int64_t ldx, const int32_t* exps, int8_t* planes, hipStream_t stream) {
  if (exact)
    hipLaunchKernelGGL((deconstruct_kernel<SIDE, true>), dim3((unsigned)blocks), dim3(256), 0, stream,
                       vecs, k, kp, X, ldx, exps, planes);
  else
    hipLaunchKernelGGL((deconstruct_kernel<SIDE, false>), dim3((unsigned)blocks), dim3(256), 0,
                       stream, vecs, k, kp, X, ldx, exps, planes);
}

}  // namespace

hipError_t launch_deconstruct(int side, int64_t vecs, int64_t k, int64_t kp, int t, const double* X,
                              int64_t ldx, const int32_t* exps, int8_t* planes,
                              hipStream_t stream) {
  if (vecs <= 0 || kp <= 0) return hipSuccess;
  const int64_t ngroups = kp / kElems;
  const bool exact = t <= 50;  // |y| <= 2^t: the quotient needs no correction
  if (side == 0) {
    const int64_t blocks = ((vecs + 3) / 4) * ((ngroups + 63) / 64);
    launch_side<0>(blocks, exact, vecs, k, kp, X, ldx, exps, planes, stream);
  } else {
    const int64_t blocks = ((vecs + 31) / 32) * ((ngroups + 7) / 8);
    launch_side<1>(blocks, exact, vecs, k, kp, X, ldx, exps, planes, stream);
  }
  return hipGetLastError();
}

}  // namespace oz
