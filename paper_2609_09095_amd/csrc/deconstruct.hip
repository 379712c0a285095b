// Deconstruction (Alg. 2): scale by 2^sigma, round to nearest even, twelve
// centred residues, limb split, packed e4m3 plane stores (every limb is an
// e4m3-exact integer, Lemma 1, so the conversion is exact).
//
// Each thread owns one vector (row of A / column of B) and 16 consecutive k,
// so every plane store is one 16-byte write.  HBM-bound: 8 bytes read and 30
// bytes written per element.
//  - A (side 0): a wavefront covers 1 row x 1024 k, so each plane store of the
//    wavefront is 1 KiB contiguous.
//  - B (side 1): a wavefront covers 32 columns x 32 k; every FP64 load of the
//    wavefront reads 256 contiguous bytes of two rows of B; a block writes 128
//    contiguous plane bytes per column.
#include <utility>

#include "device_math.hpp"
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

constexpr int kElems = 16;  // k values per thread

// four limbs as e4m3 bytes (OCP E4M3FN), the first in the low byte
__device__ __forceinline__ uint32_t pack4(int a, int b, int c, int d) {
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32((float)a, (float)b, 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32((float)c, (float)d, lo, true);
}

__device__ __forceinline__ void store16(int8_t* p, const int (&b)[kElems]) {
  uint4 w;
  w.x = pack4(b[0], b[1], b[2], b[3]);
  w.y = pack4(b[4], b[5], b[6], b[7]);
  w.z = pack4(b[8], b[9], b[10], b[11]);
  w.w = pack4(b[12], b[13], b[14], b[15]);
  *reinterpret_cast<uint4*>(p) = w;
}

// Square modulus s^2 (Eq. (pieces) with base s): d0 = centred d mod s (the
// balanced digit, [-16, 15] for s = 32), d1 = (d - d0) / s.
template <int S>
__device__ __forceinline__ void split_square(int d, int& d0, int& d1) {
  if constexpr (S == 32) {
    d0 = ((d + 16) & 31) - 16;
    d1 = (d - d0) >> 5;
  } else {
    // |d| <= 544 and s odd: d / s is never within 1/(2s) of a half integer,
    // far above the FP32 error of d * (1/s), so rint gives the nearest digit.
    constexpr float inv = 1.0f / S;
    d1 = (int)__builtin_rintf((float)d * inv);
    d0 = d - S * d1;
  }
}

// Nonsquare modulus (Lemma 1): canonical balanced base-16 split, then one
// carry when d0 + d1 is odd with |d0 + d1| >= 17 -- exactly the sums
// +-17, +-19, +-21, +-23 that e4m3 cannot hold.  d0 != 0 whenever it fires.
__device__ __forceinline__ void split_16(int d, int& d0, int& d1) {
  d0 = ((d + 8) & 15) - 8;
  d1 = (d - d0) >> 4;
  const int s = d0 + d1;
  const bool carry = (s & 1) && ((unsigned)(s + 16) > 32u);
  const int sg = d0 > 0 ? 1 : -1;
  d0 = carry ? d0 - 16 * sg : d0;
  d1 = carry ? d1 + sg : d1;
}

template <int I>
__device__ __forceinline__ void emit_modulus(const double (&y)[kElems], int8_t* planes,
                                             int64_t plane_stride, int64_t off) {
  constexpr int M = kModulus[I];
  constexpr int S = root_of(I);
  constexpr int Q = plane_base(I);
  int8_t* base = planes + (int64_t)Q * plane_stride + off;
  int l0[kElems], l1[kElems];
#pragma unroll
  for (int c = 0; c < kElems; ++c) {
    const int d = cmod_f64<M>(y[c]);
    if constexpr (S != 0)
      split_square<S>(d, l0[c], l1[c]);
    else
      split_16(d, l0[c], l1[c]);
  }
  store16(base, l0);
  store16(base + plane_stride, l1);
  if constexpr (S == 0) {
    int l2[kElems];
#pragma unroll
    for (int c = 0; c < kElems; ++c) l2[c] = l0[c] + l1[c];
    store16(base + 2 * plane_stride, l2);
  }
}

template <int... I>
__device__ __forceinline__ void emit_all(std::integer_sequence<int, I...>, const double (&y)[kElems],
                                         int8_t* planes, int64_t plane_stride, int64_t off) {
  (emit_modulus<I>(y, planes, plane_stride, off), ...);
}

template <int SIDE>
__global__ __launch_bounds__(256) void deconstruct_kernel(int64_t vecs, int64_t k, int64_t kp,
                                                          const double* __restrict__ X, int64_t ldx,
                                                          const int32_t* __restrict__ exps,
                                                          int8_t* __restrict__ planes) {
  const int64_t ngroups = kp / kElems;
  int64_t v, g;
  if constexpr (SIDE == 0) {  // block: 4 rows x 64 groups
    const int64_t gb = (ngroups + 63) / 64;
    v = (int64_t)(blockIdx.x / gb) * 4 + (threadIdx.x >> 6);
    g = (int64_t)(blockIdx.x % gb) * 64 + (threadIdx.x & 63);
  } else {  // block: 32 columns x 8 groups
    const int64_t gb = (ngroups + 7) / 8;
    v = (int64_t)(blockIdx.x / gb) * 32 + (threadIdx.x & 31);
    g = (int64_t)(blockIdx.x % gb) * 8 + (threadIdx.x >> 5);
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
  emit_all(std::make_integer_sequence<int, kR>{}, y, planes, vecs * kp, v * kp + k0);
}

}  // namespace

hipError_t launch_deconstruct(int side, int64_t vecs, int64_t k, int64_t kp, const double* X,
                              int64_t ldx, const int32_t* exps, int8_t* planes,
                              hipStream_t stream) {
  if (vecs <= 0 || kp <= 0) return hipSuccess;
  const int64_t ngroups = kp / kElems;
  if (side == 0) {
    const int64_t blocks = ((vecs + 3) / 4) * ((ngroups + 63) / 64);
    hipLaunchKernelGGL(deconstruct_kernel<0>, dim3((unsigned)blocks), dim3(256), 0, stream, vecs, k,
                       kp, X, ldx, exps, planes);
  } else {
    const int64_t blocks = ((vecs + 31) / 32) * ((ngroups + 7) / 8);
    hipLaunchKernelGGL(deconstruct_kernel<1>, dim3((unsigned)blocks), dim3(256), 0, stream, vecs, k,
                       kp, X, ldx, exps, planes);
  }
  return hipGetLastError();
}

}  // namespace oz
