// Per-modulus residue products (Eq. (residueprod)) on gfx950 int8 MFMA.
//
// For modulus i and an output tile, the three limb products of the modulus
// (square: d0e0, d0e1, d1e0 with weights {1, s, s}; nonsquare, Eq.
// (karcarry): d0e0, d1e1, (d0+d1)(e0+e1) with weights {-15, 240, 16}) run one
// after another through the same int32 MFMA accumulators.  After each product
// its accumulator is reduced modulo m_i and folded into a running centred
// residue with the product's weight, so the accumulators only ever hold one
// plain int8 dot product: |sum| <= 22^2 k < 2^31 for k <= 4 194 304.
//
// Both plane operands are K-contiguous (A rows, B columns), the layout the
// int8 MFMA wants for both sides.  v_mfma_i32_32x32x32_i8 takes 16 bytes per
// lane for each operand; the A and B register layouts mirror each other, so
// loading both with lane = row/column + 32 * (16-byte K half) pairs the same
// k on both sides whatever the hardware's internal k order.
#include <utility>

#include "device_math.hpp"
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128;         // output rows per block
constexpr int BN = 128;         // output columns per block
constexpr int BK = 64;          // k bytes per LDS stage
constexpr int kLdsStride = 80;  // bytes per LDS row: 64 + 16 pad, conflict-free b128 reads
constexpr int kStage = BM * kLdsStride;

// One limb product P of modulus I over the whole k range, for the block's
// 128 x 128 tile, folded into the running centred residues `comb`.
template <int I, int P>
__device__ __forceinline__ void product_pass(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                             const int8_t* pb, int64_t arow, int64_t brow,
                                             int8_t* lds, int (&comb)[2][2][16]) {
  constexpr int M = kModulus[I];
  constexpr int coef = product_coef(I, P);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  const int lhalf = tid & 1;
  const int lds_w = (tid >> 1) * kLdsStride + lhalf * 32;
  const int lds_ra = (wr * 64 + (lane & 31)) * kLdsStride + (lane >> 5) * 16;
  const int lds_rb = (wc * 64 + (lane & 31)) * kLdsStride + (lane >> 5) * 16;
  const int8_t* A = pa + ((int64_t)(plane_base(I) + product_plane_a(I, P)) * m + arow) * kp + lhalf * 32;
  const int8_t* B = pb + ((int64_t)(plane_base(I) + product_plane_b(I, P)) * n + brow) * kp + lhalf * 32;

  v16i acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = v16i{};

  v4i ra0 = *reinterpret_cast<const v4i*>(A), ra1 = *reinterpret_cast<const v4i*>(A + 16);
  v4i rb0 = *reinterpret_cast<const v4i*>(B), rb1 = *reinterpret_cast<const v4i*>(B + 16);
  *reinterpret_cast<v4i*>(lds + lds_w) = ra0;
  *reinterpret_cast<v4i*>(lds + lds_w + 16) = ra1;
  *reinterpret_cast<v4i*>(lds + 2 * kStage + lds_w) = rb0;
  *reinterpret_cast<v4i*>(lds + 2 * kStage + lds_w + 16) = rb1;
  __syncthreads();

  for (int64_t kk = 0; kk < kp; kk += BK) {
    const int cur = (int)((kk / BK) & 1);
    const bool next = kk + BK < kp;
    if (next) {
      ra0 = *reinterpret_cast<const v4i*>(A + kk + BK);
      ra1 = *reinterpret_cast<const v4i*>(A + kk + BK + 16);
      rb0 = *reinterpret_cast<const v4i*>(B + kk + BK);
      rb1 = *reinterpret_cast<const v4i*>(B + kk + BK + 16);
    }
    const int8_t* la = lds + cur * kStage;
    const int8_t* lb = lds + (2 + cur) * kStage;
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
      v4i af[2], bf[2];
#pragma unroll
      for (int a = 0; a < 2; ++a)
        af[a] = *reinterpret_cast<const v4i*>(la + lds_ra + a * 32 * kLdsStride + ks);
#pragma unroll
      for (int b = 0; b < 2; ++b)
        bf[b] = *reinterpret_cast<const v4i*>(lb + lds_rb + b * 32 * kLdsStride + ks);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[a], bf[b], acc[a][b], 0, 0, 0);
    }
    if (next) {
      int8_t* wa = lds + (cur ^ 1) * kStage + lds_w;
      int8_t* wb = lds + (2 + (cur ^ 1)) * kStage + lds_w;
      *reinterpret_cast<v4i*>(wa) = ra0;
      *reinterpret_cast<v4i*>(wa + 16) = ra1;
      *reinterpret_cast<v4i*>(wb) = rb0;
      *reinterpret_cast<v4i*>(wb + 16) = rb1;
    }
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = cmod_f64<M>((double)acc[a][b][v]);
        comb[a][b][v] = cmod_f64<M>((double)(comb[a][b][v] + coef * r));
      }
}

template <int I, typename OT>
__device__ __forceinline__ void residue_tile(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                             const int8_t* pb, OT* cres, int64_t tm, int64_t tn,
                                             int8_t* lds) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  // loader rows (clamped: rows past the edge load row m-1 / n-1, never stored)
  const int lrow = tid >> 1;
  const int64_t arow = tm * BM + lrow < m ? tm * BM + lrow : m - 1;
  const int64_t brow = tn * BN + lrow < n ? tn * BN + lrow : n - 1;

  int comb[2][2][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) comb[a][b][v] = 0;

  // k == 0: every product is empty and the residues stay zero.
  if (kp > 0) {
    product_pass<I, 0>(m, n, kp, pa, pb, arow, brow, lds, comb);
    product_pass<I, 1>(m, n, kp, pa, pb, arow, brow, lds, comb);
    product_pass<I, 2>(m, n, kp, pa, pb, arow, brow, lds, comb);
  }

  // 32x32 MFMA result layout: lane holds column lane%32 and rows
  // 8*(v/4) + 4*(lane/32) + v%4 of its 32x32 block.
  OT* out = cres + (int64_t)I * m * n;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int64_t col = tn * BN + wc * 64 + b * 32 + (lane & 31);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t row = tm * BM + wr * 64 + a * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        if (row < m && col < n) out[row * n + col] = (OT)comb[a][b][v];
      }
    }
}

template <typename OT, int... I>
__device__ __forceinline__ void dispatch_modulus(std::integer_sequence<int, I...>, int mod, int64_t m,
                                                 int64_t n, int64_t kp, const int8_t* pa,
                                                 const int8_t* pb, OT* cres, int64_t tm, int64_t tn,
                                                 int8_t* lds) {
  ((mod == I ? residue_tile<I, OT>(m, n, kp, pa, pb, cres, tm, tn, lds) : void()), ...);
}

template <typename OT>
__global__ __launch_bounds__(256) void residue_gemm_kernel(int64_t m, int64_t n, int64_t kp,
                                                           const int8_t* __restrict__ pa,
                                                           const int8_t* __restrict__ pb,
                                                           OT* __restrict__ cres) {
  __shared__ __attribute__((aligned(16))) int8_t lds[4 * kStage];
  const int64_t tiles_m = (m + BM - 1) / BM, tiles_n = (n + BN - 1) / BN;
  const int64_t per_mod = tiles_m * tiles_n;
  const int mod = (int)(blockIdx.x / per_mod);
  const int64_t t = blockIdx.x % per_mod;
  const int64_t tm = t / tiles_n, tn = t % tiles_n;
  dispatch_modulus<OT>(std::make_integer_sequence<int, kR>{}, mod, m, n, kp, pa, pb, cres, tm, tn,
                       lds);
}

template <typename OT>
hipError_t launch_gemm(int64_t m, int64_t n, int64_t kp, const int8_t* pa, const int8_t* pb,
                       OT* cres, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  const int64_t blocks = (int64_t)kR * ((m + BM - 1) / BM) * ((n + BN - 1) / BN);
  hipLaunchKernelGGL(residue_gemm_kernel<OT>, dim3((unsigned)blocks), dim3(256), 0, stream, m, n, kp,
                     pa, pb, cres);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_residue_gemm_i32(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                   const int8_t* pb, int32_t* cres, hipStream_t stream) {
  return launch_gemm<int32_t>(m, n, kp, pa, pb, cres, stream);
}

hipError_t launch_residue_gemm_i16(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                   const int8_t* pb, int16_t* cres, hipStream_t stream) {
  return launch_gemm<int16_t>(m, n, kp, pa, pb, cres, stream);
}

}  // namespace oz
