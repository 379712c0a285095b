// Exponent scan (the once-per-call setup of Alg. 1; Eq. (scale)): for every
// row of A / column of B the frexp exponent e of its largest magnitude, and
// sigma = t - e.  HBM-bound: one FP64 read per element.
//
// The reduction runs on the magnitude's bit pattern (|x| as uint64 is
// monotone in |x|, NaN and infinity sort above every finite value), then on
// a 32-bit order-preserving key: 0 for zero, e + 2048 for finite nonzero
// values, all ones for non-finite.
#include "kernels.hpp"

namespace oz {
namespace {

constexpr uint32_t kKeyNonfinite = 0xFFFFFFFFu;
constexpr uint64_t kAbsMask = 0x7FFFFFFFFFFFFFFFull;

__device__ __forceinline__ uint32_t exponent_key(uint64_t absbits) {
  if (absbits >= 0x7FF0000000000000ull) return kKeyNonfinite;
  if (absbits == 0) return 0;
  const int biased = (int)(absbits >> 52);
  // normal: |x| in [2^(b-1023), 2^(b-1022)); subnormal: mantissa bit p set,
  // |x| in [2^(p-1074), 2^(p-1073)).
  const int e = biased ? biased - 1022 : (63 - __builtin_clzll(absbits)) - 1073;
  return (uint32_t)(e + 2048);
}

__device__ __forceinline__ int32_t key_to_sigma(uint32_t key, int t) {
  if (key == kKeyNonfinite) return INT32_MIN;
  if (key == 0) return t;  // frexp(0) has exponent 0
  return t - ((int)key - 2048);
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = (uint32_t)__shfl_xor((int)v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}

// One block of four wavefronts per row of A; rows are contiguous, so loads
// coalesce, and short matrices (few rows, long k) still spread over the
// chip.  The waves' maxima meet in LDS.
__global__ __launch_bounds__(256) void scan_rows_kernel(int64_t vecs, int64_t k, const double* X,
                                                        int64_t ldx, int t, int32_t* exps) {
  __shared__ uint32_t part[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t v = blockIdx.x;
  const uint64_t* row = reinterpret_cast<const uint64_t*>(X + v * ldx);
  uint64_t mx0 = 0, mx1 = 0;
  int64_t l = threadIdx.x;
  for (; l + 256 < k; l += 512) {
    const uint64_t a = row[l] & kAbsMask, b = row[l + 256] & kAbsMask;
    mx0 = a > mx0 ? a : mx0;
    mx1 = b > mx1 ? b : mx1;
  }
  if (l < k) {
    const uint64_t a = row[l] & kAbsMask;
    mx0 = a > mx0 ? a : mx0;
  }
  const uint32_t key = wave_max(exponent_key(mx0 > mx1 ? mx0 : mx1));
  if (lane == 0) part[wave] = key;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t m = part[0];
    for (int w = 1; w < 4; ++w) m = part[w] > m ? part[w] : m;
    exps[v] = key_to_sigma(m, t);
  }
}

__global__ __launch_bounds__(256) void clear_keys_kernel(int64_t vecs, int32_t* keys) {
  const int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (v < vecs) keys[v] = 0;
}

// Columns of B: 64 columns per block along the lanes (coalesced row
// segments), the k range of the block split over its 4 waves, and the
// blocks of one column strip combined with an atomic max on the key.
__global__ __launch_bounds__(256) void scan_cols_kernel(int64_t vecs, int64_t k, const double* X,
                                                        int64_t ldx, int64_t rows_per_block,
                                                        int32_t* keys) {
  __shared__ uint32_t part[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t strips = (vecs + 63) / 64;
  const int64_t strip = blockIdx.x % strips, kb = blockIdx.x / strips;
  const int64_t v = strip * 64 + lane;
  const int64_t l0 = kb * rows_per_block;
  const int64_t l1 = l0 + rows_per_block < k ? l0 + rows_per_block : k;
  uint64_t mx = 0;
  if (v < vecs) {
    for (int64_t l = l0 + wave; l < l1; l += 4) {
      const uint64_t a = reinterpret_cast<const uint64_t*>(X + l * ldx)[v] & kAbsMask;
      mx = a > mx ? a : mx;
    }
  }
  part[wave][lane] = exponent_key(mx);
  __syncthreads();
  if (wave == 0 && v < vecs) {
    uint32_t key = part[0][lane];
    for (int w = 1; w < 4; ++w) key = part[w][lane] > key ? part[w][lane] : key;
    if (key) atomicMax(reinterpret_cast<unsigned int*>(keys) + v, key);
  }
}

__global__ __launch_bounds__(256) void keys_to_sigma_kernel(int64_t vecs, int t, int32_t* exps) {
  const int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (v < vecs) exps[v] = key_to_sigma((uint32_t)exps[v], t);
}

}  // namespace

hipError_t launch_scan(int side, int64_t vecs, int64_t k, const double* X, int64_t ldx, int t,
                       int32_t* exps, hipStream_t stream) {
  if (vecs <= 0) return hipSuccess;
  if (side == 0) {
    if (vecs > (int64_t)UINT32_MAX) return hipErrorInvalidValue;  // one block per row
    hipLaunchKernelGGL(scan_rows_kernel, dim3((unsigned)vecs), dim3(256), 0, stream, vecs, k, X, ldx,
                       t, exps);
    return hipGetLastError();
  }
  const unsigned vb = (unsigned)((vecs + 255) / 256);
  hipLaunchKernelGGL(clear_keys_kernel, dim3(vb), dim3(256), 0, stream, vecs, exps);
  // k blocks of 256 rows, or of 64 when that leaves fewer than 1024 blocks
  const int64_t strips = (vecs + 63) / 64;
  const int64_t rows_per_block = strips * ((k + 255) / 256) < 1024 ? 64 : 256;
  const int64_t kblocks = (k + rows_per_block - 1) / rows_per_block;
  if (kblocks > 0)
    hipLaunchKernelGGL(scan_cols_kernel, dim3((unsigned)(strips * kblocks)), dim3(256), 0, stream,
                       vecs, k, X, ldx, rows_per_block, exps);
  hipLaunchKernelGGL(keys_to_sigma_kernel, dim3(vb), dim3(256), 0, stream, vecs, t, exps);
  return hipGetLastError();
}

}  // namespace oz
