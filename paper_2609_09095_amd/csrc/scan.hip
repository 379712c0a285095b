// Exponent scan (the once-per-call setup of Alg. 1; Eq. (scale)): for every
// row of A / column of B the frexp exponent e of its largest magnitude, and
// sigma = t - e.  HBM-bound: one FP64 read per element.  The reduction key
// is in exponent_key.hpp.
#include "exponent_key.hpp"
#include "kernels.hpp"

namespace oz {
namespace {

// One block of four wavefronts per row of A; rows are contiguous, so loads
// coalesce, and short matrices (few rows, long k) still spread over the
// chip.  Each lane reads 16-byte pairs, eight independent loads in flight
// (a 64 KiB row is one unrolled sweep), from the row's first 16-byte
// boundary; the element before it (a row starting at an odd double) and
// the odd tail are read singly.  The waves' maxima meet in LDS.
//
// zero / nzero: the column keys of B to clear on the side (the first blocks
// write one zero per thread), so that B's column scan needs no launch of
// its own for that.
__global__ __launch_bounds__(256) void scan_rows_kernel(int64_t vecs, int64_t k, const double* X,
                                                        int64_t ldx, int t, int32_t* exps,
                                                        int32_t* zero, int64_t nzero) {
  __shared__ uint32_t part[4];
  if (zero) {
    const int64_t z = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (z < nzero) zero[z] = 0;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t v = blockIdx.x;
  const uint64_t* row = reinterpret_cast<const uint64_t*>(X + v * ldx);
  const int64_t head = ((uintptr_t)row & 15) ? 1 : 0;  // elements before the 16-byte boundary
  const int64_t pairs = (k - head) / 2;
  const ulonglong2* body = reinterpret_cast<const ulonglong2*>(row + head);
  uint64_t mx[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  int64_t p = threadIdx.x;
  for (; p + 7 * 256 < pairs; p += 8 * 256) {
    ulonglong2 q[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) q[u] = body[p + u * 256];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint64_t a = q[u].x & kAbsMask, b = q[u].y & kAbsMask;
      mx[u] = a > mx[u] ? a : mx[u];
      mx[u] = b > mx[u] ? b : mx[u];
    }
  }
  for (; p < pairs; p += 256) {
    const ulonglong2 q = body[p];
    const uint64_t a = q.x & kAbsMask, b = q.y & kAbsMask;
    mx[0] = a > mx[0] ? a : mx[0];
    mx[1] = b > mx[1] ? b : mx[1];
  }
  if (threadIdx.x == 0 && head) {
    const uint64_t a = row[0] & kAbsMask;
    mx[2] = a > mx[2] ? a : mx[2];
  }
  if (threadIdx.x == 1 && head + 2 * pairs < k) {
    const uint64_t a = row[k - 1] & kAbsMask;
    mx[3] = a > mx[3] ? a : mx[3];
  }
#pragma unroll
  for (int u = 1; u < 8; ++u) mx[0] = mx[u] > mx[0] ? mx[u] : mx[0];
  const uint32_t key = wave_max(exponent_key(mx[0]));
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

hipError_t launch_scan_rows(int64_t vecs, int64_t k, const double* X, int64_t ldx, int t, int32_t* exps,
                            int32_t* zero, int64_t nzero, hipStream_t stream) {
  if (vecs <= 0) return hipSuccess;
  // one block per row; the blocks also cover the keys to clear
  const int64_t zb = zero ? (nzero + 255) / 256 : 0;
  if (vecs > (int64_t)UINT32_MAX || zb > vecs) return hipErrorInvalidValue;
  hipLaunchKernelGGL(scan_rows_kernel, dim3((unsigned)vecs), dim3(256), 0, stream, vecs, k, X, ldx, t,
                     exps, zero, nzero);
  return hipGetLastError();
}

hipError_t launch_clear_keys(int64_t vecs, int32_t* keys, hipStream_t stream) {
  if (vecs <= 0) return hipSuccess;
  hipLaunchKernelGGL(clear_keys_kernel, dim3((unsigned)((vecs + 255) / 256)), dim3(256), 0, stream, vecs,
                     keys);
  return hipGetLastError();
}

hipError_t launch_scan_cols(int64_t vecs, int64_t k, const double* X, int64_t ldx, int32_t* keys,
                            hipStream_t stream) {
  if (vecs <= 0) return hipSuccess;
  // k blocks of 256 rows, or of 64 when that leaves fewer than 1024 blocks
  const int64_t strips = (vecs + 63) / 64;
  const int64_t rows_per_block = strips * ((k + 255) / 256) < 1024 ? 64 : 256;
  const int64_t kblocks = (k + rows_per_block - 1) / rows_per_block;
  if (kblocks > 0)
    hipLaunchKernelGGL(scan_cols_kernel, dim3((unsigned)(strips * kblocks)), dim3(256), 0, stream,
                       vecs, k, X, ldx, rows_per_block, keys);
  return hipGetLastError();
}

hipError_t launch_keys_to_sigma(int64_t vecs, int t, int32_t* exps, hipStream_t stream) {
  if (vecs <= 0) return hipSuccess;
  hipLaunchKernelGGL(keys_to_sigma_kernel, dim3((unsigned)((vecs + 255) / 256)), dim3(256), 0, stream,
                     vecs, t, exps);
  return hipGetLastError();
}

}  // namespace oz
