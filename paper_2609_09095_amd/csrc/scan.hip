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
//
// The magnitude digit ceil(16 |x| 2^-e) of x (its bits) given sh = 4 - e:
// exact in FP64 unless the scaled value falls below the normal range, where
// the ceiling is 1.
__device__ __forceinline__ int magnitude_digit(uint64_t bits, int sh) {
  const double a = __builtin_bit_cast(double, bits & kAbsMask);
  const double u = __builtin_ceil(__builtin_ldexp(a, sh));
  return a == 0.0 ? 0 : (u < 1.0 ? 1 : (int)u);
}

// The accurate mode's row scan for a 16-byte aligned row of at most 512 R
// elements: lane l of wavefront w holds pairs l + 64 w + 256 u (u < R) in
// registers, so the digits need no second read.  They are gathered in LDS
// (zero past k) and leave as 16-byte stores, eight to a 128-byte chunk of
// the plane.  R = 8 (rows up to 4096) keeps the registers, and so the
// occupancy, of the plain scan; R = 16 takes rows up to 8192.
constexpr int kResidentK = 8192;

template <int R>
__device__ __forceinline__ void resident_digits(int64_t vecs, int64_t k, int64_t kp, const uint64_t* row,
                                                const ulonglong2* body, int64_t pairs, int t, int32_t* exps,
                                                int8_t* digits, uint32_t* part) {
  __shared__ __attribute__((aligned(16))) uint8_t dl[kResidentK];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t v = blockIdx.x;
  ulonglong2 q[R];
  uint64_t mx = 0;
#pragma unroll
  for (int u = 0; u < R; ++u) {
    const int64_t p = threadIdx.x + u * 256;
    q[u] = p < pairs ? body[p] : ulonglong2{0, 0};
  }
#pragma unroll
  for (int u = 0; u < R; ++u) {
    const uint64_t a = q[u].x & kAbsMask, b = q[u].y & kAbsMask;
    mx = a > mx ? a : mx;
    mx = b > mx ? b : mx;
  }
  const bool tail = 2 * pairs < k;  // odd k: the last element stands alone
  const uint64_t last = (threadIdx.x == 1 && tail) ? row[k - 1] : 0;
  mx = (last & kAbsMask) > mx ? (last & kAbsMask) : mx;
  const uint32_t key = wave_max(exponent_key(mx));
  if (lane == 0) part[wave] = key;
  __syncthreads();
  uint32_t m = part[0];
  for (int w = 1; w < 4; ++w) m = part[w] > m ? part[w] : m;
  if (threadIdx.x == 0) exps[v] = key_to_sigma(m, t);
  const int32_t ne = key_to_sigma(m, 0);  // -e, or INT32_MIN
  const bool live = ne != INT32_MIN;
  const int sh = live ? 4 + ne : 0;
#pragma unroll
  for (int u = 0; u < R; ++u) {
    const int p = threadIdx.x + u * 256;
    if (p < pairs) {
      const int d0 = live ? magnitude_digit(q[u].x, sh) : 0;
      const int d1 = live ? magnitude_digit(q[u].y, sh) : 0;
      *reinterpret_cast<uint16_t*>(dl + 2 * p) = (uint16_t)(d0 | (d1 << 8));
    }
  }
  if (threadIdx.x == 1 && tail) dl[k - 1] = (uint8_t)(live ? magnitude_digit(last, sh) : 0);
  for (int l = (int)k + threadIdx.x; l < (int)kp; l += 256) dl[l] = 0;
  __syncthreads();
  // piece c of 16 bytes: chunk c / 8 of the row, its (c % 8)-th 16 bytes
  for (int c = threadIdx.x; c < (int)kp / 16; c += 256)
    *reinterpret_cast<uint4*>(digits + ((int64_t)(c >> 3) * vecs + v) * 128 + (c & 7) * 16) =
        *reinterpret_cast<const uint4*>(dl + 16 * c);
}

// DIGITS (the accurate mode, Sec. 2, Eq. (alpha)): once the row's exponent
// e is known, the block reads its row a second time -- from cache: it has
// just streamed it -- and writes the magnitude digits ceil(16 |x| 2^-e) in
// {0..16} (0 past k and on a non-finite row) as one int8 plane of the plane
// layout [kp/128][vecs][128]: each wavefront takes 128-element chunks, a
// lane two elements 64 apart, so loads and byte stores stay contiguous
// across the wavefront.
// DIG: 0 no digits; 1 digits by a second read of the row; 8 or 16 digits
// from registers (resident_digits<DIG>, chosen by the host for 16-byte
// aligned rows of at most 512 DIG elements; any other row falls back to the
// second read).
template <int DIG>
__global__ __launch_bounds__(256) void scan_rows_kernel(int64_t vecs, int64_t k, const double* X,
                                                        int64_t ldx, int t, int32_t* exps,
                                                        int32_t* zero, int64_t nzero, int64_t kp,
                                                        int8_t* digits) {
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
  if constexpr (DIG >= 8) {
    if (head == 0 && kp <= 512 * DIG) {
      resident_digits<DIG>(vecs, k, kp, row, body, pairs, t, exps, digits, part);
      return;
    }
  }
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
  uint32_t m = part[0];
  for (int w = 1; w < 4; ++w) m = part[w] > m ? part[w] : m;
  if (threadIdx.x == 0) exps[v] = key_to_sigma(m, t);
  if constexpr (DIG != 0) {
    const int32_t ne = key_to_sigma(m, 0);  // -e, or INT32_MIN
    const bool live = ne != INT32_MIN;
    const int sh = live ? 4 + ne : 0;
    const double* xr = X + v * ldx;
    const int64_t chunks = kp / 128;
    int8_t* drow = digits + v * 128 + lane;
    auto digit = [&](int64_t l) -> int {
      const uint64_t bits = (live && l < k) ? reinterpret_cast<const uint64_t*>(xr)[l < k ? l : 0] : 0;
      return magnitude_digit(bits, sh);
    };
    for (int64_t c = wave; c < chunks; c += 4) {
      const int64_t l0 = c * 128 + lane;
      const int d0 = digit(l0), d1 = digit(l0 + 64);
      int8_t* dst = drow + c * vecs * 128;
      dst[0] = (int8_t)d0;
      dst[64] = (int8_t)d1;
    }
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
                            int32_t* zero, int64_t nzero, hipStream_t stream, int8_t* digits, int64_t kp) {
  if (vecs <= 0) return hipSuccess;
  // one block per row; the blocks also cover the keys to clear
  const int64_t zb = zero ? (nzero + 255) / 256 : 0;
  if (vecs > (int64_t)UINT32_MAX || zb > vecs) return hipErrorInvalidValue;
  if (digits) {
    if (kp < k || kp % 128) return hipErrorInvalidValue;
    // every row 16-byte aligned: the digits from registers
    const bool aligned = ((uintptr_t)X & 15) == 0 && (ldx & 1) == 0;
    if (aligned && kp <= kResidentK / 2)
      hipLaunchKernelGGL(scan_rows_kernel<8>, dim3((unsigned)vecs), dim3(256), 0, stream, vecs, k, X, ldx, t,
                         exps, zero, nzero, kp, digits);
    else if (aligned && kp <= kResidentK)
      hipLaunchKernelGGL(scan_rows_kernel<16>, dim3((unsigned)vecs), dim3(256), 0, stream, vecs, k, X, ldx, t,
                         exps, zero, nzero, kp, digits);
    else
      hipLaunchKernelGGL(scan_rows_kernel<1>, dim3((unsigned)vecs), dim3(256), 0, stream, vecs, k, X, ldx, t,
                         exps, zero, nzero, kp, digits);
  } else {
    hipLaunchKernelGGL(scan_rows_kernel<0>, dim3((unsigned)vecs), dim3(256), 0, stream, vecs, k, X, ldx, t,
                       exps, zero, nzero, kp, digits);
  }
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
