// Accurate-mode scaling (Sec. 2, Eq. (alpha): one extra low-precision
// product bounds the input magnitudes).  From the totals L_ij of the bound
// product -- the largest shift with 2^L U_ij <= 2^8 (M/2 - 1), where U is
// the product of the magnitude digits ceil(16 |x| 2^-e) -- the column and
// row shifts
//     u_j = min(58, floor(min_i L_ij / 2)),   s_i = min(58, min_j (L_ij - u_j)),
// so that s_i + u_j <= L_ij everywhere and |A'B'| stays below M/2
// (Eq. (moduli)).  The exponents are then sigma_i = s_i - e_i and
// tau_j = u_j - f_j.  L is int8 [m][n] (127 where unconstrained) and the
// bound product also leaves the column minima of every 64-row group
// (colpart [groups][n]); the row pass reads L once.  HBM-bound on m n bytes.
#include "exponent_key.hpp"
#include "kernels.hpp"

namespace oz {
namespace {

constexpr int kShiftCap = 58;
constexpr int kTotalNone = 127;

// The group minima reduced over slices of groups: a block takes 64 columns
// and one slice, its four wavefronts interleave the slice's groups (each
// load reads 64 consecutive bytes of a group's row), and LDS joins them
// into colslice [slices][n].
__global__ __launch_bounds__(256) void colreduce_kernel(int64_t n, int64_t groups, int64_t per_slice,
                                                        const int8_t* __restrict__ colpart,
                                                        int8_t* __restrict__ colslice) {
  __shared__ int part[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t j = (int64_t)blockIdx.x * 64 + lane;
  const int64_t sl = blockIdx.y;
  const int64_t g0 = sl * per_slice, g1 = g0 + per_slice < groups ? g0 + per_slice : groups;
  int mn = kTotalNone;
  if (j < n) {
    for (int64_t g = g0 + wave; g < g1; g += 4) {
      const int v = colpart[g * n + j];
      mn = v < mn ? v : mn;
    }
  }
  part[wave][lane] = mn;
  __syncthreads();
  if (wave == 0 && j < n) {
    for (int w = 1; w < 4; ++w) mn = part[w][lane] < mn ? part[w][lane] : mn;
    colslice[sl * n + j] = (int8_t)mn;
  }
}

// u_j from the column minima of the slices (written as a byte, ub, for the
// row pass) and tau_j = u_j - f_j from the column scan's exponent key (a
// non-finite column keeps its flag).  A thread per column.
__global__ __launch_bounds__(256) void finalize_cols_kernel(int64_t n, int64_t groups,
                                                            const int8_t* __restrict__ colslice,
                                                            uint8_t* __restrict__ ub,
                                                            int32_t* __restrict__ keys_tau) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= n) return;
  int mn = kTotalNone;
  for (int64_t g = 0; g < groups; ++g) {
    const int v = colslice[g * n + j];
    mn = v < mn ? v : mn;
  }
  const int u = mn / 2 < kShiftCap ? mn / 2 : kShiftCap;
  ub[j] = (uint8_t)u;
  keys_tau[j] = key_to_sigma((uint32_t)keys_tau[j], u);
}

// Byte-wise minimum of four bytes below 128 each: per byte a + 128 - b
// never borrows into the next byte, and its top bit says a >= b.
__device__ __forceinline__ uint32_t min_u8x4(uint32_t a, uint32_t b) {
  const uint32_t ge = ((a | 0x80808080u) - b) & 0x80808080u;
  const uint32_t m = (ge >> 7) * 0xFFu;
  return (b & m) | (a & ~m);
}

__device__ __forceinline__ int min_bytes(uint32_t w) {
  int a = (int)(w & 0xFF), b = (int)((w >> 8) & 0xFF), c = (int)((w >> 16) & 0xFF), d = (int)(w >> 24);
  a = b < a ? b : a;
  c = d < c ? d : c;
  return c < a ? c : a;
}

// s_i: a wavefront per row, the minimum of L_ij - u_j by a butterfly, then
// sigma_i = s_i - e_i from the row scan at t = 0 (which left -e_i; a
// non-finite row keeps its flag).  VEC (n a multiple of 16): 16 columns per
// lane and load, the differences and minima four bytes at a time (every
// L_ij >= 2 u_j, so L_ij - u_j never borrows, and it stays below 128).
template <bool VEC>
__global__ __launch_bounds__(256) void finalize_rows_kernel(int64_t m, int64_t n,
                                                            const int8_t* __restrict__ L,
                                                            const uint8_t* __restrict__ ub,
                                                            int32_t* __restrict__ exps) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= m) return;
  int mn = kShiftCap;
  if constexpr (VEC) {
    const uint4* row = reinterpret_cast<const uint4*>(L + i * n);
    const uint4* uu = reinterpret_cast<const uint4*>(ub);
    uint32_t acc = 0x3A3A3A3Au;  // 58 in every byte
    for (int64_t q = lane; q < n / 16; q += 64) {
      const uint4 l = row[q], u = uu[q];
      acc = min_u8x4(acc, l.x - u.x);
      acc = min_u8x4(acc, l.y - u.y);
      acc = min_u8x4(acc, l.z - u.z);
      acc = min_u8x4(acc, l.w - u.w);
    }
    mn = min_bytes(acc);
  } else {
    const int8_t* row = L + i * n;
    for (int64_t j = lane; j < n; j += 64) {
      const int d = (int)row[j] - (int)ub[j];
      mn = d < mn ? d : mn;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const int o = __shfl_xor(mn, off, 64);
    mn = o < mn ? o : mn;
  }
  if (lane == 0) {
    const int32_t ne = exps[i];
    exps[i] = ne == INT32_MIN ? INT32_MIN : ne + mn;
  }
}

}  // namespace

int64_t accurate_slices(int64_t m, int64_t n, int64_t* per_slice) {
  // up to about 2048 blocks of 64 columns x one slice of at least 32 groups
  // (so that the final pass over the slices stays short)
  const int64_t groups = (m + 63) / 64, cb = (n + 63) / 64;
  int64_t target = 2048 / cb;
  target = target > groups / 32 ? groups / 32 : target;
  target = target < 1 ? 1 : target;
  const int64_t per = (groups + target - 1) / target;
  if (per_slice) *per_slice = per;
  return (groups + per - 1) / per;
}

hipError_t launch_accurate_shifts(int64_t m, int64_t n, const int8_t* L, const int8_t* colpart,
                                  int8_t* colslice, uint8_t* ub, int32_t* ea, int32_t* eb_keys,
                                  hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  const int64_t nb = (n + 255) / 256;
  int64_t per = 0;
  const int64_t slices = accurate_slices(m, n, &per);
  if (nb > (int64_t)UINT32_MAX || (m + 3) / 4 > (int64_t)UINT32_MAX || slices > 65535 ||
      (n + 63) / 64 > (int64_t)UINT32_MAX)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(colreduce_kernel, dim3((unsigned)((n + 63) / 64), (unsigned)slices), dim3(256), 0, stream,
                     n, (m + 63) / 64, per, colpart, colslice);
  hipLaunchKernelGGL(finalize_cols_kernel, dim3((unsigned)nb), dim3(256), 0, stream, n, slices, colslice,
                     ub, eb_keys);
  const bool vec = n % 16 == 0 && ((uintptr_t)L & 15) == 0 && ((uintptr_t)ub & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(finalize_rows_kernel<true>, dim3((unsigned)((m + 3) / 4)), dim3(256), 0, stream, m, n, L,
                       ub, ea);
  else
    hipLaunchKernelGGL(finalize_rows_kernel<false>, dim3((unsigned)((m + 3) / 4)), dim3(256), 0, stream, m, n,
                       L, ub, ea);
  return hipGetLastError();
}

}  // namespace oz
