// Accurate-mode scaling (Sec. 2, Eq. (alpha): one extra low-precision
// product bounds the input magnitudes).  From the totals L_ij of the bound
// product -- the largest shift with 2^L U_ij <= 2^8 (M/2 - 1), where U is
// the product of the magnitude digits ceil(16 |x| 2^-e) -- the column and
// row shifts
//     u_j = min(58, floor(min_i L_ij / 2)),   s_i = min(58, min_j (L_ij - u_j)),
// so that s_i + u_j <= L_ij everywhere and |A'B'| stays below M/2
// (Eq. (moduli)).  The exponents are then sigma_i = s_i - e_i and
// tau_j = u_j - f_j.  L is int8 [m][n] (127 where unconstrained); all of
// this is HBM-bound on m n bytes.
#include "exponent_key.hpp"
#include "kernels.hpp"

namespace oz {
namespace {

constexpr int kShiftCap = 58;
constexpr int kTotalNone = 127;

__global__ __launch_bounds__(256) void fill_kernel(int64_t count, int32_t value, int32_t* p) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < count) p[i] = value;
}

// Column minima of L: a thread per column, a block per 256 columns and
// rows_per_block rows (each wavefront row load reads 64 consecutive bytes),
// combined over the row blocks by an atomic min.
__global__ __launch_bounds__(256) void column_min_kernel(int64_t m, int64_t n, int64_t rows_per_block,
                                                         const int8_t* __restrict__ L,
                                                         int32_t* __restrict__ colmin) {
  const int64_t cb = (n + 255) / 256;
  const int64_t j = (int64_t)(blockIdx.x % cb) * 256 + threadIdx.x;
  const int64_t i0 = (int64_t)(blockIdx.x / cb) * rows_per_block;
  const int64_t i1 = i0 + rows_per_block < m ? i0 + rows_per_block : m;
  if (j >= n) return;
  int mn = kTotalNone;
  for (int64_t i = i0; i < i1; ++i) {
    const int v = L[i * n + j];
    mn = v < mn ? v : mn;
  }
  if (mn < kTotalNone) atomicMin(colmin + j, mn);
}

// u_j from the column minimum (kept in place of it for the row pass) and
// tau_j = u_j - f_j from the column scan's exponent key (a non-finite
// column keeps its flag).
__global__ __launch_bounds__(256) void finalize_cols_kernel(int64_t n, int32_t* __restrict__ colmin_u,
                                                            int32_t* __restrict__ keys_tau) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= n) return;
  const int half = colmin_u[j] / 2;
  const int u = half < kShiftCap ? half : kShiftCap;
  colmin_u[j] = u;
  keys_tau[j] = key_to_sigma((uint32_t)keys_tau[j], u);
}

// s_i: a wavefront per row (lanes along the row, 64 consecutive bytes per
// load), the minimum of L_ij - u_j by a butterfly; sigma_i = s_i - e_i from
// the row scan at t = 0 (which left -e_i; a non-finite row keeps its flag).
__global__ __launch_bounds__(256) void finalize_rows_kernel(int64_t m, int64_t n,
                                                            const int8_t* __restrict__ L,
                                                            const int32_t* __restrict__ u,
                                                            int32_t* __restrict__ exps) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= m) return;
  const int8_t* row = L + i * n;
  int mn = kShiftCap;
  for (int64_t j = lane; j < n; j += 64) {
    const int d = (int)row[j] - u[j];
    mn = d < mn ? d : mn;
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

hipError_t launch_accurate_shifts(int64_t m, int64_t n, const int8_t* L, int32_t* colmin, int32_t* ea,
                                  int32_t* eb_keys, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  const int64_t nb = (n + 255) / 256;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)nb), dim3(256), 0, stream, n, (int32_t)kTotalNone, colmin);
  // about 2048 blocks: rows per block a multiple of 16, at least 64
  int64_t rpb = (m * nb + 2047) / 2048;
  rpb = rpb < 64 ? 64 : (rpb + 15) / 16 * 16;
  const int64_t rb = (m + rpb - 1) / rpb;
  if (nb * rb > (int64_t)UINT32_MAX || (m + 3) / 4 > (int64_t)UINT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(column_min_kernel, dim3((unsigned)(nb * rb)), dim3(256), 0, stream, m, n, rpb, L,
                     colmin);
  hipLaunchKernelGGL(finalize_cols_kernel, dim3((unsigned)nb), dim3(256), 0, stream, n, colmin, eb_keys);
  hipLaunchKernelGGL(finalize_rows_kernel, dim3((unsigned)((m + 3) / 4)), dim3(256), 0, stream, m, n, L,
                     colmin, ea);
  return hipGetLastError();
}

}  // namespace oz
