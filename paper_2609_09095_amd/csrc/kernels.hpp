// Launchers of the gfx950 kernels (internal to the library; the C ABI in
// ozaki25.h is the public surface).  Every launcher enqueues on `stream` and
// returns the HIP error of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace oz {

// Modulus sets, as numbered by ozaki25_moduli_set.
constexpr int kSetPublished = 0;  // Eq. (moduli), FP8 limb route
constexpr int kSetBytes = 1;      // Sec. 5.1 candidate A, int8 route
// Quantisers, as numbered by ozaki25_quantiser.
constexpr int kQuantRN = 0;  // round to nearest, ties to even
constexpr int kQuantTZ = 1;  // toward zero

// Exponent scan (Alg. 1 setup): sigma_v = t - e_v, or INT32_MIN for a vector
// holding a NaN or an infinity.
//  - rows of A: exps[v] = sigma directly; `zero` (nzero int32, may be null)
//    is cleared on the side -- B's column keys, so that their scan needs no
//    clearing launch;
//  - columns of B in three steps: keys cleared to 0 (launch_clear_keys, or
//    the side job above), an atomic max of order-preserving exponent keys
//    per column (launch_scan_cols, any number of column ranges), and the
//    keys turned into sigma (launch_keys_to_sigma).  The deconstruction can
//    read the keys directly (keys_in).
// With digits (the accurate mode) the row scan also writes the rows'
// magnitude digits as one int8 plane (see launch_digits) of kp per row.
hipError_t launch_scan_rows(int64_t vecs, int64_t k, const double* X, int64_t ldx, int t, int32_t* exps,
                            int32_t* zero, int64_t nzero, hipStream_t stream, int8_t* digits = nullptr,
                            int64_t kp = 0);
hipError_t launch_clear_keys(int64_t vecs, int32_t* keys, hipStream_t stream);
hipError_t launch_scan_cols(int64_t vecs, int64_t k, const double* X, int64_t ldx, int32_t* keys,
                            hipStream_t stream);
hipError_t launch_keys_to_sigma(int64_t vecs, int t, int32_t* exps, hipStream_t stream);

// The largest scale t (|A'| <= 2^t) the residue kernels accept: t(k) of
// either set at k = 1, and the accurate mode's cap.
constexpr int kMaxScaleBits = 58;

// Alg. 2: scale, quantise, residues and the planes of one operand, given exps
// (sigma, or with keys_in the column scan's exponent keys, turned into sigma
// on load) and the scale bits t: e4m3 limb planes (published set) or int8
// residue planes (all-byte set).  vecs vectors of X, written into a plane
// layout of vstride >= vecs vectors (planes points at the first one's
// bytes), so that a run of vectors can fill its part of a larger operand's
// planes.
hipError_t launch_deconstruct(int set, int quant, int side, int64_t vecs, int64_t vstride, int64_t k,
                              int64_t kp, int t, const double* X, int64_t ldx, const int32_t* exps,
                              bool keys_in, int8_t* planes, hipStream_t stream);

// Eq. (residueprod): r centred per-modulus products [r][m][n], on FP8 MFMA
// from limb planes (published set) or int8 MFMA from residue planes
// (all-byte set).  n must not exceed kMaxResidueCols.
constexpr int64_t kMaxResidueCols = (int64_t)1 << 23;
hipError_t launch_residue_gemm_i32(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                   const int8_t* pb, int32_t* cres, hipStream_t stream);
// The fused path's compact products may split the k range (split-k) when
// the output tiles are too few to fill the chip: `splits` from
// residue_gemm_splits, and a partial buffer of splits * r * m * n elements.
// Compact int16 products (published set) are the true residues divided by
// compact_scale(i) mod m_i, reduced to |c| <= 0.51 m_i but not centred;
// launch_reconstruct_i16 takes exactly these.
constexpr int kMaxSplits = 64;
int residue_gemm_splits(int set, int64_t m, int64_t n, int64_t kp);
hipError_t launch_residue_gemm_i16(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                   const int8_t* pb, int16_t* cres, int16_t* part, int splits,
                                   hipStream_t stream);
hipError_t launch_residue_gemm_bytes_i32(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                         const int8_t* pb, int32_t* cres, hipStream_t stream);
hipError_t launch_residue_gemm_bytes_i8(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                        const int8_t* pb, int8_t* cres, int8_t* part, int splits,
                                        hipStream_t stream);

// Storage mode F for A (tall/skinny, at most 128 columns; all-byte set):
// the per-modulus products [15][m][n] (compact int8, as
// launch_residue_gemm_bytes_i8 writes them) straight from FP64 A, its row
// exponents sigma (launch_scan_rows) and B's stored planes; A is quantised
// and reduced inside the kernel.  k == 0 is not handled here.
hipError_t launch_fused_bytes(int quant, int64_t m, int64_t n, int64_t k, int64_t kp, int t,
                              const double* A, int64_t lda, const int32_t* sigma, const int8_t* pb,
                              int8_t* cres, hipStream_t stream);

// Storage mode F for A, published set (at most 128 columns): B's digit
// planes for the fused product (24 planes [kp/128][24][n][128] into pb, from
// B and its column exponents tau), then the per-modulus products [12][m][n]
// as the compact int16 residues launch_reconstruct_i16 takes, straight from
// FP64 A and its row exponents sigma.  k == 0 is not handled here.
hipError_t launch_fused_pub(int quant, int64_t m, int64_t n, int64_t k, int64_t kp, int t, const double* A,
                            int64_t lda, const int32_t* sigma, const double* B, int64_t ldb,
                            const int32_t* tau, int8_t* pb, int16_t* cres, hipStream_t stream);

// The operands of Alg. 1's last step (range check, native FP64 re-issue):
// outputs whose row of A or column of B was flagged non-finite by the
// exponent scan become the index-order FP64 dot product of that row and
// column (rounded product, then sum; no FMA).  A == nullptr (the stage API,
// stored planes): those outputs are NaN instead.
struct NativeOperands {
  const double* A = nullptr;
  int64_t lda = 0;
  const double* B = nullptr;
  int64_t ldb = 0;
  int64_t k = 0;
};

// Alg. 3: Garner, Horner, lift, single rounding (C = or C -= ).
hipError_t launch_reconstruct_i32(int64_t m, int64_t n, const int32_t* cres, const int32_t* ea,
                                  const int32_t* eb, double* C, int64_t ldc, int subtract,
                                  hipStream_t stream);
hipError_t launch_reconstruct_i16(int64_t m, int64_t n, const int16_t* cres, const int32_t* ea,
                                  const int32_t* eb, double* C, int64_t ldc, int subtract,
                                  const NativeOperands& nat, hipStream_t stream);
// the same for the fifteen residues of the all-byte set
hipError_t launch_reconstruct_bytes_i32(int64_t m, int64_t n, const int32_t* cres,
                                        const int32_t* ea, const int32_t* eb, double* C,
                                        int64_t ldc, int subtract, hipStream_t stream);
hipError_t launch_reconstruct_bytes_i8(int64_t m, int64_t n, const int8_t* cres, const int32_t* ea,
                                       const int32_t* eb, double* C, int64_t ldc, int subtract,
                                       const NativeOperands& nat, hipStream_t stream);

// Accurate mode (Sec. 2, Eq. (alpha)).
//  - launch_digits: the magnitude digits ceil(16 |x| 2^-e) of one operand as
//    a single int8 plane [kp/128][vecs][128]; exps holds -e (the scan at
//    t = 0, or with keys_in the column scan's keys);
//  - launch_bound_gemm: U = digitsA digitsB^T on int8 MFMA and, per output,
//    the total shift L (int8 [m][n]) with 2^L U <= T, T = 2^8 (M/2 - 1) of
//    bit length bt and ttop = T >> (bt - 33), plus the column minima of L
//    over each 64-row group (colpart, int8 [ceil(m/64)][n]); `splits` from
//    bound_gemm_splits, with splits * m * n int32 of `part` when above 1;
//  - launch_accurate_shifts: from colpart the column shifts (ub, n bytes,
//    16-byte aligned) and tau = u - f into eb_keys (the column scan's keys),
//    then from L sigma = s - e into ea (the row scan at t = 0).
hipError_t launch_digits(int side, int64_t vecs, int64_t k, int64_t kp, const double* X, int64_t ldx,
                         const int32_t* exps, bool keys_in, int8_t* digits, hipStream_t stream);
int bound_gemm_splits(int64_t m, int64_t n, int64_t kp);
hipError_t launch_bound_gemm(int64_t m, int64_t n, int64_t kp, const int8_t* da, const int8_t* db,
                             int8_t* total, int8_t* colpart, int32_t* part, int splits, int bt, uint64_t ttop,
                             hipStream_t stream);
// colpart is reduced in two steps: over slices of groups into colslice
// ([accurate_slices(m, n)][n] bytes), then over the slices.
int64_t accurate_slices(int64_t m, int64_t n, int64_t* per_slice);
hipError_t launch_accurate_shifts(int64_t m, int64_t n, const int8_t* L, const int8_t* colpart,
                                  int8_t* colslice, uint8_t* ub, int32_t* ea, int32_t* eb_keys,
                                  hipStream_t stream);

// C = +0.0 over an m x n block (the k == 0 product).
hipError_t launch_zero_c(int64_t m, int64_t n, double* C, int64_t ldc, hipStream_t stream);

}  // namespace oz
