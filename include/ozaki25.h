/*
 * ozaki25.h -- emulated FP64 matrix multiplication by Ozaki Scheme II on the
 * FP8 (or, for the all-byte modulus set, int8) matrix cores of an AMD
 * Instinct MI355X (gfx950).
 *
 * The method (Ozaki Scheme II, Sec. 2 of "Ozaki 2.5: Engineering the
 * Deconstruction Path of FP64-Emulated Dense Matrix Multiplication on FP8
 * Tensor Cores"):
 *   1. scale each row of A and each column of B by a power of two and round to
 *      integers, A' = RN(diag(2^sigma) A), B' = RN(B diag(2^tau))   Eq. (scale)
 *   2. reduce the integers to centred residues modulo the moduli (the published
 *      twelve, split into low-precision limbs; or fifteen byte moduli) Eq. (residueprod),
 *      Eq. (pieces), Lemma 1, Alg. 2
 *   3. form the per-modulus products C^(i) = A^(i) B^(i) mod m_i    Eq. (residueprod)
 *   4. recover A'B' by Garner's mixed-radix CRT, unscale and round once to
 *      FP64                                                          Eq. (garner),
 *      Eq. (horner), Alg. 3
 *
 * Conventions shared by every entry point:
 *  - Matrices are row-major FP64.  A is m x k with leading dimension lda >= k,
 *    B is k x n with ldb >= n, C is m x n with ldc >= n.
 *  - Every data pointer is a DEVICE pointer (memory of the current HIP device).
 *    The caller owns all memory; no entry point frees or keeps a pointer.
 *  - `stream` is a hipStream_t passed as void* (NULL: the null stream).  Work is
 *    enqueued asynchronously on it; nothing synchronises the host.
 *  - Argument errors are detected synchronously, before anything is enqueued,
 *    and nothing is written then.  No exception crosses this interface.
 *  - Residues are centred: r in [-m/2, m/2), the endpoint -m/2 included for
 *    even m (Sec. 2, the convention stated with Eq. (moduli)).
 *  - Exponents: sigma_i = t(k) - e_i where e_i is the frexp exponent of
 *    max_l |a_il| (max in [2^(e-1), 2^e); e = 0 for a zero row); likewise
 *    tau_j for the columns of B.  A row or column holding a NaN or an infinity
 *    gets OZAKI25_EXP_NONFINITE and zero planes: it is out of the range the
 *    integer quantiser can represent (the range check that ends Alg. 1 and
 *    Alg. 3).  The GEMM entry points, which see A and B (ozaki25_dgemm,
 *    ozaki25_dgemm_sub, ozaki25_dgemm_ex, ozaki25_dgemm_noalloc), re-issue
 *    every output such a row or column touches on the native FP64 path: the
 *    dot product sum_l a_il b_lj in index order l = 0..k-1 from +0, each
 *    product rounded and then added, no fused multiply-add -- so those
 *    outputs (always an infinity or a NaN) follow IEEE semantics for that
 *    order of operations.  ozaki25_reconstruct and ozaki25_dgemm_planes, which
 *    do not see A and B, write NaN there.
 *  - Rounding: the quantiser of Eq. (scale) rounds to nearest, ties to even
 *    (Ozaki-II-RN), or, where an entry point takes an ozaki25_quantiser and
 *    OZAKI25_QUANT_TZ is passed, truncates toward zero (Ozaki-II-TZ of Table
 *    variants); the final rescale rounds once to nearest even, subnormal and
 *    overflow ranges included; an exact zero gives +0.0.
 */
#ifndef OZAKI25_H
#define OZAKI25_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OZAKI25_SUCCESS = 0,
  OZAKI25_ERR_INVALID_VALUE = 1, /* bad dimension, leading dimension, pointer or enum */
  OZAKI25_ERR_UNSUPPORTED = 2,   /* k beyond OZAKI25_MAX_K or n beyond OZAKI25_MAX_N */
  OZAKI25_ERR_WORKSPACE = 3,     /* workspace too small, or its allocation failed */
  OZAKI25_ERR_HIP = 4            /* a HIP launch or runtime call failed */
} ozaki25_status;

/* The modulus sets.
 *  OZAKI25_MODULI_S12: the published set of Eq. (moduli), in its published
 *    order: 1089, 1024, 961, 841, 625, 529 (squares of 33, 32, 31, 29, 25,
 *    23), then 511, 509, 503, 499, 491, 487.  log2(prod) = 111.84.  FP8 route:
 *    limb planes as e4m3 bytes, three FP8 products per modulus.
 *  OZAKI25_MODULI_A15: the all-byte set of Sec. 5.1 (candidate A): 256, 255,
 *    253, 251, 247, 241, 239, 233, 229, 227, 223, 217, 211, 199, 197.
 *    log2(prod) = 117.8.  Int8 route: the centred residue of a byte modulus
 *    lies in [-128, 127] and is itself the int8 plane, one int8 product per
 *    modulus (the int8 substrate of Sec. 2: r + 1 = 16 products' worth of
 *    matrix work against 3r + 1 = 37).  The same scale rule gives a few more
 *    bits per operand (t(8192) = 51 against 48). */
typedef enum { OZAKI25_MODULI_S12 = 0, OZAKI25_MODULI_A15 = 1 } ozaki25_moduli_set;

/* The integer quantiser of Eq. (scale), by the variant names of Table
 * variants: OZAKI25_QUANT_RN rounds x 2^sigma to nearest, ties to even
 * (Ozaki-II-RN, the variant the error theorem covers); OZAKI25_QUANT_TZ
 * truncates it toward zero (Ozaki-II-TZ, the shipping implementation's rule,
 * whose accuracy the paper leaves as an open obligation).  Both keep the
 * same scale bits t(k) and exponents, and |A'| never exceeds the RN bound. */
typedef enum { OZAKI25_QUANT_RN = 0, OZAKI25_QUANT_TZ = 1 } ozaki25_quantiser;

#define OZAKI25_NUM_MODULI 12          /* S12 */
#define OZAKI25_NUM_PLANES 30          /* S12: 2 per square modulus + 3 per nonsquare */
#define OZAKI25_NUM_MODULI_A15 15      /* A15: also its number of planes */
#define OZAKI25_K_ALIGN 128            /* planes are zero padded to a multiple of this */
#define OZAKI25_MAX_K 4194304          /* largest k accepted (bounds grid sizes; accumulation is exact at any k) */
#define OZAKI25_MAX_N 8388608          /* columns of B / C (32-bit offsets inside a tile) */
#define OZAKI25_EXP_NONFINITE INT32_MIN
#define OZAKI25_NUM_STAGE_EVENTS 5     /* see ozaki25_dgemm_ex */
#define OZAKI25_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20) /* see ozaki25_dgemm_noalloc */

/* Text for a status code (static storage, never NULL). */
const char* ozaki25_status_string(ozaki25_status status);

/* Number of moduli r of a set (12 for S12, 15 for A15), or -1 for an unknown set. */
int ozaki25_num_moduli(ozaki25_moduli_set set);

/* Number of stored planes of a set (30 for S12, 15 for A15), or -1. */
int ozaki25_num_planes(ozaki25_moduli_set set);

/* The i-th modulus of a set (0-based, published order), or -1. */
int64_t ozaki25_modulus(ozaki25_moduli_set set, int i);

/* t(k): the largest t with k 2^(2t) <= M/2 - 1 (M the product of the
 * moduli), so that every entry of A'B' lies inside [-M/2, M/2) (Eq. (moduli):
 * M > 2 mu with mu = k 2^(2t)).  Returns -1 for k < 1 or an unknown set. */
int ozaki25_scale_bits(int64_t k, ozaki25_moduli_set set);

/* k rounded up to OZAKI25_K_ALIGN (the plane row length k_pad); 0 for k <= 0. */
int64_t ozaki25_k_pad(int64_t k);

/* Bytes of the stored planes of `vecs` rows (or columns) of length k:
 * num_planes * vecs * k_pad (layout in ozaki25_deconstruct).  0 on invalid
 * input. */
size_t ozaki25_planes_bytes(int64_t vecs, int64_t k, ozaki25_moduli_set set);

/* Deconstruction of one operand (Alg. 2 with the exponent scan of Alg. 1):
 * exponent scan, scale, round to nearest, the centred residues and, for S12,
 * the limb split of Eq. (pieces) -- squares m = s^2: balanced base-s digits
 * (d0, d1) with d0 the centred residue of d mod s; nonsquares: Lemma 1's
 * carry-corrected base-16 layout (d0, d1, d0 + d1).
 *  side 0: X is A (vecs x k, row-major, ldx >= k); vector v is row v.
 *  side 1: X is B (k x vecs, row-major, ldx >= vecs); vector v is column v.
 * Outputs (device, caller-allocated):
 *  planes: uint8 [k_pad/128][num_planes][vecs][128] -- the byte of plane q,
 *          vector v, index l sits at ((l/128) num_planes + q) vecs 128 +
 *          v 128 + l%128, so a 128-wide k block of one plane is contiguous over
 *          the vectors; entries with l >= k are zero.
 *          S12: each byte a limb (an integer in [-22, 22]) encoded as OCP FP8
 *          E4M3FN -- every limb is e4m3-exact (Lemma 1), zero is 0x00; plane
 *          q of modulus i is q = (2 per earlier square + 3 per earlier
 *          nonsquare) + limb index.
 *          A15: 15 planes, plane i the centred residue mod m_i as an int8
 *          (two's complement byte, -128 included for m = 256).
 *  exps:   int32 [vecs], sigma (side 0) or tau (side 1), or
 *          OZAKI25_EXP_NONFINITE.
 *  quant:  the quantiser (OZAKI25_QUANT_RN or OZAKI25_QUANT_TZ).
 * vecs == 0 or k == 0 is a no-op.  Errors: INVALID_VALUE (side, sizes, null
 * pointers with nonzero sizes, set, quantiser), UNSUPPORTED (k > OZAKI25_MAX_K),
 * HIP. */
ozaki25_status ozaki25_deconstruct(int side, int64_t vecs, int64_t k, const double* X,
                                   int64_t ldx, ozaki25_moduli_set set, ozaki25_quantiser quant,
                                   uint8_t* planes, int32_t* exps, void* stream);

/* Per-modulus products (Eq. (residueprod)) from stored planes.  S12: FP8
 * MFMA with FP32 accumulation, reduced mod m_i at least every 16384 k so that
 * every partial sum is an integer below 2^24 and exact: for modulus i the limb
 * products are combined with the square epilogue {1, s, s} (d1 e1 vanishes
 * mod s^2) or Eq. (karcarry)'s {-15, 16, 240}, and reduced to the centred
 * residue.  A15: one int8 MFMA product per modulus with int32 accumulation
 * (exact: terms of at most 2^14, reduced every 65536 k).
 *  planesA: uint8 [k_pad/128][num_planes][m][128] (side 0 of
 *           ozaki25_deconstruct): e4m3 limbs for S12, int8 residues for A15
 *  planesB: uint8 [k_pad/128][num_planes][n][128] (side 1)
 *  Cres:    int32 [r][m][n], centred C^(i) (written, caller-allocated)
 * m == 0 or n == 0 is a no-op; k == 0 writes zeros.  Errors as above. */
ozaki25_status ozaki25_residue_gemm(int64_t m, int64_t n, int64_t k, const uint8_t* planesA,
                                    const uint8_t* planesB, ozaki25_moduli_set set,
                                    int32_t* Cres, void* stream);

/* Reconstruction (Alg. 3, Eq. (garner), Eq. (horner)): Garner's mixed-radix
 * digits of the r centred residues (12 or 15), the integer X in [-M/2, M/2), and
 * C_ij = RN(X 2^(-sigma_i - tau_j)) rounded once; NaN where expsA[i] or
 * expsB[j] is OZAKI25_EXP_NONFINITE (the GEMM entry points re-issue those
 * outputs natively instead; see the conventions above).  With subtract != 0:
 * C_ij <- C_ij - RN(X 2^(-sigma_i - tau_j)) (the product rounded, then the
 * IEEE subtraction).
 *  Cres: int32 [r][m][n]; expsA: int32 [m]; expsB: int32 [n]; C: m x n, ldc.
 * m == 0 or n == 0 is a no-op. */
ozaki25_status ozaki25_reconstruct(int64_t m, int64_t n, const int32_t* Cres,
                                   const int32_t* expsA, const int32_t* expsB,
                                   ozaki25_moduli_set set, double* C, int64_t ldc,
                                   int subtract, void* stream);

/* Device workspace that ozaki25_dgemm_ex needs for an m x n x k product. */
size_t ozaki25_dgemm_workspace_size(int64_t m, int64_t n, int64_t k, ozaki25_moduli_set set);

/* Emulated DGEMM C = A B (Alg. 1): both operands deconstructed once into
 * planes in the workspace (storage mode M), the residue products, then the
 * reconstruction.  With n <= 128 and m >= 1024 (tall and skinny: one output
 * tile spans all of B), either set, only B's planes are stored and A is
 * quantised and reduced inside the product kernel (storage mode F for A --
 * the hybrid of Sec. 6.2); the result is the same bit for bit.  The
 * workspace is allocated and released stream-ordered on
 * `stream` (hipMallocAsync / hipFreeAsync).  m == 0 or n == 0: no-op;
 * k == 0: C = +0.  A and B must not overlap C.  Errors: INVALID_VALUE,
 * UNSUPPORTED, WORKSPACE (allocation failed), HIP. */
ozaki25_status ozaki25_dgemm(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                             const double* B, int64_t ldb, double* C, int64_t ldc,
                             ozaki25_moduli_set set, void* stream);

/* HPL trailing update C <- C - A B, same conventions (k == 0: C unchanged). */
ozaki25_status ozaki25_dgemm_sub(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                 const double* B, int64_t ldb, double* C, int64_t ldc,
                                 ozaki25_moduli_set set, void* stream);

/* Full form.  quant: the quantiser (ozaki25_dgemm and ozaki25_dgemm_sub use
 * OZAKI25_QUANT_RN).  subtract: 0 for C = A B, 1 for C <- C - A B.
 * workspace: NULL to allocate stream-ordered, else a device buffer of at least
 *   ozaki25_dgemm_workspace_size() bytes (256-byte aligned), owned by the
 *   caller and not used by anything else until the stream has passed this call.
 * stage_events: NULL, or OZAKI25_NUM_STAGE_EVENTS hipEvent_t handles (passed as
 *   void*) that are recorded on `stream` before the first kernel, after the
 *   exponent scans, after the deconstruction, after the residue products and
 *   after the reconstruction, for per-stage timing.  The scans run
 *   interleaved with the deconstruction (runs of about 256 MiB of each
 *   operand, each deconstructed right after its scan), so the first two
 *   events are recorded together and the deconstruct stage holds the scans. */
ozaki25_status ozaki25_dgemm_ex(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                const double* B, int64_t ldb, double* C, int64_t ldc,
                                ozaki25_moduli_set set, ozaki25_quantiser quant, int subtract,
                                void* workspace, size_t workspace_bytes,
                                void* const* stage_events, void* stream);

/* Device workspace that ozaki25_dgemm_planes needs for an m x n x k product
 * (the per-modulus residue products -- int16 for S12, int8 for A15 -- and,
 * when few output tiles would leave the chip idle, per-split partial
 * products of a split k range). */
size_t ozaki25_dgemm_planes_workspace_size(int64_t m, int64_t n, int64_t k, ozaki25_moduli_set set);

/* Emulated DGEMM from stored planes -- storage mode P of Sec. 6.2, principle O1
 * of Sec. 5 (planes converted once and kept across calls: a fixed A in
 * block-Krylov or iterative refinement is deconstructed once, and each call
 * pays only the residue products and the reconstruction).
 *  planesA, expsA: ozaki25_deconstruct side 0 of an m x k A;
 *  planesB, expsB: side 1 of a k x n B -- both with this k and set (either
 *    quantiser; the result is that of ozaki25_dgemm_ex with the same
 *    quantiser, bit for bit).
 *  C, ldc, subtract: as in ozaki25_dgemm_ex, except that outputs on a row or
 *    column flagged OZAKI25_EXP_NONFINITE are NaN (A and B are not at hand
 *    for the native re-issue).
 *  workspace: NULL to allocate stream-ordered, else at least
 *    ozaki25_dgemm_planes_workspace_size(m, n, k, set) bytes, 256-byte aligned.
 * m == 0 or n == 0: no-op; k == 0: C = +0 (or unchanged with subtract).
 * Errors: INVALID_VALUE, UNSUPPORTED, WORKSPACE, HIP. */
ozaki25_status ozaki25_dgemm_planes(int64_t m, int64_t n, int64_t k, const uint8_t* planesA,
                                    const int32_t* expsA, const uint8_t* planesB,
                                    const int32_t* expsB, double* C, int64_t ldc,
                                    ozaki25_moduli_set set, int subtract, void* workspace,
                                    size_t workspace_bytes, void* stream);

/* Accurate mode (Sec. 2, Eq. (alpha): one more low-precision product, an
 * estimate of the input magnitudes, so alpha = 3r + 1 products for S12).
 * Instead of the fixed t(k) of the fast mode, each row of A and column of B
 * gets its own shift from a bound on the outputs it feeds:
 *   1. digits alpha_il = ceil(16 |a_il| 2^-e_i) in {0..16} (e_i as in the
 *      conventions above), likewise beta_lj for B -- so |a_il| is at most
 *      alpha_il 2^(e_i - 4);
 *   2. U = alpha beta on int8 MFMA (exact: U <= 256 k < 2^31);
 *   3. L_ij = the largest L with 2^L U_ij <= 2^8 (M/2 - 1); column shifts
 *      u_j = min(58, floor(min_i L_ij / 2)), row shifts
 *      s_i = min(58, min_j (L_ij - u_j)); sigma_i = s_i - e_i and
 *      tau_j = u_j - f_j.
 * Since |a'_il| <= alpha_il 2^(s_i - 4), every |A'B'|_ij stays below M/2
 * (Eq. (moduli)); and since U_ij <= 256 k, s_i and u_j are never below the
 * fast mode's t(k): the accurate mode never keeps fewer bits, and on data
 * whose magnitudes vary within a row or column it keeps several more per
 * operand.  The shifts depend on all of A and all of B (a row's shift on
 * every column it meets), so they are computed per call; non-finite rows /
 * columns keep OZAKI25_EXP_NONFINITE and are re-issued natively as in the
 * fast mode.  The cap of 58 is the largest t(k) the fast mode itself uses
 * (A15 at k = 1). */

/* Device workspace of ozaki25_accurate_exponents: the digit planes of A and
 * B ((m + n) k_pad bytes), the totals L (m n bytes), their column minima per
 * 64 rows (ceil(m/64) n bytes), n bytes of column shifts, and for few output
 * tiles the split bound product's int32 partials. */
size_t ozaki25_accurate_exponents_workspace_size(int64_t m, int64_t n, int64_t k);

/* The accurate mode's sigma (expsA, m int32) and tau (expsB, n int32) for
 * C = A B, device memory; the two must not overlap.  workspace: NULL to
 * allocate stream-ordered, else at least
 * ozaki25_accurate_exponents_workspace_size() bytes, 256-byte aligned.
 * m, n or k == 0: no-op.  Errors: INVALID_VALUE, UNSUPPORTED, WORKSPACE, HIP. */
ozaki25_status ozaki25_accurate_exponents(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                          const double* B, int64_t ldb, ozaki25_moduli_set set,
                                          int32_t* expsA, int32_t* expsB, void* workspace,
                                          size_t workspace_bytes, void* stream);

/* Device workspace of ozaki25_dgemm_accurate: that of ozaki25_dgemm_ex plus
 * that of ozaki25_accurate_exponents. */
size_t ozaki25_dgemm_accurate_workspace_size(int64_t m, int64_t n, int64_t k, ozaki25_moduli_set set);

/* Emulated DGEMM in the accurate mode: ozaki25_dgemm_ex's arguments and
 * conventions (quantiser, subtract, workspace, the five stage events -- the
 * second recorded after the accurate exponents, the third after both
 * operands' planes), with the exponents of ozaki25_accurate_exponents.
 * The result is that of the fast mode's pipeline run with those exponents,
 * bit for bit.  k == 0: C = +0 (or unchanged with subtract).
 * Errors: INVALID_VALUE, UNSUPPORTED, WORKSPACE, HIP. */
ozaki25_status ozaki25_dgemm_accurate(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                      const double* B, int64_t ldb, double* C, int64_t ldc,
                                      ozaki25_moduli_set set, ozaki25_quantiser quant, int subtract,
                                      void* workspace, size_t workspace_bytes,
                                      void* const* stage_events, void* stream);

/* For callers that cannot allocate device memory -- work recorded under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc:
 * ozaki25_dgemm_ex with its workspace taken from a static device array of
 * OZAKI25_NOALLOC_SCRATCH_BYTES (128 MiB) inside the library instead of an
 * argument, and no allocation of any kind.  Each GPU the library runs on
 * holds its own copy of the array from the library's load until the process
 * ends.  The caller still passes A, B and C (device memory, as for
 * ozaki25_dgemm_ex); quant and subtract as there.
 *  - Size limit: ozaki25_dgemm_workspace_size(m, n, k, set) must not exceed
 *    OZAKI25_NOALLOC_SCRATCH_BYTES (e.g. 1024 x 1024 x 1024 fits both sets);
 *    larger products return OZAKI25_ERR_WORKSPACE before anything is
 *    enqueued.
 *  - Every call on one GPU shares that GPU's array and leaves its planes,
 *    exponents and residues there; nothing in it needs to start at zero.
 *    Calls that overlap on one GPU (other streams, other host threads) race
 *    on the array: order them, e.g. on one stream.
 *  - The first call on a device resolves the array's device address
 *    (hipGetSymbolAddress, with that device current) and keeps it; make that
 *    first call outside graph capture.
 * m == 0 or n == 0: no-op; k == 0: C = +0 (or unchanged with subtract).
 * Errors: INVALID_VALUE, UNSUPPORTED, WORKSPACE (beyond the array), HIP. */
ozaki25_status ozaki25_dgemm_noalloc(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                     const double* B, int64_t ldb, double* C, int64_t ldc,
                                     ozaki25_moduli_set set, ozaki25_quantiser quant, int subtract,
                                     void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OZAKI25_H */
