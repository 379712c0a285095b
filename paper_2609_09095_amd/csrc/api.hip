// The C ABI of ozaki25.h: argument checks, the scale-bit rule, workspace
// layout and the launch sequence of Alg. 1 on one stream, for both modulus
// sets.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>

#include "kernels.hpp"
#include "moduli.hpp"
#include "ozaki25.h"

static_assert(OZAKI25_MAX_N <= oz::kMaxResidueCols, "residue GEMM column limit");

namespace {

using u128 = unsigned __int128;

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

static_assert(OZAKI25_MODULI_S12 == oz::kSetPublished && OZAKI25_MODULI_A15 == oz::kSetBytes,
              "set numbering");
static_assert(OZAKI25_NUM_MODULI == oz::kR && OZAKI25_NUM_PLANES == oz::kPlanes &&
                  OZAKI25_NUM_MODULI_A15 == oz::kRA,
              "set sizes");

bool known_set(ozaki25_moduli_set set) {
  return set == OZAKI25_MODULI_S12 || set == OZAKI25_MODULI_A15;
}
bool bytes_set(ozaki25_moduli_set set) { return set == OZAKI25_MODULI_A15; }
bool known_quantiser(ozaki25_quantiser q) { return q == OZAKI25_QUANT_RN || q == OZAKI25_QUANT_TZ; }
static_assert(OZAKI25_QUANT_RN == oz::kQuantRN && OZAKI25_QUANT_TZ == oz::kQuantTZ, "quantiser numbering");
int num_moduli(ozaki25_moduli_set set) { return bytes_set(set) ? oz::kRA : oz::kR; }
// the all-byte set stores one int8 plane per modulus
int num_planes(ozaki25_moduli_set set) { return bytes_set(set) ? oz::kRA : oz::kPlanes; }
int64_t modulus(ozaki25_moduli_set set, int i) {
  return bytes_set(set) ? oz::kModulusA[i] : oz::kModulus[i];
}

// t(k) = max{t : k 2^(2t) <= M/2 - 1} (Eq. (moduli) with mu = k 2^(2t)).
int scale_bits(int64_t k, ozaki25_moduli_set set) {
  if (k < 1) return -1;
  u128 M = 1;
  for (int i = 0; i < num_moduli(set); ++i) M *= (u128)modulus(set, i);
  const u128 q = (M / 2 - 1) / (u128)k;
  int t = 0;
  while (((u128)1 << (2 * (t + 1))) <= q) ++t;
  return t;
}

int64_t k_pad(int64_t k) { return k <= 0 ? 0 : (k + oz::kKAlign - 1) / oz::kKAlign * oz::kKAlign; }

// Byte range [p, p + bytes) overlaps [q, q + qbytes)?
bool overlaps(const void* p, size_t bytes, const void* q, size_t qbytes) {
  const uintptr_t a = (uintptr_t)p, b = (uintptr_t)q;
  return bytes && qbytes && a < b + qbytes && b < a + bytes;
}

size_t matrix_bytes(int64_t rows, int64_t cols, int64_t ld) {
  if (rows <= 0 || cols <= 0) return 0;
  return ((size_t)(rows - 1) * (size_t)ld + (size_t)cols) * sizeof(double);
}

ozaki25_status hip_status(hipError_t e) { return e == hipSuccess ? OZAKI25_SUCCESS : OZAKI25_ERR_HIP; }

struct Workspace {
  size_t planes_a, planes_b, exps_a, exps_b, cres, part, total;
  int splits;
};

size_t cres_elem(ozaki25_moduli_set set) { return bytes_set(set) ? sizeof(int8_t) : sizeof(int16_t); }

// the compact residue products and, with split-k, the per-split partials
size_t products_bytes(int64_t m, int64_t n, int64_t k, ozaki25_moduli_set set, int* splits) {
  const int sp = oz::residue_gemm_splits((int)set, m, n, k_pad(k));
  if (splits) *splits = sp;
  const size_t one = (size_t)num_moduli(set) * m * n * cres_elem(set);
  return align_up(one) + (sp > 1 ? align_up(one * sp) : 0);
}

// Storage mode F for A (at most 128 columns, at least kFusedMinRows rows;
// either set): A is converted inside the product kernel, so the workspace
// holds no planes of A and the products need no split of k.  B's planes
// there: the all-byte set's residue planes, or for the published set the
// 24 digit planes of its fused product (fewer bytes than its 30 planes).
constexpr int64_t kFusedMinRows = 1024;
bool fused_a(int64_t m, int64_t n, ozaki25_moduli_set set) {
  return known_set(set) && n <= 128 && m >= kFusedMinRows;
}

// planes of A and B, exponents, and the residue products: int16 for the
// published set (|c| <= 0.51 m <= 556), int8 for the all-byte set (|c| <= 128)
Workspace layout(int64_t m, int64_t n, int64_t k, ozaki25_moduli_set set) {
  Workspace w;
  const int64_t kp = k_pad(k);
  const size_t np = (size_t)num_planes(set);
  const bool fused = fused_a(m, n, set);
  size_t off = 0;
  w.planes_a = off;
  off = fused ? off : align_up(off + np * m * kp);
  w.planes_b = off;
  off = align_up(off + np * n * kp);
  w.exps_a = off;
  off = align_up(off + (size_t)m * sizeof(int32_t));
  w.exps_b = off;
  off = align_up(off + (size_t)n * sizeof(int32_t));
  w.cres = off;
  const size_t one = align_up((size_t)num_moduli(set) * m * n * cres_elem(set));
  const size_t prod = fused ? one : products_bytes(m, n, k, set, &w.splits);
  if (fused) w.splits = 1;
  w.part = off + one;
  off += prod;
  w.total = off;
  return w;
}

// Exponent scan and deconstruction of one operand, in runs of whole
// 256-vector tiles holding about 256 MiB of FP64 each (the size of the
// MI355X last-level cache): each run's deconstruction reads the run right
// after its scan, from that cache rather than HBM (8192 x 8192: 1.21 ->
// 0.94 ms for both operands).  Each run writes its part of the full plane
// layout.  Columns of B: their exponent keys are cleared once (or, with
// keys_cleared, were cleared by A's scan on the side), each run's
// deconstruction reads the keys directly, and one launch turns all of them
// into tau at the end.  zero / nzero (side 0): keys to clear on the side.
hipError_t scan_and_deconstruct(ozaki25_moduli_set set, ozaki25_quantiser quant, int side, int64_t vecs,
                                int64_t k, const double* X, int64_t ldx, int t, int32_t* exps,
                                int8_t* planes, hipStream_t s, int32_t* zero = nullptr,
                                int64_t nzero = 0, bool keys_cleared = false) {
  const int64_t kp = k_pad(k);
  constexpr int64_t kRunBytes = (int64_t)256 << 20, kTile = 256;
  const int64_t per_run = kRunBytes / (kp * (int64_t)sizeof(double)) / kTile * kTile;
  const int64_t run = per_run > kTile ? per_run : kTile;
  hipError_t e = hipSuccess;
  if (side == 1 && !keys_cleared) e = oz::launch_clear_keys(vecs, exps, s);
  for (int64_t v0 = 0; v0 < vecs && e == hipSuccess; v0 += run) {
    const int64_t nv = vecs - v0 < run ? vecs - v0 : run;
    const double* Xr = side == 0 ? X + v0 * ldx : X + v0;
    if (side == 0) {
      // the first run's blocks also clear the keys (one per row: enough
      // when there are at least as many rows as keys / 256)
      const bool side_job = v0 == 0 && zero && (nzero + 255) / 256 <= nv;
      e = oz::launch_scan_rows(nv, k, Xr, ldx, t, exps + v0, side_job ? zero : nullptr,
                               side_job ? nzero : 0, s);
      if (e == hipSuccess && v0 == 0 && zero && !side_job) e = oz::launch_clear_keys(nzero, zero, s);
    } else {
      e = oz::launch_scan_cols(nv, k, Xr, ldx, exps + v0, s);
    }
    if (e == hipSuccess)
      e = oz::launch_deconstruct((int)set, (int)quant, side, nv, vecs, k, kp, t, Xr, ldx, exps + v0,
                                 side == 1, planes + v0 * oz::kKAlign, s);
  }
  if (side == 1 && e == hipSuccess) e = oz::launch_keys_to_sigma(vecs, t, exps, s);
  return e;
}

// ---- accurate mode (Sec. 2, Eq. (alpha)) ---------------------------------
// Scratch of the exponent stage: the digit planes of A and B, the totals L
// (int8 m x n), the column minima of each 64-row group of L, the column
// shifts as bytes, and the split bound product's partials.
struct AccWorkspace {
  size_t dig_a, dig_b, total, colpart, colslice, ub, part, bytes;
  int splits;
};

AccWorkspace acc_layout(int64_t m, int64_t n, int64_t k) {
  AccWorkspace w;
  const int64_t kp = k_pad(k);
  w.splits = oz::bound_gemm_splits(m, n, kp);
  size_t off = 0;
  w.dig_a = off;
  off = align_up(off + (size_t)m * kp);
  w.dig_b = off;
  off = align_up(off + (size_t)n * kp);
  w.total = off;
  off = align_up(off + (size_t)m * n);
  w.colpart = off;
  off = align_up(off + (size_t)((m + 63) / 64) * n);
  w.colslice = off;
  off = align_up(off + (size_t)(m > 0 && n > 0 ? oz::accurate_slices(m, n, nullptr) : 0) * n);
  w.ub = off;
  off = align_up(off + (size_t)n);
  w.part = off;
  off = w.splits > 1 ? align_up(off + (size_t)w.splits * m * n * sizeof(int32_t)) : off;
  w.bytes = off;
  return w;
}

// T = 2^8 (M/2 - 1): its bit length and its top 33 bits
void bound_limit(ozaki25_moduli_set set, int* bt, uint64_t* ttop) {
  u128 M = 1;
  for (int i = 0; i < num_moduli(set); ++i) M *= (u128)modulus(set, i);
  const u128 T = (M / 2 - 1) << 8;
  int b = 0;
  while (b < 128 && (T >> b) != 0) ++b;
  *bt = b;
  *ttop = (uint64_t)(T >> (b - 33));
}

// The accurate mode's exponents into ea / eb: the scans at t = 0 (A's row
// scan clears B's column keys on the side and writes A's magnitude digits),
// B's digits, the bound product and its totals, then the shifts.
hipError_t accurate_exponents(ozaki25_moduli_set set, int64_t m, int64_t n, int64_t k, const double* A,
                              int64_t lda, const double* B, int64_t ldb, int32_t* ea, int32_t* eb,
                              char* aux, const AccWorkspace& w, hipStream_t s) {
  const int64_t kp = k_pad(k);
  int8_t* da = (int8_t*)(aux + w.dig_a);
  int8_t* db = (int8_t*)(aux + w.dig_b);
  int8_t* total = (int8_t*)(aux + w.total);
  int8_t* colpart = (int8_t*)(aux + w.colpart);
  int8_t* colslice = (int8_t*)(aux + w.colslice);
  uint8_t* ub = (uint8_t*)(aux + w.ub);
  int32_t* part = w.splits > 1 ? (int32_t*)(aux + w.part) : nullptr;
  int bt = 0;
  uint64_t ttop = 0;
  bound_limit(set, &bt, &ttop);
  const bool side_job = (n + 255) / 256 <= m;
  // the row scan writes A's digits too
  hipError_t e =
      oz::launch_scan_rows(m, k, A, lda, 0, ea, side_job ? eb : nullptr, side_job ? n : 0, s, da, kp);
  if (e == hipSuccess && !side_job) e = oz::launch_clear_keys(n, eb, s);
  if (e == hipSuccess) e = oz::launch_scan_cols(n, k, B, ldb, eb, s);
  if (e == hipSuccess) e = oz::launch_digits(1, n, k, kp, B, ldb, eb, true, db, s);
  if (e == hipSuccess)
    e = oz::launch_bound_gemm(m, n, kp, da, db, total, colpart, part, w.splits, bt, ttop, s);
  if (e == hipSuccess) e = oz::launch_accurate_shifts(m, n, total, colpart, colslice, ub, ea, eb, s);
  return e;
}

// The accurate mode's shifts are at most 58: the deconstruction runs at that
// t (the residue route with one correction).
constexpr int kAccurateT = oz::kMaxScaleBits;

// The allocation-free entry point's workspace: one static array per GPU
// (each device's code object holds its own copy).  In host code `scratch`
// names a host-side stand-in, never the device memory: its device address is
// resolved per device with hipGetSymbolAddress and only that address is used.
constexpr size_t kNoallocBytes = OZAKI25_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kNoallocBytes];

constexpr int kMaxDevices = 256;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices];

// Device address of the current device's scratch array (resolved once per
// device, under a lock).
hipError_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p & (kAlign - 1))) return hipErrorInvalidSymbol;
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

const char* ozaki25_status_string(ozaki25_status s) {
  switch (s) {
    case OZAKI25_SUCCESS: return "success";
    case OZAKI25_ERR_INVALID_VALUE: return "invalid value";
    case OZAKI25_ERR_UNSUPPORTED: return "unsupported size (k or n beyond the library limits)";
    case OZAKI25_ERR_WORKSPACE: return "workspace too small or allocation failed";
    case OZAKI25_ERR_HIP: return "HIP runtime or launch error";
  }
  return "unknown status";
}

int ozaki25_num_moduli(ozaki25_moduli_set set) { return known_set(set) ? num_moduli(set) : -1; }

int ozaki25_num_planes(ozaki25_moduli_set set) { return known_set(set) ? num_planes(set) : -1; }

int64_t ozaki25_modulus(ozaki25_moduli_set set, int i) {
  return known_set(set) && i >= 0 && i < num_moduli(set) ? modulus(set, i) : -1;
}

int ozaki25_scale_bits(int64_t k, ozaki25_moduli_set set) {
  return known_set(set) ? scale_bits(k, set) : -1;
}

int64_t ozaki25_k_pad(int64_t k) { return k_pad(k); }

size_t ozaki25_planes_bytes(int64_t vecs, int64_t k, ozaki25_moduli_set set) {
  if (!known_set(set) || vecs < 0 || k < 0) return 0;
  return (size_t)num_planes(set) * (size_t)vecs * (size_t)k_pad(k);
}

ozaki25_status ozaki25_deconstruct(int side, int64_t vecs, int64_t k, const double* X, int64_t ldx,
                                   ozaki25_moduli_set set, ozaki25_quantiser quant,
                                   uint8_t* planes, int32_t* exps, void* stream) {
  if (!known_set(set) || !known_quantiser(quant) || (side != 0 && side != 1) || vecs < 0 || k < 0)
    return OZAKI25_ERR_INVALID_VALUE;
  if (k > OZAKI25_MAX_K) return OZAKI25_ERR_UNSUPPORTED;
  if (vecs == 0 || k == 0) return OZAKI25_SUCCESS;
  if (ldx < (side == 0 ? k : vecs)) return OZAKI25_ERR_INVALID_VALUE;
  if (!X || !planes || !exps) return OZAKI25_ERR_INVALID_VALUE;
  if (((uintptr_t)planes & 15) || ((uintptr_t)exps & 3) || ((uintptr_t)X & 7))
    return OZAKI25_ERR_INVALID_VALUE;
  return hip_status(scan_and_deconstruct(set, quant, side, vecs, k, X, ldx, scale_bits(k, set), exps,
                                          (int8_t*)planes, (hipStream_t)stream));
}

ozaki25_status ozaki25_residue_gemm(int64_t m, int64_t n, int64_t k, const uint8_t* planesA,
                                    const uint8_t* planesB, ozaki25_moduli_set set, int32_t* Cres,
                                    void* stream) {
  if (!known_set(set) || m < 0 || n < 0 || k < 0) return OZAKI25_ERR_INVALID_VALUE;
  if (k > OZAKI25_MAX_K || n > OZAKI25_MAX_N) return OZAKI25_ERR_UNSUPPORTED;
  if (m == 0 || n == 0) return OZAKI25_SUCCESS;
  if (!Cres || (k > 0 && (!planesA || !planesB))) return OZAKI25_ERR_INVALID_VALUE;
  if (((uintptr_t)planesA & 15) || ((uintptr_t)planesB & 15) || ((uintptr_t)Cres & 3))
    return OZAKI25_ERR_INVALID_VALUE;
  const int8_t *pa = (const int8_t*)planesA, *pb = (const int8_t*)planesB;
  hipStream_t s = (hipStream_t)stream;
  return hip_status(bytes_set(set) ? oz::launch_residue_gemm_bytes_i32(m, n, k_pad(k), pa, pb, Cres, s)
                                   : oz::launch_residue_gemm_i32(m, n, k_pad(k), pa, pb, Cres, s));
}

ozaki25_status ozaki25_reconstruct(int64_t m, int64_t n, const int32_t* Cres, const int32_t* expsA,
                                   const int32_t* expsB, ozaki25_moduli_set set, double* C,
                                   int64_t ldc, int subtract, void* stream) {
  if (!known_set(set) || m < 0 || n < 0) return OZAKI25_ERR_INVALID_VALUE;
  if (m == 0 || n == 0) return OZAKI25_SUCCESS;
  if (!Cres || !expsA || !expsB || !C || ldc < n) return OZAKI25_ERR_INVALID_VALUE;
  if (((uintptr_t)Cres & 3) || ((uintptr_t)expsA & 3) || ((uintptr_t)expsB & 3) || ((uintptr_t)C & 7))
    return OZAKI25_ERR_INVALID_VALUE;
  hipStream_t s = (hipStream_t)stream;
  const int sub = subtract ? 1 : 0;
  return hip_status(bytes_set(set)
                        ? oz::launch_reconstruct_bytes_i32(m, n, Cres, expsA, expsB, C, ldc, sub, s)
                        : oz::launch_reconstruct_i32(m, n, Cres, expsA, expsB, C, ldc, sub, s));
}

size_t ozaki25_dgemm_workspace_size(int64_t m, int64_t n, int64_t k, ozaki25_moduli_set set) {
  if (!known_set(set) || m < 0 || n < 0 || k < 0) return 0;
  return layout(m, n, k, set).total;
}

ozaki25_status ozaki25_dgemm_ex(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                const double* B, int64_t ldb, double* C, int64_t ldc,
                                ozaki25_moduli_set set, ozaki25_quantiser quant, int subtract,
                                void* workspace, size_t workspace_bytes,
                                void* const* stage_events, void* stream) {
  if (!known_set(set) || !known_quantiser(quant) || m < 0 || n < 0 || k < 0)
    return OZAKI25_ERR_INVALID_VALUE;
  if (k > OZAKI25_MAX_K || n > OZAKI25_MAX_N) return OZAKI25_ERR_UNSUPPORTED;
  if (m == 0 || n == 0) return OZAKI25_SUCCESS;
  if (!C || ldc < n || ((uintptr_t)C & 7)) return OZAKI25_ERR_INVALID_VALUE;
  if (k > 0) {
    if (!A || !B || lda < k || ldb < n || ((uintptr_t)A & 7) || ((uintptr_t)B & 7))
      return OZAKI25_ERR_INVALID_VALUE;
    const size_t cb = matrix_bytes(m, n, ldc);
    if (overlaps(A, matrix_bytes(m, k, lda), C, cb) || overlaps(B, matrix_bytes(k, n, ldb), C, cb))
      return OZAKI25_ERR_INVALID_VALUE;
  }
  hipStream_t s = (hipStream_t)stream;
  hipEvent_t* ev = (hipEvent_t*)stage_events;
  hipError_t e = hipSuccess;
  if (k == 0) {
    if (ev) e = hipEventRecord(ev[0], s);
    if (e == hipSuccess && !subtract) e = oz::launch_zero_c(m, n, C, ldc, s);
    for (int i = 1; ev && e == hipSuccess && i < OZAKI25_NUM_STAGE_EVENTS; ++i) e = hipEventRecord(ev[i], s);
    return hip_status(e);
  }

  const Workspace w = layout(m, n, k, set);
  void* ws = workspace;
  bool owned = false;
  if (ws) {
    if (workspace_bytes < w.total || ((uintptr_t)ws & (kAlign - 1))) return OZAKI25_ERR_WORKSPACE;
  } else {
    if (hipMallocAsync(&ws, w.total, s) != hipSuccess || !ws) return OZAKI25_ERR_WORKSPACE;
    owned = true;
  }
  char* base = (char*)ws;
  int8_t* pa = (int8_t*)(base + w.planes_a);
  int8_t* pb = (int8_t*)(base + w.planes_b);
  int32_t* ea = (int32_t*)(base + w.exps_a);
  int32_t* eb = (int32_t*)(base + w.exps_b);
  void* cres = base + w.cres;
  void* part = w.splits > 1 ? base + w.part : nullptr;
  const bool bytes = bytes_set(set);
  const int t = scale_bits(k, set);
  const int64_t kp = k_pad(k);

  if (ev) e = hipEventRecord(ev[0], s);
  if (fused_a(m, n, set)) {
    // storage mode F for A: its exponent scan (clearing B's column keys on
    // the side), B's scan and planes (for the published set B's scan only:
    // its digit planes come with the product), then the products straight
    // from FP64 A
    if (e == hipSuccess) e = oz::launch_scan_rows(m, k, A, lda, t, ea, eb, n, s);
    if (ev && e == hipSuccess) e = hipEventRecord(ev[1], s);
    if (bytes) {
      if (e == hipSuccess) e = scan_and_deconstruct(set, quant, 1, n, k, B, ldb, t, eb, pb, s, nullptr, 0, true);
    } else {
      if (e == hipSuccess) e = oz::launch_scan_cols(n, k, B, ldb, eb, s);
      if (e == hipSuccess) e = oz::launch_keys_to_sigma(n, t, eb, s);
    }
    if (ev && e == hipSuccess) e = hipEventRecord(ev[2], s);
    if (e == hipSuccess)
      e = bytes ? oz::launch_fused_bytes((int)quant, m, n, k, kp, t, A, lda, ea, pb, (int8_t*)cres, s)
                : oz::launch_fused_pub((int)quant, m, n, k, kp, t, A, lda, ea, B, ldb, eb, pb, (int16_t*)cres, s);
    if (ev && e == hipSuccess) e = hipEventRecord(ev[3], s);
    const oz::NativeOperands nat{A, lda, B, ldb, k};
    if (e == hipSuccess)
      e = bytes ? oz::launch_reconstruct_bytes_i8(m, n, (const int8_t*)cres, ea, eb, C, ldc, subtract ? 1 : 0, nat, s)
                : oz::launch_reconstruct_i16(m, n, (const int16_t*)cres, ea, eb, C, ldc, subtract ? 1 : 0, nat, s);
    if (ev && e == hipSuccess) e = hipEventRecord(ev[4], s);
    if (owned) {
      const hipError_t f = hipFreeAsync(ws, s);
      if (e == hipSuccess) e = f;
    }
    return hip_status(e);
  }
  // the scans run interleaved with the deconstruction (scan_and_deconstruct),
  // so the scan stage is empty and the deconstruct stage holds both
  if (ev && e == hipSuccess) e = hipEventRecord(ev[1], s);
  // A's row scan clears B's column keys on the side
  if (e == hipSuccess) e = scan_and_deconstruct(set, quant, 0, m, k, A, lda, t, ea, pa, s, eb, n);
  if (e == hipSuccess) e = scan_and_deconstruct(set, quant, 1, n, k, B, ldb, t, eb, pb, s, nullptr, 0, true);
  if (ev && e == hipSuccess) e = hipEventRecord(ev[2], s);
  if (e == hipSuccess)
    e = bytes ? oz::launch_residue_gemm_bytes_i8(m, n, kp, pa, pb, (int8_t*)cres, (int8_t*)part,
                                                 w.splits, s)
              : oz::launch_residue_gemm_i16(m, n, kp, pa, pb, (int16_t*)cres, (int16_t*)part,
                                            w.splits, s);
  if (ev && e == hipSuccess) e = hipEventRecord(ev[3], s);
  const int sub = subtract ? 1 : 0;
  // outputs on rows / columns flagged non-finite are re-issued natively
  const oz::NativeOperands nat{A, lda, B, ldb, k};
  if (e == hipSuccess)
    e = bytes ? oz::launch_reconstruct_bytes_i8(m, n, (const int8_t*)cres, ea, eb, C, ldc, sub, nat, s)
              : oz::launch_reconstruct_i16(m, n, (const int16_t*)cres, ea, eb, C, ldc, sub, nat, s);
  if (ev && e == hipSuccess) e = hipEventRecord(ev[4], s);
  if (owned) {
    const hipError_t f = hipFreeAsync(ws, s);
    if (e == hipSuccess) e = f;
  }
  return hip_status(e);
}

size_t ozaki25_accurate_exponents_workspace_size(int64_t m, int64_t n, int64_t k) {
  if (m < 0 || n < 0 || k < 0) return 0;
  return acc_layout(m, n, k).bytes;
}

ozaki25_status ozaki25_accurate_exponents(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                          const double* B, int64_t ldb, ozaki25_moduli_set set,
                                          int32_t* expsA, int32_t* expsB, void* workspace,
                                          size_t workspace_bytes, void* stream) {
  if (!known_set(set) || m < 0 || n < 0 || k < 0) return OZAKI25_ERR_INVALID_VALUE;
  if (k > OZAKI25_MAX_K || n > OZAKI25_MAX_N) return OZAKI25_ERR_UNSUPPORTED;
  if (m == 0 || n == 0 || k == 0) return OZAKI25_SUCCESS;
  if (!A || !B || !expsA || !expsB || lda < k || ldb < n) return OZAKI25_ERR_INVALID_VALUE;
  if (((uintptr_t)A & 7) || ((uintptr_t)B & 7) || ((uintptr_t)expsA & 3) || ((uintptr_t)expsB & 3))
    return OZAKI25_ERR_INVALID_VALUE;
  if (overlaps(expsA, (size_t)m * 4, expsB, (size_t)n * 4)) return OZAKI25_ERR_INVALID_VALUE;
  const AccWorkspace w = acc_layout(m, n, k);
  hipStream_t s = (hipStream_t)stream;
  void* ws = workspace;
  bool owned = false;
  if (ws) {
    if (workspace_bytes < w.bytes || ((uintptr_t)ws & (kAlign - 1))) return OZAKI25_ERR_WORKSPACE;
  } else {
    if (hipMallocAsync(&ws, w.bytes, s) != hipSuccess || !ws) return OZAKI25_ERR_WORKSPACE;
    owned = true;
  }
  hipError_t e = accurate_exponents(set, m, n, k, A, lda, B, ldb, expsA, expsB, (char*)ws, w, s);
  if (owned) {
    const hipError_t f = hipFreeAsync(ws, s);
    if (e == hipSuccess) e = f;
  }
  return hip_status(e);
}

size_t ozaki25_dgemm_accurate_workspace_size(int64_t m, int64_t n, int64_t k, ozaki25_moduli_set set) {
  if (!known_set(set) || m < 0 || n < 0 || k < 0) return 0;
  return layout(m, n, k, set).total + acc_layout(m, n, k).bytes;
}

ozaki25_status ozaki25_dgemm_accurate(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                      const double* B, int64_t ldb, double* C, int64_t ldc,
                                      ozaki25_moduli_set set, ozaki25_quantiser quant, int subtract,
                                      void* workspace, size_t workspace_bytes,
                                      void* const* stage_events, void* stream) {
  if (!known_set(set) || !known_quantiser(quant) || m < 0 || n < 0 || k < 0)
    return OZAKI25_ERR_INVALID_VALUE;
  if (k > OZAKI25_MAX_K || n > OZAKI25_MAX_N) return OZAKI25_ERR_UNSUPPORTED;
  if (m == 0 || n == 0) return OZAKI25_SUCCESS;
  if (!C || ldc < n || ((uintptr_t)C & 7)) return OZAKI25_ERR_INVALID_VALUE;
  // k == 0 needs no scaling: C = +0 (or unchanged), as in the fast mode
  if (k == 0)
    return ozaki25_dgemm_ex(m, n, k, A, lda, B, ldb, C, ldc, set, quant, subtract, nullptr, 0, stage_events,
                            stream);
  if (!A || !B || lda < k || ldb < n || ((uintptr_t)A & 7) || ((uintptr_t)B & 7))
    return OZAKI25_ERR_INVALID_VALUE;
  const size_t cb = matrix_bytes(m, n, ldc);
  if (overlaps(A, matrix_bytes(m, k, lda), C, cb) || overlaps(B, matrix_bytes(k, n, ldb), C, cb))
    return OZAKI25_ERR_INVALID_VALUE;

  const Workspace w = layout(m, n, k, set);
  const AccWorkspace aw = acc_layout(m, n, k);
  const size_t need = w.total + aw.bytes;
  hipStream_t s = (hipStream_t)stream;
  hipEvent_t* ev = (hipEvent_t*)stage_events;
  void* ws = workspace;
  bool owned = false;
  if (ws) {
    if (workspace_bytes < need || ((uintptr_t)ws & (kAlign - 1))) return OZAKI25_ERR_WORKSPACE;
  } else {
    if (hipMallocAsync(&ws, need, s) != hipSuccess || !ws) return OZAKI25_ERR_WORKSPACE;
    owned = true;
  }
  char* base = (char*)ws;
  int8_t* pa = (int8_t*)(base + w.planes_a);
  int8_t* pb = (int8_t*)(base + w.planes_b);
  int32_t* ea = (int32_t*)(base + w.exps_a);
  int32_t* eb = (int32_t*)(base + w.exps_b);
  void* cres = base + w.cres;
  void* part = w.splits > 1 ? base + w.part : nullptr;
  const bool bytes = bytes_set(set);
  const bool fused = fused_a(m, n, set);
  const int64_t kp = k_pad(k);
  const int sub = subtract ? 1 : 0;
  const oz::NativeOperands nat{A, lda, B, ldb, k};

  hipError_t e = hipSuccess;
  if (ev) e = hipEventRecord(ev[0], s);
  if (e == hipSuccess) e = accurate_exponents(set, m, n, k, A, lda, B, ldb, ea, eb, base + w.total, aw, s);
  if (ev && e == hipSuccess) e = hipEventRecord(ev[1], s);
  if (e == hipSuccess && !fused)
    e = oz::launch_deconstruct((int)set, (int)quant, 0, m, m, k, kp, kAccurateT, A, lda, ea, false, pa, s);
  // (the published set's fused product makes B's digit planes itself)
  if (e == hipSuccess && (bytes || !fused))
    e = oz::launch_deconstruct((int)set, (int)quant, 1, n, n, k, kp, kAccurateT, B, ldb, eb, false, pb, s);
  if (ev && e == hipSuccess) e = hipEventRecord(ev[2], s);
  if (e == hipSuccess) {
    if (fused && bytes)
      e = oz::launch_fused_bytes((int)quant, m, n, k, kp, kAccurateT, A, lda, ea, pb, (int8_t*)cres, s);
    else if (fused)
      e = oz::launch_fused_pub((int)quant, m, n, k, kp, kAccurateT, A, lda, ea, B, ldb, eb, pb, (int16_t*)cres, s);
    else if (bytes)
      e = oz::launch_residue_gemm_bytes_i8(m, n, kp, pa, pb, (int8_t*)cres, (int8_t*)part, w.splits, s);
    else
      e = oz::launch_residue_gemm_i16(m, n, kp, pa, pb, (int16_t*)cres, (int16_t*)part, w.splits, s);
  }
  if (ev && e == hipSuccess) e = hipEventRecord(ev[3], s);
  if (e == hipSuccess)
    e = bytes ? oz::launch_reconstruct_bytes_i8(m, n, (const int8_t*)cres, ea, eb, C, ldc, sub, nat, s)
              : oz::launch_reconstruct_i16(m, n, (const int16_t*)cres, ea, eb, C, ldc, sub, nat, s);
  if (ev && e == hipSuccess) e = hipEventRecord(ev[4], s);
  if (owned) {
    const hipError_t f = hipFreeAsync(ws, s);
    if (e == hipSuccess) e = f;
  }
  return hip_status(e);
}

size_t ozaki25_dgemm_planes_workspace_size(int64_t m, int64_t n, int64_t k, ozaki25_moduli_set set) {
  if (!known_set(set) || m < 0 || n < 0 || k < 0) return 0;
  return products_bytes(m, n, k, set, nullptr);
}

ozaki25_status ozaki25_dgemm_planes(int64_t m, int64_t n, int64_t k, const uint8_t* planesA,
                                    const int32_t* expsA, const uint8_t* planesB,
                                    const int32_t* expsB, double* C, int64_t ldc,
                                    ozaki25_moduli_set set, int subtract, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  if (!known_set(set) || m < 0 || n < 0 || k < 0) return OZAKI25_ERR_INVALID_VALUE;
  if (k > OZAKI25_MAX_K || n > OZAKI25_MAX_N) return OZAKI25_ERR_UNSUPPORTED;
  if (m == 0 || n == 0) return OZAKI25_SUCCESS;
  if (!C || ldc < n || ((uintptr_t)C & 7)) return OZAKI25_ERR_INVALID_VALUE;
  hipStream_t s = (hipStream_t)stream;
  if (k == 0) return hip_status(subtract ? hipSuccess : oz::launch_zero_c(m, n, C, ldc, s));
  if (!planesA || !planesB || !expsA || !expsB) return OZAKI25_ERR_INVALID_VALUE;
  if (((uintptr_t)planesA & 15) || ((uintptr_t)planesB & 15) || ((uintptr_t)expsA & 3) ||
      ((uintptr_t)expsB & 3))
    return OZAKI25_ERR_INVALID_VALUE;
  int splits = 1;
  const size_t need = products_bytes(m, n, k, set, &splits);
  void* ws = workspace;
  bool owned = false;
  if (ws) {
    if (workspace_bytes < need || ((uintptr_t)ws & (kAlign - 1))) return OZAKI25_ERR_WORKSPACE;
  } else {
    if (hipMallocAsync(&ws, need, s) != hipSuccess || !ws) return OZAKI25_ERR_WORKSPACE;
    owned = true;
  }
  const int64_t kp = k_pad(k);
  const int8_t *pa = (const int8_t*)planesA, *pb = (const int8_t*)planesB;
  const int sub = subtract ? 1 : 0;
  hipError_t e;
  const size_t one = align_up((size_t)num_moduli(set) * m * n * cres_elem(set));
  char* part = splits > 1 ? (char*)ws + one : nullptr;
  if (bytes_set(set)) {
    int8_t* cres = (int8_t*)ws;
    e = oz::launch_residue_gemm_bytes_i8(m, n, kp, pa, pb, cres, (int8_t*)part, splits, s);
    if (e == hipSuccess)
      e = oz::launch_reconstruct_bytes_i8(m, n, cres, expsA, expsB, C, ldc, sub, oz::NativeOperands{}, s);
  } else {
    int16_t* cres = (int16_t*)ws;
    e = oz::launch_residue_gemm_i16(m, n, kp, pa, pb, cres, (int16_t*)part, splits, s);
    if (e == hipSuccess)
      e = oz::launch_reconstruct_i16(m, n, cres, expsA, expsB, C, ldc, sub, oz::NativeOperands{}, s);
  }
  if (owned) {
    const hipError_t f = hipFreeAsync(ws, s);
    if (e == hipSuccess) e = f;
  }
  return hip_status(e);
}

ozaki25_status ozaki25_dgemm_noalloc(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                     const double* B, int64_t ldb, double* C, int64_t ldc,
                                     ozaki25_moduli_set set, ozaki25_quantiser quant, int subtract,
                                     void* stream) {
  if (!known_set(set) || !known_quantiser(quant) || m < 0 || n < 0 || k < 0)
    return OZAKI25_ERR_INVALID_VALUE;
  if (k > OZAKI25_MAX_K || n > OZAKI25_MAX_N) return OZAKI25_ERR_UNSUPPORTED;
  if (m == 0 || n == 0) return OZAKI25_SUCCESS;
  // k == 0 fills (or keeps) C without a workspace: ozaki25_dgemm_ex returns
  // before its allocation
  if (k == 0)
    return ozaki25_dgemm_ex(m, n, k, A, lda, B, ldb, C, ldc, set, quant, subtract, nullptr, 0, nullptr,
                            stream);
  if (layout(m, n, k, set).total > kNoallocBytes) return OZAKI25_ERR_WORKSPACE;
  void* ws = nullptr;
  if (scratch_address(&ws) != hipSuccess) return OZAKI25_ERR_HIP;
  return ozaki25_dgemm_ex(m, n, k, A, lda, B, ldb, C, ldc, set, quant, subtract, ws, kNoallocBytes,
                          nullptr, stream);
}

ozaki25_status ozaki25_dgemm(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                             const double* B, int64_t ldb, double* C, int64_t ldc,
                             ozaki25_moduli_set set, void* stream) {
  return ozaki25_dgemm_ex(m, n, k, A, lda, B, ldb, C, ldc, set, OZAKI25_QUANT_RN, 0, nullptr, 0,
                          nullptr, stream);
}

ozaki25_status ozaki25_dgemm_sub(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                                 const double* B, int64_t ldb, double* C, int64_t ldc,
                                 ozaki25_moduli_set set, void* stream) {
  return ozaki25_dgemm_ex(m, n, k, A, lda, B, ldb, C, ldc, set, OZAKI25_QUANT_RN, 1, nullptr, 0,
                          nullptr, stream);
}

}  // extern "C"
