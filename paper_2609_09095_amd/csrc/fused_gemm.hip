// Storage mode F for A in tall/skinny products (Alg. 1's storage modes,
// Sec. 6.2: the hybrid of a materialised small operand and a streamed large
// one), all-byte set: B's residue planes are stored once, while A is read
// as FP64 inside the product kernel -- scaled by 2^sigma, quantised and
// reduced to its byte residues per K stage (Eq. (scale), Alg. 2) straight
// into LDS, never written to HBM as planes.  For at most 128 columns one
// output tile spans all of B (lambda_A = 1: every element of A is converted
// once per modulus it serves).
//
// A block owns 128 rows of A, all (at most 128) columns and G moduli; its
// 8 wavefronts convert a 128 x 64 slab per stage (coalesced: 16 lanes per
// row, 4 consecutive k each), then multiply it with B's slabs on v_mfma_i32_32x32x32_i8
// (64 x 32 outputs per wavefront), the next slab's FP64 loads in flight
// meanwhile.  The blocks of one row strip (15 / G of them) are dealt to the
// same XCD back to back, so the strip's FP64 comes from HBM once and from
// that XCD's L2 for the others.
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int FBN = 128;   // columns of B (all of them)
constexpr int FBK = 64;    // k per stage
constexpr int kSegF = 1024;  // stages (65536 k) between reductions of the int32 sums
// residue bytes in [-128, 127]: products up to 2^14 in magnitude; the sums of
// kSegF stages, plus the largest value a reduction leaves, fit in int32
static_assert((int64_t)kSegF * FBK * 128 * 128 + 128 < (int64_t)INT32_MAX, "int32 sums exact between reductions");

__constant__ int kModF[kRA] = {kModulusA[0],  kModulusA[1],  kModulusA[2],  kModulusA[3],
                               kModulusA[4],  kModulusA[5],  kModulusA[6],  kModulusA[7],
                               kModulusA[8],  kModulusA[9],  kModulusA[10], kModulusA[11],
                               kModulusA[12], kModulusA[13], kModulusA[14]};
// RN(1/m) for the quotient route; 0 for m = 256, whose residue
// byte is the low byte of y itself
__constant__ double kInvQ[kRA] = {
    0.0,                 1.0 / kModulusA[1],  1.0 / kModulusA[2],  1.0 / kModulusA[3],
    1.0 / kModulusA[4],  1.0 / kModulusA[5],  1.0 / kModulusA[6],  1.0 / kModulusA[7],
    1.0 / kModulusA[8],  1.0 / kModulusA[9],  1.0 / kModulusA[10], 1.0 / kModulusA[11],
    1.0 / kModulusA[12], 1.0 / kModulusA[13], 1.0 / kModulusA[14]};
static_assert(kModulusA[0] == 256, "the power of two comes first");
// RN(1/m) for the reductions of the int32 sums
__constant__ double kInvF[kRA] = {
    1.0 / kModulusA[0],  1.0 / kModulusA[1],  1.0 / kModulusA[2],  1.0 / kModulusA[3],
    1.0 / kModulusA[4],  1.0 / kModulusA[5],  1.0 / kModulusA[6],  1.0 / kModulusA[7],
    1.0 / kModulusA[8],  1.0 / kModulusA[9],  1.0 / kModulusA[10], 1.0 / kModulusA[11],
    1.0 / kModulusA[12], 1.0 / kModulusA[13], 1.0 / kModulusA[14]};

constexpr double kMagicF = 6755399441055744.0;  // 1.5 * 2^52
__device__ __forceinline__ uint32_t lo32(double v) { return (uint32_t)__builtin_bit_cast(uint64_t, v); }

// y mod 2^32 of an integer-valued y with |y| <= 2^52, where y + 1.5 2^52 is
// no longer exact: h = floor(y 2^-32) (the scaling is exact), y - h 2^32 in
// [0, 2^32) by one exact FMA, converted.
__device__ __forceinline__ uint32_t low32_split(double y) {
  const double h = __builtin_floor(y * 0x1p-32);
  return (uint32_t)__builtin_fma(-h, 0x1p32, y);
}

// The centred residue of the integer-valued y modulo M, modulo 2^8 (its low
// byte is the two's complement byte; the higher bits are not defined), with
// ylo = y mod 2^32.  The FMA rounds y RN(1/M) + 1.5 2^52 once to
// 1.5 2^52 + q (|y / M| < 2^51: the sum lies where the spacing is 1), and
// |y RN(1/M) - y/M| <= |y| 2^-61 for the odd M <= 255.
//  CORR false (|y| <= 2^52): that error is at most 2^-9, below the
//  1/(2M) >= 1/510 that separates y/M from a half integer, so q is the
//  nearest quotient and ylo - q M = y - q M (mod 2^32) is the centred
//  residue, |r| < 128, whose low byte is the two's complement byte.
//  CORR true (|y| <= 2^58): the error is at most 1/8, so |y - q M| <= 5M/8
//  and one correction each way centres it (24 bits hold it exactly).
// For M = 256 (RN(1/M) taken as 0) q = 0 and the low byte of y is the
// residue byte; the corrections move it by multiples of 256, which leaves
// that byte alone.  24-bit products suffice.
template <bool CORR>
__device__ __forceinline__ uint32_t residue_byte(double y, uint32_t ylo, int M, double qinv) {
  const uint32_t q = lo32(__builtin_fma(y, qinv, kMagicF));
  // spelled out: left to itself the compiler uses a quarter-rate 32-bit
  // multiply; sext24(q) (-M) + ylo is y - q M modulo 2^24
  uint32_t r;
  asm("v_mad_i32_i24 %0, %1, %2, %3" : "=v"(r) : "v"(q), "s"(-M), "v"(ylo));
  if constexpr (CORR) {
    const int hi = (M - 1) / 2;
    int c = (int)(r << 8) >> 8;
    c = c > hi ? c - M : c;
    c = c < hi - M + 1 ? c + M : c;
    return (uint32_t)c;
  }
  return r;  // the caller keeps the low byte
}

// LDS slabs: rows of 64 bytes (one stage), the 16-byte chunk index XOR-ed
// with bits 1-2 of the row and then with bit 3, so that the fragment reads
// at one chunk of 8 consecutive rows (128 bytes a cycle) and of 16 (256
// bytes a cycle) hit distinct 16-byte bank groups.
__device__ __forceinline__ int fswz(int row) { return ((row >> 1) & 3) ^ ((row >> 3) & 1); }

// int8 fragment of a 32-row block for one 32-byte K step of a 64-byte stage:
// lane half fh takes chunk 2 ks + fh of its row
__device__ __forceinline__ v4i ffrag(const int8_t* base, int r, int ks, int fh) {
  return *reinterpret_cast<const v4i*>(base + r * FBK + (((2 * ks + fh) ^ fswz(r)) << 4));
}

__device__ __forceinline__ const int8_t* uniform_ptr_f(const int8_t* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const int8_t*)(((uint64_t)hi << 32) | lo);
}

using lds_ptr_f = __attribute__((address_space(3))) void*;

// The lane index, computed afresh where it is used. Both fused kernels run
// at the register limit, and a lane offset held across the k loop is
// spilled; its reload from scratch waits on the vector-memory counter and
// so drains the look-ahead loads with it. A volatile asm is neither hoisted
// nor merged.
__device__ __forceinline__ int lane_now() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// End of a pipeline stage. Each wave waits for its own LDS writes and its
// LDS-DMA, then the workgroup meets at the barrier. When keep_a is set, the
// last four vector loads (A's FP64 values for the stage after next, issued
// after the DMA) may stay outstanding: vmcnt(4) expcnt(0) lgkmcnt(0). Any
// other load path issues at least four loads there, and the counter retires
// in issue order. The barrier is a bare instruction behind a compiler memory
// barrier, because the release fence of __syncthreads() drains every
// outstanding vector load.
__device__ __forceinline__ void stage_barrier(bool keep_a) {
  if (keep_a)
    __builtin_amdgcn_s_waitcnt(0x0004);
  else
    __builtin_amdgcn_s_waitcnt(0);
  asm volatile("s_barrier" ::: "memory");
}

// Centred residue of an int32 sum modulo m (as cmod_i32 in the residue GEMM).
__device__ __forceinline__ int cmod_sum(int x, int m, double minv) {
  const double xd = (double)x;
  const double q = __builtin_rint(xd * minv);
  return (int)__builtin_fma(-q, (double)m, xd);
}

// 128 rows of A per block, 16 wavefronts: wavefront w converts rows
// 8 w .. 8 w + 7 of each slab and owns the 32 x 32 outputs (w / 4, w % 4) of
// every modulus of its group (one MFMA block each, so that G = 5 moduli fit
// the registers: the FP64 slab then feeds five times the matrix work).
constexpr int FBM = 128;
// MODE: the residue route by the range of y -- 1: ylo = y + 1.5 2^52
// (|y| <= 2^51); 2: ylo by low32_split (|y| <= 2^52); 3: low32_split and the
// corrected quotient (|y| <= 2^58).
template <int G, int MODE, bool TZ, bool VEC>
__global__ __launch_bounds__(1024, 1) void fused_bytes_kernel(
    int64_t m, int64_t n, int64_t k, int64_t kp, const double* __restrict__ A, int64_t lda,
    const int32_t* __restrict__ sigma, const int8_t* __restrict__ pb, int8_t* __restrict__ cres,
    int64_t strips) {
  static_assert(kRA % G == 0, "modulus groups");
  constexpr int NG = kRA / G;
  // two buffers of each, every buffer its own LDS object: the compiler then
  // tells the buffer that LDS-DMA fills from the one being read, and does
  // not wait for the DMA before the reads
  __shared__ __attribute__((aligned(1024))) int8_t lds_a0[G][FBM * FBK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_a1[G][FBM * FBK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b0[G][FBN * FBK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b1[G][FBN * FBK];
  // block -> (strip, group): the NG blocks of a strip go to one XCD (block b
  // runs on XCD b % 8), one after the other
  const uint32_t b = blockIdx.x, o = b >> 3;
  const int64_t strip = (int64_t)(o / NG) * 8 + (b & 7);
  const int grp = (int)(o % NG);
  if (strip >= strips) return;
  const int64_t row0 = strip * FBM;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave >> 2, wc = wave & 3;  // 4 x 4 wavefronts of 32 x 32 outputs
  const int fr = lane & 31, fh = lane >> 5;

  // conversion: lane l takes 4 consecutive k (4 (l % 16) ..) of row
  // 8 wave + 4 i + l / 16, i = 0, 1: 16 lanes sweep a row's 512 bytes
  const int ck = 4 * (lane & 15);
  int sg[2];
  uint32_t keep[2];  // all ones for a live row, 0 past m or for a non-finite row
  const double* arow_p[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = 8 * wave + 4 * i + (lane >> 4);
    const int64_t arow = row0 + r;
    const bool ok = arow < m;
    const int sv = ok ? sigma[arow] : 0;
    const bool live = ok && sv != INT32_MIN;
    keep[i] = live ? 0xFFFFFFFFu : 0u;
    sg[i] = live ? sv : 0;
    arow_p[i] = A + (ok ? arow : m - 1) * lda;
  }

  int mods[G];
  double qinv[G], inv[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    mods[g] = kModF[grp * G + g];
    qinv[g] = kInvQ[grp * G + g];
    inv[g] = kInvF[grp * G + g];
  }

  const int nstage = (int)(kp / FBK);
  // two register sets x0, x1: stage j's values live in x(j % 2), loaded two
  // stages ahead; x[4 i + c] is row 8 wave + 4 i + lane / 16, k = ck + c
  double x0[8], x1[8];
  // x holds the raw values (rows past m or holding a NaN or an infinity,
  // and k past the end, are masked after the conversion); whole stages take
  // the 16-byte loads, the last, partial one clamped single loads; full:
  // stage s is known to lie inside k
  auto load_a = [&](int s, double (&x)[8], bool full) __attribute__((always_inline)) {
    const int64_t k0 = (int64_t)s * FBK + 4 * (lane_now() & 15);
    if (VEC && (full || (int64_t)s * FBK + FBK <= k)) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const double2 p = *reinterpret_cast<const double2*>(arow_p[i] + k0);
        const double2 q = *reinterpret_cast<const double2*>(arow_p[i] + k0 + 2);
        x[4 * i] = p.x;
        x[4 * i + 1] = p.y;
        x[4 * i + 2] = q.x;
        x[4 * i + 3] = q.y;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          // clamped into the row; convert zeroes the digits past k
          x[4 * i + c] = arow_p[i][k0 + c < k ? k0 + c : k - 1];
        }
    }
  };
  // one dword (4 residue bytes) per row and modulus, written at chunk
  // ck / 16 of the row, swizzled
  auto convert = [&](int buf, const double (&x)[8], int t) __attribute__((always_inline)) {
    // byte c of a digit word is element k0 + c: the bytes at or past k of
    // the last (partial) stage t are cleared with the dead rows'
    uint32_t kmask = 0xFFFFFFFFu;
    if ((int64_t)(t + 1) * FBK > k) {
      const int64_t rem = k - ((int64_t)t * FBK + ck);
      kmask = rem >= 4 ? 0xFFFFFFFFu : rem <= 0 ? 0u : 0xFFFFFFFFu >> (32 - 8 * (int)rem);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = 8 * wave + 4 * i + (lane >> 4);
      double y[4];
      uint32_t ylo[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const double v = __builtin_ldexp(x[4 * i + c], sg[i]);
        y[c] = TZ ? __builtin_trunc(v) : __builtin_rint(v);
        ylo[c] = MODE == 1 ? lo32(y[c] + kMagicF) : low32_split(y[c]);
      }
      const int at = r * FBK + (((ck >> 4) ^ fswz(r)) << 4) + (ck & 15);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        // low bytes of the four residues into one dword (v_perm_b32: bytes
        // 0-3 of the second operand, 4-7 of the first)
        const uint32_t r01 =
            __builtin_amdgcn_perm(residue_byte<MODE == 3>(y[1], ylo[1], mods[g], qinv[g]),
                                  residue_byte<MODE == 3>(y[0], ylo[0], mods[g], qinv[g]), 0x0c0c0400u);
        const uint32_t r23 =
            __builtin_amdgcn_perm(residue_byte<MODE == 3>(y[3], ylo[3], mods[g], qinv[g]),
                                  residue_byte<MODE == 3>(y[2], ylo[2], mods[g], qinv[g]), 0x0c0c0400u);
        const uint32_t word = __builtin_amdgcn_perm(r23, r01, 0x05040100u);
        *reinterpret_cast<uint32_t*>(&(buf ? lds_a1 : lds_a0)[g][at]) = word & (keep[i] & kmask);
      }
    }
  };
  // B's slabs of stage s: for each of the G moduli, 128 rows x 64 bytes,
  // by LDS-DMA (eight 1 KiB loads per modulus, spread over the wavefronts):
  // lane l lands at row 16 d + l / 4, physical chunk l % 4, and fetches
  // the global chunk that the swizzle puts there; columns past n read zero.
  const int brecs = __builtin_amdgcn_readfirstlane((int)(n * 128));
  auto load_b = [&](int s, int buf) __attribute__((always_inline)) {
    const int64_t kb = s >> 1, h = s & 1;
    for (int d = wave; d < 8 * G; d += 16) {
      const int g = d >> 3, dd = d & 7;
      const int mod = grp * G + g;
      const int8_t* piece = uniform_ptr_f(pb + ((kb * kRA + mod) * n) * 128 + h * 64);
      const __amdgpu_buffer_rsrc_t rs =
          __builtin_amdgcn_make_buffer_rsrc((void*)piece, (short)0, brecs, 0x00020000);
      const int row = 16 * dd + (lane >> 2);
      const int gchunk = (lane & 3) ^ fswz(row);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_f)(&(buf ? lds_b1 : lds_b0)[g][16 * dd * FBK]), 16,
                                               row * 128 + gchunk * 16, 0, 0, 0);
    }
  };

  v16i acc[G];
#pragma unroll
  for (int g = 0; g < G; ++g) acc[g] = v16i{};

  // stage s: the loads of stage s + 2 go out, the MFMAs of stage s run on
  // the LDS buffers cur = s % 2, and stage s + 1 (loaded during stage
  // s - 1) is converted into the other buffers.
  // inner: a stage of the main loop, whose next stage exists and whose
  // look-ahead stage lies inside k. The look-ahead there is unconditional
  // and takes one load path, so that the compiler sees every look-ahead
  // register consumed and keeps the loads in flight across the barrier.
  // B's DMA goes out before A's loads, so that the end-of-stage wait can
  // leave the latter outstanding.
  auto step = [&](int s, double (&xs)[8], double (&xn)[8], int cur, bool inner)
                  __attribute__((always_inline)) {
    const int nxt = cur ^ 1;
    const bool next = inner || s + 1 < nstage;
    const bool more = inner || s + 2 < nstage;
    if (next) load_b(s + 1, nxt);
    if (more) load_a(s + 2, xs, inner);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int8_t* la = (cur ? lds_a1 : lds_a0)[g];
      const int8_t* lb = (cur ? lds_b1 : lds_b0)[g];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        acc[g] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ffrag(la, wr * 32 + fr, ks, fh),
                                                       ffrag(lb, wc * 32 + fr, ks, fh), acc[g], 0, 0, 0);
      // one modulus's fragments at a time in registers
      __builtin_amdgcn_sched_barrier(0);
    }
    if (next) convert(nxt, xn, s + 1);
    if (((s + 1) % kSegF) == 0 && next) {
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[g][v] = cmod_sum(acc[g][v], mods[g], inv[g]);
    }
    stage_barrier(more);
  };

  if (nstage > 0) {
    load_a(0, x0, false);
    load_b(0, 0);
    if (nstage > 1) load_a(1, x1, false);
    convert(0, x0, 0);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // the main loop runs while both look-ahead stages are full; the last
  // (at most four) stages take the guarded steps
  const int nfull = (int)(k / FBK);
  int s = 0;
  for (; s + 3 < nfull; s += 2) {
    step(s, x0, x1, 0, true);
    step(s + 1, x1, x0, 1, true);
  }
  for (; s < nstage; s += 2) {
    step(s, x0, x1, 0, false);
    if (s + 1 < nstage) step(s + 1, x1, x0, 1, false);
  }

  // epilogue: centred residues (+m/2 of m = 256 stores as -128), int8, into
  // the compact [15][m][n] layout of the materialised path
  const int64_t col = wc * 32 + fr;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    int8_t* out = cres + (int64_t)(grp * G + g) * m * n;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int64_t row = row0 + wr * 32 + 8 * (v >> 2) + 4 * fh + (v & 3);
      if (row < m && col < n) out[row * n + col] = (int8_t)cmod_sum(acc[g][v], mods[g], inv[g]);
    }
  }
}

template <int G, int MODE, bool TZ>
hipError_t launch_fused_g(int64_t m, int64_t n, int64_t k, int64_t kp, const double* A, int64_t lda,
                          const int32_t* sigma, const int8_t* pb, int8_t* cres, hipStream_t stream) {
  const int64_t strips = (m + FBM - 1) / FBM;
  const int64_t blocks = (strips + 7) / 8 * 8 * (kRA / G);
  if (blocks > (int64_t)UINT32_MAX) return hipErrorInvalidValue;
  // 16-byte loads when every row starts 16-byte aligned
  if ((((uintptr_t)A) & 15) == 0 && (lda & 1) == 0)
    hipLaunchKernelGGL((fused_bytes_kernel<G, MODE, TZ, true>), dim3((unsigned)blocks), dim3(1024), 0,
                       stream, m, n, k, kp, A, lda, sigma, pb, cres, strips);
  else
    hipLaunchKernelGGL((fused_bytes_kernel<G, MODE, TZ, false>), dim3((unsigned)blocks), dim3(1024), 0,
                       stream, m, n, k, kp, A, lda, sigma, pb, cres, strips);
  return hipGetLastError();
}

// ---- published set (twelve moduli) on FP8 and FP16 MFMA ---------------------
// The same storage mode F for the published moduli, in six pairs: square g
// (m = s^2) and nonsquare 6 + g.  Operands, every one exact in its format:
//  - square: the balanced base-s digits (d0, d1) of the centred residue x,
//    x = d0 + s d1, |d0|, |d1| <= 16, as e4m3; mod s^2 the product is
//    d0 e0 + s (d0 e1 + d1 e0) (d1 e1 carries the factor s^2), summed in two
//    FP32 accumulator sets (weights 1 and s) on FP8 MFMA;
//  - nonsquare (m <= 511): the centred residue itself, |x| <= 255, as fp16,
//    one product x y per k on FP16 MFMA into one FP32 set.
// Every partial sum is an integer kept below 2^24: per k the nonsquare
// products reach 255^2, so that set is reduced every kSegN = 4 stages (256
// k: 16 646 400, plus at most 256 left by the last reduction); the square
// sets (at most 256 and 512 per k) every kSegS stages.  The outputs are the
// compact residues of the published set's product path (the true ones times
// compact_scale(i)^-1 mod m_i, |c| <= 0.51 m_i), so its reconstruction takes
// them as they stand.  B's operands come from fused_b_digits_kernel in
// [kp/128][24][n][128] bytes: planes 2 g, 2 g + 1 hold square g's digits
// (the 128 k of the block, one byte each); planes 12 + 2 g + h hold
// nonsquare 6 + g's residues for k 64 h .. 64 h + 63 of the block (fp16, in
// k order).

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef __fp16 h2x __attribute__((ext_vector_type(2)));

constexpr int kPairs = 6;
constexpr int kSegS = 256;  // stages between reductions of the square sets
constexpr int kSegN = 4;    // stages between reductions of the nonsquare set
// exact FP32 sums: the products' magnitudes summed over the stages between
// reductions, plus the largest value a reduction leaves, stay below 2^24
static_assert((int64_t)kSegS * FBK * 512 + 1089 < (1 << 24), "square sets exact between reductions");
static_assert((int64_t)kSegN * FBK * 255 * 255 + 256 < (1 << 24), "nonsquare set exact between reductions");
static_assert((kSegN & (kSegN - 1)) == 0, "the stage test masks");

struct PairConst {
  int ms, s, mn;         // square modulus, its root, nonsquare modulus
  double qs, qn;         // RN(1/m) for the quotient route
  float is, ims, imn;    // RN(1/s), RN(1/ms), RN(1/mn)
  float inv16;           // 16^-1 mod mn
};
constexpr PairConst make_pair(int g) {
  return PairConst{kModulus[g],
                   root_of(g),
                   kModulus[kPairs + g],
                   1.0 / kModulus[g],
                   1.0 / kModulus[kPairs + g],
                   1.0f / (float)root_of(g),
                   1.0f / (float)kModulus[g],
                   1.0f / (float)kModulus[kPairs + g],
                   (float)inverse_mod(16, kModulus[kPairs + g])};
}
constexpr bool pairs_are_square_nonsquare() {
  for (int g = 0; g < kPairs; ++g)
    if (!root_of(g) || root_of(kPairs + g) || root_of(g) > 33 || kModulus[kPairs + g] > 511) return false;
  return true;
}
static_assert(kR == 2 * kPairs && pairs_are_square_nonsquare(),
              "six squares (s <= 33) first, then six nonsquares below 512");
static_assert(compact_scale(0) == 1 && compact_scale(kPairs) == 16, "compact scales of the product path");
__constant__ PairConst kPair[kPairs] = {make_pair(0), make_pair(1), make_pair(2),
                                        make_pair(3), make_pair(4), make_pair(5)};

// Centred residue of the integer-valued y modulo M (ylo = y mod 2^32), as a
// 24-bit signed value: the FMA quotient of y RN(1/M) + 1.5 2^52 (exact
// for M = 1024) and one 24-bit multiply-add.  MODE 1 (|y| <= 2^51): the
// quotient is the nearest one (|y| ulp(1/M) / 2 <= 2^-11 for these moduli,
// below the 1/(2M) that separates y/M from a half integer; for M = 1024 a
// tie may give +512, as good a representative).  MODE 3 (|y| <= 2^58): the
// quotient is within 5/8 of y/M, one correction each way.
template <int MODE>
__device__ __forceinline__ int residue_pub(double y, uint32_t ylo, int M, double qinv) {
  const uint32_t q = lo32(__builtin_fma(y, qinv, kMagicF));
  uint32_t r;
  asm("v_mad_i32_i24 %0, %1, %2, %3" : "=v"(r) : "v"(q), "s"(-M), "v"(ylo));
  int c = (int)(r << 8) >> 8;
  if constexpr (MODE == 3) {
    const int hi = (M - 1) / 2;
    c = c > hi ? c - M : c;
    c = c < hi - M + 1 ? c + M : c;
  }
  return c;
}

// four values (e4m3-exact integers) as OCP E4M3FN bytes, the first lowest
__device__ __forceinline__ uint32_t e4m3x4(float a, float b, float c, float d) {
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c, d, lo, true);
}

// Digits of four square residues (base s; q = rint(x / s) by one FP32
// product, which never lands on the wrong side of a half integer: x / s is
// either an exact tie -- s = 32, product exact -- or at least 1/(2s) from
// one).  Each output dword holds four bytes, the first value lowest.
__device__ __forceinline__ void square_digits(const int (&x)[4], float s, float is, uint32_t& w0,
                                              uint32_t& w1) {
  float d0[4], d1[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const float xf = (float)x[c];
    d1[c] = __builtin_rintf(xf * is);
    d0[c] = __builtin_fmaf(-d1[c], s, xf);
  }
  w0 = e4m3x4(d0[0], d0[1], d0[2], d0[3]);
  w1 = e4m3x4(d1[0], d1[1], d1[2], d1[3]);
}
// four nonsquare residues (|x| <= 255, exact in fp16) as fp16, the first in
// the low half of the first dword
__device__ __forceinline__ uint2 fp16x4(const int (&x)[4]) {
  const h2x lo = __builtin_amdgcn_cvt_pkrtz((float)x[0], (float)x[1]);
  const h2x hi = __builtin_amdgcn_cvt_pkrtz((float)x[2], (float)x[3]);
  return uint2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
}

__device__ __forceinline__ float reduce_pf(float x, float m, float minv) {
  return __builtin_fmaf(-__builtin_rintf(x * minv), m, x);
}

// fp8 fragment of a 32-row block for the 64-byte K step of a stage: lane
// half fh takes chunks fh and 2 + fh of its row (the same on both operands,
// so the MFMA pairs equal k)
__device__ __forceinline__ v8i ffrag8(const int8_t* base, int r, int fh) {
  const int8_t* row = base + r * FBK;
  const v4i lo = *reinterpret_cast<const v4i*>(row + ((fh ^ fswz(r)) << 4));
  const v4i hi = *reinterpret_cast<const v4i*>(row + (((2 + fh) ^ fswz(r)) << 4));
  return v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

__device__ __forceinline__ v16f mma8(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// The fp16 slabs: 64 k (128 bytes) per row at a row stride of 144 bytes, so
// that the rows read at one chunk by 16 lanes fall on distinct banks with
// no swizzle, and a lane's four fragments sit at immediate offsets from one
// address.  Fragment for the 16-k step ks of a stage: lane half fh takes
// chunk 2 ks + fh of its row (the same on both operands, so the MFMA pairs
// equal k).
constexpr int kNS = 144;
__device__ __forceinline__ v8h ffrag16(const int8_t* base, int r, int ks, int fh) {
  return *reinterpret_cast<const v8h*>(base + r * kNS + (2 * ks + fh) * 16);
}
__device__ __forceinline__ v16f mma16(v8h a, v8h b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// B's operands for the fused product: thread (lane, wave) of block
// (column block, 64-k group) takes column 64 cb + lane and the 16 k from
// 64 kg + 16 wave; every square plane gets one 16-byte store, every
// nonsquare residue slab two.  tau: the columns' exponents
// (OZAKI25_EXP_NONFINITE: zeros).
template <int MODE, bool TZ>
__global__ __launch_bounds__(256) void fused_b_digits_kernel(int64_t n, int64_t k, int64_t kp,
                                                             const double* __restrict__ B, int64_t ldb,
                                                             const int32_t* __restrict__ tau,
                                                             int8_t* __restrict__ digits) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t cbs = (n + 63) / 64;
  const int64_t j = (int64_t)(blockIdx.x % cbs) * 64 + lane;
  const int64_t k0 = (int64_t)(blockIdx.x / cbs) * 64 + wave * 16;
  if (j >= n || k0 >= kp) return;
  const int tj = tau[j];
  const bool live = tj != INT32_MIN;
  double y[16];
  uint32_t ylo[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const double b = (live && k0 + c < k) ? B[(k0 + c) * ldb + j] : 0.0;
    const double v = __builtin_ldexp(b, live ? tj : 0);
    y[c] = TZ ? __builtin_trunc(v) : __builtin_rint(v);
    ylo[c] = MODE == 1 ? lo32(y[c] + kMagicF) : low32_split(y[c]);
  }
  const int64_t pstride = n * 128;
  int8_t* out = digits + ((k0 / 128) * (2 * kR)) * pstride + j * 128 + (k0 % 128);
  // nonsquare g: plane 12 + 2 g + (k0 % 128) / 64, fp16 at 2 (k0 % 64)
  int8_t* outn = digits + ((k0 / 128) * (2 * kR) + 2 * kPairs + (k0 % 128) / 64) * pstride + j * 128 +
                 2 * (k0 % 64);
  for (int g = 0; g < kPairs; ++g) {
    const PairConst pc = kPair[g];
    uint32_t ws[2][4];
    uint2 wn[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      int xs[4], xn[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        xs[c] = residue_pub<MODE>(y[4 * q + c], ylo[4 * q + c], pc.ms, pc.qs);
        xn[c] = residue_pub<MODE>(y[4 * q + c], ylo[4 * q + c], pc.mn, pc.qn);
      }
      square_digits(xs, (float)pc.s, pc.is, ws[0][q], ws[1][q]);
      wn[q] = fp16x4(xn);
    }
    *reinterpret_cast<uint4*>(outn + 2 * g * pstride) = uint4{wn[0].x, wn[0].y, wn[1].x, wn[1].y};
    *reinterpret_cast<uint4*>(outn + 2 * g * pstride + 16) = uint4{wn[2].x, wn[2].y, wn[3].x, wn[3].y};
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      *reinterpret_cast<uint4*>(out + (2 * g + d) * pstride) = uint4{ws[d][0], ws[d][1], ws[d][2], ws[d][3]};
    }
  }
}

// 128 rows of A per block and one pair of moduli; 16 wavefronts: wavefront
// w converts rows 8 w .. 8 w + 7 of each 128 x 64 slab into the square
// modulus's two digit planes and the nonsquare one's fp16 residues, and
// owns the 32 x 32 outputs (w / 4, w % 4) of both moduli.  The six blocks
// of a row strip go to one XCD back to back.
// MODE: the residue route (1: |y| <= 2^51, ylo by 1.5 2^52; 3: |y| <= 2^58).
template <int MODE, bool TZ, bool VEC>
__global__ __launch_bounds__(1024, 1) void fused_pub_kernel(
    int64_t m, int64_t n, int64_t k, int64_t kp, const double* __restrict__ A, int64_t lda,
    const int32_t* __restrict__ sigma, const int8_t* __restrict__ pb, int16_t* __restrict__ cres,
    int64_t strips) {
  // [buffer][plane][slab]: the square digits; [buffer][slab]: the nonsquare
  // fp16 residues, rows kNS bytes apart (136 KiB in all)
  __shared__ __attribute__((aligned(1024))) int8_t lds_a[2][2][FBM * FBK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b[2][2][FBN * FBK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_an[2][FBM * kNS];
  __shared__ __attribute__((aligned(1024))) int8_t lds_bn[2][FBN * kNS];
  const uint32_t b = blockIdx.x, o = b >> 3;
  const int64_t strip = (int64_t)(o / kPairs) * 8 + (b & 7);
  const int grp = (int)(o % kPairs);
  if (strip >= strips) return;
  const int64_t row0 = strip * FBM;
  const PairConst pc = kPair[grp];
  const float fs = (float)pc.s, fms = (float)pc.ms, fmn = (float)pc.mn;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave >> 2, wc = wave & 3;
  const int fr = lane & 31, fh = lane >> 5;

  // conversion: lane l takes 4 consecutive k (4 (l % 16) ..) of row
  // 8 wave + 4 i + l / 16, i = 0, 1
  int sg[2];
  uint32_t keep[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = 8 * wave + 4 * i + (lane >> 4);
    const int64_t arow = row0 + r;
    const bool ok = arow < m;
    const int sv = ok ? sigma[arow] : 0;
    const bool live = ok && sv != INT32_MIN;
    keep[i] = live ? 0xFFFFFFFFu : 0u;
    sg[i] = live ? sv : 0;
  }

  const int nstage = (int)(kp / FBK);
  // whole stages (VEC) read the strip's rows through one buffer resource:
  // 32-bit byte offsets from its first row, 24-bit products (the host takes
  // this path for lda < 2^21 only, so 128 rows stay below 2^31 bytes), rows
  // past m read as zero
  const int lda8 = (int)(lda * 8);
  const int arec = VEC ? (int)((m - row0 < FBM ? m - row0 : FBM) * lda8) : 0;
  const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
      (void*)uniform_ptr_f((const int8_t*)(A + row0 * lda)), (short)0, arec, 0x00020000);
  double x0[8], x1[8];
  auto load_a = [&](int s, double (&x)[8]) {
    // the lane's offsets recomputed here, not held across the loop (the
    // kernel is at the register limit, and a spilled copy would be
    // reloaded from scratch at the start of every stage)
    const int l = lane_now();
    if (VEC && (int64_t)s * FBK + FBK <= k) {
      const int kb = (s * FBK + 4 * (l & 15)) * 8;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int off = __mul24(8 * wave + 4 * i + (l >> 4), lda8) + kb;
        const double2 p = __builtin_bit_cast(double2, __builtin_amdgcn_raw_buffer_load_b128(ars, off, 0, 0));
        const double2 q =
            __builtin_bit_cast(double2, __builtin_amdgcn_raw_buffer_load_b128(ars, off + 16, 0, 0));
        x[4 * i] = p.x;
        x[4 * i + 1] = p.y;
        x[4 * i + 2] = q.x;
        x[4 * i + 3] = q.y;
      }
    } else {
      const int64_t k0 = (int64_t)s * FBK + 4 * (l & 15);
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int64_t arow = row0 + 8 * wave + 4 * i + (l >> 4);
        const double* arow_p = A + (arow < m ? arow : m - 1) * lda;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int64_t kk = k0 + c < k ? k0 + c : k - 1;
          const double v = arow_p[kk];
          x[4 * i + c] = k0 + c < k ? v : 0.0;
        }
      }
    }
  };
  // per row one dword (4 digit bytes) into each square plane, at chunk
  // ck / 16 of the row (swizzled), and 8 bytes (4 fp16) into the nonsquare
  // slab, at byte 2 ck of the row
  auto convert = [&](int buf, const double (&x)[8]) {
    // the lane's row and k offsets recomputed, as in load_a
    const int l = lane_now(), cl = 4 * (l & 15);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = 8 * wave + 4 * i + (l >> 4);
      double y[4];
      uint32_t ylo[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const double v = __builtin_ldexp(x[4 * i + c], sg[i]);
        y[c] = TZ ? __builtin_trunc(v) : __builtin_rint(v);
        ylo[c] = MODE == 1 ? lo32(y[c] + kMagicF) : low32_split(y[c]);
      }
      int xs[4], xn[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        xs[c] = residue_pub<MODE>(y[c], ylo[c], pc.ms, pc.qs);
        xn[c] = residue_pub<MODE>(y[c], ylo[c], pc.mn, pc.qn);
      }
      uint32_t w[2];
      square_digits(xs, fs, pc.is, w[0], w[1]);
      const uint2 h = fp16x4(xn);
      const int at = r * FBK + (((cl >> 4) ^ fswz(r)) << 4) + (cl & 15);
#pragma unroll
      for (int q = 0; q < 2; ++q) *reinterpret_cast<uint32_t*>(&lds_a[buf][q][at]) = w[q] & keep[i];
      *reinterpret_cast<uint2*>(&lds_an[buf][r * kNS + 2 * cl]) = uint2{h.x & keep[i], h.y & keep[i]};
    }
  };
  // B's slabs of stage s by LDS-DMA, 1 KiB loads spread over the
  // wavefronts (columns past n read zero): loads 0-15 the two square digit
  // slabs (128 columns x 64 bytes, 16 columns a load), loads 16-33 the
  // nonsquare fp16 slab (128 columns at the kNS stride: 1152 16-byte slots
  // filled in order, slot 8 of each row, the padding, from past the end of
  // the buffer, which reads zero)
  const int brecs = __builtin_amdgcn_readfirstlane((int)(n * 128));
  auto load_b = [&](int s, int buf) {
    const int64_t kb = s >> 1, h = s & 1;
    for (int d = wave; d < 16 + FBN * kNS / 1024; d += 16) {
      if (d < 16) {
        const int q = d >> 3, dd = d & 7;
        const int8_t* piece = uniform_ptr_f(pb + ((kb * (2 * kR) + 2 * grp + q) * n) * 128 + h * 64);
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc((void*)piece, (short)0, brecs, 0x00020000);
        const int row = 16 * dd + (lane >> 2);
        const int gchunk = (lane & 3) ^ fswz(row);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_f)(&lds_b[buf][q][16 * dd * FBK]), 16,
                                                 row * 128 + gchunk * 16, 0, 0, 0);
      } else {
        const int dd = d - 16;
        const int8_t* piece = uniform_ptr_f(pb + ((kb * (2 * kR) + 2 * kPairs + 2 * grp + h) * n) * 128);
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc((void*)piece, (short)0, brecs, 0x00020000);
        const int slot = 64 * dd + lane, row = slot / 9, chunk = slot - 9 * row;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_f)(&lds_bn[buf][1024 * dd]), 16,
                                                 chunk < 8 ? row * 128 + chunk * 16 : brecs, 0, 0, 0);
      }
    }
  };

  v16f acc1 = v16f{}, accs = v16f{}, accn = v16f{};
  auto step = [&](int s, double (&xs)[8], double (&xn)[8]) {
    const int cur = s & 1, nxt = cur ^ 1;
    if (s + 2 < nstage) load_a(s + 2, xs);
    if (s + 1 < nstage) load_b(s + 1, nxt);
    // at most three fragments live at a time (registers are short here)
    const int ar = wr * 32 + fr, br = wc * 32 + fr;
    {
      const v8i a0 = ffrag8(lds_a[cur][0], ar, fh), b0 = ffrag8(lds_b[cur][0], br, fh);
      acc1 = mma8(a0, b0, acc1);
      const v8i b1 = ffrag8(lds_b[cur][1], br, fh);
      accs = mma8(a0, b1, accs);
      const v8i a1 = ffrag8(lds_a[cur][1], ar, fh);
      accs = mma8(a1, b0, accs);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      accn = mma16(ffrag16(lds_an[cur], ar, ks, fh), ffrag16(lds_bn[cur], br, ks, fh), accn);
      __builtin_amdgcn_sched_barrier(0);  // one fragment pair live at a time
    }
    __builtin_amdgcn_sched_barrier(0);
    if (s + 1 < nstage) convert(nxt, xn);
    if ((s & (kSegN - 1)) == kSegN - 1 && s + 1 < nstage) {
#pragma unroll
      for (int v = 0; v < 16; ++v) accn[v] = reduce_pf(accn[v], fmn, pc.imn);
    }
    if (((s + 1) % kSegS) == 0 && s + 1 < nstage) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        acc1[v] = reduce_pf(acc1[v], fms, pc.ims);
        accs[v] = reduce_pf(accs[v], fms, pc.ims);
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };

  if (nstage > 0) {
    load_a(0, x0);
    load_b(0, 0);
    if (nstage > 1) load_a(1, x1);
    convert(0, x0);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int s = 0; s < nstage; s += 2) {
    step(s, x0, x1);
    if (s + 1 < nstage) step(s + 1, x1, x0);
  }

  // epilogue: the compact residues -- square (acc1 + s accs) mod m; nonsquare
  // (x y summed) 16^-1 mod m -- each reduced to |c| <= 0.51 m (every value
  // here is an integer below 2^24 in magnitude), as int16 in [12][m][n]
  const int64_t col = wc * 32 + fr;
  int16_t* outs = cres + (int64_t)grp * m * n;
  int16_t* outn = cres + (int64_t)(kPairs + grp) * m * n;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int64_t row = row0 + wr * 32 + 8 * (v >> 2) + 4 * fh + (v & 3);
    const float sv = reduce_pf(reduce_pf(acc1[v], fms, pc.ims) + fs * reduce_pf(accs[v], fms, pc.ims), fms,
                               pc.ims);
    const float nv = reduce_pf(reduce_pf(accn[v], fmn, pc.imn) * pc.inv16, fmn, pc.imn);
    if (row < m && col < n) {
      outs[row * n + col] = (int16_t)(int)sv;
      outn[row * n + col] = (int16_t)(int)nv;
    }
  }
}

template <int MODE, bool TZ>
hipError_t launch_fused_pub_m(int64_t m, int64_t n, int64_t k, int64_t kp, const double* A, int64_t lda,
                              const int32_t* sigma, const double* B, int64_t ldb, const int32_t* tau,
                              int8_t* pb, int16_t* cres, hipStream_t stream) {
  const int64_t cbs = (n + 63) / 64, kgs = kp / 64;
  if (cbs * kgs > (int64_t)UINT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL((fused_b_digits_kernel<MODE, TZ>), dim3((unsigned)(cbs * kgs)), dim3(256), 0, stream, n, k,
                     kp, B, ldb, tau, pb);
  const int64_t strips = (m + FBM - 1) / FBM;
  const int64_t blocks = (strips + 7) / 8 * 8 * kPairs;
  if (blocks > (int64_t)UINT32_MAX) return hipErrorInvalidValue;
  if ((((uintptr_t)A) & 15) == 0 && (lda & 1) == 0 && lda < (1 << 21))
    hipLaunchKernelGGL((fused_pub_kernel<MODE, TZ, true>), dim3((unsigned)blocks), dim3(1024), 0, stream, m, n,
                       k, kp, A, lda, sigma, pb, cres, strips);
  else
    hipLaunchKernelGGL((fused_pub_kernel<MODE, TZ, false>), dim3((unsigned)blocks), dim3(1024), 0, stream, m,
                       n, k, kp, A, lda, sigma, pb, cres, strips);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fused_bytes(int quant, int64_t m, int64_t n, int64_t k, int64_t kp, int t,
                              const double* A, int64_t lda, const int32_t* sigma, const int8_t* pb,
                              int8_t* cres, hipStream_t stream) {
  if (n > FBN || kp % FBK || m <= 0 || n <= 0 || t > kMaxScaleBits) return hipErrorInvalidValue;
  const bool tz = quant == kQuantTZ;
  // |y| <= 2^t: the nearest quotient up to 2^52, then the corrected one
  const int mode = t <= 51 ? 1 : (t == 52 ? 2 : 3);
#define OZ_FUSED(MODE)                                                                           \
  return tz ? launch_fused_g<3, MODE, true>(m, n, k, kp, A, lda, sigma, pb, cres, stream)       \
            : launch_fused_g<3, MODE, false>(m, n, k, kp, A, lda, sigma, pb, cres, stream)
  if (mode == 1) OZ_FUSED(1);
  if (mode == 2) OZ_FUSED(2);
  OZ_FUSED(3);
#undef OZ_FUSED
}

}  // namespace oz

namespace oz {

hipError_t launch_fused_pub(int quant, int64_t m, int64_t n, int64_t k, int64_t kp, int t, const double* A,
                            int64_t lda, const int32_t* sigma, const double* B, int64_t ldb,
                            const int32_t* tau, int8_t* pb, int16_t* cres, hipStream_t stream) {
  if (n > FBN || kp % 128 || m <= 0 || n <= 0 || t > kMaxScaleBits) return hipErrorInvalidValue;
  const bool tz = quant == kQuantTZ;
  // |y| <= 2^t: the nearest quotient with ylo from 1.5 2^52 up to 2^50, the
  // corrected one beyond (as in the deconstruction of the published set)
  if (t <= 50)
    return tz ? launch_fused_pub_m<1, true>(m, n, k, kp, A, lda, sigma, B, ldb, tau, pb, cres, stream)
              : launch_fused_pub_m<1, false>(m, n, k, kp, A, lda, sigma, B, ldb, tau, pb, cres, stream);
  return tz ? launch_fused_pub_m<3, true>(m, n, k, kp, A, lda, sigma, B, ldb, tau, pb, cres, stream)
            : launch_fused_pub_m<3, false>(m, n, k, kp, A, lda, sigma, B, ldb, tau, pb, cres, stream);
}

}  // namespace oz
