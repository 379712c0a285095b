// Per-modulus residue products (Eq. (residueprod)) on gfx950 int8 MFMA.
//
// Each modulus needs three limb products of length k (square m = s^2: d0e1,
// d1e0 with weight s and d0e0 with weight 1 -- the d1e1 term vanishes mod
// s^2; nonsquare, Eq. (karcarry): d0e0, d1e1, (d0+d1)(e0+e1) with weights
// -15, 240, 16).  A block owns one 256 x 256 output tile of one modulus and
// runs the three products through ONE set of int32 MFMA accumulators: after
// product p the accumulator is reduced mod m and multiplied by
// w_p / w_{p+1} mod m (w_{p+1} is invertible whenever it differs from w_p),
// so product p+1 accumulates on top of it and
//     w_last * acc = sum_p w_p P_p   (mod m)
// at the end.  Between reductions an accumulator holds at most m plus one
// int8 dot product, |.| <= 22^2 k < 2^31 for k <= 4 194 304.
//
// Layout: both plane operands are K-contiguous (rows of A, columns of B), the
// form v_mfma_i32_32x32x32_i8 takes for both sides.  Its A and B register
// layouts mirror each other, so loading both with lane = row/column +
// 32 * (16-byte K half) pairs the same k on both sides.
//
// Tiling (4 wavefronts, 1 per SIMD): 256 x 256 block tile, 128 x 128 per
// wavefront (4 x 4 MFMA blocks of 32 x 32), K stages of 128 bytes loaded
// straight from global memory into LDS (buffer loads with the lds bit; 2 x
// 64 KiB, double buffered).  The 16 loads of stage s+1 are interleaved with
// the first half of stage s's MFMAs, so the wave never stalls on a full
// vector-memory queue with MFMAs waiting behind it.  LDS rows are 128 bytes
// with the 16-byte chunk index XOR-swizzled by the row so that the b128
// fragment reads of 8 (or 16) consecutive rows hit distinct banks.  Plane
// rows are padded to a multiple of 128 bytes, so every stage is full.
//
// At this tile size the operand stream is 64 KiB per CU per 2048 MFMA
// cycles (32 B/clk); the per-CU L2 read throughput that the counters show
// (~20 B/clk at ~530 cycles average latency) is the bound, not the MFMAs.
#include "device_math.hpp"
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 256;         // output rows per block
constexpr int BN = 256;         // output columns per block
constexpr int BK = 128;         // k bytes per stage
constexpr int kTile = BM * BK;  // bytes of one operand tile in LDS (BM == BN)
static_assert(BK == kKAlign, "every K stage is full: planes are padded to BK");
constexpr int kGroupM = 4;      // tile rows per group in the block order

// Per-modulus schedule, from the compile-time tables of moduli.hpp.
struct ModSched {
  int m;           // modulus
  int hi;          // (m - 1) / 2, top of the centred range
  int plane_a[3];  // A plane of each product, in issue order
  int plane_b[3];  // B plane of each product
  int mult[3];     // multiplier after product p (p = 2: the final weight)
};

// Issue order: squares put the two weight-s products first so they share the
// accumulator without a reduction; nonsquares keep (d0e0, d1e1, sum).
constexpr int issue_plane_a(int i, int p) {
  return root_of(i) ? plane_base(i) + (p == 1 ? 1 : 0) : plane_base(i) + p;
}
constexpr int issue_plane_b(int i, int p) {
  return root_of(i) ? plane_base(i) + (p == 0 ? 1 : 0) : plane_base(i) + p;
}
constexpr int issue_weight(int i, int p) {
  return root_of(i) ? (p == 2 ? 1 : root_of(i)) : (p == 0 ? -15 : (p == 1 ? 240 : 16));
}
constexpr int issue_mult(int i, int p) {
  const int64_t m = kModulus[i];
  if (p == 2) return (int)mod_pos(issue_weight(i, 2), m);
  const int64_t w = issue_weight(i, p), wn = issue_weight(i, p + 1);
  if (w == wn) return 1;
  return (int)(mod_pos(w, m) * inverse_mod(mod_pos(wn, m), m) % m);
}
constexpr ModSched make_sched(int i) {
  return ModSched{kModulus[i],
                  (kModulus[i] - 1) / 2,
                  {issue_plane_a(i, 0), issue_plane_a(i, 1), issue_plane_a(i, 2)},
                  {issue_plane_b(i, 0), issue_plane_b(i, 1), issue_plane_b(i, 2)},
                  {issue_mult(i, 0), issue_mult(i, 1), issue_mult(i, 2)}};
}
constexpr bool schedule_is_exact() {
  // the later multipliers applied to P_p give back its weight w_p, mod m
  for (int i = 0; i < kR; ++i) {
    const int64_t m = kModulus[i];
    for (int p = 0; p < 3; ++p) {
      int64_t f = 1;
      for (int q = p; q < 3; ++q) f = f * issue_mult(i, q) % m;
      if (f != mod_pos(issue_weight(i, p), m)) return false;
    }
  }
  return true;
}
static_assert(schedule_is_exact(), "accumulator carry schedule reproduces the epilogue weights");

__constant__ ModSched kSched[kR] = {make_sched(0), make_sched(1), make_sched(2),  make_sched(3),
                                    make_sched(4), make_sched(5), make_sched(6),  make_sched(7),
                                    make_sched(8), make_sched(9), make_sched(10), make_sched(11)};

// acc * mult reduced mod m to a representative in [-m/2, m/2]: acc * mult is
// exact in FP64 (|acc| < 2^31, mult < 2^11), its quotient by m is off from
// the nearest integer by far less than 1/(2m) (odd m: never a tie; m = 1024:
// exact), and the remainder is exact in one FMA.  Ties of the even modulus
// may land on +m/2; the final reduction maps them to -m/2.
__device__ __forceinline__ int mulmod_rt(int acc, double mult, double m, double mult_inv) {
  const double a = (double)acc;
  const double q = __builtin_rint(a * mult_inv);     // mult_inv = mult / m
  return (int)__builtin_fma(a, mult, -q * m);         // a * mult exact, q * m exact
}

__device__ __forceinline__ int swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// Block order: moduli outermost; inside a modulus, tiles go in groups of
// kGroupM tile rows, so that the ~256 blocks resident at a time cover a
// compact patch of output tiles and share their A and B panels in the L2s
// and the Infinity Cache.  (Giving each XCD a contiguous range of this order
// measured slower: it spreads the XCDs over distant tiles and moduli.)
__device__ __forceinline__ void block_coords(int64_t tiles_m, int64_t tiles_n, int& mod,
                                             int64_t& tm, int64_t& tn) {
  const int64_t id = blockIdx.x;
  const int64_t per_mod = tiles_m * tiles_n;
  mod = (int)(id / per_mod);
  const int64_t t = id % per_mod;
  const int64_t group = t / (kGroupM * tiles_n);
  const int64_t first = group * kGroupM;
  const int64_t gsz = tiles_m - first < kGroupM ? tiles_m - first : kGroupM;
  const int64_t in = t % (kGroupM * tiles_n);
  tm = first + in % gsz;
  tn = in / gsz;
}

using lds_ptr = __attribute__((address_space(3))) void*;

// Block-uniform values computed with 64-bit VALU arithmetic: pin them to
// scalar registers so buffer descriptors need no per-lane waterfall.
__device__ __forceinline__ const int8_t* uniform_ptr(const int8_t* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const int8_t*)(((uint64_t)hi << 32) | lo);
}

// One K stage: the wave's share of the A and B tiles goes straight from
// global memory into LDS.  A wave's load writes 1 KiB = 8 rows x 128 bytes,
// lane l landing at row l/8, chunk l%8 of that slab; to realise the swizzled
// layout the lane fetches the global chunk (l%8) ^ swz(row).
__device__ __forceinline__ void stage_load(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb,
                                           int8_t* la, int8_t* lb, const int (&voff)[8], int k0,
                                           int wave) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int slab = (wave * 8 + i) * 1024;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr)(la + slab), 16, voff[i], k0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr)(lb + slab), 16, voff[i], k0, 0, 0);
  }
}

__device__ __forceinline__ void load_frags(const int8_t* la, const int8_t* lb, int wr, int wc, int fr,
                                           int fh, int ks, v4i (&af)[4], v4i (&bf)[4]) {
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int r = wr * 128 + a * 32 + fr;
    af[a] = *reinterpret_cast<const v4i*>(la + r * BK + (((2 * ks + fh) ^ swz(r)) << 4));
  }
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int r = wc * 128 + b * 32 + fr;
    bf[b] = *reinterpret_cast<const v4i*>(lb + r * BK + (((2 * ks + fh) ^ swz(r)) << 4));
  }
}

// One stage of MFMAs with the next stage's 16 DMA loads spread among them:
// the fragments of step 0 first, then per K step [1 fragment read of the
// next step, 1 DMA (steps 0-1 only), 2 MFMAs] x 8.
__device__ __forceinline__ void stage_mma_dma(const int8_t* la, const int8_t* lb, int wr, int wc,
                                              int fr, int fh, v16i (&acc)[4][4],
                                              __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb,
                                              int8_t* na, int8_t* nb, const int (&voff)[8], int k0,
                                              int wave) {
  v4i af[2][4], bf[2][4];
  load_frags(la, lb, wr, wc, fr, fh, 0, af[0], bf[0]);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int slab = (wave * 8 + i) * 1024;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr)(na + slab), 16, voff[i], k0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr)(nb + slab), 16, voff[i], k0, 0, 0);
  }
#pragma unroll
  for (int ks = 0; ks < BK / 32; ++ks) {
    const int cur = ks & 1;
    if (ks + 1 < BK / 32) load_frags(la, lb, wr, wc, fr, fh, ks + 1, af[cur ^ 1], bf[cur ^ 1]);
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[cur][a], bf[cur][b], acc[a][b], 0, 0, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
  for (int ks = 0; ks < BK / 32; ++ks)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (ks + 1 < BK / 32) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (ks < 2) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
}

template <typename OT>
__global__ __launch_bounds__(256, 1) void residue_gemm_kernel(int64_t m, int64_t n, int64_t kp,
                                                              const int8_t* __restrict__ pa,
                                                              const int8_t* __restrict__ pb,
                                                              OT* __restrict__ cres) {
  // two LDS stages, each an A tile and a B tile of 256 rows x 128 bytes
  __shared__ __attribute__((aligned(1024))) int8_t lds_a0[kTile];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b0[kTile];
  __shared__ __attribute__((aligned(1024))) int8_t lds_a1[kTile];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b1[kTile];
  const int64_t tiles_m = (m + BM - 1) / BM, tiles_n = (n + BN - 1) / BN;
  int mod;
  int64_t tm, tn;
  block_coords(tiles_m, tiles_n, mod, tm, tn);
  const ModSched sc = kSched[mod];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS-DMA base in M0
  const int wr = wave >> 1, wc = wave & 1;
  const int fr = lane & 31, fh = lane >> 5;  // fragment row, 16-byte K half

  // byte offsets (within the block's 256-row panel) of the 8 slab loads
  int voff[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = wave * 64 + i * 8 + (lane >> 3);
    voff[i] = r * (int)kp + (((lane & 7) ^ swz(r)) << 4);
  }
  // rows past the matrix edge read as zero (buffer range check); they only
  // feed outputs that are never stored
  const int64_t rows_a = m - tm * BM < BM ? m - tm * BM : BM;
  const int64_t rows_b = n - tn * BN < BN ? n - tn * BN : BN;

  v16i acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = v16i{};

  const int nstage = (int)(kp / BK);
  for (int p = 0; p < 3 && nstage > 0; ++p) {
    const int8_t* A = uniform_ptr(pa + ((int64_t)sc.plane_a[p] * m + tm * BM) * kp);
    const int8_t* B = uniform_ptr(pb + ((int64_t)sc.plane_b[p] * n + tn * BN) * kp);
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        (void*)A, (short)0, __builtin_amdgcn_readfirstlane((int)(rows_a * kp)), 0x00020000);
    const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
        (void*)B, (short)0, __builtin_amdgcn_readfirstlane((int)(rows_b * kp)), 0x00020000);

    stage_load(ra, rb, lds_a0, lds_b0, voff, 0, wave);
    for (int s = 0; s < nstage; s += 2) {
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      // the DMA of the stage after the last one reads past the panel: harmless,
      // it lands in the idle buffer and is drained before the next product
      stage_mma_dma(lds_a0, lds_b0, wr, wc, fr, fh, acc, ra, rb, lds_a1, lds_b1, voff, (s + 1) * BK, wave);
      if (s + 1 >= nstage) break;
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      stage_mma_dma(lds_a1, lds_b1, wr, wc, fr, fh, acc, ra, rb, lds_a0, lds_b0, voff, (s + 2) * BK, wave);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // every wave is done with the buffers before the next product loads
    // carry: acc <- acc * mult_p mod m (a multiplier of 1 mid-way needs no reduction)
    const int mult = sc.mult[p];
    if (p == 2 || mult != 1) {
      const double dm = (double)sc.m, dmult = (double)mult, dinv = (double)mult / (double)sc.m;
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
          for (int v = 0; v < 16; ++v) acc[a][b][v] = mulmod_rt(acc[a][b][v], dmult, dm, dinv);
    }
  }

  // 32x32 MFMA result layout: lane holds column lane%32 and rows
  // 8*(v/4) + 4*(lane/32) + v%4 of its 32x32 block.  Stores use the tile's
  // scalar base and 32-bit element offsets (256 n < 2^31).
  OT* out = (OT*)uniform_ptr((const int8_t*)(cres + (int64_t)mod * m * n + tm * BM * n + tn * BN));
  const int nn = (int)n;
  const int rows_left = (int)(m - tm * BM), cols_left = (int)(n - tn * BN);
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int col = wc * 128 + b * 32 + fr;
      const int row0 = wr * 128 + a * 32 + 4 * fh;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = row0 + 8 * (v >> 2) + (v & 3);
        // representatives lie in [-m/2, m/2]: only +m/2 (even m) needs wrapping
        const int r = acc[a][b][v];
        if (row < rows_left && col < cols_left) out[row * nn + col] = (OT)(r > sc.hi ? r - sc.m : r);
      }
    }
}

template <typename OT>
hipError_t launch_gemm(int64_t m, int64_t n, int64_t kp, const int8_t* pa, const int8_t* pb,
                       OT* cres, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  // the store epilogue uses 32-bit offsets within a 256-row tile
  if (n > kMaxResidueCols) return hipErrorInvalidValue;
  const int64_t blocks = (int64_t)kR * ((m + BM - 1) / BM) * ((n + BN - 1) / BN);
  hipLaunchKernelGGL(residue_gemm_kernel<OT>, dim3((unsigned)blocks), dim3(256), 0, stream, m, n,
                     kp, pa, pb, cres);
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
