// Per-modulus residue products (Eq. (residueprod)) on gfx950 FP8 MFMA (the
// published set's limb planes) and int8 MFMA (the all-byte set's residue
// planes, further below).
//
// Each modulus needs three limb products of length k (square m = s^2: d0e1,
// d1e0 with weight s and d0e0 with weight 1 -- the d1e1 term vanishes mod
// s^2; nonsquare, Eq. (karcarry): d0e0, d1e1, (d0+d1)(e0+e1) with weights
// -15, 240, 16).  The planes hold the limbs as e4m3 bytes (every limb is
// e4m3-exact, Lemma 1), and v_mfma_f32_32x32x64_f8f6f4 multiplies them with
// FP32 accumulation, exact while every partial sum is an integer below 2^24.
//
// A block owns one output tile of one modulus and runs the three products
// through ONE set of accumulators: after product p the accumulator is
// reduced mod m and multiplied by w_p / w_{p+1} mod m (w_{p+1} is invertible
// whenever it differs from w_p), so product p+1 accumulates on top of it and
//     w_last * acc = sum_p w_p P_p   (mod m)
// at the end (the compact outputs store acc itself, reduced; the
// reconstruction applies w_last).  Products longer than kSeg stages (16384
// k) are cut into segments with a plain reduction between them, which keeps
// every sum between two reductions below 2^24: at most 0.51 m (m - 1) +
// 22^2 * 16384, or 2 * 16^2 * 16384 for the two square products that share
// an accumulator unreduced (only when each fits one segment).  This is the
// paper's chunked FP32 accumulation (its depth limit 2^24 / 22^2 = 34663),
// with the chunk at a power of two below it.
//
// Layout: planes are stored [k_pad/128][planes][rows][128] (rows of A,
// columns of B), so one 128-byte K stage of a 256-row tile is a contiguous
// 32 KiB piece; measured 6 % faster than K-contiguous rows of full length.
// The MFMA's A and B register layouts mirror each other: lane l holds
// row/column l%32 and 32 of the 64 k bytes of the step, the same 32 on both
// sides for equal l/32, so any fixed choice of those bytes pairs equal k.
//
// Tiling: a block of 16 wavefronts (4 per SIMD) owns a 256 x 256 output
// tile (512 x 128 for at most 128 columns), 64 x 64 per wavefront (2 x 2
// MFMA blocks of 32 x 32).  Four waves per
// SIMD keep the matrix core fed while other waves wait at a barrier, on LDS
// reads or on the operand stream; they cost twice the LDS reads of a 2 x 2
// layout of 128 x 128 wavefronts (measured 5-6 % faster all the same).  K
// stages of 128 bytes go straight from global memory into LDS (buffer loads
// with the lds bit; two stages, double buffered); a wave's loads for stage
// s+1 are interleaved with stage s's first MFMAs.  LDS rows are 128
// bytes with the 16-byte chunk index XOR-swizzled by the row so that the
// b128 fragment reads of 8 (or 16) consecutive rows hit distinct banks.
// k is padded to a multiple of 128 bytes, so every stage is full.
//
// At this tile size the operand stream is 64 KiB per CU per stage of 2048
// MFMA cycles (32 B/clk at the FP8 peak); direct-to-LDS loads deliver about
// 20-25 B/clk per CU, which bounds a stage (halving the stream cuts the time
// by a quarter, halving the LDS fragment reads by 2 %), and the MFMA clock
// itself drops with the switching activity of dense data.
#include "kernels.hpp"
#include "moduli.hpp"

namespace oz {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int BK = 128;  // k bytes per stage
// Block tile shapes, the kernels' template parameter S (16 waves; a wave owns
// 64 rows x 64 columns):
//  2: 256 x 256;
//  3: 512 x 128, for at most 128 columns (a 256-wide tile would leave half
//     of every MFMA idle): a stage moves 80 KiB for twice the MACs of a
//     256 x 128 tile's 48 KiB (17 % fewer operand bytes per MAC), and its two
//     stages fill the 160 KiB of LDS.
template <int S>
struct Tile {
  static_assert(S == 2 || S == 3, "tile shape");
  static constexpr int BM = S == 3 ? 512 : 256;  // output rows per block
  static constexpr int BN = S == 2 ? 256 : 128;  // output columns per block
  static constexpr int BB = 2;                   // 32-column blocks per wave
  static constexpr int WC = BN / (32 * BB);      // waves across the tile
  static constexpr int ADMA = BM / 128;          // A slabs (8 rows x 128 B) per wave and stage
  static constexpr int BDMA = BN / 128;          // B slabs per wave and stage
  static constexpr int DMA = ADMA + BDMA;
  static_assert(BM / 64 * WC == 16, "16 waves");
};
static_assert(BK == kKAlign, "every K stage is full: planes are padded to BK");
constexpr int kSeg = 128;       // K stages (16384 k) per accumulation segment

// Per-modulus schedule, from the compile-time tables of moduli.hpp.
struct ModSched {
  int m;           // modulus
  int hi;          // (m - 1) / 2, top of the centred range
  int plane_a[3];  // A plane of each product, in issue order
  int plane_b[3];  // B plane of each product
  int mult[3];     // multiplier after product p (p = 2: the final weight)
  float inv;       // RN(1/m)
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
                  {issue_mult(i, 0), issue_mult(i, 1), issue_mult(i, 2)},
                  1.0f / (float)kModulus[i]};
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
constexpr bool compact_scale_matches() {
  for (int i = 0; i < kR; ++i)
    if (issue_weight(i, 2) != compact_scale(i)) return false;
  return true;
}
static_assert(compact_scale_matches(), "compact outputs leave out the last product's weight");

__constant__ ModSched kSched[kR] = {make_sched(0), make_sched(1), make_sched(2),  make_sched(3),
                                    make_sched(4), make_sched(5), make_sched(6),  make_sched(7),
                                    make_sched(8), make_sched(9), make_sched(10), make_sched(11)};

// Modular reduction of an integer-valued fp32 accumulator, |x| < 2^24:
// q = rint(x * (1/m)) is the nearest quotient or one off (the fp32 quotient
// errs by far less than 1/100), x - q m is an integer below m in magnitude
// and comes out of the FMA exactly, so the result is congruent to x with
// |result| <= 0.51 m.
__device__ __forceinline__ float reduce_f(float x, float m, float minv) {
  const float q = __builtin_rintf(x * minv);
  return __builtin_fmaf(-q, m, x);
}

__device__ __forceinline__ int swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// Block order: moduli outermost; inside a modulus, tiles go in groups of G
// tile rows, column by column.  Blocks are dealt round-robin over the 8
// XCDs; with G = 2 and 32 tile columns the 32 blocks an XCD runs at a time
// cover 4 tile rows x 8 tile columns: 12 panels feed 32 tiles from its L2
// (G = 4: 18 panels; 8: 33).  Short k (small panels) prefers G = 1 on the
// FP8 route and G = 4 on the int8 one (gemm_group).
// Unsigned 32-bit arithmetic throughout: the grid has fewer than 2^32 blocks
// (checked at launch), so every count here fits, and 32-bit divisions cost a
// small fraction of 64-bit ones.
__device__ __forceinline__ void block_coords(uint32_t id, uint32_t tiles_m, uint32_t tiles_n,
                                             uint32_t group, int& mod, int64_t& tm, int64_t& tn) {
  const uint32_t per_mod = tiles_m * tiles_n;
  const uint32_t q = id / per_mod;
  const uint32_t t = id - q * per_mod;
  const uint32_t gw = group * tiles_n;
  const uint32_t g = t / gw;
  const uint32_t first = g * group;
  const uint32_t in = t - g * gw;
  const uint32_t gsz = tiles_m - first < group ? tiles_m - first : group;
  const uint32_t c = in / gsz;
  // uniform values: pinned to scalar registers
  mod = __builtin_amdgcn_readfirstlane((int)q);
  tm = __builtin_amdgcn_readfirstlane((int)(first + (in - c * gsz)));
  tn = __builtin_amdgcn_readfirstlane((int)c);
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

// Plane layout [k_pad/128][planes][rows][128]: K stage s of plane q of a
// 256-row tile starting at row r0 is the contiguous piece
// ((s * planes + q) * rows + r0) * 128, and consecutive stages of a plane
// are planes * rows * 128 bytes apart.  A descriptor per stage (the stage
// offset may exceed 32 bits); rows past the matrix edge fall outside its
// range and read as zero.

// One K stage: the wave's share of the A and B tiles (32 rows of each) goes
// straight from global memory into LDS.  A load writes 1 KiB = 8 rows x
// 128 bytes, lane l landing at row l/8, chunk l%8 of that slab; to realise
// the swizzled layout the lane fetches the global chunk (l%8) ^ swz(row).
// DMA d of a stage (Tile<S>::DMA per wave): d < ADMA the A slab
// wave * ADMA + d, then the B slab wave * BDMA + (d - ADMA).  voffa[i]: rows
// (wave * ADMA + i) * 8 + lane/8 of the A tile; voffb[i] likewise for B.
template <int S>
__device__ __forceinline__ void stage_dma(int d, __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb,
                                          int8_t* la, int8_t* lb, const int* voffa,
                                          const int* voffb, int wave) {
  constexpr int AD = Tile<S>::ADMA, BD = Tile<S>::BDMA;
  if (d < AD)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr)(la + (wave * AD + d) * 1024), 16, voffa[d], 0,
                                             0, 0);
  else
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr)(lb + (wave * BD + d - AD) * 1024), 16,
                                             voffb[d - AD], 0, 0, 0);
}

template <int S>
__device__ __forceinline__ void stage_load(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb,
                                           int8_t* la, int8_t* lb, const int* voffa,
                                           const int* voffb, int wave) {
#pragma unroll
  for (int d = 0; d < Tile<S>::DMA; ++d) stage_dma<S>(d, ra, rb, la, lb, voffa, voffb, wave);
}

// Byte offsets within a tile's 128-byte rows of the slab loads of a wave:
// row (wave * D + i) * 8 + lane/8, chunk (lane % 8) ^ swz(row).
template <int D>
__device__ __forceinline__ void slab_offsets(int wave, int lane, int (&voff)[D]) {
#pragma unroll
  for (int i = 0; i < D; ++i) {
    const int r = (wave * D + i) * 8 + (lane >> 3);
    voff[i] = r * BK + (((lane & 7) ^ swz(r)) << 4);
  }
}

__device__ __forceinline__ v8i cat(v4i lo, v4i hi) {
  return v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// fp8 fragment of one 32-row block for one 64-byte K step: lane half fh
// takes 16-byte chunks 4 ks + fh and 4 ks + 2 + fh of its row (the same on
// both sides, so the MFMA pairs equal k)
__device__ __forceinline__ v8i frag(const int8_t* base, int r, int ks, int fh) {
  const int8_t* row = base + r * BK;
  return cat(*reinterpret_cast<const v4i*>(row + (((4 * ks + fh) ^ swz(r)) << 4)),
             *reinterpret_cast<const v4i*>(row + (((4 * ks + 2 + fh) ^ swz(r)) << 4)));
}

// One stage: two 64-byte K steps of 2 x BB MFMAs (a wave owns 64 x 32 BB;
// four waves share each SIMD).  The next stage's DMA loads go among the
// first MFMAs.
template <int S, int NB = Tile<S>::BB>
__device__ __forceinline__ void stage_mma_dma(const int8_t* la, const int8_t* lb, int ra0, int rb0,
                                              int fh, v16f (&acc)[2][NB],
                                              __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb,
                                              int8_t* na, int8_t* nb, const int* voffa,
                                              const int* voffb, int wave) {
  constexpr int ND = Tile<S>::DMA;
  v8i af[2][2], bf[2][NB];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
    for (int x = 0; x < 2; ++x) af[ks][x] = frag(la, ra0 + 32 * x, ks, fh);
#pragma unroll
    for (int x = 0; x < NB; ++x) bf[ks][x] = frag(lb, rb0 + 32 * x, ks, fh);
  }
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int j = ks * 2 * NB + a * NB + b;  // MFMA number in issue order
        if (j < ND) stage_dma<S>(j, ra, rb, na, nb, voffa, voffb, wave);
        acc[a][b] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[ks][a], bf[ks][b], acc[a][b], 0,
                                                                    0, 0, 0, 0, 0);
      }
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
  for (int i = 0; i < ND; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 4 * NB - ND, 0);
}

// After stage s of product p:
//  - end of a segment inside a product: a plain reduction;
//  - end of product 0 or 1: reduce, then times the product's multiplier
//    (no second reduction: |result| <= 0.51 m (m - 1) < 2^20 and the next
//    segment adds at most 484 * 128 * kSeg, still below 2^24); squares skip
//    it between their two weight-s products while each fits one segment;
//  - end of product 2: reduce (|result| <= 0.51 m); with FINAL_W (true
//    residues) times the last weight and reduce again.  Without FINAL_W the
//    stored residue is the true one divided by that weight (compact outputs:
//    reconstruction folds the weight into its Garner constants).
// With FINAL_W every carry ends with a second reduction (harmless before the
// last product); the compact form is one reduction and one multiply.
template <int NB, bool FINAL_W>
__device__ __forceinline__ void carry(v16f (&acc)[2][NB], int p, int s, int nstage, int nseg, int mod,
                                      float fm, float finv) {
  static_assert((kSeg & (kSeg - 1)) == 0, "segment length is a power of two");
  const bool prod_end = s + 1 == nstage;
  if (!prod_end && ((s + 1) & (kSeg - 1)) != 0) return;
  const int mult = prod_end && (p < 2 || FINAL_W) ? kSched[mod].mult[p] : 1;
  if (mult == 1 && p < 2 && prod_end && nseg == 1) return;
  const float fmult = (float)mult;
  // one branch-free form for every carry (separate forms per case cost
  // registers at their join inside the stage loop)
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = reduce_f(acc[a][b][v], fm, finv) * fmult;
        if constexpr (FINAL_W) x = reduce_f(x, fm, finv);
        acc[a][b][v] = x;
      }
}
// the carried value times a multiplier plus one segment stays exact in fp32
static_assert((int64_t)(kModulus[0] / 2 + kModulus[0] / 50 + 1) * (kModulus[0] - 1) + 484LL * BK * kSeg <
                  (1LL << 24),
              "carry bound");
static_assert(kModulus[0] >= kModulus[kR - 1] && kModulus[0] >= kModulus[1], "largest modulus first");

// Output stores through a global (not generic) pointer; NT marks them
// streaming (measured: the FP8 kernel gains with it, the int8 one without).
template <bool NT, typename OT>
__device__ __forceinline__ void store_out(OT* p, OT v) {
  auto* g = (__attribute__((address_space(1))) OT*)p;
  if constexpr (NT)
    __builtin_nontemporal_store(v, g);
  else
    *g = v;
}

// The wave's 2 x NB blocks of outputs (value(a, b, v) of accumulator v of
// block (a, b)); 32x32 MFMA result layout: lane holds column lane%32 and
// rows 8*(v/4) + 4*(lane/32) + v%4 of its block.  Whole tiles of the compact
// outputs take 32-bit byte offsets from the tile's scalar base (row stride
// times a constant per value: one add per store, no per-value bounds test;
// offsets below 256 n size <= 2^32); edge tiles and int32 outputs test every
// value and use 32-bit element offsets (256 n < 2^31).
template <bool NT, typename OT, int S, typename F>
__device__ __forceinline__ void store_tile(OT* out, int nn, int rows_left, int cols_left, int wr,
                                           int wc, int fr, int fh, F&& value) {
  constexpr int BM = Tile<S>::BM, BN = Tile<S>::BN, NB = Tile<S>::BB;
  if constexpr (sizeof(OT) <= 2) {
    if (rows_left >= BM && cols_left >= BN) {
      char* base = (char*)out;
      const uint32_t stride = (uint32_t)nn * (uint32_t)sizeof(OT);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const uint32_t off0 = (uint32_t)(wr * 64 + a * 32 + 4 * fh) * stride +
                                (uint32_t)((wc * 32 * NB + b * 32 + fr) * (int)sizeof(OT));
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const uint32_t off = off0 + (uint32_t)(8 * (v >> 2) + (v & 3)) * stride;
            store_out<NT>((OT*)(base + off), (OT)value(a, b, v));
          }
        }
      return;
    }
  }
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int col = wc * 32 * NB + b * 32 + fr;
      const int row0 = wr * 64 + a * 32 + 4 * fh;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = row0 + 8 * (v >> 2) + (v & 3);
        if (row < rows_left && col < cols_left) store_out<NT>(out + row * nn + col, (OT)value(a, b, v));
      }
    }
}

// splits > 1 (split-k): consecutive blocks take the same tile's stage ranges,
// and block (tile, split) writes its centred partial product to the split's
// own [r][m][n] slice of cres; reduce_splits_kernel sums them mod m.
template <typename OT, int S>
__global__ __launch_bounds__(1024, 1) void residue_gemm_kernel(int64_t m, int64_t n, int64_t kp,
                                                              const int8_t* __restrict__ pa,
                                                              const int8_t* __restrict__ pb,
                                                              OT* __restrict__ cres, int splits,
                                                              int group) {
  // two LDS stages, each an A tile (BM rows x 128 bytes) and a B tile
  constexpr int BM = Tile<S>::BM, BN = Tile<S>::BN, NB = Tile<S>::BB, WC = Tile<S>::WC;
  __shared__ __attribute__((aligned(1024))) int8_t lds_a0[BM * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b0[BN * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_a1[BM * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b1[BN * BK];
  const int64_t tiles_m = (m + BM - 1) / BM, tiles_n = (n + BN - 1) / BN;
  const int split = (int)(blockIdx.x % (unsigned)splits);
  int mod;
  int64_t tm, tn;
  block_coords(blockIdx.x / (unsigned)splits, (uint32_t)tiles_m, (uint32_t)tiles_n, (uint32_t)group, mod,
               tm, tn);
  const ModSched sc = kSched[mod];
  cres += (int64_t)split * kR * m * n;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS-DMA base in M0
  const int wr = wave / WC, wc = wave % WC;  // (16 / WC) x WC waves of 64 x 32 NB
  const int fr = lane & 31, fh = lane >> 5;  // fragment row, 16-byte K half
  const int ra0 = wr * 64 + fr, rb0 = wc * 32 * NB + fr;

  // byte offsets (within the block's panels) of the slab loads
  int voffa[Tile<S>::ADMA], voffb[Tile<S>::BDMA];
  slab_offsets(wave, lane, voffa);
  slab_offsets(wave, lane, voffb);
  // rows past the matrix edge read as zero (buffer range check); they only
  // feed outputs that are never stored
  const int64_t rows_a = m - tm * BM < BM ? m - tm * BM : BM;
  const int64_t rows_b = n - tn * BN < BN ? n - tn * BN : BN;

  v16f acc[2][NB];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = v16f{};

  // The three products run as segments of at most kSeg stages: every fp32
  // accumulator sum between two reductions stays below 2^24 (at most
  // 545 + 484 * 128 * kSeg, or two square products of 16 x 16 terms when the
  // whole product fits one segment).  A segment ends with the carry (the
  // product's multiplier after its last segment, a plain reduction after the
  // others; none mid-way between the two square products of weight s while
  // they fit one segment each).
  // this block's stages [sbeg, sbeg + nstage) of each product
  const int nstage_all = (int)(kp / BK);
  // 32-bit: at most 2^15 stages times 64 splits
  const int sbeg = (int)((uint32_t)nstage_all * (uint32_t)split / (uint32_t)splits);
  const int nstage = (int)((uint32_t)nstage_all * (uint32_t)(split + 1) / (uint32_t)splits) - sbeg;
  const int nseg = nstage > 0 ? (nstage + kSeg - 1) / kSeg : 0;  // segments per product
  const int na = __builtin_amdgcn_readfirstlane((int)(rows_a * BK));
  const int nb = __builtin_amdgcn_readfirstlane((int)(rows_b * BK));
  // One pipeline over the 3 * nstage stages of the three products: the load
  // of the next stage -- the next product's first one at a product boundary
  // -- is always in flight while a stage computes, and the carry runs on the
  // registers after the last stage of a segment.
  const int total = 3 * nstage;
  // Stage cursors, advanced without divisions: the look-ahead cursor (lp,
  // ls) with the stage's A and B pieces, stepping by one K stage of the
  // plane layout and jumping to the next product's first stage at a product
  // boundary (it stays on the last stage, whose look-ahead load repeats
  // it); the carry cursor (cp, cs) follows the stage just computed.
  const int64_t step_a = (int64_t)kPlanes * m * BK, step_b = (int64_t)kPlanes * n * BK;
  auto first_a = [&](int p) {
    return pa + (((int64_t)sbeg * kPlanes + kSched[mod].plane_a[p]) * m + tm * BM) * BK;
  };
  auto first_b = [&](int p) {
    return pb + (((int64_t)sbeg * kPlanes + kSched[mod].plane_b[p]) * n + tn * BN) * BK;
  };
  int lp = 0, ls = 0, cp = 0, cs = 0;
  const int8_t* la = first_a(0);
  const int8_t* lb = first_b(0);
  auto advance = [&]() {
    if (ls + 1 < nstage) {
      ++ls;
      la += step_a;
      lb += step_b;
    } else if (lp < 2) {
      ++lp;
      ls = 0;
      la = first_a(lp);
      lb = first_b(lp);
    }
  };
  auto rsrc = [](const int8_t* p, int nrec) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(p), (short)0, nrec, 0x00020000);
  };
  const float fm = (float)sc.m, finv = sc.inv;
  auto carry_step = [&]() {
    carry<NB, sizeof(OT) == 4>(acc, cp, cs, nstage, nseg, mod, fm, finv);
    if (++cs == nstage) {
      cs = 0;
      ++cp;
    }
  };
  if (total > 0) stage_load<S>(rsrc(la, na), rsrc(lb, nb), lds_a0, lds_b0, voffa, voffb, wave);
  advance();
  for (int G = 0; G < total; G += 2) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    stage_mma_dma<S>(lds_a0, lds_b0, ra0, rb0, fh, acc, rsrc(la, na), rsrc(lb, nb), lds_a1, lds_b1,
                      voffa, voffb, wave);
    advance();
    carry_step();
    if (G + 1 >= total) break;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    stage_mma_dma<S>(lds_a1, lds_b1, ra0, rb0, fh, acc, rsrc(la, na), rsrc(lb, nb), lds_a0, lds_b0,
                      voffa, voffb, wave);
    advance();
    carry_step();
  }
  __builtin_amdgcn_s_waitcnt(0);  // the repeated look-ahead load lands before the epilogue

  OT* out = (OT*)uniform_ptr((const int8_t*)(cres + (int64_t)mod * m * n + tm * BM * n + tn * BN));
  store_tile<true, OT, S>(out, (int)n, (int)(m - tm * BM), (int)(n - tn * BN), wr, wc, fr, fh,
                           [&](int a, int b, int v) {
                             // the final carry leaves |r| <= 0.51 m: true residues
                             // are wrapped into [-(m/2), (m-1)/2]; compact ones are
                             // stored as they stand
                             const int r = (int)acc[a][b][v];
                             return sizeof(OT) == 4
                                        ? (r > sc.hi ? r - sc.m : (r < -(sc.m >> 1) ? r + sc.m : r))
                                        : r;
                           });
}

// The lane index from a volatile asm: values derived from it inside a loop
// are neither hoisted out of it nor kept live across it.
__device__ __forceinline__ int lane_id_now() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Persistent form (one block per CU, no split-k, an even number of stages
// per tile): a block takes virtual blocks blockIdx.x, + gridDim.x, ... in the
// order above (gridDim.x a multiple of 8 keeps each on its XCD).  The look-
// ahead of a tile's last stage is the next tile's first stage, so its loads
// are in flight while the tile's residues are formed and stored, and the
// block skips the launch and first-load latency of a fresh block per tile.
// The next tile's first barrier waits for every load and store (loads and
// stores share one counter, and their relative completion order is not
// relied on).  Only the compact int16 output takes this form.
template <typename OT, int S>
__global__ __launch_bounds__(1024, 1) void residue_gemm_persistent_kernel(
    int64_t m, int64_t n, int64_t kp, const int8_t* __restrict__ pa, const int8_t* __restrict__ pb,
    OT* __restrict__ cres, int group, uint32_t nvirt) {
  constexpr int BM = Tile<S>::BM, BN = Tile<S>::BN, NB = Tile<S>::BB, WC = Tile<S>::WC;
  static_assert(sizeof(OT) == 2, "the compact int16 residue output");
  __shared__ __attribute__((aligned(1024))) int8_t lds_a0[BM * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b0[BN * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_a1[BM * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b1[BN * BK];
  const int64_t tiles_m = (m + BM - 1) / BM, tiles_n = (n + BN - 1) / BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave / WC, wc = wave % WC;
  const int fr = lane & 31, fh = lane >> 5;
  const int ra0 = wr * 64 + fr, rb0 = wc * 32 * NB + fr;
  int voffa[Tile<S>::ADMA], voffb[Tile<S>::BDMA];
  slab_offsets(wave, lane, voffa);
  slab_offsets(wave, lane, voffb);

  const int nstage = (int)(kp / BK);
  const int nseg = (nstage + kSeg - 1) / kSeg;
  const int total = 3 * nstage;  // even (the host checks)
  const int64_t step_a = (int64_t)kPlanes * m * BK, step_b = (int64_t)kPlanes * n * BK;
  auto rsrc = [](const int8_t* p, int nrec) __attribute__((always_inline)) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(p), (short)0, nrec, 0x00020000);
  };
  // a tile: modulus, tile row and column, and the bytes its panels hold
  // (rows past the matrix edge read as zero)
  struct TileAt {
    int mod;
    int64_t tm, tn;
    int na, nb;
  };
  auto tile_at = [&](uint32_t v) __attribute__((always_inline)) {
    TileAt t;
    block_coords(v, (uint32_t)tiles_m, (uint32_t)tiles_n, (uint32_t)group, t.mod, t.tm, t.tn);
    const int64_t rows_a = m - t.tm * BM < BM ? m - t.tm * BM : BM;
    const int64_t rows_b = n - t.tn * BN < BN ? n - t.tn * BN : BN;
    t.na = __builtin_amdgcn_readfirstlane((int)(rows_a * BK));
    t.nb = __builtin_amdgcn_readfirstlane((int)(rows_b * BK));
    return t;
  };
  auto first_a = [&](const TileAt& t, int p) __attribute__((always_inline)) {
    return pa + ((int64_t)kSched[t.mod].plane_a[p] * m + t.tm * BM) * BK;
  };
  auto first_b = [&](const TileAt& t, int p) __attribute__((always_inline)) {
    return pb + ((int64_t)kSched[t.mod].plane_b[p] * n + t.tn * BN) * BK;
  };

  uint32_t v = blockIdx.x;
  if (v >= nvirt) return;
  TileAt cur = tile_at(v), nxt = cur;
  bool have_next = false, ahead = false;
  // look-ahead cursor: product lp, stage ls of the current tile (or, once
  // ahead, the next tile's first stage), its pieces and their tile's bytes
  int lp = 0, ls = 0, lna = cur.na, lnb = cur.nb;
  const int8_t* la = first_a(cur, 0);
  const int8_t* lb = first_b(cur, 0);
  auto advance = [&]() __attribute__((always_inline)) {
    if (ahead) return;
    if (ls + 1 < nstage) {
      ++ls;
      la += step_a;
      lb += step_b;
    } else if (lp < 2) {
      ++lp;
      ls = 0;
      la = first_a(cur, lp);
      lb = first_b(cur, lp);
    } else if (have_next) {
      ahead = true;
      la = first_a(nxt, 0);
      lb = first_b(nxt, 0);
      lna = nxt.na;
      lnb = nxt.nb;
    }
  };
  stage_load<S>(rsrc(la, lna), rsrc(lb, lnb), lds_a0, lds_b0, voffa, voffb, wave);
  for (;;) {
    const uint32_t vn = v + gridDim.x;
    have_next = vn < nvirt;
    if (have_next) nxt = tile_at(vn);
    advance();
    const ModSched sc = kSched[cur.mod];
    const float fm = (float)sc.m, finv = sc.inv;
    v16f acc[2][NB];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[a][b] = v16f{};
    int cp = 0, cs = 0;
    // every carry but the tile's last, which the store epilogue applies as
    // a bare reduction (the final weight is 1 for compact outputs)
    auto carry_step = [&]() __attribute__((always_inline)) {
      if (cp < 2 || cs + 1 < nstage) carry<NB, false>(acc, cp, cs, nstage, nseg, cur.mod, fm, finv);
      if (++cs == nstage) {
        cs = 0;
        ++cp;
      }
    };
    for (int G = 0; G < total; G += 2) {
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      stage_mma_dma<S>(lds_a0, lds_b0, ra0, rb0, fh, acc, rsrc(la, lna), rsrc(lb, lnb), lds_a1, lds_b1,
                        voffa, voffb, wave);
      advance();
      carry_step();
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      stage_mma_dma<S>(lds_a1, lds_b1, ra0, rb0, fh, acc, rsrc(la, lna), rsrc(lb, lnb), lds_a0, lds_b0,
                        voffa, voffb, wave);
      advance();
      carry_step();
    }
    OT* out = (OT*)uniform_ptr((const int8_t*)(cres + (int64_t)cur.mod * m * n + cur.tm * BM * n +
                                               cur.tn * BN));
    const int rows_left = (int)(m - cur.tm * BM), cols_left = (int)(n - cur.tn * BN);
    // the store offsets from a lane index read here: derived from the
    // loop-invariant one they would be hoisted and held across the stages
    const int el = lane_id_now() & 63;
    store_tile<true, OT, S>(out, (int)n, rows_left, cols_left, wr, wc, el & 31, el >> 5,
                             [&](int a, int b, int vv) { return (int)reduce_f(acc[a][b][vv], fm, finv); });
    if (!have_next) break;
    v = vn;
    cur = nxt;
    lp = 0;
    ls = 0;
    ahead = false;
  }
  __builtin_amdgcn_s_waitcnt(0);  // the last look-ahead (a repeat) lands before the block ends
}

// ---- all-byte set (Sec. 5.1, candidate A) on int8 MFMA --------------------
// The planes hold the centred residues themselves (|r| <= 128), so a modulus
// is ONE int8 product, accumulated in int32 by v_mfma_i32_32x32x32_i8:
// every term is at most 2^14 in magnitude, so partial sums are exact below
// 2^31.  Products longer than kSegA stages (65536 k) reduce the accumulator
// mod m between segments (|carry| <= m/2: every partial stays below
// 2^30 + 2^7).  The int8 MFMA's operand layouts mirror each other like the
// FP8 one's: lane l holds row/column l%32 and 16 of the 32 k bytes of the
// step, the same 16 on both sides for equal l/32.  Same tiling, block
// order and LDS pipeline as above; a stage is four 32-byte K steps.
constexpr int kSegA = 512;

__constant__ int kModA[kRA] = {kModulusA[0],  kModulusA[1],  kModulusA[2],  kModulusA[3],
                               kModulusA[4],  kModulusA[5],  kModulusA[6],  kModulusA[7],
                               kModulusA[8],  kModulusA[9],  kModulusA[10], kModulusA[11],
                               kModulusA[12], kModulusA[13], kModulusA[14]};
// RN(1/m) of each modulus
__constant__ double kInvA[kRA] = {
    1.0 / kModulusA[0],  1.0 / kModulusA[1],  1.0 / kModulusA[2],  1.0 / kModulusA[3],
    1.0 / kModulusA[4],  1.0 / kModulusA[5],  1.0 / kModulusA[6],  1.0 / kModulusA[7],
    1.0 / kModulusA[8],  1.0 / kModulusA[9],  1.0 / kModulusA[10], 1.0 / kModulusA[11],
    1.0 / kModulusA[12], 1.0 / kModulusA[13], 1.0 / kModulusA[14]};

// int8 fragment of one 32-row block for one 32-byte K step: lane half fh
// takes 16-byte chunk 2 ks + fh of its row
__device__ __forceinline__ v4i frag_i8(const int8_t* base, int r, int ks, int fh) {
  return *reinterpret_cast<const v4i*>(base + r * BK + (((2 * ks + fh) ^ swz(r)) << 4));
}

// Centred residue of an int32 modulo m (odd, or 256), in [-(m/2), (m-1)/2]:
// |x| < 2^31, so the FP64 quotient x RN(1/m) is within 2^-21 / m of x / m,
// far closer than the 1/(2m) that separates x / m from a half integer for
// odd m; rint gives the nearest quotient and the FMA the exact remainder.
// For m = 256 the quotient is exact and the tie +128 maps to -128 (FOLD; an
// int8 store of +128 gives -128 by itself, and a partial reduction needs
// only |r| <= m/2).
template <bool FOLD>
__device__ __forceinline__ int cmod_i32(int x, int m, double minv) {
  const double xd = (double)x;
  const double q = __builtin_rint(xd * minv);
  const int r = (int)__builtin_fma(-q, (double)m, xd);
  return FOLD && 2 * r == m ? -r : r;
}

// One stage: four 32-byte K steps of 2 x BB MFMAs; the next stage's DMA
// loads go among step 0's MFMAs, the fragment reads of step ks + 1 among
// step ks's.
template <int S, int NB = Tile<S>::BB>
__device__ __forceinline__ void stage_mma_dma_i8(const int8_t* la, const int8_t* lb, int ra0,
                                                 int rb0, int fh, v16i (&acc)[2][NB],
                                                 __amdgpu_buffer_rsrc_t ra,
                                                 __amdgpu_buffer_rsrc_t rb, int8_t* na, int8_t* nb,
                                                 const int* voffa,
                                                 const int* voffb, int wave) {
  constexpr int ND = Tile<S>::DMA;
  v4i af[4][2], bf[4][NB];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
    for (int x = 0; x < 2; ++x) af[ks][x] = frag_i8(la, ra0 + 32 * x, ks, fh);
#pragma unroll
    for (int x = 0; x < NB; ++x) bf[ks][x] = frag_i8(lb, rb0 + 32 * x, ks, fh);
  }
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int j = ks * 2 * NB + a * NB + b;  // MFMA number in issue order
        if (j < ND) stage_dma<S>(j, ra, rb, na, nb, voffa, voffb, wave);
        acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[ks][a], bf[ks][b], acc[a][b], 0, 0, 0);
      }
  __builtin_amdgcn_sched_group_barrier(0x100, ND, 0);
#pragma unroll
  for (int i = 0; i < ND; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
#pragma unroll
  for (int i = 0; i < 2 * ND; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 8 * NB - 3 * ND > 0 ? 8 * NB - 3 * ND : 0, 0);
}

// Accurate mode (Sec. 2, Eq. (alpha)): the admissible total shift of one
// output from its magnitude bound U (the exact product of the digit
// planes): the largest L with U 2^L <= T = 2^8 (M/2 - 1).  bt is the bit
// length of T and ttop = T >> (bt - 33).  For U of b bits, T >> (bt - b) =
// ttop >> (33 - b) has b bits as well, so L is bt - b when U is at most
// that and bt - b - 1 otherwise.  U = 0 stores 127, and so does any L above
// it: no shift up to the cap of 58 is then constrained.
__device__ __forceinline__ int bound_total(int u, int bt, uint64_t ttop) {
  if (u <= 0) return 127;
  const int b = 32 - __builtin_clz((unsigned)u);
  const int L = (uint64_t)u <= (ttop >> (33 - b)) ? bt - b : bt - b - 1;
  return L < 127 ? L : 127;
}

// BOUND: the bound product of the accurate mode on the same pipeline -- one
// plane of digits (0..16) per operand, the plain int32 sum (at most
// 256 k <= 2^30, no reduction), stored as the total L (int8 OT) together
// with each wavefront's column minima over its 64 rows (colpart
// [ceil(m/64)][n]: rows past m have zero digits, so their L of 127 never
// lowers a minimum), or, for a split k range, as the raw partial sums
// (int32 OT; bound_totals_kernel adds them up).
template <typename OT, int S, bool BOUND = false>
__global__ __launch_bounds__(1024, 1) void residue_gemm_bytes_kernel(int64_t m, int64_t n,
                                                                    int64_t kp,
                                                                    const int8_t* __restrict__ pa,
                                                                    const int8_t* __restrict__ pb,
                                                                    OT* __restrict__ cres,
                                                                    int splits, int group,
                                                                    int bt = 0, uint64_t ttop = 0,
                                                                    int8_t* colpart = nullptr) {
  constexpr int BM = Tile<S>::BM, BN = Tile<S>::BN, NB = Tile<S>::BB, WC = Tile<S>::WC;
  constexpr int NPL = BOUND ? 1 : kRA;  // planes in the layout
  __shared__ __attribute__((aligned(1024))) int8_t lds_a0[BM * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b0[BN * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_a1[BM * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b1[BN * BK];
  const int64_t tiles_m = (m + BM - 1) / BM, tiles_n = (n + BN - 1) / BN;
  const int split = (int)(blockIdx.x % (unsigned)splits);
  int mod;
  int64_t tm, tn;
  block_coords(blockIdx.x / (unsigned)splits, (uint32_t)tiles_m, (uint32_t)tiles_n, (uint32_t)group, mod,
               tm, tn);
  const int mm = kModA[mod];
  cres += (int64_t)split * NPL * m * n;
  const double minv = kInvA[mod];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave / WC, wc = wave % WC;
  const int fr = lane & 31, fh = lane >> 5;
  const int ra0 = wr * 64 + fr, rb0 = wc * 32 * NB + fr;
  int voffa[Tile<S>::ADMA], voffb[Tile<S>::BDMA];
  slab_offsets(wave, lane, voffa);
  slab_offsets(wave, lane, voffb);
  const int64_t rows_a = m - tm * BM < BM ? m - tm * BM : BM;
  const int64_t rows_b = n - tn * BN < BN ? n - tn * BN : BN;
  const int na = __builtin_amdgcn_readfirstlane((int)(rows_a * BK));
  const int nb = __builtin_amdgcn_readfirstlane((int)(rows_b * BK));
  auto rsrc = [](const int8_t* p, int nrec) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(p), (short)0, nrec, 0x00020000);
  };

  v16i acc[2][NB];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = v16i{};

  const int nstage_all = (int)(kp / BK);
  // 32-bit: at most 2^15 stages times 64 splits
  const int sbeg = (int)((uint32_t)nstage_all * (uint32_t)split / (uint32_t)splits);
  const int nstage = (int)((uint32_t)nstage_all * (uint32_t)(split + 1) / (uint32_t)splits);  // one past the last
  // look-ahead cursor: stage ls and its A and B pieces, one K stage of the
  // plane layout apart (it stays on the panel's last stage)
  const int64_t step_a = (int64_t)NPL * m * BK, step_b = (int64_t)NPL * n * BK;
  const int8_t* const first_a = pa + (((int64_t)sbeg * NPL + mod) * m + tm * BM) * BK;
  const int8_t* const first_b = pb + (((int64_t)sbeg * NPL + mod) * n + tn * BN) * BK;
  int ls = sbeg;
  const int8_t* la = first_a;
  const int8_t* lb = first_b;
  auto advance = [&]() {
    if (ls + 1 < nstage) {
      ++ls;
      la += step_a;
      lb += step_b;
    }
  };
  // the bound product needs no reduction: one segment
  const int seg = BOUND ? nstage - sbeg : kSegA;
  for (int s0 = sbeg; s0 < nstage; s0 += seg) {
    const int s1 = s0 + seg < nstage ? s0 + seg : nstage;
    ls = s0;
    la = first_a + (int64_t)(s0 - sbeg) * step_a;
    lb = first_b + (int64_t)(s0 - sbeg) * step_b;
    stage_load<S>(rsrc(la, na), rsrc(lb, nb), lds_a0, lds_b0, voffa, voffb, wave);
    advance();
    for (int s = s0; s < s1; s += 2) {
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      // the DMA after the segment's last stage lands in the idle buffer; past
      // the panel's last stage it repeats that stage (as above)
      stage_mma_dma_i8<S>(lds_a0, lds_b0, ra0, rb0, fh, acc, rsrc(la, na), rsrc(lb, nb), lds_a1, lds_b1,
                           voffa, voffb, wave);
      advance();
      if (s + 1 >= s1) break;
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      stage_mma_dma_i8<S>(lds_a1, lds_b1, ra0, rb0, fh, acc, rsrc(la, na), rsrc(lb, nb), lds_a0, lds_b0,
                           voffa, voffb, wave);
      advance();
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // every wave is done with the buffers before the next segment loads
    if (!BOUND && s1 < nstage) {
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int v = 0; v < 16; ++v) acc[a][b][v] = cmod_i32<false>(acc[a][b][v], mm, minv);
    }
  }

  OT* out = (OT*)uniform_ptr((const int8_t*)(cres + (int64_t)mod * m * n + tm * BM * n + tn * BN));
  store_tile<false, OT, S>(out, (int)n, (int)(m - tm * BM), (int)(n - tn * BN), wr, wc, fr, fh,
                            [&](int a, int b, int v) {
                              if constexpr (BOUND)
                                return sizeof(OT) == 1 ? bound_total(acc[a][b][v], bt, ttop)
                                                       : acc[a][b][v];
                              else
                                return cmod_i32<sizeof(OT) == 4>(acc[a][b][v], mm, minv);
                            });
  if constexpr (BOUND && sizeof(OT) == 1) {
    // lane l holds column l % 32 of each block, rows 4 (l / 32) + ... of
    // both row blocks: its minimum, then the other half's by a swap
    const int64_t g = tm * (BM / 64) + wr;
    if (g * 64 < m) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        int mn = 127;
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int L = bound_total(acc[a][b][v], bt, ttop);
            mn = L < mn ? L : mn;
          }
        const int o = __shfl_xor(mn, 32, 64);
        mn = o < mn ? o : mn;
        const int64_t col = tn * BN + wc * 32 * NB + b * 32 + fr;
        if (fh == 0 && col < n) colpart[g * n + col] = (int8_t)mn;
      }
    }
  }
}

// The split bound product's partial sums [splits][m][n], added and turned
// into totals and the column minima of each 64-row group: a thread per
// column (consecutive threads, consecutive columns), a block row per group.
__global__ __launch_bounds__(256) void bound_totals_kernel(int64_t m, int64_t n, int splits,
                                                           const int32_t* __restrict__ part,
                                                           int8_t* __restrict__ total,
                                                           int8_t* __restrict__ colpart, int bt,
                                                           uint64_t ttop) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t g = blockIdx.y;
  if (j >= n) return;
  const int64_t mn = m * n;
  const int64_t i1 = g * 64 + 64 < m ? g * 64 + 64 : m;
  int low = 127;
  for (int64_t i = g * 64; i < i1; ++i) {
    int sum = 0;
    for (int sp = 0; sp < splits; ++sp) sum += part[sp * mn + i * n + j];
    const int L = bound_total(sum, bt, ttop);
    total[i * n + j] = (int8_t)L;
    low = L < low ? L : low;
  }
  colpart[g * n + j] = (int8_t)low;
}

// Sum of the splits' centred partial products, reduced to the centred
// residue: |sum| <= splits * 545 < 2^16, exact in FP32, and the FP32
// quotient of an integer below 2^16 by m errs far less than the 1/(2m)
// that separates it from a half integer for odd m; for even m (1024, 256)
// the tie +m/2 maps to -m/2.  Grid: x over m n, y over the moduli.
template <bool BYTES, typename OT>
__global__ __launch_bounds__(256) void reduce_splits_kernel(int64_t mn, int splits,
                                                            const OT* __restrict__ part,
                                                            OT* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= mn) return;
  const int q = blockIdx.y;
  const int mm = BYTES ? kModA[q] : kSched[q].m;
  const int64_t stride = (int64_t)(BYTES ? kRA : kR) * mn;
  const int64_t at = (int64_t)q * mn + i;
  int sum = 0;
  for (int sp = 0; sp < splits; ++sp) sum += (int)part[sp * stride + at];
  const float qf = __builtin_rintf((float)sum * (1.0f / (float)mm));
  int r = sum - (int)qf * mm;
  r = 2 * r == mm ? -r : r;
  out[at] = (OT)r;
}

// Tile shape for n columns, on both routes: at most 128 columns take the
// 512 x 128 tile, more columns 256 x 256.
constexpr int gemm_shape(bool bytes, int64_t n) { return n <= 128 ? 3 : 2; }
constexpr int64_t gemm_blocks(bool bytes, int64_t m, int64_t n) {
  const bool tall = gemm_shape(bytes, n) == 3;
  const int64_t bm = tall ? Tile<3>::BM : Tile<2>::BM, bn = tall ? Tile<3>::BN : Tile<2>::BN;
  return (int64_t)(bytes ? kRA : kR) * ((m + bm - 1) / bm) * ((n + bn - 1) / bn);
}

// Persistent form of the int8 product for short k (the compact int8
// output, one segment: at most 16 stages, an even count), as the FP8 one:
// one block per CU walking virtual tiles blockIdx.x + j gridDim.x, the next
// tile's first stage loaded during the current one's last stage and its
// stores, every barrier a full wait.
template <typename OT, int S>
__global__ __launch_bounds__(1024, 1) void residue_gemm_bytes_persistent_kernel(
    int64_t m, int64_t n, int64_t kp, const int8_t* __restrict__ pa, const int8_t* __restrict__ pb,
    OT* __restrict__ cres, int group, uint32_t nvirt) {
  constexpr int BM = Tile<S>::BM, BN = Tile<S>::BN, NB = Tile<S>::BB, WC = Tile<S>::WC;
  static_assert(sizeof(OT) == 1, "the compact int8 residue output");
  __shared__ __attribute__((aligned(1024))) int8_t lds_a0[BM * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b0[BN * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_a1[BM * BK];
  __shared__ __attribute__((aligned(1024))) int8_t lds_b1[BN * BK];
  const int64_t tiles_m = (m + BM - 1) / BM, tiles_n = (n + BN - 1) / BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave / WC, wc = wave % WC;
  const int fr = lane & 31, fh = lane >> 5;
  const int ra0 = wr * 64 + fr, rb0 = wc * 32 * NB + fr;
  int voffa[Tile<S>::ADMA], voffb[Tile<S>::BDMA];
  slab_offsets(wave, lane, voffa);
  slab_offsets(wave, lane, voffb);

  const int nstage = (int)(kp / BK);  // even, at most 16 (the host checks)
  const int64_t step_a = (int64_t)kRA * m * BK, step_b = (int64_t)kRA * n * BK;
  auto rsrc = [](const int8_t* p, int nrec) __attribute__((always_inline)) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(p), (short)0, nrec, 0x00020000);
  };
  struct TileAt {
    int mod;
    int64_t tm, tn;
    int na, nb;
  };
  auto tile_at = [&](uint32_t v) __attribute__((always_inline)) {
    TileAt t;
    block_coords(v, (uint32_t)tiles_m, (uint32_t)tiles_n, (uint32_t)group, t.mod, t.tm, t.tn);
    const int64_t rows_a = m - t.tm * BM < BM ? m - t.tm * BM : BM;
    const int64_t rows_b = n - t.tn * BN < BN ? n - t.tn * BN : BN;
    t.na = __builtin_amdgcn_readfirstlane((int)(rows_a * BK));
    t.nb = __builtin_amdgcn_readfirstlane((int)(rows_b * BK));
    return t;
  };
  auto first_a = [&](const TileAt& t) __attribute__((always_inline)) {
    return pa + ((int64_t)t.mod * m + t.tm * BM) * BK;
  };
  auto first_b = [&](const TileAt& t) __attribute__((always_inline)) {
    return pb + ((int64_t)t.mod * n + t.tn * BN) * BK;
  };

  uint32_t v = blockIdx.x;
  if (v >= nvirt) return;
  TileAt cur = tile_at(v), nxt = cur;
  bool have_next = false, ahead = false;
  // look-ahead cursor: stage ls of the current tile (or, once ahead, the
  // next tile's first stage), its pieces and their tile's bytes
  int ls = 0, lna = cur.na, lnb = cur.nb;
  const int8_t* la = first_a(cur);
  const int8_t* lb = first_b(cur);
  auto advance = [&]() __attribute__((always_inline)) {
    if (ahead) return;
    if (ls + 1 < nstage) {
      ++ls;
      la += step_a;
      lb += step_b;
    } else if (have_next) {
      ahead = true;
      la = first_a(nxt);
      lb = first_b(nxt);
      lna = nxt.na;
      lnb = nxt.nb;
    }
  };
  stage_load<S>(rsrc(la, lna), rsrc(lb, lnb), lds_a0, lds_b0, voffa, voffb, wave);
  for (;;) {
    const uint32_t vn = v + gridDim.x;
    have_next = vn < nvirt;
    if (have_next) nxt = tile_at(vn);
    advance();
    v16i acc[2][NB];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[a][b] = v16i{};
    for (int G = 0; G < nstage; G += 2) {
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      stage_mma_dma_i8<S>(lds_a0, lds_b0, ra0, rb0, fh, acc, rsrc(la, lna), rsrc(lb, lnb), lds_a1, lds_b1,
                           voffa, voffb, wave);
      advance();
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      stage_mma_dma_i8<S>(lds_a1, lds_b1, ra0, rb0, fh, acc, rsrc(la, lna), rsrc(lb, lnb), lds_a0, lds_b0,
                           voffa, voffb, wave);
      advance();
    }
    const int mm = kModA[cur.mod];
    const double minv = kInvA[cur.mod];
    OT* out = (OT*)uniform_ptr((const int8_t*)(cres + (int64_t)cur.mod * m * n + cur.tm * BM * n +
                                               cur.tn * BN));
    // the store offsets from a lane index read here (as in the FP8 form)
    const int el = lane_id_now() & 63;
    store_tile<false, OT, S>(out, (int)n, (int)(m - cur.tm * BM), (int)(n - cur.tn * BN), wr, wc, el & 31,
                              el >> 5, [&](int a, int b, int vv) { return cmod_i32<false>(acc[a][b][vv], mm, minv); });
    if (!have_next) break;
    v = vn;
    cur = nxt;
    ls = 0;
    ahead = false;
  }
  __builtin_amdgcn_s_waitcnt(0);  // the last look-ahead (a repeat) lands before the block ends
}

template <bool BYTES, typename OT>
hipError_t launch_gemm(int64_t m, int64_t n, int64_t kp, const int8_t* pa, const int8_t* pb,
                       OT* cres, OT* part, int splits, hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  // the store epilogue uses 32-bit offsets within a tile (at most 256 rows
  // when n > 128)
  if (n > kMaxResidueCols) return hipErrorInvalidValue;
  const int nstage = (int)(kp / BK);
  if (splits < 1 || splits > (nstage > 1 ? nstage : 1) || (splits > 1 && !part))
    return hipErrorInvalidValue;
  const int shape = gemm_shape(BYTES, n);
  // tile rows per group of the block order: 2; short k (at most 16 stages,
  // panels of at most 512 KiB per plane) 1 on the FP8 route, 4 on the int8
  // one (measured on the 32768^2 x 1024 update: 33.7 -> 32.7 ms and 20.6 ->
  // 19.4 ms; 8192^3 and ragged 8191 x 8209 x 7937 are fastest with 2)
  const int group = kp <= 16 * BK ? (BYTES ? 4 : 1) : 2;
  const int64_t blocks = gemm_blocks(BYTES, m, n);
  OT* dst = splits > 1 ? part : cres;
  // block indices (and block_coords' arithmetic) are 32-bit
  if (blocks * splits > (int64_t)UINT32_MAX) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(blocks * splits));
  if constexpr (sizeof(OT) < 4) {
    // the persistent form for short k, where a tile's first-stage load and
    // its stores are a larger share of its time: one block per CU (a
    // multiple of 8, so a block keeps its XCD), at least two tiles each,
    // whole k, a nonzero even stage count (measured on the 32768^2 x 1024
    // update: FP8 34.7 -> 34.0 ms, int8 19.8 -> 17.9 ms; no change on
    // 8192^3, which keeps the grid of one block per tile); the tile ids
    // plus one grid stay below 2^32
    int dev = 0, cus = 0;
    if (splits == 1 && nstage >= 2 && nstage <= 16 && nstage % 2 == 0 && hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cus >= 8 && blocks >= 2 * (int64_t)(cus / 8 * 8) && blocks <= (int64_t)UINT32_MAX - cus) {
      const dim3 pgrid((unsigned)(cus / 8 * 8));
      if constexpr (BYTES) {
        if (shape == 3)
          hipLaunchKernelGGL((residue_gemm_bytes_persistent_kernel<OT, 3>), pgrid, dim3(1024), 0, stream, m,
                             n, kp, pa, pb, dst, group, (uint32_t)blocks);
        else
          hipLaunchKernelGGL((residue_gemm_bytes_persistent_kernel<OT, 2>), pgrid, dim3(1024), 0, stream, m,
                             n, kp, pa, pb, dst, group, (uint32_t)blocks);
      } else {
        if (shape == 3)
          hipLaunchKernelGGL((residue_gemm_persistent_kernel<OT, 3>), pgrid, dim3(1024), 0, stream, m, n,
                             kp, pa, pb, dst, group, (uint32_t)blocks);
        else
          hipLaunchKernelGGL((residue_gemm_persistent_kernel<OT, 2>), pgrid, dim3(1024), 0, stream, m, n,
                             kp, pa, pb, dst, group, (uint32_t)blocks);
      }
      return hipGetLastError();
    }
  }
  if constexpr (BYTES) {
    if (shape == 3)
      hipLaunchKernelGGL((residue_gemm_bytes_kernel<OT, 3>), grid, dim3(1024), 0, stream, m, n, kp, pa,
                         pb, dst, splits, group);
    else
      hipLaunchKernelGGL((residue_gemm_bytes_kernel<OT, 2>), grid, dim3(1024), 0, stream, m, n, kp, pa,
                         pb, dst, splits, group);
  } else {
    if (shape == 3)
      hipLaunchKernelGGL((residue_gemm_kernel<OT, 3>), grid, dim3(1024), 0, stream, m, n, kp, pa, pb,
                         dst, splits, group);
    else
      hipLaunchKernelGGL((residue_gemm_kernel<OT, 2>), grid, dim3(1024), 0, stream, m, n, kp, pa, pb,
                         dst, splits, group);
  }
  if (splits > 1) {
    const int64_t mn = m * n;
    hipLaunchKernelGGL((reduce_splits_kernel<BYTES, OT>),
                       dim3((unsigned)((mn + 255) / 256), (unsigned)(BYTES ? kRA : kR)), dim3(256), 0,
                       stream, mn, splits, part, cres);
  }
  return hipGetLastError();
}

}  // namespace

namespace {

// Split the k range when the output tiles leave most of the chip idle.  A
// block holds a whole CU, so blocks run in rounds of kCUs; the split count
// minimises rounds x (fixed cost of a block + its stages), the fixed cost
// (prologue, carries, epilogue) measured at about seven stage times, with
// at least 2 stages of each product per block (4 for the single-product
// int8 kernel).
int best_splits(int64_t blocks, int64_t nstage, bool bytes) {
  constexpr int64_t kCUs = 256, kFixedStages = 7;
  if (blocks >= 512) return 1;
  int64_t cap = nstage / (bytes ? 4 : 2);
  if (cap > kMaxSplits) cap = kMaxSplits;
  const int64_t prods = bytes ? 1 : 3;
  int64_t best = -1, best_s = 1;
  for (int64_t s = 1; s <= cap; ++s) {
    const int64_t rounds = (blocks * s + kCUs - 1) / kCUs;
    const int64_t t = rounds * (kFixedStages + prods * ((nstage + s - 1) / s));
    if (best < 0 || t < best) {
      best = t;
      best_s = s;
    }
  }
  return (int)best_s;
}

}  // namespace

int residue_gemm_splits(int set, int64_t m, int64_t n, int64_t kp) {
  if (m <= 0 || n <= 0) return 1;
  const bool bytes = set == kSetBytes;
  return best_splits(gemm_blocks(bytes, m, n), kp / BK, bytes);
}

int bound_gemm_splits(int64_t m, int64_t n, int64_t kp) {
  if (m <= 0 || n <= 0) return 1;
  return best_splits(gemm_blocks(true, m, n) / kRA, kp / BK, true);
}

hipError_t launch_bound_gemm(int64_t m, int64_t n, int64_t kp, const int8_t* da, const int8_t* db,
                             int8_t* total, int8_t* colpart, int32_t* part, int splits, int bt, uint64_t ttop,
                             hipStream_t stream) {
  if (m <= 0 || n <= 0) return hipSuccess;
  if (n > kMaxResidueCols) return hipErrorInvalidValue;
  const int nstage = (int)(kp / BK);
  if (nstage < 1 || splits < 1 || splits > nstage || (splits > 1 && !part)) return hipErrorInvalidValue;
  const int shape = gemm_shape(true, n);
  const int group = kp <= 16 * BK ? 4 : 2;
  const int64_t blocks = gemm_blocks(true, m, n) / kRA;
  if (blocks * splits > (int64_t)UINT32_MAX) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(blocks * splits));
  if (splits == 1) {
    if (shape == 3)
      hipLaunchKernelGGL((residue_gemm_bytes_kernel<int8_t, 3, true>), grid, dim3(1024), 0, stream, m, n,
                         kp, da, db, total, 1, group, bt, ttop, colpart);
    else
      hipLaunchKernelGGL((residue_gemm_bytes_kernel<int8_t, 2, true>), grid, dim3(1024), 0, stream, m, n,
                         kp, da, db, total, 1, group, bt, ttop, colpart);
  } else {
    if (shape == 3)
      hipLaunchKernelGGL((residue_gemm_bytes_kernel<int32_t, 3, true>), grid, dim3(1024), 0, stream, m, n,
                         kp, da, db, part, splits, group, bt, ttop);
    else
      hipLaunchKernelGGL((residue_gemm_bytes_kernel<int32_t, 2, true>), grid, dim3(1024), 0, stream, m, n,
                         kp, da, db, part, splits, group, bt, ttop);
    const int64_t groups = (m + 63) / 64;
    if ((n + 255) / 256 > (int64_t)UINT32_MAX || groups > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL(bound_totals_kernel, dim3((unsigned)((n + 255) / 256), (unsigned)groups), dim3(256), 0,
                       stream, m, n, splits, part, total, colpart, bt, ttop);
  }
  return hipGetLastError();
}

hipError_t launch_residue_gemm_i32(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                   const int8_t* pb, int32_t* cres, hipStream_t stream) {
  return launch_gemm<false, int32_t>(m, n, kp, pa, pb, cres, nullptr, 1, stream);
}

hipError_t launch_residue_gemm_i16(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                   const int8_t* pb, int16_t* cres, int16_t* part, int splits,
                                   hipStream_t stream) {
  return launch_gemm<false, int16_t>(m, n, kp, pa, pb, cres, part, splits, stream);
}

hipError_t launch_residue_gemm_bytes_i32(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                         const int8_t* pb, int32_t* cres, hipStream_t stream) {
  return launch_gemm<true, int32_t>(m, n, kp, pa, pb, cres, nullptr, 1, stream);
}

hipError_t launch_residue_gemm_bytes_i8(int64_t m, int64_t n, int64_t kp, const int8_t* pa,
                                        const int8_t* pb, int8_t* cres, int8_t* part, int splits,
                                        hipStream_t stream) {
  return launch_gemm<true, int8_t>(m, n, kp, pa, pb, cres, part, splits, stream);
}

}  // namespace oz
