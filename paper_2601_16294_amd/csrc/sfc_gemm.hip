// Persistent MFMA GEMM for gfx950 (bf16 operands, or OCP FP8 E4M3 operands)
// whose output blocks are taken in space-filling-curve order, with the
// communication-avoiding K split.
//
// What it computes (Listing 1, Section II.D): the task space has gm*gn*layers
// entries; task t is layer l = t / (gm*gn) and curve position s = t % (gm*gn);
// the curve table maps s to the output block (im, in); layer l contracts the
// l-th contiguous range of K blocks (64 deep for bf16, 128 for fp8) into its
// own copy of the block.
// With one layer the copy is C itself (fp32 or bf16); with several it is an
// fp32 workspace layer that a separate reduction sums.
//
// Mapping to the chip:
//   * one workgroup = 4 waves (one per SIMD; 1 x 4 for blocks 256 columns
//     wide, except fp8 256x256, else 2 x 2), each wave owning its sub-block as
//     16x16 fp32 MFMA accumulators;
//   * the grid is persistent: P workgroups, P = CUs x occupancy, each looping
//     over tasks.  Hardware deals workgroup b to chiplet (XCD) b % 8; ranks are
//     renumbered so that each XCD's workgroups hold consecutive ranks, and with
//     the interleaved schedule the P tasks in flight are one contiguous curve
//     segment whose XCD sub-segments are compact patches sharing A rows and B
//     columns in that XCD's L2;
//   * fast path (16-byte aligned rows): A and B go straight from global memory
//     into LDS with buffer loads (lanes outside the matrix read zeros), A in a
//     ring of three 64-deep block slots [BM][64], B in a ring of four 32-deep
//     stage slots [32][BN], with one barrier per 64-deep block.  Every
//     32-deep step has a fixed plan: one MFMA per group, beside it at most one
//     fragment read of the next step and one load operation for the blocks
//     ahead, and small pieces of the scalar bookkeeping (a wave issues one
//     instruction every 4 cycles, a 16x16x32 MFMA takes 16);
//   * general path (any alignment): elements assembled in registers, two
//     64-deep LDS buffers;
//   * the MFMA B operand is read from [k][n] with the transposing LDS read
//     (ds_read_b64_tr_b16); 16-byte chunks are XOR-swizzled so that the
//     fragment reads and the staging writes are free of bank conflicts on the
//     64-bank LDS;
//   * bf16 MFMA 16x16x32 with fp32 accumulation (Section III.A's BRGEMM role).
//     With random operands it holds a higher clock than 32x32x16 for the same
//     work per clock;
//   * bf16 output: v_permlane16_swap pairs two fragments so that every lane
//     stores 8 consecutive columns (16 bytes); a store instruction costs about
//     the same whatever its width, so this halves the epilogue.
//   * fp8 operands (F8 = 1 + a + 2b with a, b the OCP formats of A and B, 0 for
//     E4M3 and 1 for E5M2; F8 = 0 for bf16): the rings hold the same bytes (an A block row is 128
//     fp8, a B stage 64 rows of BN fp8); each 64-deep step is MFMA 32x32x64
//     f8f6f4 per 32x32 fragment, fed by two 16-byte A reads and four
//     ds_read_b64_tr_b8 B reads per fragment, and the 32x32 accumulators are
//     stored by store_tile32.
#include <type_traits>
#include <utility>

#include "sfc_params.h"

namespace sfc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) const bf16x8 lds_bf16x8;

// ---- chiplet-aware rank ------------------------------------------------------
// Workgroup b runs on XCD b % 8.  Ranks give each XCD a contiguous range.
__device__ __forceinline__ int xcd_rank(int b, int P) {
  constexpr int X = 8;
  const int x = b % X, i = b / X;
  const int q = P / X, r = P % X;
  return x * q + (x < r ? x : r) + i;
}

// ---- LDS layouts ---------------------------------------------------------------
// A block: [BM rows][64 k] bf16, 8 chunks of 16 B per row; chunk c of row r is
// stored at chunk c ^ ((r >> 1) & 7).  The 16 consecutive rows that one quarter
// of a wave reads at one logical chunk land on 16 distinct 16-byte bank groups.
__device__ __forceinline__ int a_off(int row, int chunk) {
  return row * kBK + ((chunk ^ ((row >> 1) & 7)) << 3);
}
// B block: [K k][BN n] bf16 (K = 64 or 32); chunk c (8 columns) of row k is
// stored at chunk c ^ b_swz(k).  One pass of the transposing read (32 lanes)
// touches rows k0..k0+3 and k0+8..k0+11 at 2 chunks; the swizzle puts those 16
// pieces on 16 distinct 16-byte bank groups.
__device__ __forceinline__ int b_swz(int k) { return ((k & 3) << 2) | (((k >> 3) & 1) << 1); }
template <int BN>
__device__ __forceinline__ int b_off(int k, int n) {
  return k * BN + ((((n >> 3) ^ b_swz(k))) << 3) + (n & 7);
}

// ---- global -> register staging -------------------------------------------------
template <bool VEC>
__device__ __forceinline__ u32x4 load_chunk(const uint16_t* base, int64_t ld, int64_t row,
                                            int64_t col, int64_t rows, int64_t cols) {
  u32x4 v = {0u, 0u, 0u, 0u};
  if (VEC) {
    // cols is a multiple of 8 and rows are 16-byte aligned: a chunk is all in or all out.
    if (row < rows && col < cols) v = *reinterpret_cast<const u32x4*>(base + row * ld + col);
  } else {
    if (row < rows) {
      const uint16_t* p = base + row * ld;
      uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t h = (col + e < cols) ? (uint32_t)p[col + e] : 0u;
        w[e >> 1] |= h << ((e & 1) * 16);
      }
      v[0] = w[0]; v[1] = w[1]; v[2] = w[2]; v[3] = w[3];
    }
  }
  return v;
}

// ---- direct global -> LDS loads (fast path) ----------------------------------------
// buffer_load_dwordx4 ... offset:O lds: every lane fetches 16 bytes at (descriptor
// base + its voffset + O) and the wave writes them to LDS at M0 + O + 16*lane.  A
// lane whose voffset + O lies at or beyond the descriptor's num_records fetches
// zeros.  The instruction is issued from inline assembly so that the compiler
// does not serialise later LDS reads behind it; the kernel orders it explicitly
// with s_waitcnt vmcnt and workgroup barriers.  Raw buffer descriptor: 48-bit
// base, stride 0, num_records, word 3 = 0x00020000 on gfx9 parts.
typedef int i32x4 __attribute__((ext_vector_type(4)));
constexpr int kOobOffset = 0x7FFFFFF0;   // largest num_records; a lane at this offset reads zeros

// One 32-bit scalar load from global memory (the table written by an earlier
// dispatch), waited for at once.
__device__ __forceinline__ int load_scalar_i32(const int32_t* p) {
  int v;
  asm volatile("s_load_dword %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(v) : "s"(p) : "memory");
  return v;
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

template <int N>
__device__ __forceinline__ void wait_vmem_at_most() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}
__device__ __forceinline__ void wait_lds_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }


// ---- MFMA 16x16x32 fragments -------------------------------------------------------------
// The MFMA takes the B fragment as its first operand, so it computes the
// transposed 16x16 block: lane l ends with row l%16 of the fragment and its 4
// consecutive columns 4*(l/16) .. +3.
// NW = 4 waves per workgroup (one per SIMD) in a WGM x WGN grid.  A wave's
// fragment reads per 32-deep step are FM b128 reads of A and 2*FN transposing
// reads of B.  A transposing read takes about twice the LDS time of a b128
// read per byte and, unlike b128 reads, slows the global-to-LDS loads that run
// beside it, so blocks 256 columns wide put the 4 waves side by side (1 x 4:
// 128x64 or, for bf16 256x256, 256x64 per wave, a quarter of B each) and the
// narrower blocks keep 2 x 2.  (fp8 256x256 blocks stay 2 x 2: 1 x 4 measured
// 1.5 % slower there.)
template <int BM, int BN, int NW, int F8>
struct Tile {
  static_assert(NW == 4, "4 waves");
  static constexpr int THREADS = NW * 64;
  static constexpr int WGM = (BN == 256 && (BM == 128 || F8 == 0)) ? 1 : 2;  // waves along M
  static constexpr int WGN = NW / WGM;                // waves along N
  static constexpr int WTM = BM / WGM, WTN = BN / WGN;  // wave sub-block
  // fragments per wave: 16x16 (bf16, MFMA 16x16x32) or 32x32 (fp8, MFMA 32x32x64)
  static constexpr int FS = F8 ? 32 : 16;
  static constexpr int FM = WTM / FS, FN = WTN / FS;
  static constexpr int A_ELEMS = BM * kBK, B_ELEMS = kBK * BN;
  static constexpr int A_CH = BM * kBK / 8 / THREADS;   // 16-byte chunks per thread
  static constexpr int B_CH = kBK * BN / 8 / THREADS;
};

// One accumulator fragment: 16x16 fp32 (4 per lane) or 32x32 fp32 (16 per lane).
template <int F8>
using AccFrag = typename std::conditional<(F8 != 0), f32x16, f32x4>::type;
template <int BM, int BN, int NW, int F8>
using Acc = AccFrag<F8>[Tile<BM, BN, NW, F8>::FM][Tile<BM, BN, NW, F8>::FN];

// Operand fragments of one step: 8 bf16 per lane (16x32), or 32 fp8 bytes per
// lane (32x64).
template <int F8>
using OpFrag = typename std::conditional<(F8 != 0), i32x8, bf16x8>::type;
template <int BM, int BN, int NW, int F8>
struct Frags {
  OpFrag<F8> a[Tile<BM, BN, NW, F8>::FM];
  OpFrag<F8> b[Tile<BM, BN, NW, F8>::FN];
};

// Per-lane LDS element offsets of the fragment reads of one 32-deep step:
// A fragment i of step ks (0 or 1 within a 64-deep block) is 16 rows x 32 k,
// lane l holding row l%16, k = 8*(l/16) .. +8; the swizzle does not depend on
// i, so fragment i sits i*16*64 elements further.  B fragment j is 32 k x 16
// columns, lane l holding column l%16, k = 8*(l/16) .. +8, assembled from two
// transposing reads of 4 rows each (the second 4 rows further).
__device__ __forceinline__ int a_frag_off(int wm_rows, int lane, int ks) {
  const int row = wm_rows + (lane & 15);
  return a_off(row, ks * 4 + (lane >> 4));
}
template <int BN>
__device__ __forceinline__ int b_frag_off(int wn_cols, int lane, int kbase, int j) {
  // Lane (g = l/16, jj = l%16) points at row 8g + jj/4, columns n .. n+3 with
  // n = 16j + 4*(jj%4); the transposing read returns column jj of the 4 rows
  // to lane jj of each group of 16.
  const int g = lane >> 4, jj = lane & 15;
  const int k = kbase + 8 * g + (jj >> 2);
  const int n = wn_cols + j * 16 + ((jj & 3) << 2);
  return b_off<BN>(k, n);
}

__device__ __forceinline__ bf16x8 read_b_pair(const uint16_t* p, int half_stride) {
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + half_stride));
  const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// All operand fragments of one 32-deep step from an A block [BM][64] (step
// ks) and a B buffer [..][BN] (rows kbase .. kbase+31).
template <int BM, int BN, int NW, int F8>
__device__ __forceinline__ void load_frags(const uint16_t* As, const uint16_t* Bs, int wm, int wn,
                                           int lane, int ks, int kbase, Frags<BM, BN, NW, F8>& f) {
  using T = Tile<BM, BN, NW, F8>;
  const int ao = a_frag_off(wm * T::WTM, lane, ks);
#pragma unroll
  for (int i = 0; i < T::FM; ++i) f.a[i] = *reinterpret_cast<const bf16x8*>(As + ao + i * 16 * kBK);
#pragma unroll
  for (int j = 0; j < T::FN; ++j) f.b[j] = read_b_pair(Bs + b_frag_off<BN>(wn * T::WTN, lane, kbase, j), 4 * BN);
}

// acc += one 32-deep step.
template <int BM, int BN, int NW, int F8>
__device__ __forceinline__ void mma_step(const Frags<BM, BN, NW, F8>& cur, Acc<BM, BN, NW, F8>& acc) {
  using T = Tile<BM, BN, NW, F8>;
#pragma unroll
  for (int i = 0; i < T::FM; ++i)
#pragma unroll
    for (int j = 0; j < T::FN; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur.b[j], cur.a[i], acc[i][j], 0, 0, 0);
}

// ---- fast path: rings of LDS slots ---------------------------------------------------------
// A is staged per 64-deep block, in three slots of [BM][64]: a row of a block is
// one full 128-byte line of A.  B is staged per 32-deep stage, in four slots of
// [32][BN].  A 32-deep stage is one MFMA step.  Loads are buffer loads of 1 KiB
// (16 B per lane) written straight into LDS.  Wave w loads A segments w*APB ..
// +APB-1 (8 rows each) of a block and B segments w*BPW .. +BPW-1 of a stage; a
// wave's segments are consecutive KiB, so up to four share one M0 value and
// differ only in the instruction offset, which the hardware adds to both the
// LDS address and the memory address.  The per-lane voffset is biased by kBias
// - offset and the descriptor base lowered by kBias to cancel the memory side.
//
// Every instruction of the loop counts: with one wave per SIMD a wave issues
// at most one instruction per four clocks, so the loop keeps its other work
// (LDS reads, loads, address arithmetic) to a few instructions per MFMA,
// spread evenly.
constexpr int kSK = 32;        // K depth of one B stage (one MFMA step)
constexpr int kBias = 4096;    // bytes; keeps every biased voffset positive

// The rings hold the same bytes for both element types: a block row is 128
// bytes (64 bf16 or 128 fp8 elements of K), a B stage is 64*BN bytes (32 rows
// of BN bf16 or 64 rows of BN fp8).  K depth, in elements, of a block and of a
// B stage:
template <int F8>
constexpr int block_k() { return F8 ? 128 : kBK; }
template <int F8>
constexpr int stage_k() { return F8 ? 64 : kSK; }
// fp8 B stages: chunk c (16 columns) of row k is stored at chunk c ^ (2*(k&7));
// a transposing read of 8 consecutive rows at two adjacent chunks (2m, 2m+1)
// then touches 16 distinct 16-byte bank groups.
__device__ __forceinline__ int b_swz8(int k) { return (k & 7) << 1; }

// The loads of block b+D are issued during block b (prefetch depth D): the A
// ring has D+1 block slots, the B ring 2D stage slots.  By default D = 3 where
// the LDS holds that at the same occupancy (128x256: exactly 160 KiB), else 2.
// 128x128 blocks run two workgroups per CU at D = 2 (80 KiB each); when a grid
// has no more blocks than CUs that occupancy buys nothing, and a kernel with
// D = 4 (144 KiB, one workgroup per CU) keeps twice the blocks in flight, which
// is what a short grid with long K is bound by (the latency of its operand
// stream).
template <int BM, int BN>
constexpr int default_depth() { return (BM == 128 && BN == 256) ? 3 : 2; }

template <int BM, int BN, int NW, int F8, int DEPTH = default_depth<BM, BN>()>
struct Ring {
  static constexpr int A_BLK = BM * kBK;                 // elements of one A block
  static constexpr int B_STG = kSK * BN;                 // elements of one B stage
  static constexpr int A_BYTES = A_BLK * 2, B_BYTES = B_STG * 2;
  static constexpr int D = DEPTH;
  static constexpr int NA = D + 1, NB = 2 * D;           // A block slots, B stage slots
  static constexpr int B_OFF = NA * A_BYTES;             // byte offset of the B slots
  static constexpr int APB = A_BYTES / 1024 / NW;        // A loads per wave per block
  static constexpr int BPW = B_BYTES / 1024 / NW;        // B loads per wave per stage
  static constexpr int ELEMS = NA * A_BLK + NB * B_STG;
  // loads younger than block b+1's, when block b's barrier waits for it
  static constexpr int IN_FLIGHT = (D - 2) * (APB + 2 * BPW) + APB;
  static_assert(APB % 4 == 0 && (BPW == 2 || BPW == 4), "tile shape");
  static_assert(ELEMS * 2 <= 160 * 1024, "LDS of one CU");
  static_assert(IN_FLIGHT <= 63, "vmcnt range");
  static_assert(D >= 2 && D <= 4, "ring depth");
};

// Two loads sharing M0: LDS M0+OFF+16*lane and M0+OFF+1024+16*lane.
template <int OFF>
__device__ __forceinline__ void dma16_pair(i32x4 rsrc, uint32_t m0_value, int v0, int v1) {
  static_assert(OFF + 1024 <= 4095, "instruction offset range");
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\t"
               "buffer_load_dwordx4 %1, %3, 0 offen offset:%4 lds\n\t"
               "buffer_load_dwordx4 %2, %3, 0 offen offset:%5 lds"
               :: "s"(m0_value), "v"(v0), "v"(v1), "s"(rsrc), "n"(OFF), "n"(OFF + 1024) : "memory");
}

// Make a scalar opaque to the optimiser, so that an update stays where the code
// puts it (induction-variable rewriting would otherwise move the per-block
// address updates together to the end of the loop body).
template <typename V>
__device__ __forceinline__ void pin_scalar(V& v) {
  asm volatile("" : "+s"(v));
}

__device__ __forceinline__ i32x4 make_rsrc_addr(uint64_t a, uint32_t num_records) {
  i32x4 r = {(int)(uint32_t)a, (int)((uint32_t)(a >> 32) & 0xFFFFu), (int)num_records, 0x00020000};
  r[0] = __builtin_amdgcn_readfirstlane(r[0]);
  r[1] = __builtin_amdgcn_readfirstlane(r[1]);
  r[2] = __builtin_amdgcn_readfirstlane(r[2]);
  return r;
}
// The same descriptor in two steps, for code that spreads scalar work thinly:
// the address words first (wave-uniform values), then the descriptor.
__device__ __forceinline__ void rsrc_words(uint64_t a, uint32_t& lo, uint32_t& hi) {
  lo = (uint32_t)a;
  hi = (uint32_t)(a >> 32) & 0xFFFFu;
}
__device__ __forceinline__ i32x4 rsrc_of_words(uint32_t lo, uint32_t hi, uint32_t num_records) {
  return i32x4{(int)lo, (int)hi, (int)num_records, 0x00020000};
}

// Per-lane, per-task load offsets (bytes, biased).
template <int BM, int BN, int NW, int F8>
struct RingLanes {
  int a_voff[Ring<BM, BN, NW, F8>::APB];
  int b_voff[Ring<BM, BN, NW, F8>::BPW];
};

// K index (within a block, in elements) at which A load j of this lane starts.
template <int F8>
__device__ __forceinline__ int a_load_k(int wave, int apb, int j, int lane) {
  const int row = (wave * apb + j) * 8 + (lane >> 3);
  return ((lane & 7) ^ ((row >> 1) & 7)) * (F8 ? 16 : 8);
}

template <int BM, int BN, int NW, int F8>
__device__ __forceinline__ void ring_lanes(const GemmParams& p, int64_t m0, int64_t n0, int wave,
                                           int lane, RingLanes<BM, BN, NW, F8>& L) {
  using R = Ring<BM, BN, NW, F8>;
#pragma unroll
  for (int j = 0; j < R::APB; ++j) {
    const int row = (wave * R::APB + j) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    if constexpr (F8 != 0)
      L.a_voff[j] = (m0 + row < p.M) ? (int)(row * p.lda + c * 16) + kBias - (j & 3) * 1024 : kOobOffset;
    else
      L.a_voff[j] = (m0 + row < p.M) ? (int)((row * p.lda + c * 8) * 2) + kBias - (j & 3) * 1024 : kOobOffset;
  }
#pragma unroll
  for (int j = 0; j < R::BPW; ++j) {
    if constexpr (F8 != 0) {
      const int eb = (wave * R::BPW + j) * 1024 + lane * 16;   // byte offset in the [64][BN] stage
      const int k = eb / BN;
      const int c = ((eb % BN) >> 4) ^ b_swz8(k);
      L.b_voff[j] = (n0 + c * 16 < p.N) ? (int)(k * p.ldb + c * 16) + kBias - j * 1024 : kOobOffset;
    } else {
      const int e = (wave * R::BPW + j) * 512 + lane * 8;   // element index in the [32][BN] stage
      const int k = e / BN;
      const int c = ((e % BN) >> 3) ^ b_swz(k);
      L.b_voff[j] = (n0 + c * 8 < p.N) ? (int)((k * p.ldb + c * 8) * 2) + kBias - j * 1024 : kOobOffset;
    }
  }
}

// Turn the A lanes whose load starts at a K index >= kin (within the block)
// into out-of-range lanes, for the loads of a block that runs past K.
template <int BM, int BN, int NW, int F8>
__device__ __forceinline__ void mask_a_lanes(RingLanes<BM, BN, NW, F8>& L, int wave, int lane, int kin) {
  using R = Ring<BM, BN, NW, F8>;
#pragma unroll
  for (int j = 0; j < R::APB; ++j)
    if (a_load_k<F8>(wave, R::APB, j, lane) >= kin) L.a_voff[j] = kOobOffset;
}

// The same without a branch: masks only when `on` (wave-uniform).
template <int BM, int BN, int NW, int F8>
__device__ __forceinline__ void mask_a_lanes_if(RingLanes<BM, BN, NW, F8>& L, int wave, int lane, int kin, bool on) {
  using R = Ring<BM, BN, NW, F8>;
#pragma unroll
  for (int j = 0; j < R::APB; ++j)
    L.a_voff[j] = (on && a_load_k<F8>(wave, R::APB, j, lane) >= kin) ? kOobOffset : L.a_voff[j];
}

// Per-lane LDS byte offsets of the fragment reads: A fragment i of step ks at
// a_rd[ks] + i*2048 within its slot; the two halves of B fragment j at
// b_rd[j] and b_rd[j] + 8*BN in B slot 0 (LDS byte addresses; slot s adds
// s times the slot size, an immediate offset of the read).
// fp8: A fragment i of step ks is two 16-byte reads, at a_rd[ks] + i*4096 and
// a_d further (the next chunk, +-16 bytes under the swizzle); B fragment j is
// four transposing reads of 8 rows, at b_rd[j] + q*8*BN.
template <int BM, int BN, int NW, int F8>
struct ReadOffsets {
  uint32_t a_rd[2];
  uint32_t a_d;
  uint32_t b_rd[Tile<BM, BN, NW, F8>::FN];
};

template <int BM, int BN, int NW, int F8>
__device__ __forceinline__ void read_offsets(int wm, int wn, int lane, uint32_t b_ring, ReadOffsets<BM, BN, NW, F8>& o) {
  using T = Tile<BM, BN, NW, F8>;
  if constexpr (F8 != 0) {
    // A: lane l holds row l%32 of the fragment and K bytes 32*(l/32) .. +31 of
    // the 64-deep step, i.e. chunks 4ks + 2h and 4ks + 2h + 1 (h = l/32)
    const int row = wm * T::WTM + (lane & 31), h = lane >> 5;
    const int swz = (row >> 1) & 7;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) o.a_rd[ks] = (uint32_t)(row * 128 + 16 * ((4 * ks + 2 * h) ^ swz));
    o.a_d = (uint32_t)(16 * ((2 * h + 1) ^ swz) - 16 * ((2 * h) ^ swz));
    // B: in each group of 16 lanes (g = l/16, m = l%16), lanes 2r and 2r+1 point
    // at the two 8-byte halves of row r of an 8-row x 16-column block; the
    // transposing read gives lane m column m of the 8 rows.  Group g covers
    // columns 16*(g&1) of the fragment and rows 32*(g>>1) of the step, so lane
    // j + 32h ends with column j, K bytes 32h .. 32h+31 over the four reads.
    const int g = lane >> 4, m = lane & 15;
    const int k = 32 * (g >> 1) + (m >> 1);
#pragma unroll
    for (int j = 0; j < T::FN; ++j) {
      const int n = wn * T::WTN + 32 * j + 16 * (g & 1) + 8 * (m & 1);
      o.b_rd[j] = b_ring + (uint32_t)(k * BN + 16 * ((n >> 4) ^ b_swz8(k)) + (n & 15));
    }
  } else {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) o.a_rd[ks] = (uint32_t)(a_frag_off(wm * T::WTM, lane, ks) * 2);
    o.a_d = 0;
#pragma unroll
    for (int j = 0; j < T::FN; ++j) o.b_rd[j] = b_ring + (uint32_t)(b_frag_off<BN>(wn * T::WTN, lane, 0, j) * 2);
  }
}

typedef __attribute__((address_space(3))) i32x4 lds_i32x4;
typedef __attribute__((address_space(3))) i32x2 lds_i32x2;

// fp8 operand pieces: half p of A fragment i, quarter q of B fragment j.
__device__ __forceinline__ void read_a8(uint32_t a_base, uint32_t a_d, int i, int p, i32x8& f) {
  const i32x4 v = *(const lds_i32x4*)(uintptr_t)(a_base + (uint32_t)(i * 32 * 128) + (p ? a_d : 0u));
  f[4 * p + 0] = v[0];
  f[4 * p + 1] = v[1];
  f[4 * p + 2] = v[2];
  f[4 * p + 3] = v[3];
}
template <int BN>
__device__ __forceinline__ void read_b8(uint32_t addr, int q, i32x8& f) {
  const i32x2 v = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(uintptr_t)(addr + (uint32_t)(q * 8 * BN)));
  f[2 * q] = v[0];
  f[2 * q + 1] = v[1];
}

// Read item t of a step, in the order the next step's MFMAs consume them:
// A0, B0, B1, .., B(FN-1), A1, .., A(FM-1).
template <int BM, int BN, int NW, int F8>
__device__ __forceinline__ void read_item(int t, uint32_t a_base, uint32_t a_d, uint32_t b_slot, const uint32_t* b_rd,
                                          Frags<BM, BN, NW, F8>& f) {
  using T = Tile<BM, BN, NW, F8>;
  if constexpr (F8 != 0) {
    if (t == 0 || t > T::FN) {
      const int i = t == 0 ? 0 : t - T::FN;
      read_a8(a_base, a_d, i, 0, f.a[i]);
      read_a8(a_base, a_d, i, 1, f.a[i]);
    } else {
      const int j = t - 1;
      const uint32_t b_addr = b_slot + b_rd[j];
#pragma unroll
      for (int q = 0; q < 4; ++q) read_b8<BN>(b_addr, q, f.b[j]);
    }
  } else {
  if (t == 0 || t > T::FN) {
    const int i = t == 0 ? 0 : t - T::FN;
    f.a[i] = *(lds_bf16x8*)(uintptr_t)(a_base + (uint32_t)(i * 16 * kBK * 2));
  } else {
    const int j = t - 1;
    // the slot offset is added here, beside the reads, rather than for all
    // fragments at once at the start of a step
    const uint32_t b_addr = b_slot + b_rd[j];
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(uintptr_t)b_addr);
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(uintptr_t)(b_addr + 8 * BN));
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    f.b[j] = __builtin_bit_cast(bf16x8, v);
  }
  }
}

// Loads of one A block or one B stage: descriptor and M0 of this wave's first segment.
struct SlotDma {
  i32x4 rsrc;
  uint32_t m0;
};

// Load pair q (loads 2q, 2q+1) of an A block (OP 1) or a B stage (OP 2).
template <int BM, int BN, int NW, int F8, int OP, int Q>
__device__ __forceinline__ void dma_pair(const SlotDma& d, const RingLanes<BM, BN, NW, F8>& L) {
  constexpr int j = 2 * Q;
  if constexpr (OP == 1)
    dma16_pair<(j & 3) * 1024>(d.rsrc, d.m0 + (uint32_t)((j >> 2) * 4096), L.a_voff[j], L.a_voff[j + 1]);
  else
    dma16_pair<j * 1024>(d.rsrc, d.m0, L.b_voff[j], L.b_voff[j + 1]);
}

// All loads of an A block (OP 1) or a B stage (OP 2).
template <int BM, int BN, int NW, int F8, int OP>
__device__ __forceinline__ void dma_all(const SlotDma& d, const RingLanes<BM, BN, NW, F8>& L) {
  using R = Ring<BM, BN, NW, F8>;
  [&]<int... q>(std::integer_sequence<int, q...>) {
    (dma_pair<BM, BN, NW, F8, OP, q>(d, L), ...);
  }(std::make_integer_sequence<int, (OP == 1 ? R::APB : R::BPW) / 2>{});
}

// Instruction plan of one 32-deep step: FM*FN groups, each one MFMA of the
// current fragments plus at most one fragment read for the next step (two in
// the shorter steps of the smaller bf16 blocks) and at most one load
// operation.  With one wave per SIMD a wave issues one instruction every 4
// cycles, so a 16-cycle MFMA hides three others; two LDS reads in one group
// already cost extra cycles (both measured on gfx950).
//   reads:  A0, B0 low, B0 high, B1 low, .., B(FN-1) high, A1, .., A(FM-1)
//           (the order the next step's MFMAs consume them), spread evenly over
//           the first half of the step (bf16) or the whole step (fp8);
//   loads:  each load pair becomes three operations (set M0, load, load) in
//           consecutive groups from evenly spaced starting groups, so that the
//           MFMA between M0 and the first load covers the wait M0 needs; a
//           step with fewer free groups than that needs (fp8 128x256: 8 MFMAs
//           of 64 cycles) issues each pair whole in one group, evenly spaced.
template <int BM, int BN, int NW, int F8, int OP>
struct StepPlan {
  using T = Tile<BM, BN, NW, F8>;
  static constexpr int G = T::FM * T::FN;
  // fragment reads of the next step: bf16 one A read and two B reads per
  // fragment; fp8 two A reads and four B reads per fragment
  static constexpr int NR = F8 ? 2 * T::FM + 4 * T::FN : T::FM + 2 * T::FN;
  static constexpr int NP0 = OP == 1 ? Ring<BM, BN, NW, F8>::APB / 2 : Ring<BM, BN, NW, F8>::BPW / 2;   // pairs from d0
  static constexpr int NP1 = OP == 1 ? 0 : Ring<BM, BN, NW, F8>::BPW / 2;                      // pairs from d1
  static constexpr int NP = NP0 + NP1;
  // the B step opens with G0 groups of MFMAs alone and then waits at the
  // block's barrier: those MFMAs need nothing the barrier publishes, and they
  // keep the matrix core busy while the waves meet and while the A step's last
  // fragment reads (which the barrier waits for) complete; steps of 32 MFMAs
  // open with 4 (measured best of 2, 4, 6, 8), the 64-MFMA steps of bf16
  // 256x256 blocks and shorter steps with 2
  static constexpr int G0 = OP == 2 ? (T::FM * T::FN == 32 ? 4 : 2) : 0;
  // whole pairs: one operation per pair (M0, a wait state and both loads)
  static constexpr bool WHOLE = 3 * NP > G - G0;
  static constexpr int ND = WHOLE ? NP : 3 * NP;
  // bf16 reads of 32-group steps run over the first half of the step's groups:
  // the next step's first MFMAs need them, and the LDS returns them late under
  // the step's own loads (2 % faster on 8192^3 than spread over the whole step
  // with 2 x 2 waves, measured); fp8 and the 64-group steps of bf16 256x256
  // blocks (1 x 4 waves, fewer transposing reads) spread them over the whole
  // step (0.2-1.6 % faster there than the first half, measured)
  static constexpr int read_group(int r) {
    return (F8 || G >= 64) ? G0 + (r * (G - G0)) / NR : G0 + (r * (G - G0)) / (2 * NR);
  }
  static constexpr int dma_group(int o) {
    if (WHOLE) return G0 + ((2 * o + 1) * (G - G0)) / (2 * NP);
    int g = G0 - 1;
    for (int i = 0; i <= o; ++i) {
      const int start = G0 + ((2 * (i / 3) + 1) * (G - G0)) / (2 * NP) - 1 + i % 3;
      g = g + 1 > start ? g + 1 : start;
    }
    return g;
  }
  // groups that issue neither a read nor a load operation (nor, in the A
  // step, one of the K-mask selects of the first APB groups)
  static constexpr bool busy(int g) {
    if (OP == 1 && g < Ring<BM, BN, NW, F8>::APB) return true;
    for (int r = 0; r < NR; ++r)
      if (read_group(r) == g) return true;
    for (int o = 0; o < ND; ++o)
      if (dma_group(o) == g) return true;
    return false;
  }
  // group of scalar stage s of ns: spread over the free groups
  static constexpr int stage_group(int s, int ns) {
    int nfree = 0;
    for (int g = 0; g < G; ++g) nfree += busy(g) ? 0 : 1;
    if (nfree >= ns) {
      const int want = (s * nfree) / ns;
      int k = 0;
      for (int g = 0; g < G; ++g) {
        if (busy(g)) continue;
        if (k == want) return g;
        ++k;
      }
    }
    return (s * G) / ns;
  }
  // the first load of A pair q (lanes 2q, 2q+1) comes after the K-mask
  // selects of those lanes, which run on groups 2q and 2q+1
  static constexpr bool a_loads_after_masks() {
    for (int q = 0; q < NP; ++q)
      if (dma_group(WHOLE ? q : 3 * q + 1) <= 2 * q + 1) return false;
    return true;
  }
  // bf16: at most two reads beside each 16-cycle MFMA; fp8: up to three beside
  // each 64-cycle MFMA
  static_assert(F8 ? NR <= 3 * (G - G0) : NR <= G - G0, "reads per group");
  static_assert(ND == 0 || dma_group(ND - 1) < G, "loads fit in the step");
  static_assert(OP != 1 || a_loads_after_masks(), "A loads after their K-mask selects");
};

// Per-step state of the split B reads: address and low half of each fragment.
template <int BM, int BN, int NW, int F8>
struct BReads {
  uint32_t addr[Tile<BM, BN, NW, F8>::FN];
  i16x4 lo[Tile<BM, BN, NW, F8>::FN];
  uint32_t a_d;   // fp8: offset of the second half of an A fragment
};

template <int BM, int BN, int NW, int F8, int OP, int r>
__device__ __forceinline__ void step_read(uint32_t a_base, uint32_t b_slot, const uint32_t* b_rd, BReads<BM, BN, NW, F8>& br,
                                          Frags<BM, BN, NW, F8>& nxt) {
  using T = Tile<BM, BN, NW, F8>;
  if constexpr (F8 != 0) {
    // A0 (halves 0, 1), B0 .. B(FN-1) (quarters 0..3 each), A1 .. A(FM-1)
    if constexpr (r < 2) {
      read_a8(a_base, br.a_d, 0, r, nxt.a[0]);
    } else if constexpr (r < 2 + 4 * T::FN) {
      constexpr int j = (r - 2) / 4, q = (r - 2) % 4;
      if constexpr (q == 0) br.addr[j] = b_slot + b_rd[j];
      read_b8<BN>(br.addr[j], q, nxt.b[j]);
    } else {
      constexpr int i = 1 + (r - 2 - 4 * T::FN) / 2, h = (r - 2 - 4 * T::FN) % 2;
      read_a8(a_base, br.a_d, i, h, nxt.a[i]);
    }
  } else if constexpr (r == 0 || r > 2 * T::FN) {
    constexpr int i = r == 0 ? 0 : r - 2 * T::FN;
    nxt.a[i] = *(lds_bf16x8*)(uintptr_t)(a_base + (uint32_t)(i * 16 * kBK * 2));
  } else if constexpr ((r - 1) % 2 == 0) {
    constexpr int j = (r - 1) / 2;
    br.addr[j] = b_slot + b_rd[j];
    br.lo[j] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(uintptr_t)br.addr[j]);
  } else {
    constexpr int j = (r - 1) / 2;
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(uintptr_t)(br.addr[j] + 8 * BN));
    const i16x4 lo = br.lo[j];
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    nxt.b[j] = __builtin_bit_cast(bf16x8, v);
  }
}

template <int BM, int BN, int NW, int F8, int OP, int g, int... r>
__device__ __forceinline__ void group_reads(uint32_t a_base, uint32_t b_slot, const uint32_t* b_rd,
                                            BReads<BM, BN, NW, F8>& br, Frags<BM, BN, NW, F8>& nxt, std::integer_sequence<int, r...>) {
  using P = StepPlan<BM, BN, NW, F8, OP>;
  ((void)(P::read_group(r) == g ? (step_read<BM, BN, NW, F8, OP, r>(a_base, b_slot, b_rd, br, nxt), 0) : 0), ...);
}

// Load operation o of a step: o = 3q + k for load pair q (k 0: set M0, k 1
// and 2: the pair's loads), or load pair o whole.
template <int BM, int BN, int NW, int F8, int OP, int o>
__device__ __forceinline__ void step_dma(const SlotDma& d0, const SlotDma& d1, const RingLanes<BM, BN, NW, F8>& L) {
  using P = StepPlan<BM, BN, NW, F8, OP>;
  if constexpr (P::WHOLE) {
    // operation o is load pair o, whole
    if constexpr (o < P::NP0) dma_pair<BM, BN, NW, F8, OP, o>(d0, L);
    else dma_pair<BM, BN, NW, F8, OP, o - P::NP0>(d1, L);
  } else {
    constexpr int q = o / 3, k = o % 3;
    constexpr bool first = q < P::NP0;
    constexpr int qq = first ? q : q - P::NP0;
    const SlotDma& d = first ? d0 : d1;
    constexpr int j = 2 * qq + (k == 2 ? 1 : 0);
    if constexpr (k == 0) {
      const uint32_t m0v = OP == 1 ? d.m0 + (uint32_t)((j >> 2) * 4096) : d.m0;
      asm volatile("s_mov_b32 m0, %0" :: "s"(m0v) : "memory");
    } else {
      constexpr int off = OP == 1 ? (j & 3) * 1024 : j * 1024;
      static_assert(off <= 4095, "instruction offset range");
      const int v = OP == 1 ? L.a_voff[j] : L.b_voff[j];
      asm volatile("buffer_load_dwordx4 %0, %1, 0 offen offset:%2 lds" :: "v"(v), "s"(d.rsrc), "n"(off) : "memory");
    }
  }
}

template <int BM, int BN, int NW, int F8, int OP, int g, int... o>
__device__ __forceinline__ void group_dma(const SlotDma& d0, const SlotDma& d1, const RingLanes<BM, BN, NW, F8>& L,
                                          std::integer_sequence<int, o...>) {
  using P = StepPlan<BM, BN, NW, F8, OP>;
  ((void)(P::dma_group(o) == g ? (step_dma<BM, BN, NW, F8, OP, o>(d0, d1, L), 0) : 0), ...);
}

template <int BM, int BN, int NW, int F8, int D, int OP, int g, typename X>
__device__ __forceinline__ void ring_group(Acc<BM, BN, NW, F8>& acc, const Frags<BM, BN, NW, F8>& cur, Frags<BM, BN, NW, F8>& nxt,
                                           uint32_t a_base, uint32_t b_slot, const uint32_t* b_rd,
                                           BReads<BM, BN, NW, F8>& br, const SlotDma& d0, const SlotDma& d1,
                                           const RingLanes<BM, BN, NW, F8>& L, X& ex) {
  using T = Tile<BM, BN, NW, F8>;
  using P = StepPlan<BM, BN, NW, F8, OP>;
  constexpr int i = g / T::FN, j = g % T::FN;
  if constexpr (F8 != 0)   // the first operand is B (format b), the second A (format a); unit scales (E8M0 127)
    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(cur.b[j], cur.a[i], acc[i][j], (F8 - 1) >> 1,
                                                                (F8 - 1) & 1, 0, 127, 0, 127);
  else
    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur.b[j], cur.a[i], acc[i][j], 0, 0, 0);
  // bf16: the group's other instructions follow its 16-cycle MFMA (left free,
  // the compiler hoists the next group's reads above it and packs up to 7
  // instructions between two MFMAs); a 64-cycle fp8 MFMA hides them anyway and
  // its steps run faster with the compiler's order
  if constexpr (F8 == 0) __builtin_amdgcn_sched_barrier(0);
  if constexpr (OP == 2 && g == P::G0) {
    // the block's barrier: A block b+1 and B stages x0+2, x0+3 have landed for
    // every wave (only the A block loaded in the A step may be in flight), and
    // every wave's reads issued in the A step are done (among them the last
    // reads of the B slot this step loads into, and of the A slot the next A
    // step loads into)
    wait_vmem_at_most<Ring<BM, BN, NW, F8, D>::IN_FLIGHT>();
    wait_lds_all();
    __syncthreads();
  }
  group_reads<BM, BN, NW, F8, OP, g>(a_base, b_slot, b_rd, br, nxt, std::make_integer_sequence<int, P::NR>{});
  group_dma<BM, BN, NW, F8, OP, g>(d0, d1, L, std::make_integer_sequence<int, P::ND>{});
  ex.template operator()<g>();
  __builtin_amdgcn_sched_barrier(0);
}

template <int BM, int BN, int NW, int F8, int D, int OP, typename X, int... g>
__device__ __forceinline__ void ring_groups(Acc<BM, BN, NW, F8>& acc, const Frags<BM, BN, NW, F8>& cur, Frags<BM, BN, NW, F8>& nxt,
                                            uint32_t a_base, uint32_t b_slot, const uint32_t* b_rd,
                                            BReads<BM, BN, NW, F8>& br, const SlotDma& d0, const SlotDma& d1,
                                            const RingLanes<BM, BN, NW, F8>& L, X& ex, std::integer_sequence<int, g...>) {
  (ring_group<BM, BN, NW, F8, D, OP, g>(acc, cur, nxt, a_base, b_slot, b_rd, br, d0, d1, L, ex), ...);
}

// One 32-deep step with a fixed instruction order (the plan above): MFMAs of
// `cur` (i-major), reads of `nxt`, the loads of an A block d0 (OP 1) or of two
// B stages d0 and d1 (OP 2), and the scalar work `ex` puts on each group
// (ex.operator()<g>() runs in group g).  The groups are generated as
// straight-line code (a loop this long is not always unrolled, and the
// accumulators must stay in registers).
template <int BM, int BN, int NW, int F8, int D, int OP, typename X>
__device__ __forceinline__ void ring_step(Acc<BM, BN, NW, F8>& acc, const Frags<BM, BN, NW, F8>& cur, Frags<BM, BN, NW, F8>& nxt,
                                          uint32_t a_base, uint32_t b_slot, const ReadOffsets<BM, BN, NW, F8>& o,
                                          const SlotDma& d0, const SlotDma& d1, const RingLanes<BM, BN, NW, F8>& L,
                                          X&& ex) {
  using T = Tile<BM, BN, NW, F8>;
  BReads<BM, BN, NW, F8> br;
  br.a_d = o.a_d;
  ring_groups<BM, BN, NW, F8, D, OP>(acc, cur, nxt, a_base, b_slot, o.b_rd, br, d0, d1, L, ex,
                          std::make_integer_sequence<int, T::FM * T::FN>{});
}

// Where the blocks and stages of one task come from and go to.  Everything
// here is wave-uniform (scalar registers).
struct RingAddr {
  uint64_t a0, b0;           // byte address of the first block's A origin and B origin, minus kBias
  uint64_t b_step;           // bytes between consecutive B stages (32 rows of B)
  int x_part;                // first B stage that is not wholly before the task's K end
  uint32_t lim_part;         // its num_records: its rows before that end, plus the bias
  uint32_t lds0;             // LDS byte address of the ring
  int wave;
};

// num_records of B stage x: rows at or past the task's K end (row K, or the
// end of its layer's K range) fall outside and read zeros (a stage wholly past
// that end reads nothing from memory)
__device__ __forceinline__ uint32_t b_stage_limit(const RingAddr& ra, int x) {
  return x < ra.x_part ? (uint32_t)kOobOffset : x == ra.x_part ? ra.lim_part : (uint32_t)kBias;
}

// The K loop of one task over nb 64-deep blocks.  Block b = A block b and B
// stages x0 = 2b, x0+1, one 32-deep MFMA step each.  Each step runs the MFMAs
// of one stage while it reads the operands of the next:
//   step 1 (MFMAs of x0, reads A b/1 and B x0+1):  loads: A block b+D
//   step 2 (MFMAs of x0+1, reads A b+1/0 and B x0+2): loads: B stages x0+2D, x0+2D+1
//     after its first MFMAs: wait until A block b+1 and B stages x0+2, x0+3
//     have landed (the loads issued after them may still be in flight) and
//     this wave's reads are done, barrier b; then the reads and loads of step 2
// A block kb lives in A slot kb mod (D+1), B stage x in B slot x mod 2D.  Every
// load goes into a slot whose last reads were done before the barrier that
// precedes the load; the shortest lead from a load to the barrier that
// publishes it is 2D-3 steps.  The prologue issues blocks 0 .. D-1; the last
// blocks still issue their loads, for blocks and stages past K, with empty
// ranges (no memory is read, zeros land in slots that are not read again), so
// that the loop has no branches.
//
// The scalar bookkeeping (slot addresses, descriptors, limits) is carried from
// block to block and updated in small pieces on chosen groups of the steps:
// step 1 builds the B descriptors step 2 loads with; step 2 advances the state
// to the next block.
//
// When the last block runs past K (kin_last < 64): B rows at or past K fall
// outside the B descriptors' ranges and read zeros; A block nb-1 is loaded with
// its lanes past K masked (selects on the first groups of the step that issues
// those loads, or in the prologue when nb <= D).
template <int BM, int BN, int NW, int F8, int D>
__device__ __forceinline__ void main_loop_ring(const RingAddr& ra, int nb, int kin_last,
                                               const ReadOffsets<BM, BN, NW, F8>& o, RingLanes<BM, BN, NW, F8>& L, int lane,
                                               Acc<BM, BN, NW, F8>& acc) {
  using R = Ring<BM, BN, NW, F8, D>;
  using T = Tile<BM, BN, NW, F8>;
  using P1 = StepPlan<BM, BN, NW, F8, 1>;
  using P2 = StepPlan<BM, BN, NW, F8, 2>;
  constexpr uint32_t BB = (uint32_t)R::B_BYTES;
  const int wave = ra.wave;
  const bool masked = kin_last < block_k<F8>();
  const uint32_t a_m0w = ra.lds0 + (uint32_t)(wave * R::APB * 1024);            // this wave's segment, A slot 0
  const uint32_t b_m0w = ra.lds0 + (uint32_t)(R::B_OFF + wave * R::BPW * 1024);  // this wave's segment, B slot 0
  auto a_dma = [&](uint64_t addr, int slot, uint32_t lim) {
    SlotDma d;
    d.rsrc = make_rsrc_addr(addr, lim);
    d.m0 = a_m0w + (uint32_t)(slot * R::A_BYTES);
    return d;
  };
  auto b_dma = [&](uint64_t addr, int x, int slot) {
    SlotDma d;
    d.rsrc = make_rsrc_addr(addr, b_stage_limit(ra, x));
    d.m0 = b_m0w + (uint32_t)(slot * R::B_BYTES);
    return d;
  };

  // prologue: blocks 0 .. D-1 (A block k into A slot k, B stages 2k, 2k+1 into
  // B slots 2k, 2k+1), then wait for block 0.  Depth 2 loads block 1 only when
  // there is one; deeper rings load blocks past K with empty ranges.
  if constexpr (D == 2) {
    if (masked && nb == 1) mask_a_lanes<BM, BN, NW, F8>(L, wave, lane, kin_last);
    dma_all<BM, BN, NW, F8, 1>(a_dma(ra.a0, 0, kOobOffset), L);
    dma_all<BM, BN, NW, F8, 2>(b_dma(ra.b0, 0, 0), L);
    dma_all<BM, BN, NW, F8, 2>(b_dma(ra.b0 + ra.b_step, 1, 1), L);
    if (nb > 1) {
      if (masked && nb == 2) mask_a_lanes<BM, BN, NW, F8>(L, wave, lane, kin_last);
      dma_all<BM, BN, NW, F8, 1>(a_dma(ra.a0 + kBK * 2, 1, kOobOffset), L);
      dma_all<BM, BN, NW, F8, 2>(b_dma(ra.b0 + 2 * ra.b_step, 2, 2), L);
      dma_all<BM, BN, NW, F8, 2>(b_dma(ra.b0 + 3 * ra.b_step, 3, 3), L);
      wait_vmem_at_most<R::APB + 2 * R::BPW>();
    } else {
      wait_vmem_at_most<0>();
    }
  } else {
#pragma unroll
    for (int k = 0; k < D; ++k) {
      if (masked) mask_a_lanes_if<BM, BN, NW, F8>(L, wave, lane, kin_last, k == nb - 1);
      dma_all<BM, BN, NW, F8, 1>(a_dma(ra.a0 + (uint64_t)k * (kBK * 2), k, k < nb ? (uint32_t)kOobOffset : 0u), L);
      dma_all<BM, BN, NW, F8, 2>(b_dma(ra.b0 + (uint64_t)(2 * k) * ra.b_step, 2 * k, 2 * k), L);
      dma_all<BM, BN, NW, F8, 2>(b_dma(ra.b0 + (uint64_t)(2 * k + 1) * ra.b_step, 2 * k + 1, 2 * k + 1), L);
    }
    wait_vmem_at_most<(D - 1) * (R::APB + 2 * R::BPW)>();
  }
  __syncthreads();

  Frags<BM, BN, NW, F8> f0, f1;
  {
    const uint32_t as = ra.lds0 + o.a_rd[0];
    // B slot 0, as an opaque register value: with a literal 0 the compiler
    // would keep b_rd[j] + 8*BN in registers across tasks
    uint32_t bs0;
    asm volatile("s_mov_b32 %0, 0" : "=s"(bs0));
    // same order as the reads issued by the loop's last step, so that the
    // first MFMAs wait only for their own operands on either path into the loop
#pragma unroll
    for (int t = 0; t < T::FM + T::FN; ++t) {
      read_item<BM, BN, NW, F8>(t, as, o.a_d, bs0, o.b_rd, f0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // per-lane K-mask condition of each A load (used on block nb-1-D, whose A
  // step loads A block nb-1; for nb <= D the prologue has masked)
  bool mk[R::APB];
#pragma unroll
  for (int j = 0; j < R::APB; ++j) mk[j] = a_load_k<F8>(wave, R::APB, j, lane) >= kin_last;
  const int mask_b = masked ? nb - 1 - D : -1;

  // scalar state of block b
  // A slots of blocks b, b+1, .., b+D
  uint32_t la0 = 0, la1 = R::A_BYTES, la2 = 2 * R::A_BYTES, la3 = 3 * R::A_BYTES, la4 = 4 * R::A_BYTES;
  uint32_t sb = 0, lb1 = BB, lb2 = 2 * BB;  // B slots of stages x0 (and x0+2D), x0+1 (and x0+2D+1), x0+2
  uint64_t a_nx = ra.a0 + D * kBK * 2;      // A block b+D
  uint64_t b_nx = ra.b0 + 2 * D * ra.b_step; // B stage x0+2D
  int xb = 2 * D;                           // x0+2D
  bool mnow = mask_b == 0;                  // block b applies the K mask
  SlotDma da = a_dma(a_nx, D, D < nb ? (uint32_t)kOobOffset : 0u), db0, db1;

  uint32_t lim0, lim1, lt0, lt1, w_lo, w_hi, a_lim;
  int x1;
  uint64_t b_nx1;
  for (int b = 0; b < nb; ++b) {
    ring_step<BM, BN, NW, F8, D, 1>(acc, f0, f1, ra.lds0 + la0 + o.a_rd[1], lb1, o, da, da, L, [&]<int g>() {
      if constexpr (g < R::APB) {
        if (mnow && mk[g]) L.a_voff[g] = kOobOffset;
      }
      // the scalar work in pieces of at most three instructions, one piece per
      // group: an MFMA of 16 cycles hides three others, each one more costs 4
      constexpr int NS1 = 10;
      // (the stage limits are b_stage_limit in two selects)
      if constexpr (g == P1::stage_group(0, NS1)) { lt0 = xb == ra.x_part ? ra.lim_part : (uint32_t)kBias; pin_scalar(lt0); }
      if constexpr (g == P1::stage_group(1, NS1)) { lim0 = xb < ra.x_part ? (uint32_t)kOobOffset : lt0; pin_scalar(lim0); }
      if constexpr (g == P1::stage_group(2, NS1)) { rsrc_words(b_nx, w_lo, w_hi); pin_scalar(w_lo); pin_scalar(w_hi); }
      if constexpr (g == P1::stage_group(3, NS1)) db0.rsrc = rsrc_of_words(w_lo, w_hi, lim0);
      if constexpr (g == P1::stage_group(4, NS1)) {
        db0.m0 = b_m0w + sb;
        db1.m0 = b_m0w + lb1;
      }
      if constexpr (g == P1::stage_group(5, NS1)) { x1 = xb + 1; lt1 = x1 == ra.x_part ? ra.lim_part : (uint32_t)kBias; pin_scalar(lt1); }
      if constexpr (g == P1::stage_group(6, NS1)) { lim1 = x1 < ra.x_part ? (uint32_t)kOobOffset : lt1; pin_scalar(lim1); }
      if constexpr (g == P1::stage_group(7, NS1)) { b_nx1 = b_nx + ra.b_step; pin_scalar(b_nx1); }
      if constexpr (g == P1::stage_group(8, NS1)) { rsrc_words(b_nx1, w_lo, w_hi); pin_scalar(w_lo); pin_scalar(w_hi); }
      if constexpr (g == P1::stage_group(9, NS1)) db1.rsrc = rsrc_of_words(w_lo, w_hi, lim1);
    });
    ring_step<BM, BN, NW, F8, D, 2>(acc, f1, f0, ra.lds0 + la1 + o.a_rd[0], lb2, o, db0, db1, L, [&]<int g>() {
      if constexpr (g == P2::stage_group(0, 8)) {
        const uint32_t t = la0;
        la0 = la1;
        la1 = la2;
        if constexpr (D == 2) {
          la2 = t;
        } else if constexpr (D == 3) {
          la2 = la3;
          la3 = t;
        } else {
          la2 = la3;
          la3 = la4;
          la4 = t;
        }
      }
      if constexpr (g == P2::stage_group(1, 8)) {
        if constexpr (R::NB == 4) {
          sb ^= 2 * BB;
          lb1 ^= 2 * BB;
          lb2 ^= 2 * BB;
        } else {
          sb = lb2;
          lb1 = lb2 + BB;
          lb2 = lb2 + 2 * BB == (uint32_t)R::NB * BB ? 0u : lb2 + 2 * BB;
        }
      }
      if constexpr (g == P2::stage_group(2, 8)) {
        a_nx += kBK * 2;
        pin_scalar(a_nx);
      }
      if constexpr (g == P2::stage_group(3, 8)) { a_lim = b + 1 + D < nb ? (uint32_t)kOobOffset : 0u; pin_scalar(a_lim); }
      if constexpr (g == P2::stage_group(4, 8)) { rsrc_words(a_nx, w_lo, w_hi); pin_scalar(w_lo); pin_scalar(w_hi); }
      if constexpr (g == P2::stage_group(5, 8)) {
        da.rsrc = rsrc_of_words(w_lo, w_hi, a_lim);
        da.m0 = a_m0w + (D == 2 ? la2 : D == 3 ? la3 : la4);
      }
      if constexpr (g == P2::stage_group(6, 8)) {
        b_nx += 2 * ra.b_step;
        pin_scalar(b_nx);
      }
      if constexpr (g == P2::stage_group(7, 8)) {
        xb += 2;
        pin_scalar(xb);
        mnow = b + 1 == mask_b;
      }
    });
  }
  // the last blocks' empty-range loads still write zeros into the ring: let
  // them land before the next task's prologue loads into the same slots
  wait_vmem_at_most<0>();
  wait_lds_all();
  __syncthreads();
}

// ---- main loop, general path: element loads staged in registers ---------------------------
template <int BM, int BN, int NW, int F8>
__device__ __forceinline__ void main_loop_staged(const GemmParams& p, uint16_t* smem, int64_t m0,
                                                 int64_t n0, int kt0, int kt1, int tid, Acc<BM, BN, NW, F8>& acc) {
  using T = Tile<BM, BN, NW, F8>;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / T::WGN, wn = wave % T::WGN;
  u32x4 ra[T::A_CH], rb[T::B_CH];
  auto load_blocks = [&](int kt) {
    const int64_t k0 = (int64_t)kt * kBK;
#pragma unroll
    for (int i = 0; i < T::A_CH; ++i) {
      const int q = tid + T::THREADS * i;
      ra[i] = load_chunk<false>(p.A, p.lda, m0 + (q >> 3), k0 + (q & 7) * 8, p.M, p.K);
    }
#pragma unroll
    for (int i = 0; i < T::B_CH; ++i) {
      const int q = tid + T::THREADS * i;
      rb[i] = load_chunk<false>(p.B, p.ldb, k0 + q / (BN / 8), n0 + (q % (BN / 8)) * 8, p.K, p.N);
    }
  };
  auto store_blocks = [&](int buf) {
    uint16_t* As = smem + buf * (T::A_ELEMS + T::B_ELEMS);
    uint16_t* Bs = As + T::A_ELEMS;
#pragma unroll
    for (int i = 0; i < T::A_CH; ++i) {
      const int q = tid + T::THREADS * i;
      *reinterpret_cast<u32x4*>(As + a_off(q >> 3, q & 7)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < T::B_CH; ++i) {
      const int q = tid + T::THREADS * i;
      *reinterpret_cast<u32x4*>(Bs + b_off<BN>(q / (BN / 8), (q % (BN / 8)) * 8)) = rb[i];
    }
  };
  load_blocks(kt0);
  store_blocks(0);
  __syncthreads();
  for (int kt = kt0; kt < kt1; ++kt) {
    const int buf = (kt - kt0) & 1;
    const bool more = kt + 1 < kt1;
    if (more) load_blocks(kt + 1);
    const uint16_t* As = smem + buf * (T::A_ELEMS + T::B_ELEMS);
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      Frags<BM, BN, NW, F8> f;
      load_frags<BM, BN, NW, F8>(As, As + T::A_ELEMS, wm, wn, lane, ks, 32 * ks, f);
      mma_step<BM, BN, NW, F8>(f, acc);
    }
    if (more) store_blocks(buf ^ 1);
    __syncthreads();
  }
}

// ---- epilogue ---------------------------------------------------------------------------------
// Fragment (i, j) of the wave: lane l holds row 16i + l%16 and columns
// 16j + 4*(l/16) .. +3 of the wave's sub-block.
// Two bf16-packed fragments (j, j+1) of one 16-row strip, each lane holding 4
// consecutive columns (two dwords) of each, rearranged so that each lane holds
// 8 consecutive columns of one of them: v_permlane16_swap exchanges the odd
// 16-lane rows of its first operand with the even rows of its second, so lane
// group q ends with columns 16*(q&1) + 8*(q>>1) .. +7 of the pair.
__device__ __forceinline__ u32x4 pair_to_row8(const f32x4& x, const f32x4& y) {
  const bf16x4 xb = {(__bf16)x[0], (__bf16)x[1], (__bf16)x[2], (__bf16)x[3]};
  const bf16x4 yb = {(__bf16)y[0], (__bf16)y[1], (__bf16)y[2], (__bf16)y[3]};
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
  const u32x2 xw = __builtin_bit_cast(u32x2, xb), yw = __builtin_bit_cast(u32x2, yb);
  const auto s0 = __builtin_amdgcn_permlane16_swap(xw[0], yw[0], false, false);
  const auto s1 = __builtin_amdgcn_permlane16_swap(xw[1], yw[1], false, false);
  return u32x4{s0[0], s1[0], s0[1], s1[1]};
}

// Epilogue of the fp8 kernels (MFMA 32x32x64, B fragment first): fragment
// (i, j) of the wave, lane l, accumulator v holds row 32i + l%32 and column
// 32j + 8*(v/4) + 4*(l/32) + v%4 -- four runs of 4 consecutive columns.  For
// bf16 output, runs (g, g+1) are exchanged between the lane halves with
// v_permlane32_swap so that each lane stores 8 consecutive columns (16 bytes).
template <int BM, int BN, int NW, bool OUT_BF16>
__device__ __forceinline__ void store_tile32(const GemmParams& p, const Acc<BM, BN, NW, 1>& acc, int64_t m0,
                                             int64_t n0, int64_t lstride, int wm, int wn, int lane, bool fast,
                                             bool fast16) {
  using T = Tile<BM, BN, NW, 1>;
  typedef typename std::conditional<OUT_BF16, __bf16, float>::type OutT;
  OutT* out = reinterpret_cast<OutT*>(p.out) + lstride;
  const int h = lane >> 5;
  const int64_t r0 = m0 + wm * T::WTM + (lane & 31);
  const int64_t cb = n0 + wn * T::WTN;
  if (OUT_BF16 && fast16) {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
      OutT* row = out + (r0 + i * 32) * p.ldo + cb + 8 * h;
#pragma unroll
      for (int j = 0; j < T::FN; ++j) {
#pragma unroll
        for (int g = 0; g < 4; g += 2) {
          const f32x16& a = acc[i][j];
          const bf16x4 xb = {(__bf16)a[4 * g], (__bf16)a[4 * g + 1], (__bf16)a[4 * g + 2], (__bf16)a[4 * g + 3]};
          const bf16x4 yb = {(__bf16)a[4 * g + 4], (__bf16)a[4 * g + 5], (__bf16)a[4 * g + 6], (__bf16)a[4 * g + 7]};
          const u32x2 xw = __builtin_bit_cast(u32x2, xb), yw = __builtin_bit_cast(u32x2, yb);
          const auto s0 = __builtin_amdgcn_permlane32_swap(xw[0], yw[0], false, false);
          const auto s1 = __builtin_amdgcn_permlane32_swap(xw[1], yw[1], false, false);
          *reinterpret_cast<u32x4*>(row + j * 32 + 8 * g) = u32x4{s0[0], s1[0], s0[1], s1[1]};
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    return;
  }
  if (fast) {
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
      OutT* row = out + (r0 + i * 32) * p.ldo + cb + 4 * h;
#pragma unroll
      for (int j = 0; j < T::FN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x16& a = acc[i][j];
          if (OUT_BF16) {
            const bf16x4 v = {(__bf16)a[4 * g], (__bf16)a[4 * g + 1], (__bf16)a[4 * g + 2], (__bf16)a[4 * g + 3]};
            *reinterpret_cast<bf16x4*>(row + j * 32 + 8 * g) = v;
          } else {
            const f32x4 v = {a[4 * g], a[4 * g + 1], a[4 * g + 2], a[4 * g + 3]};
            *reinterpret_cast<f32x4*>(row + j * 32 + 8 * g) = v;
          }
        }
      if (OUT_BF16) __builtin_amdgcn_sched_barrier(0);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < T::FM; ++i) {
    const int64_t r = r0 + i * 32;
    if (r >= p.M) continue;
    OutT* row = out + r * p.ldo;
#pragma unroll
    for (int j = 0; j < T::FN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t c = cb + j * 32 + 8 * g + 4 * h;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (c + e < p.N) row[c + e] = (OutT)acc[i][j][4 * g + e];
      }
    if (OUT_BF16) __builtin_amdgcn_sched_barrier(0);
  }
}

// ---- stores of layer copies that the fused reduction reads ------------------------------------
// With `co` set, a store is made at device scope: written through this
// chiplet's L2 to the device's coherence point, so that once the wave's stores
// have completed (vmcnt 0) a workgroup on another chiplet can read them with
// device-scope loads, without an L2 write-back or invalidation.  `co` is
// wave-uniform; the choice is a scalar branch inside the store itself, so that
// the compiler keeps one copy of the epilogue (two copies raise the register
// pressure of the kernel past its budget).  The compiler treats the data
// registers as free once the statement ends, but a 16-byte store still reads
// them after it issues: the trailing s_nop keeps the next vector instruction
// from overwriting them too early (the compiler inserts the same wait states
// after its own stores).
__device__ __forceinline__ void st16_co(void* p, u32x4 v, int co) {
  asm volatile("s_cmp_eq_u32 %2, 0\n\t"
               "s_cbranch_scc1 1f\n\t"
               "global_store_dwordx4 %0, %1, off sc1\n\t"
               "s_branch 2f\n"
               "1:\n\t"
               "global_store_dwordx4 %0, %1, off\n"
               "2:\n\t"
               "s_nop 1"
               :: "v"(p), "v"(v), "s"(__builtin_amdgcn_readfirstlane(co)) : "memory", "scc");
}
// 16 bytes of an epilogue store: device scope when the kernel may fuse the
// reduction (fp32 layer copies) and `co` is set, else a plain store.
template <bool FUSABLE>
__device__ __forceinline__ void st16(void* p, u32x4 v, int co) {
  if constexpr (FUSABLE) st16_co(p, v, co);
  else *reinterpret_cast<u32x4*>(p) = v;
}
__device__ __forceinline__ void st_f32(float* p, float v, int co) {
  if (co) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else *p = v;
}

// ---- epilogue through LDS (fast path) ------------------------------------------------------
// After a task's K loop the rings are free.  Each wave writes its sub-block to
// its own LDS region, rows padded by 16 bytes (the fragment writes, 16 rows at
// one column, then hit 16 distinct bank groups), reads it back 16 bytes per
// lane with 16 lanes on one row segment, and stores 16 bytes per lane: a store
// instruction then covers 1024 / (row bytes) whole row segments instead of 16
// or 32 rows of 32-64 bytes, and the store path issues it faster (measured on
// MI355X: about a third less time for the block's stores).  Interior blocks
// with 16-byte aligned rows only; a sub-block that does not fit the rings at
// once goes in several row passes.  The caller synchronises the workgroup
// before the rings are written again.
template <int BM, int BN, int NW, int F8, bool OUT_BF16>
struct Staging {
  using T = Tile<BM, BN, NW, F8>;
  static constexpr int ES = OUT_BF16 ? 2 : 4;                 // bytes per output element
  static constexpr int ROWB = T::WTN * ES;                     // bytes of a sub-block row
  static constexpr int RS = ROWB + 16;                         // LDS row stride
  static constexpr int RING = Ring<BM, BN, NW, F8>::ELEMS * 2; // bytes of LDS
  static constexpr int PASS_ROWS = NW * T::WTM * RS <= RING ? T::WTM : T::WTM / 2;
  static constexpr int PASSES = T::WTM / PASS_ROWS;
  static constexpr int CPR = ROWB / 16;                        // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;                         // rows per store instruction
  static_assert(NW * PASS_ROWS * RS <= RING, "staging fits the rings");
  // used where the whole sub-block fits at once, and for the fp8 kernels; the
  // two-pass form makes the register allocator shuffle the 16x16 accumulators
  // inside the bf16 K loop (fp32 output of 256x256 and 256x128 blocks), which
  // costs more than the stores gain, so those keep the direct stores
  static constexpr bool USE = PASSES == 1 || F8;
  static_assert(PASS_ROWS % T::FS == 0 && PASS_ROWS % RPI == 0, "whole fragments and rows per pass");
};

__device__ __forceinline__ void lds_write16(uint32_t addr, u32x4 v) {
  typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
  *(lds_u32x4*)(uintptr_t)addr = v;
}
__device__ __forceinline__ u32x4 lds_read16(uint32_t addr) {
  typedef __attribute__((address_space(3))) const u32x4 lds_u32x4c;
  return *(lds_u32x4c*)(uintptr_t)addr;
}

template <int BM, int BN, int NW, int F8, bool OUT_BF16>
__device__ __forceinline__ void store_tile_staged(const GemmParams& p, const Acc<BM, BN, NW, F8>& acc, int64_t m0,
                                                  int64_t n0, int64_t lstride, int wm, int wn, int wave, int lane,
                                                  uint32_t lds0, int co) {
  using T = Tile<BM, BN, NW, F8>;
  using S = Staging<BM, BN, NW, F8, OUT_BF16>;
  typedef typename std::conditional<OUT_BF16, __bf16, float>::type OutT;
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
  OutT* out = reinterpret_cast<OutT*>(p.out) + lstride;
  const uint32_t base = lds0 + (uint32_t)(wave * S::PASS_ROWS * S::RS);
  const int64_t row0 = m0 + wm * T::WTM, col0 = n0 + wn * T::WTN;
#pragma unroll
  for (int pass = 0; pass < S::PASSES; ++pass) {
    // fragments of sub-block rows [pass*PASS_ROWS, +PASS_ROWS) into LDS
    if constexpr (F8 != 0) {
      // 32x32 fragments: lane l, run g: row 32i + l%32, columns 32j + 8g + 4(l/32)
      const int h = lane >> 5, r = lane & 31;
#pragma unroll
      for (int ii = 0; ii < S::PASS_ROWS / 32; ++ii) {
        const int i = pass * (S::PASS_ROWS / 32) + ii;
        const uint32_t rowa = base + (uint32_t)((32 * ii + r) * S::RS);
#pragma unroll
        for (int j = 0; j < T::FN; ++j) {
          const f32x16& a = acc[i][j];
          if constexpr (OUT_BF16) {
#pragma unroll
            for (int g = 0; g < 4; g += 2) {
              const bf16x4 xb = {(__bf16)a[4 * g], (__bf16)a[4 * g + 1], (__bf16)a[4 * g + 2], (__bf16)a[4 * g + 3]};
              const bf16x4 yb = {(__bf16)a[4 * g + 4], (__bf16)a[4 * g + 5], (__bf16)a[4 * g + 6], (__bf16)a[4 * g + 7]};
              const u32x2 xw = __builtin_bit_cast(u32x2, xb), yw = __builtin_bit_cast(u32x2, yb);
              const auto s0 = __builtin_amdgcn_permlane32_swap(xw[0], yw[0], false, false);
              const auto s1 = __builtin_amdgcn_permlane32_swap(xw[1], yw[1], false, false);
              lds_write16(rowa + (uint32_t)((32 * j + 8 * g + 8 * h) * 2), u32x4{s0[0], s1[0], s0[1], s1[1]});
            }
          } else {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const f32x4 v = {a[4 * g], a[4 * g + 1], a[4 * g + 2], a[4 * g + 3]};
              lds_write16(rowa + (uint32_t)((32 * j + 8 * g + 4 * h) * 4), __builtin_bit_cast(u32x4, v));
            }
          }
        }
      }
    } else {
      // 16x16 fragments: lane l: row 16i + l%16, columns 16j + 4(l/16)
      const int q = lane >> 4, r = lane & 15;
#pragma unroll
      for (int ii = 0; ii < S::PASS_ROWS / 16; ++ii) {
        const int i = pass * (S::PASS_ROWS / 16) + ii;
        const uint32_t rowa = base + (uint32_t)((16 * ii + r) * S::RS);
        if constexpr (OUT_BF16) {
#pragma unroll
          for (int j = 0; j < T::FN; j += 2)
            lds_write16(rowa + (uint32_t)((16 * j + 16 * (q & 1) + 8 * (q >> 1)) * 2),
                        pair_to_row8(acc[i][j], acc[i][j + 1]));
        } else {
#pragma unroll
          for (int j = 0; j < T::FN; ++j)
            lds_write16(rowa + (uint32_t)((16 * j + 4 * q) * 4), __builtin_bit_cast(u32x4, acc[i][j]));
        }
      }
    }
    wait_lds_all();
    // whole row segments back out: lane l reads chunk l % CPR of row l / CPR
    const int rr = lane / S::CPR, cc = lane % S::CPR;
#pragma unroll
    for (int t = 0; t < S::PASS_ROWS / S::RPI; t += 4) {
      u32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (t + u < S::PASS_ROWS / S::RPI) v[u] = lds_read16(base + (uint32_t)(((t + u) * S::RPI + rr) * S::RS + cc * 16));
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (t + u < S::PASS_ROWS / S::RPI) {
          const int64_t row = row0 + pass * S::PASS_ROWS + (t + u) * S::RPI + rr;
          st16<!OUT_BF16 && F8 == 0>(out + row * p.ldo + col0 + cc * (16 / S::ES), v[u], co);
        }
    }
    if (pass + 1 < S::PASSES) wait_lds_all();   // this wave's reads are done before its next writes
  }
}

template <int BM, int BN, int NW, int F8, bool OUT_BF16>
__device__ __forceinline__ void store_tile(const GemmParams& p, const Acc<BM, BN, NW, F8>& acc, int64_t m0, int64_t n0,
                                           int64_t lstride, int wm, int wn, int lane, bool fast, bool fast16, int co) {
  if constexpr (F8 != 0) {
    store_tile32<BM, BN, NW, OUT_BF16>(p, acc, m0, n0, lstride, wm, wn, lane, fast, fast16);
    return;
  } else {

  using T = Tile<BM, BN, NW, F8>;
  typedef typename std::conditional<OUT_BF16, __bf16, float>::type OutT;
  OutT* out = reinterpret_cast<OutT*>(p.out) + lstride;
  const int64_t r0 = m0 + wm * T::WTM + (lane & 15);
  const int64_t c0 = n0 + wn * T::WTN + 4 * (lane >> 4);
  if constexpr (OUT_BF16 && T::FN % 2 == 0) {
    if (fast16) {
      // whole block inside C, 16-byte aligned rows: one 16-byte store per lane
      // covers 16 rows x 32 columns (half the store instructions of the
      // 8-byte path)
      const int q = lane >> 4;
      const int64_t c8 = n0 + wn * T::WTN + 16 * (q & 1) + 8 * (q >> 1);
#pragma unroll
      for (int i = 0; i < T::FM; ++i) {
        OutT* row = out + (r0 + i * 16) * p.ldo + c8;
#pragma unroll
        for (int j = 0; j < T::FN; j += 2)
          *reinterpret_cast<u32x4*>(row + j * 16) = pair_to_row8(acc[i][j], acc[i][j + 1]);
        __builtin_amdgcn_sched_barrier(0);
      }
      return;
    }
  }
  if (fast) {
    // whole block inside C and 4-element aligned rows: no checks
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
      OutT* row = out + (r0 + i * 16) * p.ldo + c0;
#pragma unroll
      for (int j = 0; j < T::FN; ++j) {
        if (OUT_BF16) {
          bf16x4 v = {(__bf16)acc[i][j][0], (__bf16)acc[i][j][1], (__bf16)acc[i][j][2], (__bf16)acc[i][j][3]};
          *reinterpret_cast<bf16x4*>(row + j * 16) = v;
        } else {
          if (F8 == 0 && co) {
            // device scope, as two 8-byte atomic stores (an inline-assembly
            // store would copy the accumulators out of their registers first)
            typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
            const u64x2 w = __builtin_bit_cast(u64x2, acc[i][j]);
            uint64_t* q = reinterpret_cast<uint64_t*>(row + j * 16);
            __hip_atomic_store(q, w[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(q + 1, w[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          } else {
            *reinterpret_cast<f32x4*>(row + j * 16) = acc[i][j];
          }
        }
      }
      // keep the scheduler from converting every accumulator before storing any
      if (OUT_BF16) __builtin_amdgcn_sched_barrier(0);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < T::FM; ++i) {
    const int64_t r = r0 + i * 16;
    if (r >= p.M) continue;
    OutT* row = out + r * p.ldo;
#pragma unroll
    for (int j = 0; j < T::FN; ++j) {
      const int64_t c = c0 + j * 16;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (c + e < p.N) {
          if constexpr (OUT_BF16) row[c + e] = (OutT)acc[i][j][e];
          else st_f32(reinterpret_cast<float*>(row) + c + e, acc[i][j][e], co);
        }
    }
    if (OUT_BF16) __builtin_amdgcn_sched_barrier(0);
  }
  }
}

// ---- fused reduction of the layer copies ------------------------------------------------
// Listing 1's final add-reduce over the K layers, done inside the GEMM launch
// instead of by a separate kernel.  A workgroup stores its layer copy of a
// block with device-scope stores (written through its chiplet's L2), waits
// until they have completed, and counts the copy on the block's arrival
// counter with a device-scope vector atomic: no L2 write-back is needed on
// this side.  The workgroup whose count completes the block (the last of its
// c_eff layers to finish) invalidates its chiplet's L2 (an acquire fence at
// device scope: lines that other chiplets have since overwritten are not read
// stale), reads every copy and sums them in ascending layer order in fp32,
// exactly as the separate reduction does (same bits), stores C, and resets
// the counter to zero for the next launch.  No workgroup ever waits for
// another.  `flag` is an LDS word that is free at this point (the ring is idle
// between tasks).
template <int BM, int BN, int NW>
__device__ __forceinline__ void fused_finish(const GemmParams& p, int cell, int64_t m0, int64_t n0, int tid,
                                             int* flag) {
  constexpr int THREADS = NW * 64;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's copy has reached the coherence point
  __syncthreads();
  if (tid == 0) *flag = __hip_atomic_fetch_add(p.counters + cell, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const int arrived = *flag;
  __syncthreads();   // every wave has read the flag before the next task's loads reuse the LDS
  if (arrived != p.layers - 1) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");

  const float* W = reinterpret_cast<const float*>(p.out);   // layer copies: dense M x N, ld = N
  const int64_t ls = p.out_layer_stride;
  const int layers = p.layers;
  const int rows = (int)(p.M - m0 < BM ? p.M - m0 : BM);
  const int cols = (int)(p.N - n0 < BN ? p.N - n0 : BN);
  const int esz = p.c_bf16 ? 2 : 4;
  const bool vec = (p.N % 4) == 0 && (p.ldc % 4) == 0 && ((uintptr_t)p.C % (4 * esz)) == 0;
  if (vec) {
    // 4 consecutive columns per thread, BN/4 threads per row, U rows per
    // thread in flight; rows past the block's last re-read that row (in
    // bounds) and are not stored, so the loads carry no branches
    constexpr int TPR = BN / 4, RPP = THREADS / TPR, U = 8;
    const int cg = tid % TPR, r0 = tid / TPR;
    if (4 * cg < cols) {
      const int64_t col = n0 + 4 * cg;
      for (int rb = 0; rb < rows; rb += RPP * U) {
        const float* src[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int r = rb + u * RPP + r0;
          src[u] = W + (m0 + (r < rows ? r : rows - 1)) * p.N + col;
        }
        f32x4 acc[U];
#pragma unroll
        for (int u = 0; u < U; ++u) acc[u] = *reinterpret_cast<const f32x4*>(src[u]);
        for (int l = 1; l < layers; ++l) {
          f32x4 v[U];
#pragma unroll
          for (int u = 0; u < U; ++u) v[u] = *reinterpret_cast<const f32x4*>(src[u] + l * ls);
#pragma unroll
          for (int u = 0; u < U; ++u) {
            acc[u][0] += v[u][0];
            acc[u][1] += v[u][1];
            acc[u][2] += v[u][2];
            acc[u][3] += v[u][3];
          }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int r = rb + u * RPP + r0;
          if (r < rows) {
            const int64_t row = m0 + r;
            if (p.c_bf16) {
              const bf16x4 b = {(__bf16)acc[u][0], (__bf16)acc[u][1], (__bf16)acc[u][2], (__bf16)acc[u][3]};
              *reinterpret_cast<bf16x4*>(reinterpret_cast<__bf16*>(p.C) + row * p.ldc + col) = b;
            } else {
              *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(p.C) + row * p.ldc + col) = acc[u];
            }
          }
        }
      }
    }
  } else {
    // one element per thread, BN (or all) threads per row
    constexpr int TPR = BN < THREADS ? BN : THREADS, RPP = THREADS / TPR;
    const int cc0 = tid % TPR, r0 = tid / TPR;
    for (int rr = r0; rr < rows; rr += RPP)
      for (int cc = cc0; cc < cols; cc += TPR) {
        const int64_t idx = (m0 + rr) * p.N + n0 + cc;
        float sum = W[idx];
        for (int l = 1; l < layers; ++l) sum += W[l * ls + idx];
        if (p.c_bf16) reinterpret_cast<__bf16*>(p.C)[(m0 + rr) * p.ldc + n0 + cc] = (__bf16)sum;
        else reinterpret_cast<float*>(p.C)[(m0 + rr) * p.ldc + n0 + cc] = sum;
      }
  }
  if (tid == 0) __hip_atomic_store(p.counters + cell, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int BM, int BN, int NW, int F8, bool OUT_BF16, bool VEC, int D = default_depth<BM, BN>()>
__global__ __launch_bounds__(NW * 64, 1) void sfc_gemm_kernel(GemmParams p) {
  using T = Tile<BM, BN, NW, F8>;
  static_assert(T::A_CH >= 1 && T::B_CH >= 1, "tile too small for the workgroup");
  static_assert(!F8 || VEC, "fp8 operands take the fast path only");
  // fast path: the rings of A block and B stage slots; general path: two 64-deep blocks
  constexpr int kSmem = VEC ? Ring<BM, BN, NW, F8, D>::ELEMS : 2 * (T::A_ELEMS + T::B_ELEMS);
  __shared__ __attribute__((aligned(16))) uint16_t smem[kSmem];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / T::WGN, wn = wave % T::WGN;
  ReadOffsets<BM, BN, NW, F8> ro;
  if constexpr (VEC) read_offsets<BM, BN, NW, F8>(wm, wn, lane, lds_addr(smem) + (uint32_t)Ring<BM, BN, NW, F8, D>::B_OFF, ro);

  const int P = gridDim.x;
  // SFC_SCHED_INTERLEAVED_PLAIN keeps the hardware order (comparison only)
  const int rank = p.sched == 2 ? (int)blockIdx.x : xcd_rank(blockIdx.x, P);
  // task counts are below 2^31 (the library checks it), so 32-bit indices do
  const int NT = (int)p.tasks;
  int t_begin, t_end, t_step;
  if (p.sched == 1) {                  // block partition
    t_begin = (int)((int64_t)NT * rank / P);
    t_end = (int)((int64_t)NT * (rank + 1) / P);
    t_step = 1;
  } else {                             // interleaved
    t_begin = rank;
    t_end = NT;
    t_step = P;
  }
  const int cells = p.gm * p.gn;
  // 4-wide stores need 4-element aligned rows (and layer copies).
  const int esize = OUT_BF16 ? 2 : 4;
  const bool vec_store = ((uintptr_t)p.out % (4 * esize)) == 0 && (p.ldo % 4) == 0 &&
                         (p.out_layer_stride % 4) == 0;
  // 8-element (16-byte) aligned rows for the paired bf16 stores
  const bool vec16_store = ((uintptr_t)p.out % 16) == 0 && (p.ldo % 8) == 0 && (p.out_layer_stride % 8) == 0;

  for (int t = t_begin; t < t_end; t += t_step) {
    // Per-lane values are recomputed for every task rather than kept live
    // across the whole kernel (that costs registers the main loop needs).
    int lane_t;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane_t));
    const int layer = t / cells;
    const int s = t - layer * cells;
    // scalar load: a vector load here would wait for the previous task's stores
    const int cell = load_scalar_i32(p.table + s);
    const int im = cell / p.gn, in = cell - im * p.gn;
    const int64_t m0 = (int64_t)im * BM, n0 = (int64_t)in * BN;
    const int kt0 = (int)((unsigned)layer * (unsigned)p.nk / (unsigned)p.layers);
    const int kt1 = (int)((unsigned)(layer + 1) * (unsigned)p.nk / (unsigned)p.layers);

    Acc<BM, BN, NW, F8> acc;
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
      for (int j = 0; j < T::FN; ++j) {
        if constexpr (F8 != 0) acc[i][j] = f32x16{};
        else acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      }

    if (kt0 < kt1) {
      if constexpr (VEC) {
        constexpr int ESZ = F8 ? 1 : 2;          // bytes per element
        constexpr int SK = stage_k<F8>();
        const int64_t k0 = (int64_t)kt0 * block_k<F8>();
        RingLanes<BM, BN, NW, F8> L;
        ring_lanes<BM, BN, NW, F8>(p, m0, n0, wave, lane_t, L);
        RingAddr ra;
        const uint8_t* Ab = reinterpret_cast<const uint8_t*>(p.A);
        const uint8_t* Bb = reinterpret_cast<const uint8_t*>(p.B);
        ra.a0 = reinterpret_cast<uint64_t>(Ab + (m0 * p.lda + k0) * ESZ) - kBias;
        ra.b0 = reinterpret_cast<uint64_t>(Bb + (k0 * p.ldb + n0) * ESZ) - kBias;
        ra.b_step = (uint64_t)SK * (uint64_t)p.ldb * ESZ;
        {
          // rows of B from the task's first stage to the end of its layer's K
          // range (row K for the last layer): the stages that the ring loads
          // ahead past that point get empty ranges and fetch nothing
          const int64_t k_end = (int64_t)kt1 * block_k<F8>() < p.K ? (int64_t)kt1 * block_k<F8>() : p.K;
          const int b_rows = (int)(k_end - k0);
          ra.x_part = b_rows / SK;
          ra.lim_part = (uint32_t)((b_rows % SK) * (int)(p.ldb * ESZ) + kBias);
        }
        ra.lds0 = lds_addr(smem);
        ra.wave = wave;
        // K elements of the task's last block that lie before K (a full
        // block unless the block runs past K), in 32 bits: the per-lane K-mask
        // compares then stay single registers
        const int64_t kin64 = p.K - (int64_t)(kt1 - 1) * block_k<F8>();
        const int kin_last = kin64 < block_k<F8>() ? (int)kin64 : block_k<F8>();
        main_loop_ring<BM, BN, NW, F8, D>(ra, kt1 - kt0, kin_last, ro, L, lane_t, acc);
      } else if constexpr (!F8) {
        main_loop_staged<BM, BN, NW, F8>(p, smem, m0, n0, kt0, kt1, tid, acc);
      }
    }

    const int64_t lstride = p.out_layer_stride * layer;
    const bool interior = m0 + BM <= p.M && n0 + BN <= p.N;
    // layer copies that this launch reduces itself are stored coherently
    constexpr bool kFusable = !OUT_BF16 && F8 == 0;
    const bool fused = kFusable && p.counters != nullptr;
    if (VEC && Staging<BM, BN, NW, F8, OUT_BF16>::USE && interior && (OUT_BF16 ? vec16_store : vec_store)) {
      if constexpr (VEC && Staging<BM, BN, NW, F8, OUT_BF16>::USE) {
        store_tile_staged<BM, BN, NW, F8, OUT_BF16>(p, acc, m0, n0, lstride, wm, wn, wave, lane_t, lds_addr(smem),
                                                    fused ? 1 : 0);
        // every wave has read its staging rows before the next task's loads
        // land in the rings
        wait_lds_all();
        __syncthreads();
      }
    } else {
      store_tile<BM, BN, NW, F8, OUT_BF16>(p, acc, m0, n0, lstride, wm, wn, lane_t, interior && vec_store,
                                        interior && vec16_store, fused ? 1 : 0);
    }
    if constexpr (kFusable) {
      if (fused) fused_finish<BM, BN, NW>(p, cell, m0, n0, tid, reinterpret_cast<int*>(smem));
    }
  }
}

// ---- dispatch ---------------------------------------------------------------------
// Every variant runs 4 waves per workgroup.  (256x256 blocks with 8 waves, two
// per SIMD and 128x64 each, needed ~3.5 % fewer cycles per launch on MI355X
// but read 1.5x the LDS bytes and ran at a lower clock for the same time.)
constexpr int kWaves = 4;

template <int BM, int BN, int NW, int F8, bool OB, bool VEC, int D = default_depth<BM, BN>()>
static const void* kernel_ptr() {
  return reinterpret_cast<const void*>(&sfc_gemm_kernel<BM, BN, NW, F8, OB, VEC, D>);
}

// fp8 operands (f8 = 1 + a + 2b, a and b the formats of A and B: 0 OCP E4M3,
// 1 OCP E5M2): 256x256 or 128x256 blocks, fast path only.
static const void* select_kernel_f8(int tile, bool ob, int f8) {
  if (tile != kT256x256 && tile != kT128x256) return nullptr;
  const bool wide = tile == kT256x256;
#define SFC_K8(F_)                                                                                        \
  return wide ? (ob ? kernel_ptr<256, 256, 4, F_, true, true>() : kernel_ptr<256, 256, 4, F_, false, true>()) \
              : (ob ? kernel_ptr<128, 256, 4, F_, true, true>() : kernel_ptr<128, 256, 4, F_, false, true>())
  switch (f8) {
    case 1: SFC_K8(1);
    case 2: SFC_K8(2);
    case 3: SFC_K8(3);
    case 4: SFC_K8(4);
    default: return nullptr;
  }
#undef SFC_K8
}

// deep: the 4-deep ring of 128x128 blocks (fast path), for grids of at most
// one block per CU.
static const void* select_kernel(int tile, bool ob, bool vec, bool deep) {
  if (deep) {
    if (tile != kT128x128 || !vec) return nullptr;
    return ob ? kernel_ptr<128, 128, kWaves, 0, true, true, 4>() : kernel_ptr<128, 128, kWaves, 0, false, true, 4>();
  }
#define SFC_K(BM_, BN_, NW_)                                                                   \
  return ob ? (vec ? kernel_ptr<BM_, BN_, NW_, 0, true, true>() : kernel_ptr<BM_, BN_, 4, 0, true, false>()) \
            : (vec ? kernel_ptr<BM_, BN_, NW_, 0, false, true>() : kernel_ptr<BM_, BN_, 4, 0, false, false>())
  switch (tile) {
    case kT128x128: SFC_K(128, 128, kWaves);
    case kT256x128: SFC_K(256, 128, kWaves);
    case kT128x256: SFC_K(128, 256, kWaves);
    case kT256x256: SFC_K(256, 256, kWaves);
    default: return nullptr;
  }
#undef SFC_K
}

static int threads_of(int, bool) { return kWaves * 64; }

hipError_t launch_gemm(int tile, bool out_bf16, bool vec, const GemmParams& p, int grid,
                       hipStream_t stream, int f8, bool deep) {
  const void* k = f8 ? select_kernel_f8(tile, out_bf16, f8) : select_kernel(tile, out_bf16, vec, deep);
  if (!k) return hipErrorInvalidValue;
  GemmParams local = p;
  void* args[] = {&local};
  return hipLaunchKernel(k, dim3(grid), dim3(threads_of(tile, vec)), args, 0, stream);
}

hipError_t gemm_occupancy(int tile, bool out_bf16, bool vec, int* blocks_per_cu, int f8, bool deep) {
  const void* k = f8 ? select_kernel_f8(tile, out_bf16, f8) : select_kernel(tile, out_bf16, vec, deep);
  if (!k) return hipErrorInvalidValue;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, k, threads_of(tile, vec), 0);
}

}  // namespace sfc
