// Persistent bf16 MFMA GEMM for gfx950 whose output blocks are taken in
// space-filling-curve order, with the communication-avoiding K split.
//
// What it computes (Listing 1, Section II.D): the task space has gm*gn*layers
// entries; task t is layer l = t / (gm*gn) and curve position s = t % (gm*gn);
// the curve table maps s to the output block (im, in); layer l contracts the
// l-th contiguous range of 64-deep K blocks into its own copy of the block.
// With one layer the copy is C itself (fp32 or bf16); with several it is an
// fp32 workspace layer that a separate reduction sums.
//
// Mapping to the chip:
//   * one workgroup = 4 waves (2 x 2), each wave owns a (BM/2) x (BN/2)
//     sub-block held as 32x32 fp32 MFMA accumulators;
//   * the grid is persistent: P workgroups, P = CUs x occupancy, each looping
//     over tasks.  Hardware deals workgroup b to chiplet (XCD) b % 8; ranks are
//     renumbered so that each XCD's workgroups hold consecutive ranks, and with
//     the interleaved schedule the P tasks in flight are one contiguous curve
//     segment whose XCD sub-segments are compact patches sharing A rows and B
//     columns in that XCD's L2;
//   * A and B K-blocks are staged through LDS, double buffered, with one
//     barrier per K block.  On the fast path (16-byte aligned rows) they go
//     straight from global memory into LDS with buffer loads (lanes outside
//     the matrix read zeros), so no registers hold staged data; otherwise
//     they are assembled element by element in registers.  A is kept
//     row-major [BM][64]; B is kept as loaded,
//     [64][BN], and the MFMA B operand is assembled with the transposing LDS
//     read (ds_read_b64_tr_b16).  16-byte chunks are XOR-swizzled so that both
//     the fragment reads and the staging writes are free of bank conflicts on
//     the 64-bank LDS;
//   * bf16 MFMA 32x32x16 with fp32 accumulation (Section III.A's BRGEMM role).
#include <type_traits>

#include "sfc_params.h"

namespace sfc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// ---- chiplet-aware rank ------------------------------------------------------
// Workgroup b runs on XCD b % 8.  Ranks give each XCD a contiguous range.
__device__ __forceinline__ int xcd_rank(int b, int P) {
  constexpr int X = 8;
  const int x = b % X, i = b / X;
  const int q = P / X, r = P % X;
  return x * q + (x < r ? x : r) + i;
}

// ---- LDS layouts ---------------------------------------------------------------
// A block: [BM rows][64 k] bf16 = 8 chunks of 16 B per row; chunk c of row r is
// stored at chunk c ^ ((r >> 1) & 7).  Sixteen consecutive rows read at one
// logical chunk then hit 16 distinct 16-byte bank groups.
__device__ __forceinline__ int a_off(int row, int chunk) {
  return row * kBK + ((chunk ^ ((row >> 1) & 7)) << 3);
}
// B block: [64 k][BN n] bf16; chunk c (8 columns) of row k is stored at chunk
// c ^ ((k & 3) << 2).  The transposing read touches 4 rows x 4 chunks per
// 32 lanes, which this spreads over all 16 bank groups.
template <int BN>
__device__ __forceinline__ int b_off(int k, int n) {
  return k * BN + ((((n >> 3) ^ ((k & 3) << 2))) << 3) + (n & 7);
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
// buffer_load_dwordx4 ... lds: every lane fetches 16 bytes at (descriptor base +
// its voffset) and the wave writes them to LDS at M0 + 16*lane.  A lane whose
// voffset lies at or beyond the descriptor's num_records fetches zeros.  The
// instruction is issued from inline assembly so that the compiler does not
// serialise later LDS reads behind it; the kernel orders it explicitly with
// s_waitcnt vmcnt and workgroup barriers.
typedef int i32x4 __attribute__((ext_vector_type(4)));
constexpr int kOobOffset = 0x7FFFFFF0;   // num_records; a lane at this offset reads zeros

__device__ __forceinline__ i32x4 make_rsrc(const void* base) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  // raw buffer: 48-bit base, stride 0, num_records, word 3 = 0x00020000 on gfx9 parts
  i32x4 r = {(int)(uint32_t)a, (int)((uint32_t)(a >> 32) & 0xFFFFu), kOobOffset, 0x00020000};
  r[0] = __builtin_amdgcn_readfirstlane(r[0]);
  r[1] = __builtin_amdgcn_readfirstlane(r[1]);
  return r;
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

__device__ __forceinline__ void dma16(i32x4 rsrc, uint32_t lds_byte_addr, int voffset) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(lds_byte_addr), "v"(voffset), "s"(rsrc) : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmem_at_most() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}
__device__ __forceinline__ void wait_lds_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// ---- one K block of MFMA work ----------------------------------------------------------
template <int BM, int BN>
struct Tile {
  static constexpr int WTM = BM / 2, WTN = BN / 2;   // wave sub-block (2 x 2 waves)
  static constexpr int FM = WTM / 32, FN = WTN / 32; // 32x32 fragments per wave
  static constexpr int A_ELEMS = BM * kBK, B_ELEMS = kBK * BN;
  static constexpr int A_CH = BM * kBK / 8 / kThreads;   // 16-byte chunks per thread
  static constexpr int B_CH = kBK * BN / 8 / kThreads;
};

template <int BM, int BN>
struct Frags {
  bf16x8 a[Tile<BM, BN>::FM];
  bf16x8 b[Tile<BM, BN>::FN];
};

// Operand fragments of k sub-step ks (16 deep) for this lane.
template <int BM, int BN>
__device__ __forceinline__ void load_frags(const uint16_t* As, const uint16_t* Bs, int wm, int wn,
                                           int lane, int ks, Frags<BM, BN>& f) {
  using T = Tile<BM, BN>;
#pragma unroll
  for (int i = 0; i < T::FM; ++i) {
    // A operand: lane holds row lane%32, k = 8*(lane/32) .. +8
    const int row = wm * T::WTM + i * 32 + (lane & 31);
    const int c = ks * 2 + (lane >> 5);
    f.a[i] = *reinterpret_cast<const bf16x8*>(As + a_off(row, c));
  }
#pragma unroll
  for (int j = 0; j < T::FN; ++j) {
    // B operand: lane holds column lane%32, k = 8*(lane/32) .. +8.  Lane
    // (g = lane/16, jj = lane%16) points at row k, columns n..n+3; the
    // transposing read returns column n0 + jj of rows k0..k0+3 to lane jj.
    const int g = lane >> 4, jj = lane & 15;
    const int n = wn * T::WTN + j * 32 + ((g & 1) << 4) + ((jj & 3) << 2);
    const int k = ks * 16 + ((g >> 1) << 3) + (jj >> 2);
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(Bs + b_off<BN>(k, n)));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(Bs + b_off<BN>(k + 4, n)));
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    f.b[j] = __builtin_bit_cast(bf16x8, v);
  }
}

// acc += one 16-deep step, with the fragment reads of the following step
// interleaved between the MFMAs (one LDS read after each of the first MFMAs).
template <int BM, int BN>
__device__ __forceinline__ void mma_step(const Frags<BM, BN>& cur,
                                         f32x16 (&acc)[Tile<BM, BN>::FM][Tile<BM, BN>::FN]) {
  using T = Tile<BM, BN>;
#pragma unroll
  for (int i = 0; i < T::FM; ++i)
#pragma unroll
    for (int j = 0; j < T::FN; ++j)
      // B fragment as the first operand: the accumulator holds the transposed
      // 32x32 block, so each lane ends with runs of 4 consecutive columns.
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.b[j], cur.a[i], acc[i][j], 0, 0, 0);
}

template <int BM, int BN>
__device__ __forceinline__ void interleave_reads_with_mfma() {
  using T = Tile<BM, BN>;
  constexpr int kMfma = T::FM * T::FN;
  constexpr int kReads = T::FM + 2 * T::FN;
  constexpr int kPaired = kReads < kMfma ? kReads : kMfma;
#pragma unroll
  for (int r = 0; r < kPaired; ++r) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
  }
  if (kMfma > kPaired) __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kPaired, 0);
  if (kReads > kPaired) __builtin_amdgcn_sched_group_barrier(0x100, kReads - kPaired, 0);
}

// ---- main loop, fast path: buffer loads straight into LDS ---------------------------------
// Wave w fills LDS 1 KiB segments w, w+4, w+8, ...; lane l of a segment holds
// physical 16-byte chunk l of it, i.e. it loads the logical chunk that the
// swizzle stores there.  Lanes outside M, N or K use an offset past the
// buffer's range and write zeros.
//
// Software pipeline (two LDS buffers, one barrier per 64-deep block):
//   step 0..2 of block kt: MFMAs of step s, reads of step s+1 from buffer b;
//   step 3: wait for this wave's loads of block kt+1 and its reads of step 3,
//           barrier (block kt+1 is now visible and buffer b is free), issue the
//           loads of block kt+2 into b, then the MFMAs of step 3 with the reads
//           of step 0 of block kt+1 from buffer b^1.
template <int BM, int BN>
__device__ __forceinline__ void main_loop_direct(const GemmParams& p, uint16_t* smem, int64_t m0,
                                                 int64_t n0, int kt0, int kt1, int wave, int lane,
                                                 f32x16 (&acc)[Tile<BM, BN>::FM][Tile<BM, BN>::FN]) {
  using T = Tile<BM, BN>;
  constexpr int kStage = T::A_ELEMS + T::B_ELEMS;
  constexpr int kLoads = T::A_CH + T::B_CH;
  const int wm = wave >> 1, wn = wave & 1;
  int a_voff[T::A_CH], a_k[T::A_CH], b_voff[T::B_CH], b_k[T::B_CH];
#pragma unroll
  for (int i = 0; i < T::A_CH; ++i) {
    const int seg = i * 4 + wave;               // rows 8*seg .. 8*seg+7
    const int row = seg * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    a_k[i] = c * 8;
    a_voff[i] = (m0 + row < p.M) ? (int)((row * p.lda + c * 8) * 2) : kOobOffset;
  }
#pragma unroll
  for (int i = 0; i < T::B_CH; ++i) {
    const int seg = i * 4 + wave;
    const int e = seg * 512 + lane * 8;         // element index in the [64][BN] block
    const int k = e / BN;
    const int c = ((e % BN) >> 3) ^ ((k & 3) << 2);
    b_k[i] = k;
    b_voff[i] = (n0 + c * 8 < p.N) ? (int)((k * p.ldb + c * 8) * 2) : kOobOffset;
  }
  const uint32_t smem_lds = lds_addr(smem);
  auto issue = [&](int kt, int buf) {
    const int64_t k0 = (int64_t)kt * kBK;
    const i32x4 ra = make_rsrc(p.A + m0 * p.lda + k0);
    const i32x4 rb = make_rsrc(p.B + k0 * p.ldb + n0);
    const uint32_t a_base = smem_lds + (uint32_t)(buf * kStage) * 2u;
    const uint32_t b_base = a_base + (uint32_t)T::A_ELEMS * 2u;
#pragma unroll
    for (int i = 0; i < T::A_CH; ++i)
      dma16(ra, a_base + (uint32_t)((i * 4 + wave) * 1024),
            (k0 + a_k[i] < p.K) ? a_voff[i] : kOobOffset);
#pragma unroll
    for (int i = 0; i < T::B_CH; ++i)
      dma16(rb, b_base + (uint32_t)((i * 4 + wave) * 1024),
            (k0 + b_k[i] < p.K) ? b_voff[i] : kOobOffset);
  };

  issue(kt0, 0);
  if (kt0 + 1 < kt1) {
    issue(kt0 + 1, 1);
    wait_vmem_at_most<kLoads>();
  } else {
    wait_vmem_at_most<0>();
  }
  __syncthreads();

  Frags<BM, BN> f0, f1;
  load_frags<BM, BN>(smem, smem + T::A_ELEMS, wm, wn, lane, 0, f0);
  for (int kt = kt0; kt < kt1; ++kt) {
    const int buf = (kt - kt0) & 1;
    const uint16_t* As = smem + buf * kStage;
    const uint16_t* Bs = As + T::A_ELEMS;
    load_frags<BM, BN>(As, Bs, wm, wn, lane, 1, f1);
    mma_step<BM, BN>(f0, acc);
    interleave_reads_with_mfma<BM, BN>();
    load_frags<BM, BN>(As, Bs, wm, wn, lane, 2, f0);
    mma_step<BM, BN>(f1, acc);
    interleave_reads_with_mfma<BM, BN>();
    load_frags<BM, BN>(As, Bs, wm, wn, lane, 3, f1);
    mma_step<BM, BN>(f0, acc);
    interleave_reads_with_mfma<BM, BN>();
    // Step 3 runs the same way on the last block (one MFMA chain, no copies
    // of the accumulators); the reads of the other buffer are then unused.
    wait_vmem_at_most<0>();
    wait_lds_all();
    __syncthreads();
    if (kt + 2 < kt1) issue(kt + 2, buf);
    const uint16_t* An = smem + (buf ^ 1) * kStage;
    load_frags<BM, BN>(An, An + T::A_ELEMS, wm, wn, lane, 0, f0);
    mma_step<BM, BN>(f1, acc);
    interleave_reads_with_mfma<BM, BN>();
  }
  // the next task's first loads overwrite both buffers
  wait_lds_all();
  __syncthreads();
}

// ---- main loop, general path: element loads staged in registers ---------------------------
template <int BM, int BN>
__device__ __forceinline__ void main_loop_staged(const GemmParams& p, uint16_t* smem, int64_t m0,
                                                 int64_t n0, int kt0, int kt1, int tid,
                                                 f32x16 (&acc)[Tile<BM, BN>::FM][Tile<BM, BN>::FN]) {
  using T = Tile<BM, BN>;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  u32x4 ra[T::A_CH], rb[T::B_CH];
  auto load_blocks = [&](int kt) {
    const int64_t k0 = (int64_t)kt * kBK;
#pragma unroll
    for (int i = 0; i < T::A_CH; ++i) {
      const int q = tid + kThreads * i;
      ra[i] = load_chunk<false>(p.A, p.lda, m0 + (q >> 3), k0 + (q & 7) * 8, p.M, p.K);
    }
#pragma unroll
    for (int i = 0; i < T::B_CH; ++i) {
      const int q = tid + kThreads * i;
      rb[i] = load_chunk<false>(p.B, p.ldb, k0 + q / (BN / 8), n0 + (q % (BN / 8)) * 8, p.K, p.N);
    }
  };
  auto store_blocks = [&](int buf) {
    uint16_t* As = smem + buf * (T::A_ELEMS + T::B_ELEMS);
    uint16_t* Bs = As + T::A_ELEMS;
#pragma unroll
    for (int i = 0; i < T::A_CH; ++i) {
      const int q = tid + kThreads * i;
      *reinterpret_cast<u32x4*>(As + a_off(q >> 3, q & 7)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < T::B_CH; ++i) {
      const int q = tid + kThreads * i;
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
    for (int ks = 0; ks < kBK / 16; ++ks) {
      Frags<BM, BN> f;
      load_frags<BM, BN>(As, As + T::A_ELEMS, wm, wn, lane, ks, f);
      mma_step<BM, BN>(f, acc);
    }
    if (more) store_blocks(buf ^ 1);
    __syncthreads();
  }
}

// ---- epilogue ---------------------------------------------------------------------------------
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

template <int BM, int BN, bool OUT_BF16>
__device__ __forceinline__ void store_tile(const GemmParams& p,
                                           const f32x16 (&acc)[Tile<BM, BN>::FM][Tile<BM, BN>::FN],
                                           int64_t m0, int64_t n0, int64_t lstride, int wm, int wn,
                                           int lane, bool fast) {
  using T = Tile<BM, BN>;
  typedef typename std::conditional<OUT_BF16, __bf16, float>::type OutT;
  OutT* out = reinterpret_cast<OutT*>(p.out) + lstride;
  const int col_lane = 4 * (lane >> 5);
  if (fast) {
    // whole block inside C and 4-element aligned rows: no checks
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
      OutT* row = out + (m0 + wm * T::WTM + i * 32 + (lane & 31)) * p.ldo + n0 + wn * T::WTN + col_lane;
#pragma unroll
      for (int j = 0; j < T::FN; ++j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          OutT* dst = row + j * 32 + q * 8;
          if (OUT_BF16) {
            bf16x4 v = {(__bf16)acc[i][j][4 * q], (__bf16)acc[i][j][4 * q + 1],
                        (__bf16)acc[i][j][4 * q + 2], (__bf16)acc[i][j][4 * q + 3]};
            *reinterpret_cast<bf16x4*>(dst) = v;
          } else {
            f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            *reinterpret_cast<f32x4*>(dst) = v;
          }
        }
        // keep the scheduler from converting every accumulator before storing any
        if (OUT_BF16) __builtin_amdgcn_sched_barrier(0);
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < T::FM; ++i) {
    const int64_t r = m0 + wm * T::WTM + i * 32 + (lane & 31);
    if (r >= p.M) continue;
    OutT* row = out + r * p.ldo;
#pragma unroll
    for (int j = 0; j < T::FN; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t c = n0 + wn * T::WTN + j * 32 + q * 8 + col_lane;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (c + e < p.N) row[c + e] = (OutT)acc[i][j][4 * q + e];
      }
      if (OUT_BF16) __builtin_amdgcn_sched_barrier(0);
    }
  }
}

template <int BM, int BN, bool OUT_BF16, bool VEC>
__global__ __launch_bounds__(kThreads, 1) void sfc_gemm_kernel(GemmParams p) {
  using T = Tile<BM, BN>;
  static_assert(T::A_CH >= 1 && T::B_CH >= 1, "tile too small for 256 threads");
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (T::A_ELEMS + T::B_ELEMS)];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  const int P = gridDim.x;
  const int rank = xcd_rank(blockIdx.x, P);
  const int64_t NT = p.tasks;
  int64_t t_begin, t_end, t_step;
  if (p.sched == 1) {                  // block partition
    t_begin = NT * rank / P;
    t_end = NT * (rank + 1) / P;
    t_step = 1;
  } else {                             // interleaved
    t_begin = rank;
    t_end = NT;
    t_step = P;
  }
  const int64_t cells = (int64_t)p.gm * p.gn;
  // 4-wide stores need 4-element aligned rows (and layer copies).
  const int esize = OUT_BF16 ? 2 : 4;
  const bool vec_store = ((uintptr_t)p.out % (4 * esize)) == 0 && (p.ldo % 4) == 0 &&
                         (p.out_layer_stride % 4) == 0;

  for (int64_t t = t_begin; t < t_end; t += t_step) {
    const int layer = (int)(t / cells);
    const int s = (int)(t - (int64_t)layer * cells);
    const int cell = p.table[s];
    const int im = cell / p.gn, in = cell - im * p.gn;
    const int64_t m0 = (int64_t)im * BM, n0 = (int64_t)in * BN;
    const int kt0 = (int)((int64_t)layer * p.nk / p.layers);
    const int kt1 = (int)((int64_t)(layer + 1) * p.nk / p.layers);

    f32x16 acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
      for (int j = 0; j < T::FN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    if (kt0 < kt1) {
      if constexpr (VEC) main_loop_direct<BM, BN>(p, smem, m0, n0, kt0, kt1, wave, lane, acc);
      else main_loop_staged<BM, BN>(p, smem, m0, n0, kt0, kt1, tid, acc);
    }

    // Epilogue.  Accumulator element e of fragment (i, j) is row lane%32 and
    // column 8*(e/4) + 4*(lane/32) + e%4 of that 32x32 fragment.
    const int64_t lstride = p.out_layer_stride * layer;
    const bool interior = m0 + BM <= p.M && n0 + BN <= p.N;
    store_tile<BM, BN, OUT_BF16>(p, acc, m0, n0, lstride, wm, wn, lane, interior && vec_store);
  }
}

// ---- dispatch ---------------------------------------------------------------------
template <int BM, int BN, bool OB, bool VEC>
static const void* kernel_ptr() {
  return reinterpret_cast<const void*>(&sfc_gemm_kernel<BM, BN, OB, VEC>);
}

static const void* select_kernel(int tile, bool ob, bool vec) {
#define SFC_K(BM_, BN_)                                                        \
  return ob ? (vec ? kernel_ptr<BM_, BN_, true, true>() : kernel_ptr<BM_, BN_, true, false>()) \
            : (vec ? kernel_ptr<BM_, BN_, false, true>() : kernel_ptr<BM_, BN_, false, false>())
  switch (tile) {
    case kT128x128: SFC_K(128, 128);
    case kT256x128: SFC_K(256, 128);
    case kT128x256: SFC_K(128, 256);
    case kT256x256: SFC_K(256, 256);
    default: return nullptr;
  }
#undef SFC_K
}

hipError_t launch_gemm(int tile, bool out_bf16, bool vec, const GemmParams& p, int grid,
                       hipStream_t stream) {
  const void* k = select_kernel(tile, out_bf16, vec);
  if (!k) return hipErrorInvalidValue;
  GemmParams local = p;
  void* args[] = {&local};
  return hipLaunchKernel(k, dim3(grid), dim3(kThreads), args, 0, stream);
}

hipError_t gemm_occupancy(int tile, bool out_bf16, bool vec, int* blocks_per_cu) {
  const void* k = select_kernel(tile, out_bf16, vec);
  if (!k) return hipErrorInvalidValue;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, k, kThreads, 0);
}

}  // namespace sfc
