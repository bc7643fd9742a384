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
//     barrier per K block.  A is kept row-major [BM][64]; B is kept as loaded,
//     [64][BN], and the MFMA B operand is assembled with the transposing LDS
//     read (ds_read_b64_tr_b16).  16-byte chunks are XOR-swizzled so that both
//     the fragment reads and the staging writes are free of bank conflicts on
//     the 64-bank LDS;
//   * bf16 MFMA 32x32x16 with fp32 accumulation (Section III.A's BRGEMM role).
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

template <int BM, int BN, bool OUT_BF16, bool VEC>
__global__ __launch_bounds__(kThreads, 1) void sfc_gemm_kernel(GemmParams p) {
  constexpr int WTM = BM / 2, WTN = BN / 2;       // wave sub-block
  constexpr int FM = WTM / 32, FN = WTN / 32;     // 32x32 fragments per wave
  constexpr int A_CH = BM * kBK / 8 / kThreads;   // 16-byte chunks per thread
  constexpr int B_CH = kBK * BN / 8 / kThreads;
  constexpr int A_ELEMS = BM * kBK, B_ELEMS = kBK * BN;
  static_assert(A_CH >= 1 && B_CH >= 1, "tile too small for 256 threads");

  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (A_ELEMS + B_ELEMS)];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const int P = gridDim.x;
  const int rank = xcd_rank(blockIdx.x, P);
  const int64_t T = p.tasks;
  int64_t t_begin, t_end, t_step;
  if (p.sched == 1) {                  // block partition
    t_begin = T * rank / P;
    t_end = T * (rank + 1) / P;
    t_step = 1;
  } else {                             // interleaved
    t_begin = rank;
    t_end = T;
    t_step = P;
  }
  const int64_t cells = (int64_t)p.gm * p.gn;

  for (int64_t t = t_begin; t < t_end; t += t_step) {
    const int layer = (int)(t / cells);
    const int s = (int)(t - (int64_t)layer * cells);
    const int cell = p.table[s];
    const int im = cell / p.gn, in = cell - im * p.gn;
    const int64_t m0 = (int64_t)im * BM, n0 = (int64_t)in * BN;
    const int kt0 = (int)((int64_t)layer * p.nk / p.layers);
    const int kt1 = (int)((int64_t)(layer + 1) * p.nk / p.layers);

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    if (kt0 < kt1) {
      u32x4 ra[A_CH], rb[B_CH];
      auto load_blocks = [&](int kt) {
        const int64_t k0 = (int64_t)kt * kBK;
#pragma unroll
        for (int i = 0; i < A_CH; ++i) {
          const int q = tid + kThreads * i;
          const int row = q >> 3, c = q & 7;
          ra[i] = load_chunk<VEC>(p.A, p.lda, m0 + row, k0 + c * 8, p.M, p.K);
        }
#pragma unroll
        for (int i = 0; i < B_CH; ++i) {
          const int q = tid + kThreads * i;
          const int k = q / (BN / 8), c = q % (BN / 8);
          rb[i] = load_chunk<VEC>(p.B, p.ldb, k0 + k, n0 + c * 8, p.K, p.N);
        }
      };
      auto store_blocks = [&](int buf) {
        uint16_t* As = smem + buf * (A_ELEMS + B_ELEMS);
        uint16_t* Bs = As + A_ELEMS;
#pragma unroll
        for (int i = 0; i < A_CH; ++i) {
          const int q = tid + kThreads * i;
          const int row = q >> 3, c = q & 7;
          *reinterpret_cast<u32x4*>(As + a_off(row, c)) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < B_CH; ++i) {
          const int q = tid + kThreads * i;
          const int k = q / (BN / 8), c = q % (BN / 8);
          *reinterpret_cast<u32x4*>(Bs + b_off<BN>(k, c * 8)) = rb[i];
        }
      };

      load_blocks(kt0);
      store_blocks(0);
      __syncthreads();

      for (int kt = kt0; kt < kt1; ++kt) {
        const int buf = (kt - kt0) & 1;
        const bool more = kt + 1 < kt1;
        if (more) load_blocks(kt + 1);

        const uint16_t* As = smem + buf * (A_ELEMS + B_ELEMS);
        const uint16_t* Bs = As + A_ELEMS;
#pragma unroll
        for (int ks = 0; ks < kBK / 16; ++ks) {
          bf16x8 af[FM], bfr[FN];
#pragma unroll
          for (int i = 0; i < FM; ++i) {
            const int row = wm * WTM + i * 32 + (lane & 31);
            const int c = ks * 2 + (lane >> 5);
            af[i] = *reinterpret_cast<const bf16x8*>(As + a_off(row, c));
          }
#pragma unroll
          for (int j = 0; j < FN; ++j) {
            // Lane (g = lane/16, jj = lane%16) points at row k, columns n..n+3; the
            // transposing read returns column (n0 + jj) of rows k0..k0+3 to lane jj.
            const int g = lane >> 4, jj = lane & 15;
            const int n = wn * WTN + j * 32 + ((g & 1) << 4) + ((jj & 3) << 2);
            const int k = ks * 16 + ((g >> 1) << 3) + (jj >> 2);
            const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_i16x4*)(Bs + b_off<BN>(k, n)));
            const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_i16x4*)(Bs + b_off<BN>(k + 4, n)));
            const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            bfr[j] = __builtin_bit_cast(bf16x8, v);
          }
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }

        if (more) store_blocks(buf ^ 1);
        __syncthreads();
      }
    }

    // Epilogue: element e of a 32x32 accumulator sits at row (e/4)*8 + (lane/32)*4 + e%4,
    // column lane%32 of the fragment.
    const int64_t lstride = p.out_layer_stride * layer;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int64_t col = n0 + wn * WTN + j * 32 + (lane & 31);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int64_t row = m0 + wm * WTM + i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
          if (row < p.M && col < p.N) {
            if (OUT_BF16) {
              const __bf16 h = (__bf16)acc[i][j][e];
              reinterpret_cast<__bf16*>(p.out)[lstride + row * p.ldo + col] = h;
            } else {
              reinterpret_cast<float*>(p.out)[lstride + row * p.ldo + col] = acc[i][j][e];
            }
          }
        }
      }
    }
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
