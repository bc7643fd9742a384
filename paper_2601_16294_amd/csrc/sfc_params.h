// Internal interface between the C-ABI layer and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sfc {

constexpr int kBK = 64;          // depth of one K block (the paper's bk)

enum TileId { kT128x128 = 0, kT256x128 = 1, kT128x256 = 2, kT256x256 = 3, kNumTiles = 4 };

inline int tile_bm(int t) { return (t == kT256x128 || t == kT256x256) ? 256 : 128; }
inline int tile_bn(int t) { return (t == kT128x256 || t == kT256x256) ? 256 : 128; }

struct GemmParams {
  int64_t M, N, K;
  const uint16_t* A;
  int64_t lda;
  const uint16_t* B;
  int64_t ldb;
  void* out;                 // C (layers == 1) or the fp32 workspace (layers > 1)
  int64_t ldo;               // leading dimension of `out`
  int64_t out_layer_stride;  // elements between layer copies of `out` (0 when layers == 1)
  const int32_t* table;      // gm*gn curve positions -> im*gn + in
  int gm, gn;
  int layers;                // c_eff
  int nk;                    // ceil(K / kBK)
  int64_t tasks;             // gm * gn * layers
  int sched;                 // SFC_SCHED_*
  // Fused reduction (layers > 1 and counters != nullptr): the workgroup that
  // finishes a block's last layer copy sums the copies into C itself.
  int c_bf16;                // C holds bf16 (else fp32)
  int32_t* counters;         // per block (im*gn + in): layer copies finished; zero between launches
  void* C;                   // the final output
  int64_t ldc;
};

// Curve table of a gm x gn grid into dev_out (gm*gn int32), order = SFC_ORDER_*.
hipError_t launch_sfc_order(int gm, int gn, int order, int32_t* dev_out, hipStream_t stream);

// Persistent GEMM.  out_bf16 selects the epilogue; vec selects 128-bit loads
// (needs 16-byte aligned A and B, lda, ldb, K and N multiples of 8).
// f8 = 0: bf16 operands; f8 = 1 + a + 2b: A and B hold OCP fp8 bytes of format a
// and b (0 E4M3, 1 E5M2; lda, ldb in elements = bytes); 256x256 only.
// deep = true: 128x128 blocks on the fast path with a 4-deep ring (one
// workgroup per CU), for grids of at most one block per CU.
hipError_t launch_gemm(int tile, bool out_bf16, bool vec, const GemmParams& p, int grid,
                       hipStream_t stream, int f8 = 0, bool deep = false);
// Workgroups of the given kernel variant that fit on one CU.
hipError_t gemm_occupancy(int tile, bool out_bf16, bool vec, int* blocks_per_cu, int f8 = 0, bool deep = false);

// p[0 .. n) = v (a fill kernel: usable where a memset node is not wanted).
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t stream);

// C[i][j] = sum_l W[l][i][j] (ascending l, fp32), W dense M x N per layer.
hipError_t launch_reduce(const float* W, int layers, int64_t M, int64_t N, void* C, int64_t ldc,
                         bool out_bf16, hipStream_t stream);

// Register-only MFMA probe (256 workgroups x 4 waves); dev_out holds
// 256*256 + 256 floats (the last 256: shader clock per workgroup in MHz).
hipError_t run_mfma_probe(int random_operands, int iters, float* dev_out, double* ms);

}  // namespace sfc
