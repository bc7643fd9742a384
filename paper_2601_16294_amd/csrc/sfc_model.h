// Analytical choice of the block shape and of the number of K layers
// (Section III.B's fine-grained roofline, Eq. 1-4, used as in Section III.C,
// option 2: evaluate every decomposition and keep the fastest).
//
// The paper's model, per core: the critical path is the sum of the BRGEMM
// times on it, each max(G*gamma, beta*(S_A + S_B)) for the panels that come
// from slow memory (Eq. 1; Eq. 2-4 drop the panels already in fast memory),
// plus the reads and writes of C and, with several layers, of the C copies.
// On the GPU a "core" is a CU running `occ` persistent workgroups; one BRGEMM
// is one 64-deep block of one task; fast memory is the L2 of an XCD, which the
// workgroups of that XCD share, and slow memory is HBM.  With the interleaved
// schedule the tasks in flight on one XCD form a compact patch of the curve,
// about sqrt(P) x sqrt(P) blocks for P tasks, so per block a workgroup brings
// (S_A + S_B) / sqrt(P) bytes from HBM (each panel is fetched once per patch).
// Every candidate is evaluated with the same constants; the smallest time wins.
#pragma once
#include <cstdint>

namespace sfc {

// Calibration on MI355X (fast path, bf16 in, fp32 accumulate).
struct ModelConst {
  double flops_per_clk_cu = 4096.0 * 0.74;   // dense bf16 MFMA peak x achieved fraction (256x256)
  double rate[4] = {0.60, 0.80, 0.86, 1.0};  // per shape, relative to 256x256 (index: kT* order)
  double hbm_bytes_per_clk = 3500.0;         // whole chip, at the loaded shader clock
  double launch_clk = 10000.0;               // per kernel launch (about 5 us)
  int xcds = 8;
};

constexpr int kModelMaxLayers = 16;          // the candidates are c = 1, 2, 4, 8, 16

struct ModelChoice {
  int tile;          // kT* index
  int layers;        // effective layer count
  double clk;        // estimated time in shader clocks
};

// Best (tile, layers) for C[M x N] = A[M x K] B[K x N].  occ[t] = workgroups
// per CU of shape t (kT* index).  tile_fixed = -1 and layers_fixed = 0 leave
// the choice free; otherwise only the fixed value is evaluated.
ModelChoice model_choose(int64_t M, int64_t N, int64_t K, int out_bytes, int num_cus,
                         const int occ[4], int tile_fixed, int layers_fixed,
                         const ModelConst& k = ModelConst());

}  // namespace sfc
