// Analytical choice of the block shape and the layer count (see sfc_model.h).
#include "sfc_model.h"

#include <cmath>

#include "sfc_params.h"

namespace sfc {

namespace {

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Estimated shader clocks of one candidate.  pad = output elements computed,
// ragged edges included (the first tie-breaker).
double candidate_clk(int64_t M, int64_t N, int64_t nk, int out_bytes, int num_cus, int occ, int t, int c,
                     const ModelConst& k, double* pad) {
  const int64_t bm = tile_bm(t), bn = tile_bn(t);
  const int64_t tasks = cdiv(M, bm) * cdiv(N, bn) * c;
  const int64_t slots = (int64_t)num_cus * occ;
  const int64_t rounds = cdiv(tasks, slots);
  const int64_t nb = cdiv(nk, c);                       // blocks of the longest layer
  const int64_t active = tasks < slots ? tasks : slots;  // workgroups streaming at once
  // one BRGEMM (64-deep block): G flops, panels S_A + S_B bytes
  const double g = 2.0 * (double)bm * (double)bn * 64.0;
  const double s_ab = 2.0 * 64.0 * (double)(bm + bn);
  // gamma: a workgroup gets 1/w of its CU's MFMA rate, w the workgroups that
  // share the CU: the dispatcher spreads a grid over the CUs before it puts a
  // second workgroup on one (and a grid of at most one 128x128 block per CU
  // runs the one-per-CU kernel)
  int64_t w = cdiv(active, num_cus);
  if (w > occ) w = occ;
  if (w < 1) w = 1;
  const double t_compute = g * (double)w / (k.flops_per_clk_cu * k.rate[t]);
  // beta: HBM shared by the active workgroups; each panel read once per XCD patch
  double patch = (double)active / (double)k.xcds;
  if (patch < 1.0) patch = 1.0;
  const double t_memory = s_ab / std::sqrt(patch) * (double)active / k.hbm_bytes_per_clk;
  const double t_block = t_compute > t_memory ? t_compute : t_memory;   // Eq. 1
  // C written once; with layers, the copies written and read back, then C
  const double mn = (double)M * (double)N;
  const double c_bytes = c == 1 ? mn * out_bytes : 2.0 * c * mn * 4.0 + mn * out_bytes;
  *pad = (double)tasks * (double)(bm * bn);
  return k.launch_clk * (c == 1 ? 1.0 : 2.0) + (double)rounds * (double)nb * t_block +
         c_bytes / k.hbm_bytes_per_clk;
}

}  // namespace

ModelChoice model_choose(int64_t M, int64_t N, int64_t K, int out_bytes, int num_cus, const int occ[4],
                         int tile_fixed, int layers_fixed, const ModelConst& k) {
  static const int order[4] = {kT256x256, kT128x256, kT256x128, kT128x128};
  const int64_t nk = K > 0 ? cdiv(K, 64) : 0;
  ModelChoice best{kT256x256, 1, 1e300};
  double best_pad = 1e300;
  for (int i = 0; i < 4; ++i) {
    const int t = order[i];
    if (tile_fixed >= 0 && t != tile_fixed) continue;
    int last_c = 0;
    for (int c0 = 1; c0 <= kModelMaxLayers; c0 *= 2) {
      if (layers_fixed > 0 && c0 != 1) break;
      int c = layers_fixed > 0 ? layers_fixed : c0;
      if (c > nk) c = nk > 0 ? (int)nk : 1;               // effective layer count
      if (c == last_c) continue;
      last_c = c;
      double pad = 0.0;
      const double clk = candidate_clk(M, N, nk, out_bytes, num_cus, occ[t] < 1 ? 1 : occ[t], t, c, k, &pad);
      // relative tolerance: candidates this close are ties, settled by the
      // padded work, then by the order of evaluation (shape order above, then
      // ascending layer counts)
      const double tol = 1e-9 * best.clk;
      const bool take = clk < best.clk - tol || (clk <= best.clk + tol && pad < best_pad);
      if (take) {
        best = ModelChoice{t, c, clk};
        best_pad = pad;
      }
    }
  }
  return best;
}

}  // namespace sfc
