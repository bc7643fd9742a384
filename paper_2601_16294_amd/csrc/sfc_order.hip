// Generalized Hilbert order of an arbitrary gm x gn block grid, computed on the
// device one curve position per thread (Section II.B; the map of Listing 1).
//
// The curve is defined recursively on a rectangle given by a start cell, a
// major vector (the direction the walk advances) and a minor vector:
//   * a strip one cell thick is walked straight;
//   * when 2*major > 3*minor the rectangle is cut across the major axis into
//     two parts walked in turn with the same orientation;
//   * otherwise it is cut into three parts: the near half of the minor side
//     with the axes exchanged, the far half of the minor side, and the rest
//     walked back towards the far corner;
//   * halves are taken rounding toward minus infinity and an odd half of a
//     side longer than 2 is grown by one cell.
// Instead of enumerating the whole curve, each thread descends the recursion
// for its own position: at every level it counts the cells of the parts, picks
// the part that holds its position, and rebases.  The depth is O(log(gm+gn)).
#include "sfc_params.h"

namespace sfc {

__host__ __device__ __forceinline__ int sgn(int v) { return (v > 0) - (v < 0); }
__host__ __device__ __forceinline__ int iabs(int v) { return v < 0 ? -v : v; }

// Cell (x, y) = (im, in) at curve position s of the gm x gn grid.
__host__ __device__ void curve_cell(int gm, int gn, int s, int* out_x, int* out_y) {
  int x = 0, y = 0;
  int ax, ay, bx, by;                    // major and minor vectors
  if (gm >= gn) { ax = gm; ay = 0; bx = 0; by = gn; }
  else          { ax = 0; ay = gn; bx = gm; by = 0; }
  for (;;) {
    const int w = iabs(ax + ay), h = iabs(bx + by);
    const int dax = sgn(ax), day = sgn(ay), dbx = sgn(bx), dby = sgn(by);
    if (h == 1) { x += s * dax; y += s * day; break; }
    if (w == 1) { x += s * dbx; y += s * dby; break; }
    // Arithmetic right shift halves rounding toward minus infinity.
    int hax = ax >> 1, hay = ay >> 1, hbx = bx >> 1, hby = by >> 1;
    int hw = iabs(hax + hay), hh = iabs(hbx + hby);
    if (2 * w > 3 * h) {
      if ((hw & 1) && w > 2) { hax += dax; hay += day; hw += 1; }
      const int first = hw * h;
      if (s < first) { ax = hax; ay = hay; }
      else { s -= first; x += hax; y += hay; ax -= hax; ay -= hay; }
    } else {
      if ((hh & 1) && h > 2) { hbx += dbx; hby += dby; hh += 1; }
      const int first = hh * hw;          // major = half minor side, minor = half major side
      const int second = w * (h - hh);
      if (s < first) {
        const int nax = hbx, nay = hby;
        bx = hax; by = hay; ax = nax; ay = nay;
      } else if (s < first + second) {
        s -= first; x += hbx; y += hby; bx -= hbx; by -= hby;
      } else {
        s -= first + second;
        const int nx = x + (ax - dax) + (hbx - dbx), ny = y + (ay - day) + (hby - dby);
        const int nbx = -(ax - hax), nby = -(ay - hay);
        x = nx; y = ny; ax = -hbx; ay = -hby; bx = nbx; by = nby;
      }
    }
  }
  *out_x = x;
  *out_y = y;
}

__global__ void sfc_order_kernel(int gm, int gn, int order, int32_t* out) {
  const int64_t total = (int64_t)gm * gn;
  for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < total;
       s += (int64_t)gridDim.x * blockDim.x) {
    if (order == 1) { out[s] = (int32_t)s; continue; }
    int x, y;
    curve_cell(gm, gn, (int)s, &x, &y);
    out[s] = x * gn + y;
  }
}

hipError_t launch_sfc_order(int gm, int gn, int order, int32_t* dev_out, hipStream_t stream) {
  const int64_t total = (int64_t)gm * gn;
  int blocks = (int)((total + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(sfc_order_kernel, dim3(blocks), dim3(256), 0, stream, gm, gn, order, dev_out);
  return hipGetLastError();
}

}  // namespace sfc
