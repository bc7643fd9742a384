// Argument checks of the C ABI, kept free of any HIP dependency so that they
// run (and are tested) without a GPU.  Every check happens before the library
// touches the device.
#pragma once
#include <stdint.h>
#include <stdio.h>

#include "sfcgemm.h"

namespace sfc {

constexpr int kMaxLayers = 64;
constexpr int kAutoLayers = 16;                  // largest layer count SFC_CA_AUTO picks
constexpr int64_t kMaxDim = (int64_t)1 << 31;   // block indices are int32

struct Checked {
  int code;
  char msg[160];
};

inline Checked ok() { Checked c; c.code = SFC_OK; c.msg[0] = 0; return c; }
inline Checked fail(int code, const char* what) {
  Checked c;
  c.code = code;
  snprintf(c.msg, sizeof c.msg, "%s", what);
  return c;
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Layers actually used: min(c, number of 64-deep K blocks), at least 1.
inline int effective_layers(int64_t K, int c, int bk) {
  const int64_t nk = K > 0 ? ceil_div(K, bk) : 0;
  int64_t e = c < nk ? c : nk;
  return e < 1 ? 1 : (int)e;
}

inline Checked check_order_args(int gm, int gn, int order, const void* out) {
  if (gm <= 0 || gn <= 0) return fail(SFC_ERR_INVALID_ARG, "grid sides must be >= 1");
  if (order != SFC_ORDER_HILBERT && order != SFC_ORDER_ROW_MAJOR)
    return fail(SFC_ERR_INVALID_ARG, "unknown order");
  if (!out) return fail(SFC_ERR_INVALID_ARG, "out_idx is NULL");
  if ((int64_t)gm * gn >= kMaxDim) return fail(SFC_ERR_UNSUPPORTED, "gm*gn must be < 2^31");
  return ok();
}

inline Checked check_gemm_args(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                               const void* B, int64_t ldb, const void* C, int64_t ldc,
                               int out_type, int ca_layers, int tile, int order, int sched,
                               const void* ws, size_t ws_bytes) {
  if (M < 0 || N < 0 || K < 0) return fail(SFC_ERR_INVALID_ARG, "M, N, K must be >= 0");
  if (out_type != SFC_OUT_F32 && out_type != SFC_OUT_BF16)
    return fail(SFC_ERR_INVALID_ARG, "unknown out_type");
  if (ca_layers < 0 || ca_layers > kMaxLayers)
    return fail(SFC_ERR_INVALID_ARG, "ca_layers must be 0 (chosen by the model) or in [1, 64]");
  if (tile < SFC_TILE_AUTO || tile > SFC_TILE_256x256) return fail(SFC_ERR_INVALID_ARG, "unknown tile");
  if (order != SFC_ORDER_HILBERT && order != SFC_ORDER_ROW_MAJOR)
    return fail(SFC_ERR_INVALID_ARG, "unknown order");
  if (sched != SFC_SCHED_INTERLEAVED && sched != SFC_SCHED_BLOCK && sched != SFC_SCHED_INTERLEAVED_PLAIN)
    return fail(SFC_ERR_INVALID_ARG, "unknown sched");
  if (M == 0 || N == 0) return ok();   // nothing to write
  if (!C) return fail(SFC_ERR_INVALID_ARG, "C is NULL");
  if (ldc < N) return fail(SFC_ERR_INVALID_ARG, "ldc < N");
  if (K > 0) {
    if (!A) return fail(SFC_ERR_INVALID_ARG, "A is NULL");
    if (!B) return fail(SFC_ERR_INVALID_ARG, "B is NULL");
    if (lda < K) return fail(SFC_ERR_INVALID_ARG, "lda < K");
    if (ldb < N) return fail(SFC_ERR_INVALID_ARG, "ldb < N");
    if (((uintptr_t)A & 1) || ((uintptr_t)B & 1))
      return fail(SFC_ERR_UNSUPPORTED, "A and B must be 2-byte aligned");
  }
  const uintptr_t calign = out_type == SFC_OUT_F32 ? 4 : 2;
  if ((uintptr_t)C % calign) return fail(SFC_ERR_UNSUPPORTED, "C is not aligned to its element size");
  if (M >= kMaxDim || N >= kMaxDim || K >= kMaxDim)
    return fail(SFC_ERR_UNSUPPORTED, "M, N and K must be < 2^31");
  // the smallest block is 128 x 128
  if (ceil_div(M, 128) * ceil_div(N, 128) >= kMaxDim)
    return fail(SFC_ERR_UNSUPPORTED, "too many output blocks");
  // the model chooses at most kAutoLayers layers: check the largest case
  const int ce = effective_layers(K, ca_layers == 0 ? kAutoLayers : ca_layers, 64);
  // task indices (blocks x layers) are 32-bit in the kernel
  if (ceil_div(M, 128) * ceil_div(N, 128) * ce >= kMaxDim)
    return fail(SFC_ERR_UNSUPPORTED, "too many output blocks x layers");
  if (ce > 1 && ws) {
    const uint64_t need = (uint64_t)ce * (uint64_t)M * (uint64_t)N * 4u;
    if (ws_bytes < need) return fail(SFC_ERR_WORKSPACE, "workspace smaller than sfc_gemm_ws_size()");
    if ((uintptr_t)ws % 16) return fail(SFC_ERR_UNSUPPORTED, "workspace must be 16-byte aligned");
  }
  return ok();
}

inline size_t ws_size(int64_t M, int64_t N, int64_t K, int ca_layers) {
  if (M < 0 || N < 0 || K < 0 || ca_layers < 0 || ca_layers > kMaxLayers) return 0;
  const int ce = effective_layers(K, ca_layers == 0 ? kAutoLayers : ca_layers, 64);
  if (ce <= 1) return 0;
  return (size_t)ce * (size_t)M * (size_t)N * 4u;
}

// Block columns that a half-height strip takes over (0: none).  A grid of
// gm x gn blocks on `slots` resident workgroups leaves r = gm*gn mod slots
// blocks in its last round; when 0 < r <= slots/2 the last w = ceil(r/gm)
// block columns go to blocks of half the height, `half_rows` rows of them,
// provided those fit in one round of `half_slots` workgroups and w < gn.
inline int strip_columns(int gm, int gn, int64_t slots, int64_t half_rows, int64_t half_slots) {
  if (gm <= 0 || gn <= 0 || slots <= 0) return 0;
  const int64_t T = (int64_t)gm * gn;
  const int64_t r = T % slots;
  if (T <= slots || r == 0 || 2 * r > slots) return 0;
  const int64_t w = ceil_div(r, gm);
  if (w >= gn || half_rows * w > half_slots) return 0;
  return (int)w;
}

// Whether a launch takes the 4-deep ring of 128x128 blocks: the fast path,
// bf16 operands, 128x128 blocks and no more tasks (blocks x layers) than CUs,
// so that one workgroup per CU (instead of two) loses nothing.
inline bool deep_ring(int tile_128x128, bool vec, int f8, int64_t tasks, int64_t num_cus) {
  return tile_128x128 && vec && f8 == 0 && tasks > 0 && tasks <= num_cus;
}

// 16-byte loads are legal when every row starts 16-byte aligned and the K and
// N extents end on whole 8-element chunks.
inline bool vector_loads_ok(const void* A, int64_t lda, const void* B, int64_t ldb, int64_t K,
                            int64_t N) {
  // Per-lane byte offsets within a block are 32-bit: 256 rows of A, 64 of B.
  return ((uintptr_t)A % 16 == 0) && ((uintptr_t)B % 16 == 0) && (lda % 8 == 0) &&
         (ldb % 8 == 0) && (K % 8 == 0) && (N % 8 == 0) && lda < ((int64_t)1 << 20) &&
         ldb < ((int64_t)1 << 22);
}

// fp8 (OCP E4M3) operands take the 16-byte load path only: 16-byte aligned
// rows, and K and N ending on whole 16-element chunks.
inline bool f8_loads_ok(const void* A, int64_t lda, const void* B, int64_t ldb, int64_t K, int64_t N) {
  return ((uintptr_t)A % 16 == 0) && ((uintptr_t)B % 16 == 0) && (lda % 16 == 0) && (ldb % 16 == 0) &&
         (K % 16 == 0) && (N % 16 == 0) && lda < ((int64_t)1 << 21) && ldb < ((int64_t)1 << 23);
}

inline Checked check_gemm_f8_args(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                                  const void* B, int64_t ldb, const void* C, int64_t ldc,
                                  int out_type, int ca_layers, int tile, int order, int sched,
                                  const void* ws, size_t ws_bytes) {
  Checked c = check_gemm_args(M, N, K, A, lda, B, ldb, C, ldc, out_type, ca_layers, tile, order, sched, ws,
                              ws_bytes);
  if (c.code != SFC_OK || M == 0 || N == 0) return c;
  if (tile != SFC_TILE_AUTO && tile != SFC_TILE_256x256 && tile != SFC_TILE_128x256)
    return fail(SFC_ERR_UNSUPPORTED, "fp8 operands run on 256x256 or 128x256 blocks");
  if (K > 0 && !f8_loads_ok(A, lda, B, ldb, K, N))
    return fail(SFC_ERR_UNSUPPORTED,
                "fp8 operands need 16-byte aligned A and B and lda, ldb, K, N multiples of 16");
  return ok();
}

}  // namespace sfc
