// C ABI of the SFC-CA GEMM (declarations and contracts in include/sfcgemm.h).
//
// Host-side duties: argument checks (before any HIP call), choice of the block
// shape, the per-device cache of curve tables (built once per grid on the
// device and kept), the per-stream internal workspace for layer copies and
// arrival counters, and the launches.  Nothing here computes any part of the
// product.  No entry point synchronises the device or a stream: new curve
// tables and workspaces are made stream-ordered (events, hipMallocAsync /
// hipFreeAsync).
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>
#include <string>
#include <tuple>

#include "sfc_model.h"
#include "sfc_params.h"
#include "sfc_validate.h"
#include "sfcgemm.h"

namespace {

thread_local std::string g_last_error;

// A curve table on the device, written by a kernel on the stream of the call
// that first needed it; `ready` marks its completion for calls on other streams.
struct Table {
  int32_t* d = nullptr;
  hipEvent_t ready = nullptr;
  bool done = false;        // `ready` has been seen complete
};

// Library-owned memory of one stream: the layer copies of calls that pass no
// workspace, and the arrival counters of fused reductions (kept zero between
// launches).  Only work on that stream touches it, so calls on different
// streams never share it; it grows stream-ordered.
struct StreamMem {
  void* ws = nullptr;
  size_t ws_bytes = 0;
  int32_t* counters = nullptr;
  int64_t n_counters = 0;
};

struct DeviceState {
  std::map<std::tuple<int, int, int>, Table> tables;   // (gm, gn, order) -> device table
  std::map<hipStream_t, StreamMem> streams;
  char* scratch = nullptr;   // this device's copy of `scratch` (see sfc_gemm_noalloc_ex)
  int num_cus = 0;
  int occupancy[sfc::kNumTiles][2][2][2] = {};               // [tile][bf16 out][vec][fp8 in], 0 = unknown
  int occupancy_deep[2] = {};                                  // 4-deep 128x128 ring, [bf16 out]
};

std::mutex g_mu;
std::map<int, DeviceState> g_devices;

int set_error(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return set_error(SFC_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

// Must be called with g_mu held.
int device_state(DeviceState** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  DeviceState& st = g_devices[dev];
  if (st.num_cus == 0) {
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    st.num_cus = cus;
  }
  *out = &st;
  return SFC_OK;
}

// Curve table of a gm x gn grid on the current device.  The first call for a
// grid allocates it and enqueues the generator on `stream` (no wait); a later
// call on another stream waits for that kernel on the device, until the table
// is known to be complete.  Must be called with g_mu held.
int get_table(DeviceState& st, int gm, int gn, int order, hipStream_t stream, const int32_t** out) {
  auto key = std::make_tuple(gm, gn, order);
  auto it = st.tables.find(key);
  if (it != st.tables.end()) {
    Table& t = it->second;
    if (!t.done) {
      hipError_t e = hipEventQuery(t.ready);
      if (e == hipSuccess) {
        t.done = true;
      } else if (e == hipErrorNotReady) {
        (void)hipGetLastError();   // not an error: do not leave it for the next check
        e = hipStreamWaitEvent(stream, t.ready, 0);
        if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent(curve table)");
      } else {
        return hip_fail(e, "hipEventQuery(curve table)");
      }
    }
    *out = t.d;
    return SFC_OK;
  }
  Table t;
  hipError_t e = hipMalloc(&t.d, sizeof(int32_t) * (size_t)gm * (size_t)gn);
  if (e != hipSuccess) return hip_fail(e, "hipMalloc(curve table)");
  e = sfc::launch_sfc_order(gm, gn, order, t.d, stream);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&t.ready, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventRecord(t.ready, stream);
  if (e != hipSuccess) {
    // the generator may be queued: the table is kept (never used) rather than freed under it
    return hip_fail(e, "curve table");
  }
  st.tables[key] = t;
  *out = t.d;
  return SFC_OK;
}

// At least `bytes` of layer workspace owned by `stream`.  A smaller buffer is
// released stream-ordered (after the work already queued on the stream that
// uses it) and a larger one allocated in stream order.  Must be called with
// g_mu held.
int stream_workspace(DeviceState& st, hipStream_t stream, size_t bytes, void** out) {
  StreamMem& m = st.streams[stream];
  if (m.ws_bytes < bytes) {
    if (m.ws) {
      hipError_t e = hipFreeAsync(m.ws, stream);
      m.ws = nullptr;
      m.ws_bytes = 0;
      if (e != hipSuccess) return hip_fail(e, "hipFreeAsync(workspace)");
    }
    hipError_t e = hipMallocAsync(&m.ws, bytes, stream);
    if (e != hipSuccess) {
      m.ws = nullptr;
      return hip_fail(e, "hipMallocAsync(workspace)");
    }
    m.ws_bytes = bytes;
  }
  *out = m.ws;
  return SFC_OK;
}

// At least n arrival counters owned by `stream`, all zero when the next
// launch on the stream starts (new ones are cleared by a fill kernel; the
// fused reduction leaves every counter it used at zero).  Must be called with
// g_mu held.
int stream_counters(DeviceState& st, hipStream_t stream, int64_t n, int32_t** out) {
  StreamMem& m = st.streams[stream];
  if (m.n_counters < n) {
    if (m.counters) {
      hipError_t e = hipFreeAsync(m.counters, stream);
      m.counters = nullptr;
      m.n_counters = 0;
      if (e != hipSuccess) return hip_fail(e, "hipFreeAsync(counters)");
    }
    const int64_t cap = n < 4096 ? 4096 : n;
    hipError_t e = hipMallocAsync(reinterpret_cast<void**>(&m.counters), (size_t)cap * 4u, stream);
    if (e != hipSuccess) {
      m.counters = nullptr;
      return hip_fail(e, "hipMallocAsync(counters)");
    }
    e = sfc::launch_fill_i32(m.counters, cap, 0, stream);
    if (e != hipSuccess) return hip_fail(e, "counter fill");
    m.n_counters = cap;
  }
  *out = m.counters;
  return SFC_OK;
}

int get_occupancy(DeviceState& st, int tile, bool ob, bool vec, int* occ, int f8 = 0, bool deep = false) {
  int& o = deep ? st.occupancy_deep[ob] : st.occupancy[tile][ob][vec][f8 != 0];
  if (o == 0) {
    int v = 0;
    hipError_t e = sfc::gemm_occupancy(tile, ob, vec, &v, f8, deep);
    if (e != hipSuccess) return hip_fail(e, "occupancy query");
    o = v < 1 ? 1 : v;
  }
  *occ = o;
  return SFC_OK;
}

int tile_from_api(int t) {
  switch (t) {
    case SFC_TILE_128x128: return sfc::kT128x128;
    case SFC_TILE_256x128: return sfc::kT256x128;
    case SFC_TILE_128x256: return sfc::kT128x256;
    case SFC_TILE_256x256: return sfc::kT256x256;
    default: return -1;
  }
}

struct Plan {
  int tile, bm, bn, gm, gn, ce, nk, grid, occ;
  bool vec;
  bool deep = false;   // 128x128 blocks with the 4-deep ring (one workgroup per CU)
};

int make_plan(DeviceState& st, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
              const void* B, int64_t ldb, bool ob, int ca_layers, int tile_api, Plan* pl, int f8 = 0) {
  int rc = SFC_OK;
  if (f8) {
    // fp8 operands (checked by check_gemm_f8_args): 256x256 or 128x256 blocks,
    // 128-deep K blocks.  A 128-deep fp8 block moves the bytes of a 64-deep
    // bf16 block and takes the same MFMA time, so the free knobs are chosen by
    // the model for the bf16 problem with the same number of blocks, over the
    // two fp8 block shapes (256x256 first: it keeps a tie).
    pl->vec = true;
    int occ[sfc::kNumTiles];
    for (int t = 0; t < sfc::kNumTiles; ++t) occ[t] = 1;
    static const int kF8Tiles[2] = {sfc::kT256x256, sfc::kT128x256};
    for (int t : kF8Tiles) {
      rc = get_occupancy(st, t, ob, true, &occ[t], f8);
      if (rc != SFC_OK) return rc;
    }
    int tile = tile_api == SFC_TILE_AUTO ? -1 : tile_from_api(tile_api);
    int layers = ca_layers;
    if (tile < 0 || ca_layers == SFC_CA_AUTO) {
      const int64_t k_equiv = (K > 0 ? sfc::ceil_div(K, 128) : 0) * sfc::kBK;
      sfc::ModelChoice best{-1, 1, 0.0};
      for (int t : kF8Tiles) {
        if (tile >= 0 && t != tile) continue;
        const sfc::ModelChoice ch = sfc::model_choose(M, N, k_equiv, ob ? 2 : 4, st.num_cus, occ, t, ca_layers);
        if (best.tile < 0 || ch.clk < best.clk) best = ch;
      }
      tile = best.tile;
      layers = best.layers;
    }
    pl->tile = tile;
    pl->ce = sfc::effective_layers(K, layers, 128);
    pl->bm = sfc::tile_bm(tile);
    pl->bn = sfc::tile_bn(tile);
    pl->gm = (int)sfc::ceil_div(M, pl->bm);
    pl->gn = (int)sfc::ceil_div(N, pl->bn);
    pl->nk = (int)(K > 0 ? sfc::ceil_div(K, 128) : 0);
    rc = get_occupancy(st, pl->tile, ob && pl->ce == 1, true, &pl->occ, f8);
    if (rc != SFC_OK) return rc;
    const int64_t tasks = (int64_t)pl->gm * pl->gn * pl->ce;
    const int64_t slots = (int64_t)st.num_cus * pl->occ;
    pl->grid = (int)(tasks < slots ? tasks : slots);
    return SFC_OK;
  }
  // the fast path needs at least one K block per task
  pl->vec = K > 0 && sfc::vector_loads_ok(A, lda, B, ldb, K, N);
  if (tile_api == SFC_TILE_AUTO || ca_layers == SFC_CA_AUTO) {
    // the analytical model evaluates the free knobs (block shape, layers)
    int occ[sfc::kNumTiles];
    for (int t = 0; t < sfc::kNumTiles; ++t) {
      rc = get_occupancy(st, t, ob && ca_layers == 1, pl->vec, &occ[t]);
      if (rc != SFC_OK) return rc;
    }
    const sfc::ModelChoice ch =
        sfc::model_choose(M, N, K, ob ? 2 : 4, st.num_cus, occ,
                          tile_api == SFC_TILE_AUTO ? -1 : tile_from_api(tile_api), ca_layers);
    pl->tile = ch.tile;
    pl->ce = sfc::effective_layers(K, ch.layers, sfc::kBK);
  } else {
    pl->tile = tile_from_api(tile_api);
    pl->ce = sfc::effective_layers(K, ca_layers, sfc::kBK);
  }
  pl->bm = sfc::tile_bm(pl->tile);
  pl->bn = sfc::tile_bn(pl->tile);
  pl->gm = (int)sfc::ceil_div(M, pl->bm);
  pl->gn = (int)sfc::ceil_div(N, pl->bn);
  pl->nk = (int)(K > 0 ? sfc::ceil_div(K, sfc::kBK) : 0);
  // layer copies are fp32 whatever the output type
  const bool kernel_bf16 = ob && pl->ce == 1;
  const int64_t tasks = (int64_t)pl->gm * pl->gn * pl->ce;
  // a grid of at most one 128x128 block per CU runs the deep-ring kernel
  pl->deep = sfc::deep_ring(pl->tile == sfc::kT128x128, pl->vec, 0, tasks, st.num_cus);
  rc = get_occupancy(st, pl->tile, kernel_bf16, pl->vec, &pl->occ, 0, pl->deep);
  if (rc != SFC_OK) return rc;
  int64_t slots = (int64_t)st.num_cus * pl->occ;
  pl->grid = (int)(tasks < slots ? tasks : slots);
  return SFC_OK;
}

// Wave quantisation of the last round.  With T = gm*gn blocks and S resident
// workgroups the last of ceil(T/S) rounds holds r = T mod S blocks.  When r <= S/2
// and a kernel with half-height blocks of the same width exists, the last
// w = ceil(r/gm) block columns go to a second launch with half-height blocks: their
// 2*gm*w <= S blocks form one round that takes about half as long, and the first
// launch keeps at most floor(T/S) full rounds.  Every element is still one full
// ascending K pass of the same MFMA sequence, so no result bit changes.
struct Split {
  bool on = false;
  int w = 0;      // block columns moved to the strip
  Plan strip;     // the strip's plan (half-height blocks)
};

int plan_tail_split(DeviceState& st, const Plan& pl, int64_t M, int64_t N, int64_t K, const void* A,
                    int64_t lda, const void* B, int64_t ldb, bool ob, Split* sp) {
  sp->on = false;
  if (pl.ce != 1 || !pl.vec) return SFC_OK;
  int half;
  if (pl.tile == sfc::kT256x256) half = sfc::kT128x256;
  else if (pl.tile == sfc::kT256x128) half = sfc::kT128x128;
  else return SFC_OK;
  int occ2 = 1;
  int rc = get_occupancy(st, half, ob, true, &occ2);
  if (rc != SFC_OK) return rc;
  const int64_t half_rows = sfc::ceil_div(M, sfc::tile_bm(half));
  const int w = sfc::strip_columns(pl.gm, pl.gn, (int64_t)st.num_cus * pl.occ, half_rows,
                                   (int64_t)st.num_cus * occ2);
  if (w == 0) return SFC_OK;
  Plan& q = sp->strip;
  q.tile = half;
  q.bm = sfc::tile_bm(half);
  q.bn = sfc::tile_bn(half);
  const int64_t n1 = (int64_t)(pl.gn - w) * pl.bn;
  q.gm = (int)half_rows;
  q.gn = (int)sfc::ceil_div(N - n1, q.bn);
  q.ce = 1;
  q.nk = pl.nk;
  q.occ = occ2;
  q.vec = sfc::vector_loads_ok(A, lda, static_cast<const uint16_t*>(B) + n1, ldb, K, N - n1);
  if (!q.vec) return SFC_OK;
  q.grid = (int)((int64_t)q.gm * q.gn);
  sp->w = w;
  sp->on = true;
  return SFC_OK;
}

// The fused reduction's part of a launch: C and the arrival counters (none:
// the layer copies are summed by the separate reduction kernel).
struct Fuse {
  int32_t* counters = nullptr;
  void* C = nullptr;
  int64_t ldc = 0;
  bool bf16 = false;
};

// One GEMM launch of plan pl into out (C, or the layer copies when pl.ce > 1),
// blocks taken in the order of `table`.  Must be called with g_mu held.
int launch_plan(const Plan& pl, const int32_t* table, int64_t M, int64_t N, int64_t K, const void* A,
                int64_t lda, const void* B, int64_t ldb, void* out, int64_t ldo, int64_t layer_stride,
                bool out_bf16, int sched, const Fuse& fu, hipStream_t stream, int f8) {
  sfc::GemmParams p;
  p.M = M; p.N = N; p.K = K;
  p.A = reinterpret_cast<const uint16_t*>(A); p.lda = lda;
  p.B = reinterpret_cast<const uint16_t*>(B); p.ldb = ldb;
  p.out = out; p.ldo = ldo; p.out_layer_stride = layer_stride;
  p.table = table;
  p.gm = pl.gm; p.gn = pl.gn;
  p.layers = pl.ce;
  p.nk = pl.nk;
  p.tasks = (int64_t)pl.gm * pl.gn * pl.ce;
  p.sched = sched;
  p.c_bf16 = fu.bf16 ? 1 : 0;
  p.counters = fu.counters;
  p.C = fu.C;
  p.ldc = fu.ldc;
  hipError_t e = sfc::launch_gemm(pl.tile, out_bf16, pl.vec, p, pl.grid, stream, f8, pl.deep);
  if (e != hipSuccess) return hip_fail(e, "GEMM launch");
  return SFC_OK;
}

// How the layer copies of a call with c_eff > 1 are summed.
enum Reduce { kReduceSeparate = 0, kReduceFused = 1 };

int gemm_impl(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B,
              int64_t ldb, void* C, int64_t ldc, int out_type, int ca_layers, int tile, int order,
              int sched, void* ws, size_t ws_bytes, void* stream_ptr, int f8 = 0, int reduce = kReduceSeparate) {
  const sfc::Checked chk =
      f8 ? sfc::check_gemm_f8_args(M, N, K, A, lda, B, ldb, C, ldc, out_type, ca_layers, tile, order, sched, ws,
                                   ws_bytes)
         : sfc::check_gemm_args(M, N, K, A, lda, B, ldb, C, ldc, out_type, ca_layers, tile, order, sched, ws,
                                ws_bytes);
  if (chk.code != SFC_OK) return set_error(chk.code, chk.msg);
  if (M == 0 || N == 0) return SFC_OK;
  hipStream_t stream = reinterpret_cast<hipStream_t>(stream_ptr);
  const bool ob = out_type == SFC_OUT_BF16;

  std::lock_guard<std::mutex> lock(g_mu);
  DeviceState* st = nullptr;
  int rc = device_state(&st);
  if (rc != SFC_OK) return rc;
  Plan pl;
  rc = make_plan(*st, M, N, K, A, lda, B, ldb, ob, ca_layers, tile, &pl, f8);
  if (rc != SFC_OK) return rc;

  // the block shape is the library's to choose: a half-height strip may take
  // a partial last round
  Split sp;
  if (tile == SFC_TILE_AUTO && !f8) {
    rc = plan_tail_split(*st, pl, M, N, K, A, lda, B, ldb, ob, &sp);
    if (rc != SFC_OK) return rc;
  }
  const Fuse none;
  if (sp.on) {
    Plan main = pl;
    main.gn -= sp.w;
    const int64_t tasks = (int64_t)main.gm * main.gn;
    const int64_t slots = (int64_t)st->num_cus * main.occ;
    main.grid = (int)(tasks < slots ? tasks : slots);
    const int64_t n1 = (int64_t)main.gn * main.bn;
    const int32_t *t_main = nullptr, *t_strip = nullptr;
    rc = get_table(*st, main.gm, main.gn, order, stream, &t_main);
    if (rc == SFC_OK) rc = get_table(*st, sp.strip.gm, sp.strip.gn, order, stream, &t_strip);
    if (rc != SFC_OK) return rc;
    rc = launch_plan(main, t_main, M, n1, K, A, lda, B, ldb, C, ldc, 0, ob, sched, none, stream, 0);
    if (rc != SFC_OK) return rc;
    const size_t esz = ob ? 2 : 4;
    return launch_plan(sp.strip, t_strip, M, N - n1, K, A, lda, static_cast<const uint16_t*>(B) + n1, ldb,
                       static_cast<char*>(C) + (size_t)n1 * esz, ldc, 0, ob, sched, none, stream, 0);
  }

  const int32_t* table = nullptr;
  rc = get_table(*st, pl.gm, pl.gn, order, stream, &table);
  if (rc != SFC_OK) return rc;
  if (pl.ce == 1) return launch_plan(pl, table, M, N, K, A, lda, B, ldb, C, ldc, 0, ob, sched, none, stream, f8);

  // layer copies: the caller's workspace, or this stream's own
  void* W = ws;
  if (!W) {
    rc = stream_workspace(*st, stream, (size_t)pl.ce * (size_t)M * (size_t)N * 4u, &W);
    if (rc != SFC_OK) return rc;
  }
  Fuse fu;
  if (reduce == kReduceFused) {
    rc = stream_counters(*st, stream, (int64_t)pl.gm * pl.gn, &fu.counters);
    if (rc != SFC_OK) return rc;
    fu.C = C;
    fu.ldc = ldc;
    fu.bf16 = ob;
  }
  rc = launch_plan(pl, table, M, N, K, A, lda, B, ldb, W, N, M * N, false, sched, fu, stream, f8);
  if (rc != SFC_OK || reduce == kReduceFused) return rc;
  hipError_t e = sfc::launch_reduce(static_cast<const float*>(W), pl.ce, M, N, C, ldc, ob, stream);
  if (e != hipSuccess) return hip_fail(e, "reduction launch");
  return SFC_OK;
}

// ---- the entry point that allocates nothing ---------------------------------------------
// sfc_gemm_noalloc_ex keeps everything it needs beyond the caller's buffers in
// this file-scope device array: the layer copies of a ca_layers > 1 call
// (kNoAllocWsBytes) and the curve tables of its launches (two of at most
// kNoAllocCells entries: the main grid and the half-height strip).  Each
// device holds its own copy until the process ends.  In host code `scratch`
// only names the array: its address on a device comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kNoAllocWsBytes = SFC_NOALLOC_WS_BYTES;
constexpr int64_t kNoAllocCells = SFC_NOALLOC_MAX_BLOCKS;
constexpr size_t kNoAllocTableOffset = kNoAllocWsBytes;
constexpr size_t kScratchBytes = kNoAllocWsBytes + 2 * (size_t)kNoAllocCells * 4;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// The current device's address of `scratch`.  Must be called with g_mu held.
int scratch_address(DeviceState& st, char** out) {
  if (!st.scratch) {
    void* ptr = nullptr;
    hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    st.scratch = static_cast<char*>(ptr);
  }
  *out = st.scratch;
  return SFC_OK;
}

int gemm_noalloc_impl(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B, int64_t ldb,
                      void* C, int64_t ldc, int out_type, int ca_layers, int tile, int order, int sched,
                      void* stream_ptr) {
  const sfc::Checked chk =
      sfc::check_gemm_args(M, N, K, A, lda, B, ldb, C, ldc, out_type, ca_layers, tile, order, sched, nullptr, 0);
  if (chk.code != SFC_OK) return set_error(chk.code, chk.msg);
  if (M == 0 || N == 0) return SFC_OK;
  // the layer copies must fit (for SFC_CA_AUTO: the largest count the model picks)
  const size_t need = sfc::ws_size(M, N, K, ca_layers);
  if (need > kNoAllocWsBytes)
    return set_error(SFC_ERR_WORKSPACE, "sfc_gemm_noalloc_ex: the layer copies need " + std::to_string(need) +
                                            " bytes; its workspace holds " + std::to_string(kNoAllocWsBytes));
  hipStream_t stream = reinterpret_cast<hipStream_t>(stream_ptr);
  const bool ob = out_type == SFC_OUT_BF16;

  std::lock_guard<std::mutex> lock(g_mu);
  DeviceState* st = nullptr;
  int rc = device_state(&st);
  if (rc != SFC_OK) return rc;
  char* base = nullptr;
  rc = scratch_address(*st, &base);
  if (rc != SFC_OK) return rc;
  int32_t* tables = reinterpret_cast<int32_t*>(base + kNoAllocTableOffset);
  float* W = reinterpret_cast<float*>(base);

  Plan pl;
  rc = make_plan(*st, M, N, K, A, lda, B, ldb, ob, ca_layers, tile, &pl);
  if (rc != SFC_OK) return rc;
  if (pl.ce > 1 && (size_t)pl.ce * (size_t)M * (size_t)N * 4u > kNoAllocWsBytes)
    return set_error(SFC_ERR_WORKSPACE, "sfc_gemm_noalloc_ex: the planned layer copies exceed its workspace");
  Split sp;
  if (tile == SFC_TILE_AUTO) {
    rc = plan_tail_split(*st, pl, M, N, K, A, lda, B, ldb, ob, &sp);
    if (rc != SFC_OK) return rc;
  }
  Plan main = pl;
  if (sp.on) {
    main.gn -= sp.w;
    const int64_t tasks = (int64_t)main.gm * main.gn;
    const int64_t slots = (int64_t)st->num_cus * main.occ;
    main.grid = (int)(tasks < slots ? tasks : slots);
  }
  if ((int64_t)main.gm * main.gn > kNoAllocCells || (sp.on && (int64_t)sp.strip.gm * sp.strip.gn > kNoAllocCells))
    return set_error(SFC_ERR_UNSUPPORTED, "sfc_gemm_noalloc_ex: more output blocks than its curve table holds (" +
                                              std::to_string(kNoAllocCells) + ")");
  // the curve tables are written on the stream for every call: the array
  // keeps only what the last call left there
  hipError_t e = sfc::launch_sfc_order(main.gm, main.gn, order, tables, stream);
  if (e != hipSuccess) return hip_fail(e, "curve table");
  const Fuse none;
  if (sp.on) {
    int32_t* t_strip = tables + kNoAllocCells;
    e = sfc::launch_sfc_order(sp.strip.gm, sp.strip.gn, order, t_strip, stream);
    if (e != hipSuccess) return hip_fail(e, "curve table");
    const int64_t n1 = (int64_t)main.gn * main.bn;
    rc = launch_plan(main, tables, M, n1, K, A, lda, B, ldb, C, ldc, 0, ob, sched, none, stream, 0);
    if (rc != SFC_OK) return rc;
    const size_t esz = ob ? 2 : 4;
    return launch_plan(sp.strip, t_strip, M, N - n1, K, A, lda, static_cast<const uint16_t*>(B) + n1, ldb,
                       static_cast<char*>(C) + (size_t)n1 * esz, ldc, 0, ob, sched, none, stream, 0);
  }
  if (pl.ce == 1) return launch_plan(pl, tables, M, N, K, A, lda, B, ldb, C, ldc, 0, ob, sched, none, stream, 0);
  rc = launch_plan(pl, tables, M, N, K, A, lda, B, ldb, W, N, M * N, false, sched, none, stream, 0);
  if (rc != SFC_OK) return rc;
  e = sfc::launch_reduce(W, pl.ce, M, N, C, ldc, ob, stream);
  if (e != hipSuccess) return hip_fail(e, "reduction launch");
  return SFC_OK;
}

}  // namespace

extern "C" {

int sfc_version(void) { return 1; }

const char* sfc_strerror(int code) {
  switch (code) {
    case SFC_OK: return "success";
    case SFC_ERR_INVALID_ARG: return "invalid argument";
    case SFC_ERR_UNSUPPORTED: return "unsupported argument";
    case SFC_ERR_WORKSPACE: return "workspace too small";
    case SFC_ERR_HIP: return "HIP runtime error";
    default: return "unknown error code";
  }
}

const char* sfc_last_error(void) { return g_last_error.c_str(); }

size_t sfc_gemm_ws_size(int64_t M, int64_t N, int64_t K, int ca_layers) {
  return sfc::ws_size(M, N, K, ca_layers);
}

int sfc_tile_order_ex(int gm, int gn, int order, int32_t* out_idx) {
  const sfc::Checked chk = sfc::check_order_args(gm, gn, order, out_idx);
  if (chk.code != SFC_OK) return set_error(chk.code, chk.msg);
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceState* st = nullptr;
  int rc = device_state(&st);
  if (rc != SFC_OK) return rc;
  const int32_t* table = nullptr;
  rc = get_table(*st, gm, gn, order, nullptr, &table);
  if (rc != SFC_OK) return rc;
  // a synchronous copy on the null stream: it follows the generator (get_table
  // made the null stream wait for it if it was enqueued on another stream)
  hipError_t e = hipMemcpy(out_idx, table, sizeof(int32_t) * (size_t)gm * (size_t)gn,
                           hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy(curve table)");
  return SFC_OK;
}

int sfc_tile_order(int gm, int gn, int32_t* out_idx) {
  return sfc_tile_order_ex(gm, gn, SFC_ORDER_HILBERT, out_idx);
}

int sfc_gemm_ex(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B,
                int64_t ldb, void* C, int64_t ldc, int out_type, int ca_layers, int tile, int order,
                int sched, void* ws, size_t ws_bytes, void* stream) {
  return gemm_impl(M, N, K, A, lda, B, ldb, C, ldc, out_type, ca_layers, tile, order, sched, ws,
                   ws_bytes, stream);
}

int sfc_gemm_f8_ex(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B,
                   int64_t ldb, void* C, int64_t ldc, int out_type, int ca_layers, int tile, int order,
                   int sched, void* ws, size_t ws_bytes, void* stream) {
  return gemm_impl(M, N, K, A, lda, B, ldb, C, ldc, out_type, ca_layers, tile, order, sched, ws,
                   ws_bytes, stream, 1);
}

int sfc_gemm_f8_fmt_ex(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B,
                       int64_t ldb, void* C, int64_t ldc, int out_type, int a_format, int b_format,
                       int ca_layers, int tile, int order, int sched, void* ws, size_t ws_bytes, void* stream) {
  if ((a_format != SFC_FP8_E4M3 && a_format != SFC_FP8_E5M2) || (b_format != SFC_FP8_E4M3 && b_format != SFC_FP8_E5M2))
    return set_error(SFC_ERR_INVALID_ARG, "unknown fp8 format");
  return gemm_impl(M, N, K, A, lda, B, ldb, C, ldc, out_type, ca_layers, tile, order, sched, ws,
                   ws_bytes, stream, 1 + a_format + 2 * b_format);
}

int sfc_gemm_noalloc_ex(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B,
                        int64_t ldb, void* C, int64_t ldc, int out_type, int ca_layers, int tile, int order,
                        int sched, void* stream) {
  return gemm_noalloc_impl(M, N, K, A, lda, B, ldb, C, ldc, out_type, ca_layers, tile, order, sched, stream);
}

int sfc_gemm_fused_ex(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B,
                      int64_t ldb, void* C, int64_t ldc, int out_type, int ca_layers, int tile, int order,
                      int sched, void* ws, size_t ws_bytes, void* stream) {
  return gemm_impl(M, N, K, A, lda, B, ldb, C, ldc, out_type, ca_layers, tile, order, sched, ws,
                   ws_bytes, stream, 0, kReduceFused);
}

int sfc_gemm(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B, int64_t ldb,
             void* C, int64_t ldc, int ca_layers, void* stream) {
  return gemm_impl(M, N, K, A, lda, B, ldb, C, ldc, SFC_OUT_F32, ca_layers, SFC_TILE_AUTO,
                   SFC_ORDER_HILBERT, SFC_SCHED_INTERLEAVED, nullptr, 0, stream);
}

int sfc_gemm_bf16out(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B,
                     int64_t ldb, void* C, int64_t ldc, int ca_layers, void* stream) {
  return gemm_impl(M, N, K, A, lda, B, ldb, C, ldc, SFC_OUT_BF16, ca_layers, SFC_TILE_AUTO,
                   SFC_ORDER_HILBERT, SFC_SCHED_INTERLEAVED, nullptr, 0, stream);
}

int sfc_probe_mfma(int random_operands, int iterations, double* tflops, double* mhz) {
  if (iterations < 1 || !tflops || !mhz) return set_error(SFC_ERR_INVALID_ARG, "invalid probe arguments");
  const size_t n = 256 * 256 + 256;
  float* d = nullptr;
  hipError_t e = hipMalloc(&d, n * sizeof(float));
  if (e != hipSuccess) return hip_fail(e, "hipMalloc(probe)");
  double ms = 0.0;
  e = sfc::run_mfma_probe(random_operands ? 1 : 0, iterations, d, &ms);
  float clk[256];
  if (e == hipSuccess) e = hipMemcpy(clk, d + 256 * 256, sizeof clk, hipMemcpyDeviceToHost);
  (void)hipFree(d);
  if (e != hipSuccess) return hip_fail(e, "MFMA probe");
  double sum = 0.0;
  for (int i = 0; i < 256; ++i) sum += clk[i];
  *mhz = sum / 256.0;
  // per wave and round: 64 MFMA 16x16x32
  const double flops = 256.0 * 4.0 * (double)iterations * 64.0 * (2.0 * 16 * 16 * 32);
  *tflops = ms > 0.0 ? flops / (ms * 1e-3) / 1e12 : 0.0;
  return SFC_OK;
}

int sfc_gemm_plan(int64_t M, int64_t N, int64_t K, int ca_layers, int tile, int64_t plan[7]) {
  if (!plan) return set_error(SFC_ERR_INVALID_ARG, "plan is NULL");
  if (M <= 0 || N <= 0 || K < 0 || ca_layers < 0 || ca_layers > sfc::kMaxLayers ||
      tile < SFC_TILE_AUTO || tile > SFC_TILE_256x256)
    return set_error(SFC_ERR_INVALID_ARG, "invalid plan arguments");
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceState* st = nullptr;
  int rc = device_state(&st);
  if (rc != SFC_OK) return rc;
  Plan pl;
  // aligned dummy pointers: the plan of the vector-load path
  rc = make_plan(*st, M, N, K, reinterpret_cast<const void*>(256), (K + 7) / 8 * 8,
                 reinterpret_cast<const void*>(256), (N + 7) / 8 * 8, false, ca_layers, tile, &pl);
  if (rc != SFC_OK) return rc;
  plan[0] = pl.bm; plan[1] = pl.bn; plan[2] = pl.gm; plan[3] = pl.gn;
  plan[4] = pl.ce; plan[5] = pl.grid; plan[6] = pl.occ;
  return SFC_OK;
}

int sfc_gemm_f8_plan(int64_t M, int64_t N, int64_t K, int ca_layers, int tile, int64_t plan[7]) {
  if (!plan) return set_error(SFC_ERR_INVALID_ARG, "plan is NULL");
  if (M <= 0 || N <= 0 || K < 0 || ca_layers < 0 || ca_layers > sfc::kMaxLayers ||
      (tile != SFC_TILE_AUTO && tile != SFC_TILE_128x256 && tile != SFC_TILE_256x256))
    return set_error(SFC_ERR_INVALID_ARG, "invalid plan arguments");
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceState* st = nullptr;
  int rc = device_state(&st);
  if (rc != SFC_OK) return rc;
  Plan pl;
  rc = make_plan(*st, M, N, K, nullptr, 0, nullptr, 0, false, ca_layers, tile, &pl, 1);
  if (rc != SFC_OK) return rc;
  plan[0] = pl.bm; plan[1] = pl.bn; plan[2] = pl.gm; plan[3] = pl.gn;
  plan[4] = pl.ce; plan[5] = pl.grid; plan[6] = pl.occ;
  return SFC_OK;
}

int sfc_gemm_model(int64_t M, int64_t N, int64_t K, int out_type, int ca_layers, int tile, int num_cus,
                   const int32_t occupancy[4], int64_t choice[3]) {
  if (!choice || !occupancy) return set_error(SFC_ERR_INVALID_ARG, "NULL model argument");
  if (M < 0 || N < 0 || K < 0 || num_cus < 1 || ca_layers < 0 || ca_layers > sfc::kMaxLayers ||
      tile < SFC_TILE_AUTO || tile > SFC_TILE_256x256 || (out_type != SFC_OUT_F32 && out_type != SFC_OUT_BF16))
    return set_error(SFC_ERR_INVALID_ARG, "invalid model arguments");
  int occ[sfc::kNumTiles];
  for (int t = 0; t < sfc::kNumTiles; ++t) {
    if (occupancy[t] < 1) return set_error(SFC_ERR_INVALID_ARG, "occupancy must be >= 1");
    occ[t] = occupancy[t];
  }
  const sfc::ModelChoice ch = sfc::model_choose(M, N, K, out_type == SFC_OUT_BF16 ? 2 : 4, num_cus, occ,
                                                tile == SFC_TILE_AUTO ? -1 : tile_from_api(tile), ca_layers);
  choice[0] = ch.tile + 1;   // SFC_TILE_* code
  choice[1] = sfc::effective_layers(K, ch.layers, sfc::kBK);
  choice[2] = (int64_t)(ch.clk + 0.5);
  return SFC_OK;
}

}  // extern "C"
