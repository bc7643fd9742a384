/*
 * sfcgemm.h -- C ABI of the MI355X (gfx950) space-filling-curve,
 * communication-avoiding bf16 GEMM.
 *
 * The operation is the GEMM of the paper's Section II.A, C = A * B with A of
 * M x K and B of K x N, executed as in Listing 1 (Section II.D): the M x N
 * output is cut into BM x BN blocks; the blocks are visited in generalized
 * Hilbert order (Section II.B); with ca_layers = c > 1 the contraction is
 * split into c contiguous K ranges, each computing a full copy of C, and the
 * copies are summed (Section II.C / II.D).  C is overwritten (Listing 1 zeroes
 * each block before the first contraction); there is no alpha or beta.
 *
 * Conventions for every entry point below
 *   - Matrices are row-major.  A[i][k] is at A[i*lda + k], B[k][j] at
 *     B[k*ldb + j], C[i][j] at C[i*ldc + j].  bf16 elements are 16-bit
 *     patterns (the upper half of an IEEE binary32).
 *   - A, B, C and workspace pointers are DEVICE pointers on the current HIP
 *     device; the caller owns them and keeps them alive until the work on
 *     `stream` has finished.  `stream` is a hipStream_t (NULL = null stream).
 *   - GEMM calls are asynchronous: they validate, enqueue kernels on `stream`
 *     and return.  Faults during execution surface at the next synchronisation.
 *   - On any error nothing is enqueued and C is not touched.
 *   - Elements of C outside the M x N region (ldc padding) are never written;
 *     elements of A and B outside their M x K and K x N regions are never used.
 *   - Accumulation is fp32 in every case.  For a fixed tile shape and layer
 *     count the result is bitwise reproducible and independent of the tile
 *     order and schedule.
 */
#ifndef SFCGEMM_H
#define SFCGEMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ------------------------------------------------------ */
#define SFC_OK               0
#define SFC_ERR_INVALID_ARG (-1) /* negative size, ld too small, null pointer, bad enum */
#define SFC_ERR_UNSUPPORTED (-2) /* misaligned element pointer, size beyond int32 tile indexing */
#define SFC_ERR_WORKSPACE   (-3) /* caller workspace smaller than sfc_gemm_ws_size() */
#define SFC_ERR_HIP         (-4) /* HIP runtime error; sfc_last_error() has the text */

/* ---- output element type (reading A8: fp32 accumulate, fp32 or bf16 out) */
#define SFC_OUT_F32  0           /* C holds float */
#define SFC_OUT_BF16 1           /* C holds bf16, rounded to nearest even */

/* ---- block (tile) shape BM x BN of the output grid --------------------- */
#define SFC_TILE_AUTO    0       /* chosen from M, N, K and ca_layers.  With one
                                    layer, 256-row blocks and a last round of
                                    blocks at most half full, the last block columns
                                    that make up that round are computed by a second
                                    launch (same stream) with 128-row blocks of the
                                    same width, which fill one round in about half
                                    the time; result bits are those of the single
                                    launch */
#define SFC_TILE_128x128 1
#define SFC_TILE_256x128 2       /* BM = 256, BN = 128 */
#define SFC_TILE_128x256 3       /* BM = 128, BN = 256 */
#define SFC_TILE_256x256 4

/* ---- number of K layers (copies of C) ---------------------------------- */
#define SFC_CA_AUTO      0       /* ca_layers = 0: chosen with the block shape by the
                                    analytical model (Section III.B Eq. 1-4, used as in
                                    Section III.C's second option), among 1, 2, 4, 8, 16 */

/* ---- order of the output blocks ---------------------------------------- */
#define SFC_ORDER_HILBERT   0    /* generalized Hilbert curve (Section II.B) */
#define SFC_ORDER_ROW_MAJOR 1    /* plain row-major; for comparison only */

/* ---- how curve positions are dealt to the persistent workgroups --------- */
#define SFC_SCHED_INTERLEAVED 0  /* workgroup r takes positions r, r+P, ...: the blocks
                                    in flight form one contiguous curve segment, and each
                                    chiplet (XCD) owns a contiguous sub-segment of it */
#define SFC_SCHED_BLOCK       1  /* workgroup r takes the r-th contiguous range of
                                    positions (the block partition of Section III.A) */
#define SFC_SCHED_INTERLEAVED_PLAIN 2  /* as SFC_SCHED_INTERLEAVED with r = the
                                    hardware workgroup index, so consecutive positions
                                    go to different chiplets; for comparison only */

/*
 * sfc_tile_order -- the block order of a gm x gn grid (Section II.B; the map
 * built by create_sfc_map in Listing 1).
 *   gm, gn   grid sides (blocks along M and along N), both >= 1, gm*gn < 2^31.
 *   out_idx  HOST buffer of gm*gn int32, caller-owned.  On return out_idx[s]
 *            = im*gn + in for the block (im, in) visited at curve position s.
 * The table is produced on the current device by the same generator the GEMM
 * uses, then copied back; the call is synchronous.
 * Returns SFC_OK, SFC_ERR_INVALID_ARG (bad sides, NULL out_idx),
 * SFC_ERR_UNSUPPORTED (gm*gn too large) or SFC_ERR_HIP.
 */
int sfc_tile_order(int gm, int gn, int32_t *out_idx);

/* As sfc_tile_order, with an explicit SFC_ORDER_* mode. */
int sfc_tile_order_ex(int gm, int gn, int order, int32_t *out_idx);

/*
 * sfc_gemm -- C = A * B, fp32 output (Section II.A, Listing 1).
 *   M, N, K    >= 0.  M == 0 or N == 0: nothing to do, SFC_OK.  K == 0: C = 0.
 *   A, lda     bf16, M x K, lda >= K (A may be NULL when M*K == 0).
 *   B, ldb     bf16, K x N, ldb >= N (B may be NULL when K*N == 0).
 *   C, ldc     float, M x N, ldc >= N.
 *   ca_layers  c in [1, 64]: number of K ranges / copies of C.  The K blocks
 *              (64 deep) are split into min(c, ceil(K/64)) contiguous ranges,
 *              range l holding blocks [floor(l*nK/c), floor((l+1)*nK/c)).  For
 *              c > 1 the partial copies live in a workspace of
 *              sfc_gemm_ws_size() bytes that the library keeps per stream: it
 *              is allocated, and grown, in stream order (hipMallocAsync /
 *              hipFreeAsync on `stream`), and only work on that stream uses
 *              it, so calls on different streams may run concurrently.  It is
 *              kept, keyed by the stream handle, until the process ends.
 *              SFC_CA_AUTO (0): the model picks c (see sfc_gemm_model).
 *   stream     hipStream_t or NULL.
 * No GEMM entry point synchronises the device or a stream.  The first call for
 * a block grid allocates its curve table (hipMalloc) and enqueues the
 * generator on `stream`; calls on other streams wait for it on the device.
 */
int sfc_gemm(int64_t M, int64_t N, int64_t K,
             const void *A, int64_t lda,
             const void *B, int64_t ldb,
             void *C, int64_t ldc,
             int ca_layers, void *stream);

/* As sfc_gemm with a bf16 C (rounded to nearest even from the fp32 sums). */
int sfc_gemm_bf16out(int64_t M, int64_t N, int64_t K,
                     const void *A, int64_t lda,
                     const void *B, int64_t ldb,
                     void *C, int64_t ldc,
                     int ca_layers, void *stream);

/*
 * sfc_gemm_ws_size -- bytes of fp32 workspace that a ca_layers = c call needs
 * for the replicated C of Section II.C / II.D (Listing 1 keeps K_layers copies
 * of C, one per K range, and reduces them): c_eff dense M x N fp32 copies,
 * c_eff * M * N * 4 bytes with c_eff = min(c, ceil(K/64)) when c_eff > 1, else 0.
 * For c = SFC_CA_AUTO: the size for the largest count the model picks (16), a
 * bound that holds whatever it chooses.  Returns 0 for invalid arguments as well.
 */
size_t sfc_gemm_ws_size(int64_t M, int64_t N, int64_t K, int ca_layers);

/*
 * sfc_gemm_ex -- the general entry point behind sfc_gemm / sfc_gemm_bf16out.
 *   out_type   SFC_OUT_F32 or SFC_OUT_BF16.
 *   tile       SFC_TILE_*; order SFC_ORDER_*; sched SFC_SCHED_*.
 *   ws         device workspace of ws_bytes bytes, or NULL to use the library's
 *              internal one.  When c_eff > 1, layer l of the partial result is
 *              left in ws as a dense fp32 M x N matrix at ws + l*M*N floats.
 * Tile order and schedule never change the result bits; tile shape and layer
 * count change only the fp32 summation grouping.
 */
int sfc_gemm_ex(int64_t M, int64_t N, int64_t K,
                const void *A, int64_t lda,
                const void *B, int64_t ldb,
                void *C, int64_t ldc,
                int out_type, int ca_layers, int tile, int order, int sched,
                void *ws, size_t ws_bytes, void *stream);

/*
 * sfc_gemm_fused_ex -- sfc_gemm_ex with the reduction of the layer copies
 * fused into the GEMM launch (Listing 1's final add-reduce, Section II.D,
 * done by the GEMM's own workgroups): the workgroup that finishes a block's
 * layer copy publishes it (a release fence at device scope) and counts it on
 * the block's arrival counter (a device-scope atomic); the workgroup that
 * completes the count reads the c_eff copies of that block and sums them in
 * ascending layer order in fp32, so C is bit-identical to sfc_gemm_ex's.  No
 * workgroup waits for another.  One launch instead of two; the c_eff-way sum of
 * a block runs on one compute unit.  The counters are library memory kept per
 * stream (zero between launches; a call never leaves one raised), so `ws`, if
 * given, still needs only sfc_gemm_ws_size() bytes.  With c_eff = 1 this is
 * sfc_gemm_ex.  Arguments, errors and the contents left in ws as for
 * sfc_gemm_ex.
 */
int sfc_gemm_fused_ex(int64_t M, int64_t N, int64_t K,
                      const void *A, int64_t lda,
                      const void *B, int64_t ldb,
                      void *C, int64_t ldc,
                      int out_type, int ca_layers, int tile, int order, int sched,
                      void *ws, size_t ws_bytes, void *stream);

/*
 * sfc_gemm_noalloc_ex -- sfc_gemm_ex for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same kernels and results, bit for bit, with no
 * allocation and no synchronisation in the call.  Instead of the library's
 * per-stream workspace and cached curve tables it uses one static device
 * array per GPU, held until the process ends: SFC_NOALLOC_WS_BYTES of fp32
 * layer copies and two curve tables of SFC_NOALLOC_MAX_BLOCKS entries, which
 * every call rewrites on `stream` (a small kernel before the GEMM).
 *   Arguments and errors as for sfc_gemm_ex without a workspace, plus:
 *   SFC_ERR_WORKSPACE   sfc_gemm_ws_size(M, N, K, ca_layers) exceeds
 *                       SFC_NOALLOC_WS_BYTES (checked before any HIP call);
 *   SFC_ERR_UNSUPPORTED the block grid has more than SFC_NOALLOC_MAX_BLOCKS
 *                       blocks.
 * Every call on a GPU uses that GPU's one array, whose contents are those the
 * last call left: calls that overlap on one GPU (on different streams, or
 * from different threads) race on it and must be ordered by the caller.  The
 * first call on a device looks up the array's address (hipGetSymbolAddress).
 */
#define SFC_NOALLOC_WS_BYTES   ((size_t)64 << 20)   /* 64 MiB of layer copies */
#define SFC_NOALLOC_MAX_BLOCKS (1 << 17)            /* blocks per curve table */
int sfc_gemm_noalloc_ex(int64_t M, int64_t N, int64_t K,
                        const void *A, int64_t lda,
                        const void *B, int64_t ldb,
                        void *C, int64_t ldc,
                        int out_type, int ca_layers, int tile, int order, int sched,
                        void *stream);

/*
 * sfc_gemm_f8_ex -- C = A * B with 8-bit float operands (the paper leaves the
 * data type a parameter of the method, Section III.A): A and B hold OCP FP8
 * E4M3 bytes (1 sign, 4 exponent bits with bias 7, 3 mantissa bits; no
 * infinities, 0x7F / 0xFF are NaN), row-major, lda and ldb in elements (=
 * bytes).  The products are exact in fp32 and the sums are fp32, as in
 * sfc_gemm_ex; C is fp32 or bf16 (out_type).  Same blocks-along-the-curve and
 * K-layer scheme, with K blocks 128 deep: ca_layers = c uses min(c,
 * ceil(K/128)) layers, whose workspace sfc_gemm_ws_size(M, N, K, c) bounds.
 * Restrictions (else SFC_ERR_UNSUPPORTED, nothing enqueued): A and B 16-byte
 * aligned, lda, ldb, K and N multiples of 16; tile SFC_TILE_AUTO,
 * SFC_TILE_256x256 or SFC_TILE_128x256.  SFC_TILE_AUTO and SFC_CA_AUTO pick the
 * free knobs with the model of sfc_gemm_model over those two block shapes,
 * evaluated on the bf16 problem with the same number of K blocks (K' =
 * 64*ceil(K/128)): a 128-deep fp8 block moves the bytes of a 64-deep bf16
 * block and takes the same MFMA time (ties go to 256x256).  Other arguments and
 * errors as for sfc_gemm_ex.
 */
int sfc_gemm_f8_ex(int64_t M, int64_t N, int64_t K,
                   const void *A, int64_t lda,
                   const void *B, int64_t ldb,
                   void *C, int64_t ldc,
                   int out_type, int ca_layers, int tile, int order, int sched,
                   void *ws, size_t ws_bytes, void *stream);

/* ---- 8-bit float formats --------------------------------------------------- */
#define SFC_FP8_E4M3 0   /* OCP E4M3: bias 7, 3 mantissa bits, no infinities, 0x7F/0xFF NaN */
#define SFC_FP8_E5M2 1   /* OCP E5M2: bias 15, 2 mantissa bits, 0x7C/0xFC = +-inf,
                            0x7D-0x7F/0xFD-0xFF NaN (the IEEE-style 8-bit format) */

/*
 * sfc_gemm_f8_fmt_ex -- sfc_gemm_f8_ex with the format of each operand chosen:
 * a_format and b_format are SFC_FP8_E4M3 or SFC_FP8_E5M2 (the two 8-bit float
 * formats of the same matrix instruction; mixed pairs allowed).  Every value of
 * either format is a bf16 value, so products are exact in fp32 as for E4M3.
 * Errors: SFC_ERR_INVALID_ARG for another format code, else as sfc_gemm_f8_ex.
 * sfc_gemm_f8_ex is this call with both formats SFC_FP8_E4M3.
 */
int sfc_gemm_f8_fmt_ex(int64_t M, int64_t N, int64_t K,
                       const void *A, int64_t lda,
                       const void *B, int64_t ldb,
                       void *C, int64_t ldc,
                       int out_type, int a_format, int b_format,
                       int ca_layers, int tile, int order, int sched,
                       void *ws, size_t ws_bytes, void *stream);

/*
 * sfc_gemm_plan -- what sfc_gemm_ex would launch, without launching
 * (fp32 output, 16-byte aligned operands).  ca_layers may be SFC_CA_AUTO and
 * tile SFC_TILE_AUTO; the plan then shows the model's choice (for the whole
 * grid: a half-height strip that SFC_TILE_AUTO may add is not shown).
 *   plan[0] = BM, plan[1] = BN, plan[2] = gm, plan[3] = gn, plan[4] = c_eff,
 *   plan[5] = number of persistent workgroups, plan[6] = workgroups per CU.
 * Needs a device (it queries the CU count and kernel occupancy).
 */
int sfc_gemm_plan(int64_t M, int64_t N, int64_t K, int ca_layers, int tile, int64_t plan[7]);

/*
 * sfc_gemm_f8_plan -- what sfc_gemm_f8_ex (and sfc_gemm_f8_fmt_ex) would
 * launch, without launching (fp32 output); plan[] as for sfc_gemm_plan.  tile
 * is SFC_TILE_AUTO, SFC_TILE_128x256 or SFC_TILE_256x256, else
 * SFC_ERR_INVALID_ARG.  Needs a device.
 */
int sfc_gemm_f8_plan(int64_t M, int64_t N, int64_t K, int ca_layers, int tile, int64_t plan[7]);

/*
 * sfc_gemm_model -- the analytical model behind SFC_TILE_AUTO and SFC_CA_AUTO,
 * evaluated for given device parameters (host only: no device is touched).
 * The paper's fine-grained roofline (Section III.B, Eq. 1-4) on the GPU: a core
 * is a CU running `occupancy` persistent workgroups, one BRGEMM is one 64-deep
 * block of one task, at max(G*gamma, beta*(S_A + S_B)) with the panels of a
 * block shared by the tasks in flight on one XCD; the critical path is the
 * rounds of tasks times the blocks of the longest layer, plus the C traffic
 * (and, with layers, the copies written and read back) and the launches.
 * Every candidate (block shape x c in {1, 2, 4, 8, 16}, or only the fixed ones) is
 * evaluated and the fastest kept; near ties go to less padded work, then to
 * 256x256, 128x256, 256x128, 128x128 in that order, then to fewer layers.
 *   out_type   SFC_OUT_F32 or SFC_OUT_BF16 (bytes of C).
 *   ca_layers  SFC_CA_AUTO (0) or a fixed count in [1, 64].
 *   tile       SFC_TILE_AUTO or a fixed SFC_TILE_*.
 *   num_cus    compute units (>= 1).
 *   occupancy  host array: workgroups per CU of SFC_TILE_128x128, _256x128,
 *              _128x256, _256x256 (each >= 1).
 *   choice     host out: [0] SFC_TILE_* code, [1] effective layer count,
 *              [2] estimated shader clocks.
 * Returns SFC_OK or SFC_ERR_INVALID_ARG.
 */
int sfc_gemm_model(int64_t M, int64_t N, int64_t K, int out_type, int ca_layers, int tile, int num_cus,
                   const int32_t occupancy[4], int64_t choice[3]);

/*
 * sfc_probe_mfma -- measurement aid for the roofline (the counterpart of the
 * paper's compute micro-benchmark, Section III.B): register-only bf16 MFMA
 * 16x16x32 throughput (the GEMM kernel's instruction) of the current device,
 * 256 workgroups x 4 waves, each wave running `iterations` rounds of 64
 * independent MFMAs.
 *   random_operands  1: operands drawn at random (they change between MFMAs, as
 *                    in a GEMM); 0: constant operands.
 *   tflops, mhz      out: achieved TFLOP/s and the mean shader clock sampled
 *                    during the loop (MHz).  Host pointers.
 * Synchronous (null stream); allocates and frees a 257 KiB device buffer.
 * Returns SFC_OK, SFC_ERR_INVALID_ARG (iterations < 1, NULL outputs) or
 * SFC_ERR_HIP.
 */
int sfc_probe_mfma(int random_operands, int iterations, double *tflops, double *mhz);

/* Static text of a return code. */
const char *sfc_strerror(int code);

/* Text of the last error raised on the calling thread ("" if none). */
const char *sfc_last_error(void);

/* ABI version: 1. */
int sfc_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SFCGEMM_H */
