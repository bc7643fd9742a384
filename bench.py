#!/usr/bin/env python3
"""Benchmark of the SFC-CA bf16 GEMM on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Prints ONE JSON line.  The headline `value` is TFLOP/s of the 8192^3 bf16
GEMM (256x256 blocks, a 32x32 block grid in generalized Hilbert order, bf16
output), timed over K back-to-back calls with inputs resident in HBM.  The
line also carries:
  * roofline   -- the GEMM kernel's own average duration (HIP events on the
                  launch stream over the timed steps) against the bf16 dense
                  MFMA peak, HBM bytes per launch from committed counter runs,
                  the sustained MFMA probe, and the same kernel on constant
                  operands (full clock: the kernel's per-clock efficiency);
  * cpu_baseline -- the CPU oracle on a bounded row sample of the same GEMM;
  * workloads  -- every measured workload (TFLOP/s, cold and warm, the paper's
                  protocol of 10 cold repetitions) and their flop-weighted
                  harmonic mean; for the K-dominant one also the layers placed
                  on whole chiplets against the hardware workgroup order;
  * fp8_square8192 -- the same 8192^3 GEMM with OCP FP8 E4M3 operands
                  (sfc_gemm_f8_ex, bf16 output), timed like the headline,
                  against the fp8 dense MFMA peak, with the vendor library's
                  fp8 GEMM beside it and an E5M2 line (sfc_gemm_f8_fmt_ex);
  * sweep      -- with --sweep: the paper's 125-shape cube sweep (Section IV.A),
                  per shape the library's own choice of block shape and layer
                  count (10 cold repetitions), the best of a small autotune
                  over the layer count, the fraction of the shape's roofline,
                  and the flop-weighted harmonic mean.
Inputs are synthetic (seeded, see paper_2601_16294_amd/inputs.py).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
METRIC = "bf16 GEMM TFLOP/s per shape + weighted harmonic mean; % of MFMA peak"
# MI355X bf16 dense MFMA peak: 256 CUs x 4096 FLOP/clock x 2.4 GHz.
PEAK_BF16_TFLOPS = 2516.6
PEAK_HBM_GBS = 8000.0
# MI355X fp8 dense MFMA peak (the published 5.0 PFLOP/s): twice the bf16 rate.
PEAK_FP8_TFLOPS = 5033.2
HEADLINE = "square8192_bf16out_t256"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_square8192_gemm.json")
GEMM_SRC = os.path.join(ROOT, "paper_2601_16294_amd", "csrc", "sfc_gemm.hip")


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--reps", type=int, default=10, help="cold repetitions per workload")
    ap.add_argument("--no-workloads", action="store_true", help="headline only")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--order", default="hilbert", choices=["hilbert", "row_major"])
    ap.add_argument("--sched", default="interleaved", choices=["interleaved", "block", "interleaved_plain"])
    ap.add_argument("--only", default=None,
                    help="run the kernel of one workload (or fp8_square8192) K times and exit")
    ap.add_argument("--sweep", action="store_true", help="also run the 125-shape sweep")
    ap.add_argument("--sweep-reps", type=int, default=3, help="cold repetitions per autotune candidate")
    ap.add_argument("--tune-reps", type=int, default=5,
                    help="cold repetitions per candidate of the per-workload autotune")
    ap.add_argument("--no-autotune", action="store_true", help="skip the per-workload model-vs-autotune check")
    ap.add_argument("--only-layers", type=int, default=None, help="with --only: ca_layers (0: the model's)")
    ap.add_argument("--only-tile", default=None, help="with --only: block shape (default: the workload's)")
    ap.add_argument("--warm-clock-ms", type=float, default=200.0,
                    help="back-to-back calls of a workload before it is timed (sweep shapes: a quarter)")
    ap.add_argument("--cold", action="store_true",
                    help="with --only: clear a 512 MiB buffer before every call (for counter runs: the "
                         "timed cold runs of the bench rotate over operand copies instead)")
    ap.add_argument("--fused", action="store_true", help="with --only: sum the layer copies inside the GEMM")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="with --only: also run a plain device copy of MIB MiB (counter calibration)")
    return ap.parse_args()


def counter_record():
    """Per-launch figures of the headline kernel from committed rocprofv3
    counter runs (HBM bytes, shader cycles per XCD, MFMA busy), valid only
    while the GEMM kernel source is the one the counters were taken on."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return {}
    sha = hashlib.sha256(open(GEMM_SRC, "rb").read()).hexdigest()
    if rec.get("kernel_src_sha256") != sha:
        return {}
    return rec


def roofline_tflops(M, N, K, out_bytes):
    """min(MFMA peak, OI x HBM bandwidth) with compulsory bytes A + B + C."""
    oi = 2.0 * M * N * K / (2.0 * M * K + 2.0 * K * N + out_bytes * M * N)
    hbm = oi * PEAK_HBM_GBS / 1e3
    return ("hbm", hbm) if hbm < PEAK_BF16_TFLOPS else ("mfma", PEAK_BF16_TFLOPS)


def warm_clock(torch, stream, fn, min_ms):
    """Run fn back to back for at least min_ms of wall time and return the
    time per call of the first and of the last batch (HIP events).  A GPU that
    sat idle while the host drew a workload's inputs runs its first tens of
    milliseconds of work at a lower clock; the cold protocol clears the caches
    between repetitions, it is not meant to time that clock ramp."""
    t0 = time.perf_counter()
    first = last = None
    while True:
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record(stream)
        for _ in range(4):
            fn()
        e.record(stream)
        torch.cuda.synchronize()
        last = s.elapsed_time(e) / 4
        if first is None:
            first = last
        if (time.perf_counter() - t0) * 1e3 >= min_ms:
            return round(first, 4), round(last, 4)


ROTATION_BYTES = 1 << 30


def gpu_backlog(torch, us):
    """Keep the GPU busy for about `us` microseconds (a spin kernel that touches
    no memory) while the host enqueues what follows, so that a timed call
    starts as soon as its start event does: for calls of a few microseconds the
    host's enqueue time would otherwise sit between the two."""
    torch.cuda._sleep(int(us * 2000))


class ColdSets:
    """The cold protocol of Section IV.A: copies of one GEMM's A, B and C,
    enough of them (at least 2, together at least 1 GiB: past the 256 MiB
    Infinity Cache and the 8 x 4 MiB of L2) that a call taken in rotation
    finds none of its operands in a cache.  Nothing runs between the calls but
    the other copies' GEMMs (no flush kernel, whose dirty lines the timed call
    would have to write back)."""

    def __init__(self, torch, a, b, c):
        set_bytes = a.numel() * a.element_size() + b.numel() * b.element_size() + c.numel() * c.element_size()
        n = max(2, -(-ROTATION_BYTES // max(set_bytes, 1)))
        self.sets = [(a, b, c)] + [(a.clone(), b.clone(), torch.empty_like(c)) for _ in range(n - 1)]
        self.next = 0

    def time_ms(self, torch, stream, fn, reps):
        """Mean time of `reps` calls fn(a, b, c), each on the set least recently
        used (HIP events around each call); every set is used once, untimed,
        before the first timed call."""
        n = len(self.sets)
        for _ in range(n):
            fn(*self.sets[self.next])
            self.next = (self.next + 1) % n
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for s0, s1 in ev:
            gpu_backlog(torch, 50)
            s0.record(stream)
            fn(*self.sets[self.next])
            s1.record(stream)
            self.next = (self.next + 1) % n
        torch.cuda.synchronize()
        return sum(x.elapsed_time(y) for x, y in ev) / reps


def run_sweep(args, sg, torch, stream, dev):
    """The 125-shape sweep: the library's choice (SFC_TILE_AUTO, SFC_CA_AUTO),
    timed cold (10 repetitions in rotation over copies of the operands), and an
    autotune over ca_layers in {1, 2, 4, 8, 16} with the model's block shape for
    each count."""
    from paper_2601_16294_amd.inputs import draw, sweep_gemms
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    occ = tuple(sg.sfc_gemm_plan(8192, 8192, 64, 1, t)["per_cu"] for t in ("128x128", "256x128", "128x256", "256x256"))
    mats = {}

    def mat(rows, cols, dist, seed):
        if seed not in mats:
            mats[seed] = sg.to_device_bf16(draw(rows, cols, dist, seed))
        return mats[seed]

    def cold(sets, layers, tile, reps):
        return sets.time_ms(torch, stream,
                            lambda a, b, c: sg.sfc_gemm_ex(a, b, c, ca_layers=layers, tile=tile, stream=stream), reps)

    rows = []
    num = den = 0.0
    for g in sweep_gemms():
        a = mat(g.M, g.K, g.dist_a, g.seed_a)
        b = mat(g.K, g.N, g.dist_b, g.seed_b)
        c = torch.empty((g.M, g.N), dtype=torch.bfloat16, device=dev)
        choice = sg.sfc_gemm_model(g.M, g.N, g.K, out="bf16", num_cus=cus, occupancy=occ)
        warm_clock(torch, stream, lambda: sg.sfc_gemm_ex(a, b, c, ca_layers=0, tile="auto", stream=stream),
                   args.warm_clock_ms / 4)
        sets = ColdSets(torch, a, b, c)
        ms = cold(sets, 0, "auto", args.reps)
        tuned = []
        for layers in (1, 2, 4, 8, 16):
            t = sg.sfc_gemm_model(g.M, g.N, g.K, out="bf16", ca_layers=layers, num_cus=cus, occupancy=occ)["tile"]
            sg.sfc_gemm_ex(a, b, c, ca_layers=layers, tile=t, stream=stream)
            tuned.append((cold(sets, layers, t, args.sweep_reps), t, layers))
        best = min(tuned)
        bound, roof = roofline_tflops(g.M, g.N, g.K, 2)
        tf = g.flops / (ms * 1e-3) / 1e12
        rows.append({"M": g.M, "N": g.N, "K": g.K, "tile": choice["tile"], "ca_layers": choice["layers"],
                     "ms": round(ms, 4), "tflops": round(tf, 1), "bound": bound,
                     "frac_roofline": round(tf / roof, 4),
                     "best": {"tile": best[1], "ca_layers": best[2], "ms": round(best[0], 4),
                              "tflops": round(g.flops / (best[0] * 1e-3) / 1e12, 1)}})
        num += g.flops
        den += g.flops / tf
        log(f"[sweep] {g.M}x{g.N}x{g.K} {choice} {tf:.1f} TFLOP/s, best {rows[-1]['best']}")
        del c, sets
    del mats
    torch.cuda.empty_cache()
    best_num = sum(2.0 * r["M"] * r["N"] * r["K"] for r in rows)
    best_den = sum(2.0 * r["M"] * r["N"] * r["K"] / r["best"]["tflops"] for r in rows)
    ratio = [r["tflops"] / r["best"]["tflops"] for r in rows]
    return {"protocol": f"bf16 in, fp32 accumulate, bf16 out, U(-1,1); mean of {args.reps} cold reps "
                        f"(in rotation over >= 1 GiB of operand copies) of the library's choice; autotune: ca_layers in "
                        f"{{1,2,4,8,16}} with the model's block shape, {args.sweep_reps} cold reps each",
            "whm_tflops": round(num / den, 2), "whm_tflops_autotuned": round(best_num / best_den, 2),
            "model_over_autotune_mean": round(sum(ratio) / len(ratio), 4),
            "model_over_autotune_min": round(min(ratio), 4),
            "worst_frac_roofline": min(r["frac_roofline"] for r in rows),
            "shapes": rows}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(this build has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2601_16294_amd import sfcgemm as sg
    from paper_2601_16294_amd.inputs import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    W = {w.name: w for w in workloads()}

    def run_once(dA, dB, C, w, c, sched=None, tile=None, fused=False):
        f = sg.sfc_gemm_fused_ex if fused else sg.sfc_gemm_ex
        f(dA, dB, C, ca_layers=c, tile=tile or w.tile, order=args.order, sched=sched or args.sched, stream=stream)

    def prepare(g):
        A, B = g.operands()
        dA, dB = sg.to_device_bf16(A), sg.to_device_bf16(B)
        dtype = torch.float32 if g.out == "f32" else torch.bfloat16
        C = torch.empty((g.M, g.N), dtype=dtype, device=dev)
        return A, B, dA, dB, C

    if args.only == "fp8_square8192":
        from paper_2601_16294_amd.inputs import draw_e4m3
        a8 = sg.to_device_u8(draw_e4m3(8192, 8192, ("normal", 0.0, 1.0), 2101))
        b8 = sg.to_device_u8(draw_e4m3(8192, 8192, ("normal", 0.0, 1.0), 2102))
        c8 = torch.empty((8192, 8192), dtype=torch.bfloat16, device=dev)
        for _ in range(args.steps):
            sg.sfc_gemm_f8_ex(a8, b8, c8, stream=stream)
        torch.cuda.synchronize()
        log(f"[bench] ran fp8_square8192 {args.steps} times")
        return
    if args.only:
        # one workload's GEMMs (each called --steps times, in turn), for
        # profilers: --only-layers picks the layer count (default: the last of
        # the workload's list), --only-tile the block shape, --cold clears
        # 512 MiB before every call (operands out of the caches for counter
        # runs), --fused sums the layer copies in the GEMM
        ow = W[args.only]
        c_only = ow.ca_layers[-1] if args.only_layers is None else args.only_layers
        flush = torch.empty(512 * 1024 * 1024 // 4, dtype=torch.float32, device=dev) if args.cold else None
        for og in ow.gemms:
            _, _, oA, oB, oC = prepare(og)
            for _ in range(args.steps):
                if flush is not None:
                    flush.zero_()
                run_once(oA, oB, oC, ow, c_only, tile=args.only_tile, fused=args.fused)
            torch.cuda.synchronize()
            log(f"[bench] ran {args.only} {og.M}x{og.N}x{og.K} ca_layers={c_only} order={args.order} "
                f"{'cold ' if args.cold else ''}{args.steps} times")
            del oA, oB, oC
        if args.calibrate_copy:
            n = args.calibrate_copy * 1024 * 1024 // 4
            src = torch.ones(n, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            dst.copy_(src)
            torch.cuda.synchronize()
            log(f"[bench] copied {args.calibrate_copy} MiB")
        return

    # ---------------------------------------------------------------- headline
    w = W[HEADLINE]
    g = w.gemms[0]
    log(f"[bench] preparing {HEADLINE} {g.M}x{g.N}x{g.K}")
    A_host, B_host, dA, dB, C = prepare(g)
    plan = sg.sfc_gemm_plan(g.M, g.N, g.K, 1, w.tile)
    # the GPU idled while the host drew the inputs: bring it to its loaded
    # clock before the warm-up steps (reported in the line as clock_warmup)
    head_ramp = warm_clock(torch, stream, lambda: run_once(dA, dB, C, w, 1), args.warm_clock_ms)
    log(f"[bench] clock warm-up: ms per call {head_ramp[0]} (first batch) -> {head_ramp[1]} (last)")
    for _ in range(args.warmup):
        run_once(dA, dB, C, w, 1)
    torch.cuda.synchronize()
    log(f"[bench] warmup done; timing {args.steps} steps")
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        run_once(dA, dB, C, w, 1)
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = sum(s.elapsed_time(e) for s, e in zip(starts, ends)) / args.steps
    ms_per_step = wall * 1e3 / args.steps
    value = g.flops / (ms_per_step * 1e-3) / 1e12
    achieved = g.flops / (kern_ms * 1e-3) / 1e12
    log(f"[bench] headline {value:.1f} TFLOP/s (wall), kernel {kern_ms:.3f} ms -> {achieved:.1f} TFLOP/s")

    # The vendor library on the same operands (torch.matmul -> hipBLASLt), timed
    # the same way: a reference point, not part of the path.
    ref = torch.empty_like(C)
    for _ in range(args.warmup):
        torch.matmul(dA, dB, out=ref)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for s0, s1 in ev:
        s0.record(stream)
        torch.matmul(dA, dB, out=ref)
        s1.record(stream)
    torch.cuda.synchronize()
    lib_ms = sum(a.elapsed_time(b) for a, b in ev) / args.steps
    library = {"call": "torch.matmul (hipBLASLt), bf16 in, bf16 out", "ms": round(lib_ms, 4),
               "tflops": round(g.flops / (lib_ms * 1e-3) / 1e12, 1)}
    log(f"[bench] library {library}")

    # The same kernel and launch on constant operands (A = 0.25, B = 0.5): the
    # cycle count is the same, but with no data toggling the chip holds its
    # full clock, so this separates the kernel's per-clock efficiency from the
    # clock that random operands leave it (a diagnostic, not the metric).
    cA, cB = torch.full_like(dA, 0.25), torch.full_like(dB, 0.5)
    for _ in range(args.warmup):
        run_once(cA, cB, C, w, 1)
    torch.cuda.synchronize()
    evc = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for s0, s1 in evc:
        s0.record(stream)
        run_once(cA, cB, C, w, 1)
        s1.record(stream)
    torch.cuda.synchronize()
    const_ms = sum(a.elapsed_time(b) for a, b in evc) / args.steps
    const_tf = g.flops / (const_ms * 1e-3) / 1e12
    constant = {"call": "the same kernel, A = 0.25 and B = 0.5 everywhere", "ms": round(const_ms, 4),
                "tflops": round(const_tf, 1), "frac": round(const_tf / PEAK_BF16_TFLOPS, 4)}
    log(f"[bench] constant operands {constant}")
    del dA, dB, C, ref, cA, cB
    torch.cuda.empty_cache()

    # ------------------------------------------------- fp8 operands, same shape
    from paper_2601_16294_amd.inputs import draw_e4m3
    log("[bench] fp8 operands")
    a8 = sg.to_device_u8(draw_e4m3(g.M, g.K, ("normal", 0.0, 1.0), 2101))
    b8 = sg.to_device_u8(draw_e4m3(g.K, g.N, ("normal", 0.0, 1.0), 2102))
    c8 = torch.empty((g.M, g.N), dtype=torch.bfloat16, device=dev)
    warm_clock(torch, stream, lambda: sg.sfc_gemm_f8_ex(a8, b8, c8, stream=stream), args.warm_clock_ms)
    for _ in range(args.warmup):
        sg.sfc_gemm_f8_ex(a8, b8, c8, stream=stream)
    torch.cuda.synchronize()
    ev8 = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for s0, s1 in ev8:
        s0.record(stream)
        sg.sfc_gemm_f8_ex(a8, b8, c8, stream=stream)
        s1.record(stream)
    torch.cuda.synchronize()
    f8_ms = sum(x.elapsed_time(y) for x, y in ev8) / args.steps
    f8_tf = g.flops / (f8_ms * 1e-3) / 1e12
    fp8 = {"call": "sfc_gemm_f8_ex, E4M3 A and B ~ N(0,1), bf16 out, 256x256 blocks", "ms": round(f8_ms, 4),
           "tflops": round(f8_tf, 1), "peak": PEAK_FP8_TFLOPS, "frac": round(f8_tf / PEAK_FP8_TFLOPS, 4)}
    # the vendor library on the same E4M3 operands (torch._scaled_mm -> hipBLASLt),
    # when this torch build offers it: a reference point, not part of the path
    try:
        fa = a8.view(torch.float8_e4m3fn)
        fb = b8.view(torch.float8_e4m3fn).t().contiguous().t()   # column-major B, as the call requires
        one = torch.ones((), dtype=torch.float32, device=dev)
        for _ in range(args.warmup):
            torch._scaled_mm(fa, fb, scale_a=one, scale_b=one, out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        evl = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for s0, s1 in evl:
            s0.record(stream)
            torch._scaled_mm(fa, fb, scale_a=one, scale_b=one, out_dtype=torch.bfloat16)
            s1.record(stream)
        torch.cuda.synchronize()
        lib8_ms = sum(x.elapsed_time(y) for x, y in evl) / args.steps
        fp8["library_same_workload"] = {"call": "torch._scaled_mm (hipBLASLt), E4M3 in, bf16 out",
                                        "ms": round(lib8_ms, 4),
                                        "tflops": round(g.flops / (lib8_ms * 1e-3) / 1e12, 1)}
        del fa, fb
    except (RuntimeError, TypeError) as e:   # not offered by this torch build / device
        fp8["library_same_workload"] = {"unavailable": str(e)[:120]}
    # the same shape with OCP E5M2 operands (sfc_gemm_f8_fmt_ex)
    from paper_2601_16294_amd.inputs import draw_fp8
    a5 = sg.to_device_u8(draw_fp8(g.M, g.K, ("normal", 0.0, 1.0), 2101, fmt="e5m2"))
    b5 = sg.to_device_u8(draw_fp8(g.K, g.N, ("normal", 0.0, 1.0), 2102, fmt="e5m2"))
    warm_clock(torch, stream, lambda: sg.sfc_gemm_f8_ex(a5, b5, c8, stream=stream, a_format="e5m2", b_format="e5m2"),
               args.warm_clock_ms / 2)
    for _ in range(args.warmup):
        sg.sfc_gemm_f8_ex(a5, b5, c8, stream=stream, a_format="e5m2", b_format="e5m2")
    torch.cuda.synchronize()
    ev5 = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for s0, s1 in ev5:
        s0.record(stream)
        sg.sfc_gemm_f8_ex(a5, b5, c8, stream=stream, a_format="e5m2", b_format="e5m2")
        s1.record(stream)
    torch.cuda.synchronize()
    f5_ms = sum(x.elapsed_time(y) for x, y in ev5) / args.steps
    fp8["e5m2"] = {"call": "sfc_gemm_f8_fmt_ex, E5M2 A and B ~ N(0,1), bf16 out", "ms": round(f5_ms, 4),
                   "tflops": round(g.flops / (f5_ms * 1e-3) / 1e12, 1)}
    # the fp8 block shapes on a ragged grid: the model's choice (128x256 here)
    # against 256x256 blocks, warm, E4M3 in and bf16 out
    rM, rN, rK = 3000, 7008, 2048
    ra8 = sg.to_device_u8(draw_e4m3(rM, rK, ("normal", 0.0, 1.0), 2103))
    rb8 = sg.to_device_u8(draw_e4m3(rK, rN, ("normal", 0.0, 1.0), 2104))
    rc8 = torch.empty((rM, rN), dtype=torch.bfloat16, device=dev)
    shapes8 = {}
    for t in ("auto", "256x256"):
        fn8 = lambda: sg.sfc_gemm_f8_ex(ra8, rb8, rc8, tile=t, stream=stream)
        warm_clock(torch, stream, fn8, args.warm_clock_ms / 4)
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record(stream)
        for _ in range(20):
            fn8()
        s1.record(stream)
        torch.cuda.synchronize()
        ms8 = s0.elapsed_time(s1) / 20
        key = "model_choice" if t == "auto" else t
        shapes8[key] = {"ms": round(ms8, 4), "tflops": round(2.0 * rM * rN * rK / (ms8 * 1e-3) / 1e12, 1)}
    pl8 = sg.sfc_gemm_f8_plan(rM, rN, rK, 1, "auto")
    shapes8["model_choice"]["tile"] = f"{pl8['BM']}x{pl8['BN']}"
    fp8["ragged3000x7008x2048"] = shapes8
    log(f"[bench] fp8 {fp8}")
    del a8, b8, c8, a5, b5, ra8, rb8, rc8
    torch.cuda.empty_cache()

    # ---------------------------------------------- sustained MFMA throughput
    # Register-only MFMA loops: the clock the chip holds depends on how much the
    # operand bits toggle, so the achievable ceiling for random data sits well
    # below the published peak.
    probe = {"random_operands": sg.sfc_probe_mfma(True, 200000),
             "constant_operands": sg.sfc_probe_mfma(False, 200000)}
    for v in probe.values():
        v["tflops"] = round(v["tflops"], 1)
        v["mhz"] = round(v["mhz"], 0)
    log(f"[bench] MFMA probe {probe}")

    # --------------------------------------------------------------- workloads
    table = None
    if not args.no_workloads:
        table = {}
        whm_num = whm_den = 0.0
        for name, wl in W.items():
            entry = {"flops": wl.flops, "tile": wl.tile, "gemms": [list((x.M, x.N, x.K)) for x in wl.gemms]}
            # what the library's analytical model picks for each GEMM (SFC_CA_AUTO)
            entry["model_choice"] = []
            for x in wl.gemms:
                pm = sg.sfc_gemm_plan(x.M, x.N, x.K, 0, wl.tile)
                entry["model_choice"].append({"tile": f"{pm['BM']}x{pm['BN']}", "ca_layers": pm["layers"]})
            ops = [prepare(gg)[2:] for gg in wl.gemms]
            c_first = wl.ca_layers[0]
            ramp = warm_clock(torch, stream,
                              lambda: [run_once(a, b, cc, wl, c_first) for a, b, cc in ops], args.warm_clock_ms)
            entry["clock_warmup"] = {"ms": args.warm_clock_ms, "first_batch_ms": ramp[0], "last_batch_ms": ramp[1]}
            log(f"[bench] {name} clock warm-up: ms per call {ramp[0]} (first batch) -> {ramp[1]} (last)")

            cold_sets = [ColdSets(torch, *op) for op in ops]

            def cold_ms(gi, c, reps, sched=None, tile=None, fused=False):
                """Mean of `reps` cold calls (in rotation over copies of the operands)."""
                return cold_sets[gi].time_ms(torch, stream,
                                             lambda a, b, cc: run_once(a, b, cc, wl, c, sched, tile, fused), reps)

            def timed(c, sched=None, tile=None, fused=False):
                cold_t = warm_t = 0.0
                for gi in range(len(wl.gemms)):
                    a, b, cc = ops[gi]
                    for _ in range(3):
                        run_once(a, b, cc, wl, c, sched, tile, fused)
                    torch.cuda.synchronize()
                    cold_t += cold_ms(gi, c, args.reps, sched, tile, fused)
                    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    gpu_backlog(torch, 40 * args.reps)
                    s.record(stream)
                    for _ in range(args.reps):
                        run_once(a, b, cc, wl, c, sched, tile, fused)
                    e.record(stream)
                    torch.cuda.synchronize()
                    warm_t += s.elapsed_time(e) / args.reps
                return {"cold_ms": round(cold_t, 4), "warm_ms": round(warm_t, 4),
                        "tflops_cold": round(wl.flops / (cold_t * 1e-3) / 1e12, 2),
                        "tflops_warm": round(wl.flops / (warm_t * 1e-3) / 1e12, 2)}

            def autotune():
                """The model's choice (SFC_TILE_AUTO, SFC_CA_AUTO) against the best of
                the four block shapes x ca_layers in {1, 2, 4, 8, 16} (layer copies
                up to 2 GiB), each timed cold, per GEMM: the GPU counterpart of
                Section III.C's knob prediction checked against autotuning."""
                best_t = model_t = 0.0
                rows = []
                for gi, x in enumerate(wl.gemms):
                    a, b, cc = ops[gi]
                    cands = []
                    # the model's choice is timed before and after the candidates
                    # (mean of the two): the candidates run for a while, and the
                    # chip's state drifts over that time
                    run_once(a, b, cc, wl, 0, None, "auto")
                    mt0 = cold_ms(gi, 0, args.tune_reps, None, "auto")
                    for t in ("128x128", "256x128", "128x256", "256x256"):
                        for c in (1, 2, 4, 8, 16):
                            if c > 1 and c * x.M * x.N * 4 > (2 << 30):
                                continue
                            run_once(a, b, cc, wl, c, None, t)
                            cands.append((cold_ms(gi, c, args.tune_reps, None, t), t, c))
                    mt = 0.5 * (mt0 + cold_ms(gi, 0, args.tune_reps, None, "auto"))
                    bt = min(cands)
                    pm = sg.sfc_gemm_plan(x.M, x.N, x.K, 0, "auto")
                    rows.append({"gemm": [x.M, x.N, x.K],
                                 "model": {"tile": f"{pm['BM']}x{pm['BN']}", "ca_layers": pm["layers"],
                                           "cold_ms": round(mt, 4)},
                                 "best": {"tile": bt[1], "ca_layers": bt[2], "cold_ms": round(bt[0], 4)},
                                 "candidates": len(cands)})
                    best_t += bt[0]
                    model_t += mt
                return {"protocol": f"each candidate: mean of {args.tune_reps} cold calls; the model's choice: "
                                    f"the same, before and after the candidates, averaged", "per_gemm": rows,
                        "model_over_best": round(best_t / model_t, 4)}

            per_c = {}
            for c in wl.ca_layers:
                label = "auto" if c == 0 else c
                per_c[label] = timed(c)
                log(f"[bench] {name} c={label}: {per_c[label]}")
            if len(wl.ca_layers) > 1:
                # chiplet-aware placement of the layers against the hardware
                # workgroup order, at the model's layer count
                entry["layer_placement"] = {"chiplet_aware": per_c["auto"],
                                            "hardware_order": timed(0, "interleaved_plain")}
                log(f"[bench] {name} placement: {entry['layer_placement']}")
                # the layer copies summed inside the GEMM launch (sfc_gemm_fused_ex)
                # against the separate reduction kernel, per layer count
                entry["fused_reduction"] = {("auto" if c == 0 else c): timed(c, fused=True)
                                            for c in wl.ca_layers if c != 1}
                log(f"[bench] {name} fused reduction: {entry['fused_reduction']}")
            if wl.tile != "auto":
                # the configuration pins the block shape and one layer; the
                # library's own choice on the same GEMM, for comparison
                entry["model_choice_timed"] = timed(0, tile="auto")
                log(f"[bench] {name} at the model's choice: {entry['model_choice_timed']}")
            if not args.no_autotune:
                entry["model_vs_autotune"] = autotune()
                log(f"[bench] {name} model vs autotune: {entry['model_vs_autotune']['model_over_best']}")
            del ops, cold_sets
            best_c = max(per_c, key=lambda k: per_c[k]["tflops_cold"])
            best = per_c[best_c]
            # roofline of the workload: min(MFMA peak, OI x HBM) per GEMM with its
            # compulsory bytes (A, B and C once), times summed over the GEMMs
            roofs = [roofline_tflops(x.M, x.N, x.K, 2 if x.out == "bf16" else 4) for x in wl.gemms]
            t_roof = sum(2.0 * x.M * x.N * x.K / (r[1] * 1e12) for x, r in zip(wl.gemms, roofs))
            roof = wl.flops / t_roof / 1e12
            entry.update({"per_ca_layers": per_c if len(per_c) > 1 else None, "best_ca_layers": best_c,
                          "tflops": best["tflops_cold"], "tflops_warm": best["tflops_warm"],
                          "frac_of_mfma_peak": round(best["tflops_cold"] / PEAK_BF16_TFLOPS, 4),
                          "roofline_bound": "hbm" if any(r[0] == "hbm" for r in roofs) else "mfma",
                          "roofline_tflops": round(roof, 1),
                          "frac_of_roofline": round(best["tflops_cold"] / roof, 4)})
            table[name] = entry
            whm_num += wl.flops
            whm_den += wl.flops / best["tflops_cold"]
            torch.cuda.empty_cache()
        whm = whm_num / whm_den
        best_shape = max(v["tflops"] for v in table.values())
        tuned = [v["model_vs_autotune"]["model_over_best"] for v in table.values() if "model_vs_autotune" in v]
        table = {"protocol": f"mean of {args.reps} cold reps (in rotation over >= 1 GiB of copies of A, B and C), "
                             "best ca_layers",
                 "shapes": table, "whm_tflops": round(whm, 2),
                 "whm_over_best_shape": round(whm / best_shape, 4)}
        if tuned:
            table["model_over_autotune_mean"] = round(sum(tuned) / len(tuned), 4)
            table["model_over_autotune_min"] = round(min(tuned), 4)

    sweep = run_sweep(args, sg, torch, stream, dev) if args.sweep else None

    # ------------------------------------------------------------ cpu baseline
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import gemm as ogemm
        threads = ogemm.threads()
        rows = 4 * threads                 # every thread busy while calibrating
        t = time.perf_counter()
        ogemm.gemm_ref_rows(A_host, B_host, g.N, g.K, g.K, g.N, row0=0, nrows=rows)
        dt = time.perf_counter() - t
        rows = int(max(8, min(g.M, rows * args.cpu_seconds / max(dt, 1e-3))))
        log(f"[bench] cpu oracle: {rows} rows on {threads} threads")
        t = time.perf_counter()
        ogemm.gemm_ref_rows(A_host, B_host, g.N, g.K, g.K, g.N, row0=0, nrows=rows)
        dt = time.perf_counter() - t
        cpu_model = "unknown"
        try:
            for ln in open("/proc/cpuinfo"):
                if ln.startswith("model name"):
                    cpu_model = ln.split(":", 1)[1].strip()
                    break
        except OSError:
            pass
        cpu = {"value": round(2.0 * rows * g.N * g.K / dt / 1e12, 6), "unit": "TFLOP/s",
               "cores": threads, "kind": "oracle", "cpu_model": cpu_model,
               "host_cpus": os.cpu_count(),
               "sample": f"rows 0..{rows - 1} of the {g.M}x{g.N}x{g.K} GEMM "
                         f"({rows}x{g.N} outputs, fp64, {dt:.1f} s)"}

    counters = counter_record()
    # The kernel's shader cycles per launch do not depend on the box or the
    # operands (committed counter runs); its duration follows the clock the
    # board holds under load.  Cycles / duration is that clock, and 4096 flop
    # per CU per clock at that clock is the MFMA ceiling of this very run.
    clock = None
    if counters.get("cycles_per_xcd_per_launch"):
        ghz = counters["cycles_per_xcd_per_launch"] / (kern_ms * 1e-3) / 1e9
        ceiling = PEAK_BF16_TFLOPS * ghz / 2.4
        clock = {"ghz_implied": round(ghz, 3), "mfma_ceiling_at_that_clock": round(ceiling, 1),
                 "frac_of_that_ceiling": round(achieved / ceiling, 4),
                 "cycles_per_xcd_per_launch": counters["cycles_per_xcd_per_launch"],
                 "mfma_busy_per_clock": counters.get("mfma_busy")}
    cold_c2 = None
    if table is not None:
        e2 = table["shapes"][HEADLINE]
        cold_c2 = {"protocol": table["protocol"], "tflops": e2["tflops"],
                   "frac_of_mfma_peak": e2["frac_of_mfma_peak"], "tflops_warm_10": e2["tflops_warm"]}
    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "clock_warmup": {"ms": args.warm_clock_ms, "first_batch_ms_per_step": head_ramp[0],
                         "last_batch_ms_per_step": head_ramp[1]},
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "accumulate": "f32", "data": "synthetic",
        "config": {"workload": HEADLINE, "M": g.M, "N": g.N, "K": g.K, "out": g.out,
                   "tile": w.tile, "grid": [plan["gm"], plan["gn"]], "ca_layers": 1,
                   "order": args.order, "sched": args.sched, "workgroups": plan["workgroups"],
                   "dist": "A, B ~ N(0,1) rounded to bf16"},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": counters.get("hbm_bytes_per_launch"),
                     "kernel": "sfc_gemm_kernel<256,256,bf16 out>",
                     "kernel_ms": round(kern_ms, 4),
                     "mfma_probe": probe,
                     "frac_of_probe_random": round(achieved / probe["random_operands"]["tflops"], 4),
                     "same_kernel_constant_operands": constant,
                     "loaded_clock": clock},
        "headline_cold": cold_c2,
        "cpu_baseline": cpu,
        "library_same_workload": library,
        "fp8_square8192": fp8,
        "workloads": table,
    }
    if sweep is not None:
        line["sweep"] = sweep
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
